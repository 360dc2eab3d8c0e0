#pragma once
// WBMM kernels for gfx950 (MI355X, CDNA4): device code and per-shape host
// launchers.  Included by wbmm_inst.hip, which instantiates it for one dtype
// and a range of window sizes per translation unit.
//
// Operator (Alg. 1; eq. index_computation; eq. index_select; Theorem 3.2):
//   Y_window[j] = sum_i X_window[i] * T[c, I(i, j)],
//   I(i, j) = (h_i - h_j + w - 1)(2w - 1) + (w_i - w_j + w - 1)
// with i the input and j the output position inside one w x w window.
//
// Data layout inside the kernels
// ------------------------------
// Window positions are stored "row padded": position (h, x) of a window sits at
// p = h * RP + x with RP = 8 (w <= 8) or 16 (w <= 16); the columns x >= w and
// the rows h >= w are zero.  A 16-wide tile of p is then one padded window row
// (RP = 16) or two (RP = 8), which is what makes the matrix M_c cheap to
// produce on chip: M_c is block-Toeplitz (Theorem 3.2), the block linking input
// row h_i to output row h_j depends only on h_i - h_j, so every matrix-core
// B fragment of M_c depends only on (2 * kstep - ntile) and a kernel needs at
// most 2S + NT - 2 distinct fragments (26 at w = 14) instead of all of M_c.
//
// Global memory is read and written in aligned 16-byte chunks of window
// "bands" (w consecutive image rows of one (b, c) plane, contiguous in NCHW);
// each element is routed to its LDS slot by its (row, column).  Chunks that
// straddle the edge of a band fall back to element accesses, so no byte
// outside the caller's tensors is touched.
//
// Forward / backward-input kernel: one workgroup = (channel, tile of
// windows).  X tile -> LDS (window-major); T[c] -> LDS; Toeplitz blocks
// TB[dh][x_out][x_in] -> LDS; each wave keeps the distinct B fragments in
// registers and runs 16-window sub-tiles through v_mfma_f32_16x16x32_{bf16,
// f16} (or v_mfma_f32_16x16x4_f32); results go back through LDS to coalesced
// band stores.  The input gradient reuses it with the table read reversed,
// because M_c^T is the matrix of the reversed table.
//
// Backward-table kernel: one workgroup = (channel, slab of windows).  X and dY
// chunks -> LDS position-major (windows contiguous), so matrix-core fragments
// of X^T and dY are contiguous.  The accumulator for the 16x16 block pair
// (input tile pi, output tile po) only matters through pi - po, so all pairs
// with equal pi - po share one accumulator (27 16x16 fp32 tiles at w = 14),
// split across the four waves.  Diagonal sums of those tiles give dT.  Slabs
// are combined by a second kernel in a fixed order (no atomics anywhere).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wbmm_internal.h"

namespace wbmm {

typedef unsigned short u16;
typedef u16 u16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // 4 waves of 64
constexpr int kWaves = 4;

__host__ __device__ constexpr int rp_of(int w) { return w <= 8 ? 8 : 16; }
__host__ __device__ constexpr int rup(int a, int b) { return (a + b - 1) / b * b; }
__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

// ----------------------------------------------------------------- dtypes

struct TagF32 {
  typedef float S;   // storage
  typedef float Frag;  // matrix-core operand per lane
  static constexpr int ES = 4;
  static constexpr bool W16 = false;
  static constexpr int KS = 4;  // K per MFMA
};
struct TagBF16 {
  typedef u16 S;
  typedef u16x8 Frag;
  static constexpr int ES = 2;
  static constexpr bool W16 = true;
  static constexpr int KS = 32;
};
struct TagF16 {
  typedef u16 S;
  typedef u16x8 Frag;
  static constexpr int ES = 2;
  static constexpr bool W16 = true;
  static constexpr int KS = 32;
};

__device__ inline float bf16_to_f(u16 v) { return __uint_as_float((uint32_t)v << 16); }
__device__ inline u16 f_to_bf16(float f) {  // round to nearest even
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u16)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (u16)(u >> 16);
}
__device__ inline u16 f_to_f16(float f) { return __builtin_bit_cast(u16, (_Float16)f); }

template <class Tag> __device__ inline typename Tag::S from_f32(float f);
template <> __device__ inline float from_f32<TagF32>(float f) { return f; }
template <> __device__ inline u16 from_f32<TagBF16>(float f) { return f_to_bf16(f); }
template <> __device__ inline u16 from_f32<TagF16>(float f) { return f_to_f16(f); }

template <class Tag> __device__ inline f32x4 mma(typename Tag::Frag a, typename Tag::Frag b, f32x4 c);
template <> __device__ inline f32x4 mma<TagF32>(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
template <> __device__ inline f32x4 mma<TagBF16>(u16x8 a, u16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <> __device__ inline f32x4 mma<TagF16>(u16x8 a, u16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// Element u of a 16-byte chunk held as uint4.
template <int ES> __device__ inline uint32_t chunk_elem(const uint4 &v, int u);
template <> __device__ inline uint32_t chunk_elem<4>(const uint4 &v, int u) {
  return u == 0 ? v.x : u == 1 ? v.y : u == 2 ? v.z : v.w;
}
template <> __device__ inline uint32_t chunk_elem<2>(const uint4 &v, int u) {
  const uint32_t d = (u >> 1) == 0 ? v.x : (u >> 1) == 1 ? v.y : (u >> 1) == 2 ? v.z : v.w;
  return (u & 1) ? (d >> 16) : (d & 0xffffu);
}

// ------------------------------------------------------------- geometry

struct KArgs {
  int64_t B, C, H, W;
  int64_t NH, NW, N;
  int64_t tile;          // windows per workgroup tile (forward) / per slab (dtable)
  int64_t tiles_per_ch;  // tiles (slabs) per channel
  int dense;             // H and W are multiples of w
};

// One aligned 16-byte chunk of a band.  The band of window-row index bi of
// channel c covers image rows [wy*w, wy*w + rows) of plane (b, c); it is
// contiguous in NCHW.  Chunk ci of the band starts at the 16-byte boundary at
// or below the band start.  On success: ca = chunk address, elements [u0, u1)
// of the chunk belong to the band, and (r, x) = band row / image column of
// element u0.
template <int WIN, int ES>
__device__ inline bool band_chunk(const KArgs &a, int64_t c, int64_t bi, int ci, uintptr_t base,
                                  uintptr_t &ca, int &u0, int &u1, int &r, int &x) {
  constexpr int VE = 16 / ES;
  const int64_t b = bi / a.NH;
  const int64_t wy = bi - b * a.NH;
  const int64_t rows64 = a.H - wy * WIN;
  const int rows = rows64 < WIN ? (int)rows64 : WIN;
  const int64_t estart = ((b * a.C + c) * a.H + wy * WIN) * a.W;
  const int64_t elen = (int64_t)rows * a.W;
  const uintptr_t bs = base + (uintptr_t)(estart * ES);
  const uintptr_t be = bs + (uintptr_t)(elen * ES);
  ca = (bs & ~(uintptr_t)15) + (uintptr_t)ci * 16u;
  if (ca >= be) return false;
  const int64_t e_ca = ((int64_t)ca - (int64_t)bs) / ES;  // may be negative
  u0 = e_ca < 0 ? (int)(-e_ca) : 0;
  const int64_t rem = elen - e_ca;
  u1 = rem < VE ? (int)rem : VE;
  const int e0 = (int)(e_ca + u0);
  const int Wi = (int)a.W;
  r = e0 / Wi;
  x = e0 - r * Wi;
  return true;
}

template <int WIN, int ES>
__device__ inline int chunks_per_band(const KArgs &a) {
  return (int)((WIN * a.W * ES) / 16) + 2;
}

// Load a chunk: whole-vector when the chunk lies inside the band, otherwise
// only the band's elements.
template <int ES>
__device__ inline uint4 load_chunk(uintptr_t ca, int u0, int u1) {
  constexpr int VE = 16 / ES;
  if (u0 == 0 && u1 == VE) return *reinterpret_cast<const uint4 *>(ca);
  uint4 v = make_uint4(0, 0, 0, 0);
  uint32_t w4[4] = {0, 0, 0, 0};
#pragma unroll
  for (int u = 0; u < VE; ++u) {
    if (u >= u0 && u < u1) {
      uint32_t e;
      if (ES == 4) e = *reinterpret_cast<const uint32_t *>(ca + 4 * u);
      else e = *reinterpret_cast<const u16 *>(ca + 2 * u);
      if (ES == 4) w4[u] = e;
      else w4[u >> 1] |= (u & 1) ? (e << 16) : e;
    }
  }
  v.x = w4[0]; v.y = w4[1]; v.z = w4[2]; v.w = w4[3];
  return v;
}

// ======================================================= forward kernel

template <class Tag, int WIN>
struct FwdCfg {
  static constexpr int RP = rp_of(WIN);
  static constexpr int PP = WIN * RP;                 // padded positions
  static constexpr int KP = rup(PP, Tag::KS);         // padded K
  static constexpr int S = KP / Tag::KS;              // K steps
  static constexpr int NT = cdiv(PP, 16);             // 16-wide output tiles
  static constexpr int NB = 2 * S + NT - 2;           // distinct B fragments (16-bit)
  // LDS row stride (elements) of the window-major tile, chosen so 16 lanes
  // reading one fragment each hit distinct banks.
  static constexpr int LDSW = Tag::W16 ? KP + 8 : KP + ((4 - KP) % 64 + 64) % 64;
  static constexpr int K1 = 2 * WIN - 1;
  static constexpr int K2 = K1 * K1;
  static constexpr int TS_LEN = rup(K2, 8);
  static constexpr int TB_LEN = Tag::W16 ? K1 * RP * RP : 0;
};

template <class Tag, int WIN>
__host__ __device__ constexpr size_t fwd_lds_bytes(int64_t tile) {
  typedef FwdCfg<Tag, WIN> G;
  return (size_t)tile * G::LDSW * Tag::ES + (size_t)(G::TS_LEN + G::TB_LEN) * Tag::ES;
}

template <class Tag, int WIN, bool REV>
__global__ __launch_bounds__(kThreads) void wbmm_fwd_kernel(const typename Tag::S *__restrict__ x,
                                                            const typename Tag::S *__restrict__ tab,
                                                            typename Tag::S *__restrict__ y, KArgs a) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RP = G::RP, KP = G::KP, LDSW = G::LDSW, K1 = G::K1, K2 = G::K2;
  constexpr int VE = 16 / Tag::ES;

  extern __shared__ __align__(16) unsigned char smem[];
  S *tile = reinterpret_cast<S *>(smem);
  S *Ts = tile + a.tile * LDSW;
  S *TB = Ts + G::TS_LEN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t c = blockIdx.x / a.tiles_per_ch;
  const int64_t tix = blockIdx.x - c * a.tiles_per_ch;
  const int64_t n0 = tix * a.tile;
  const int64_t n1 = (n0 + a.tile < a.N) ? n0 + a.tile : a.N;
  const int nwin = (int)(n1 - n0);

  // ---- 1. zero what the scatter will not write; stage the table
  const bool full = a.dense && nwin == a.tile;
  if (!full) {
    uint4 *t4 = reinterpret_cast<uint4 *>(tile);
    const int n16 = (int)((a.tile * LDSW * Tag::ES) / 16);
    for (int i = tid; i < n16; i += kThreads) t4[i] = make_uint4(0, 0, 0, 0);
  } else {
    constexpr int PADS = KP - WIN * WIN;  // padded slots per window
    constexpr int PADC = RP - WIN;        // padded columns per row
    if constexpr (PADS > 0) {
      for (int i = tid; i < nwin * PADS; i += kThreads) {
        const int v = i / PADS;
        const int q = i - v * PADS;
        int p;
        if constexpr (PADC > 0) {
          if (q < WIN * PADC) {
            const int h = q / PADC;
            p = h * RP + WIN + (q - h * PADC);
          } else {
            p = WIN * RP + (q - WIN * PADC);
          }
        } else {
          p = WIN * RP + q;
        }
        tile[v * LDSW + p] = (S)0;
      }
    }
  }
  for (int k = tid; k < K2; k += kThreads) Ts[k] = tab[c * K2 + (REV ? K2 - 1 - k : k)];
  if (!full) __syncthreads();

  // ---- 2. scatter the X tile: bands -> window-major LDS
  {
    const int64_t bi0 = n0 / a.NW, bi1 = (n1 - 1) / a.NW;
    const int nb = (int)(bi1 - bi0 + 1);
    const int cpb = chunks_per_band<WIN, Tag::ES>(a);
    const int total = nb * cpb;
    const uintptr_t xb = reinterpret_cast<uintptr_t>(x);
    constexpr int U = 4;
    for (int s0 = tid; s0 < total; s0 += kThreads * U) {
      uint4 v[U];
      uintptr_t ca[U];
      int u0[U], u1[U], r[U], xx[U];
      bool ok[U];
      int64_t bi[U];
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int slot = s0 + k * kThreads;
        ok[k] = false;
        if (slot < total) {
          const int bl = slot / cpb;
          const int ci = slot - bl * cpb;
          bi[k] = bi0 + bl;
          ok[k] = band_chunk<WIN, Tag::ES>(a, c, bi[k], ci, xb, ca[k], u0[k], u1[k], r[k], xx[k]);
          if (ok[k]) v[k] = load_chunk<Tag::ES>(ca[k], u0[k], u1[k]);
        }
      }
#pragma unroll
      for (int k = 0; k < U; ++k) {
        if (!ok[k]) continue;
        int rr = r[k], cx = xx[k];
#pragma unroll
        for (int u = 0; u < VE; ++u) {
          if (u >= u0[k] && u < u1[k]) {
            const int wx = cx / WIN;
            const int xi = cx - wx * WIN;
            const int64_t n = bi[k] * a.NW + wx;
            if (n >= n0 && n < n1) {
              const uint32_t e = chunk_elem<Tag::ES>(v[k], u);
              S val;
              if constexpr (Tag::ES == 4) val = __uint_as_float(e);
              else val = (u16)e;
              tile[(int)(n - n0) * LDSW + rr * RP + xi] = val;
            }
            if (++cx == (int)a.W) { cx = 0; ++rr; }
          }
        }
      }
    }
  }
  __syncthreads();

  // ---- 3. Toeplitz blocks of M_c (16-bit path): TB[dh][x_out][x_in]
  if constexpr (Tag::W16) {
    for (int i = tid; i < G::TB_LEN; i += kThreads) {
      const int dhi = i / (RP * RP);
      const int rem = i - dhi * RP * RP;
      const int xo = rem / RP;
      const int xi = rem - xo * RP;
      TB[i] = (xo < WIN && xi < WIN) ? Ts[dhi * K1 + xi - xo + WIN - 1] : (S)0;
    }
    __syncthreads();
  }

  // ---- 4. matrix-core products, 16 windows at a time per wave
  const int g = lane >> 4;   // lane group
  const int ln = lane & 15;  // row (A) / column (B, C) inside a 16x16 tile
  if constexpr (Tag::W16) {
    constexpr int S_ = G::S, NT = G::NT, NB = G::NB;
    Frag bf[NB];
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int d0 = q - (NT - 1);  // = 2*kstep - ntile
      int dh, xi0;
      if (RP == 16) { dh = d0 + (g >> 1); xi0 = 8 * (g & 1); }
      else { dh = 2 * d0 + g - (ln >> 3); xi0 = 0; }
      const int xo = ln & (RP - 1);
      if (dh >= -(WIN - 1) && dh <= WIN - 1)
        bf[q] = *reinterpret_cast<const Frag *>(&TB[((dh + WIN - 1) * RP + xo) * RP + xi0]);
      else
        bf[q] = Frag{0, 0, 0, 0, 0, 0, 0, 0};
    }
    const int nsub = (nwin + 15) >> 4;
    for (int sub = wave; sub < nsub; sub += kWaves) {
      S *rowp = tile + (sub * 16) * LDSW;
      Frag af[S_];
#pragma unroll
      for (int s = 0; s < S_; ++s)
        af[s] = *reinterpret_cast<const Frag *>(&rowp[ln * LDSW + s * 32 + 8 * g]);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < S_; ++s) acc = mma<Tag>(af[s], bf[2 * s - t + NT - 1], acc);
        const int p = 16 * t + ln;
        const int ho = p / RP, xo = p - (p / RP) * RP;
        if (ho < WIN && xo < WIN) {
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) rowp[(4 * g + rr) * LDSW + p] = from_f32<Tag>(acc[rr]);
        }
      }
    }
  } else {
    constexpr int S_ = G::S, NT = G::NT;
    const int nsub = (nwin + 15) >> 4;
    for (int sub = wave; sub < nsub; sub += kWaves) {
      S *rowp = tile + (sub * 16) * LDSW;
      float af[S_];
#pragma unroll
      for (int s = 0; s < S_; ++s) af[s] = rowp[ln * LDSW + 4 * s + g];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        const int pn = 16 * t + ln;
        const int ho = pn / RP, xo = pn - (pn / RP) * RP;
#pragma unroll
        for (int s = 0; s < S_; ++s) {
          const int k = 4 * s + g;
          const int hi = k / RP, xi = k - (k / RP) * RP;
          const int dh = hi - ho;
          float bv = 0.f;
          if (xo < WIN && xi < WIN && dh >= -(WIN - 1) && dh <= WIN - 1)
            bv = Ts[(dh + WIN - 1) * K1 + xi - xo + WIN - 1];
          acc = mma<Tag>(af[s], bv, acc);
        }
        if (ho < WIN && xo < WIN) {
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) rowp[(4 * g + rr) * LDSW + pn] = acc[rr];
        }
      }
    }
  }
  __syncthreads();

  // ---- 5. store the Y tile: window-major LDS -> bands
  {
    const int64_t bi0 = n0 / a.NW, bi1 = (n1 - 1) / a.NW;
    const int nb = (int)(bi1 - bi0 + 1);
    const int cpb = chunks_per_band<WIN, Tag::ES>(a);
    const int total = nb * cpb;
    const uintptr_t yb = reinterpret_cast<uintptr_t>(y);
    for (int slot = tid; slot < total; slot += kThreads) {
      const int bl = slot / cpb;
      const int ci = slot - bl * cpb;
      const int64_t bi = bi0 + bl;
      uintptr_t ca;
      int u0, u1, rr, cx;
      if (!band_chunk<WIN, Tag::ES>(a, c, bi, ci, yb, ca, u0, u1, rr, cx)) continue;
      uint32_t w4[4] = {0, 0, 0, 0};
      int mask = 0;
#pragma unroll
      for (int u = 0; u < VE; ++u) {
        if (u >= u0 && u < u1) {
          const int wx = cx / WIN;
          const int xi = cx - wx * WIN;
          const int64_t n = bi * a.NW + wx;
          if (n >= n0 && n < n1) {
            const S val = tile[(int)(n - n0) * LDSW + rr * RP + xi];
            uint32_t e;
            if constexpr (Tag::ES == 4) e = __float_as_uint(val);
            else e = (uint32_t)val;
            if (Tag::ES == 4) w4[u] = e;
            else w4[u >> 1] |= (u & 1) ? (e << 16) : e;
            mask |= 1 << u;
          }
          if (++cx == (int)a.W) { cx = 0; ++rr; }
        }
      }
      if (mask == (1 << VE) - 1) {
        *reinterpret_cast<uint4 *>(ca) = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      } else {
#pragma unroll
        for (int u = 0; u < VE; ++u) {
          if (mask & (1 << u)) {
            if (Tag::ES == 4) *reinterpret_cast<uint32_t *>(ca + 4 * u) = w4[u];
            else *reinterpret_cast<u16 *>(ca + 2 * u) = (u16)((u & 1) ? (w4[u >> 1] >> 16) : (w4[u >> 1] & 0xffffu));
          }
        }
      }
    }
  }
}

// ===================================================== dtable kernel

template <class Tag, int WIN>
struct DtCfg {
  static constexpr int RP = rp_of(WIN);
  static constexpr int PP = WIN * RP;
  static constexpr int NPT = cdiv(PP, 16);        // 16-position tiles
  static constexpr int KPT = NPT * 16;            // padded positions
  static constexpr int R = 16 / RP;               // window rows per tile
  static constexpr int CW = Tag::W16 ? 32 : 16;   // windows per LDS chunk
  static constexpr int CWS = Tag::W16 ? CW + 8 : CW + 4;  // row stride (elements)
  static constexpr int NACC = 2 * NPT - 1;        // accumulators: pi - po
  static constexpr int K1 = 2 * WIN - 1;
  static constexpr int K2 = K1 * K1;
  static constexpr int NBT = (2 * R - 1) * K1;    // bins per accumulator tile
  static constexpr int BUF = KPT * CWS;           // elements per operand buffer
};

// Accumulator tiles are assigned to waves by longest-processing-time: tile P
// (= pi - po) carries NPT - |P| block products per K step.
template <int NPT>
struct PAssign {
  int count[kWaves];
  int list[kWaves][2 * NPT - 1];
};

template <int NPT>
__host__ __device__ constexpr PAssign<NPT> make_passign() {
  PAssign<NPT> pa{};
  int load[kWaves] = {0, 0, 0, 0};
  for (int w = 0; w < kWaves; ++w) pa.count[w] = 0;
  // work NPT - |P|, P = 0, 1, -1, 2, -2, ...: already in non-increasing work order
  for (int i = 0; i < 2 * NPT - 1; ++i) {
    const int P = (i & 1) ? (i + 1) / 2 : -(i / 2);
    int best = 0;
    for (int w = 1; w < kWaves; ++w)
      if (load[w] < load[best] || (load[w] == load[best] && pa.count[w] < pa.count[best])) best = w;
    pa.list[best][pa.count[best]++] = P + NPT - 1;
    load[best] += NPT - (P < 0 ? -P : P);
  }
  return pa;
}

template <class Tag, int WIN>
__host__ __device__ constexpr size_t dt_lds_bytes() {
  typedef DtCfg<Tag, WIN> G;
  const size_t ops = 2 * (size_t)G::BUF * Tag::ES;
  const size_t bins = (size_t)(kWaves * 16 * 17 + G::NACC * G::NBT) * 4;
  return ops > bins ? ops : bins;
}

// Scatter one chunk of windows [m0, m1) of channel c from tensor `src` into
// the position-major buffer dst[p * CWS + (n - m0)].
template <class Tag, int WIN>
__device__ inline void dt_scatter(const KArgs &a, int64_t c, int64_t m0, int64_t m1,
                                  uintptr_t src, typename Tag::S *dst, int tid) {
  typedef typename Tag::S S;
  typedef DtCfg<Tag, WIN> G;
  constexpr int RP = G::RP, CWS = G::CWS;
  constexpr int VE = 16 / Tag::ES;
  const int64_t bi0 = m0 / a.NW, bi1 = (m1 - 1) / a.NW;
  const int nb = (int)(bi1 - bi0 + 1);
  const int cpb = chunks_per_band<WIN, Tag::ES>(a);
  const int total = nb * cpb;
  constexpr int U = 4;
  for (int s0 = tid; s0 < total; s0 += kThreads * U) {
    uint4 v[U];
    uintptr_t ca[U];
    int u0[U], u1[U], r[U], xx[U];
    bool ok[U];
    int64_t bi[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int slot = s0 + k * kThreads;
      ok[k] = false;
      if (slot < total) {
        const int bl = slot / cpb;
        const int ci = slot - bl * cpb;
        bi[k] = bi0 + bl;
        ok[k] = band_chunk<WIN, Tag::ES>(a, c, bi[k], ci, src, ca[k], u0[k], u1[k], r[k], xx[k]);
        if (ok[k]) v[k] = load_chunk<Tag::ES>(ca[k], u0[k], u1[k]);
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      if (!ok[k]) continue;
      int rr = r[k], cx = xx[k];
#pragma unroll
      for (int u = 0; u < VE; ++u) {
        if (u >= u0[k] && u < u1[k]) {
          const int wx = cx / WIN;
          const int xi = cx - wx * WIN;
          const int64_t n = bi[k] * a.NW + wx;
          if (n >= m0 && n < m1) {
            const uint32_t e = chunk_elem<Tag::ES>(v[k], u);
            S val;
            if constexpr (Tag::ES == 4) val = __uint_as_float(e);
            else val = (u16)e;
            dst[(rr * RP + xi) * CWS + (int)(n - m0)] = val;
          }
          if (++cx == (int)a.W) { cx = 0; ++rr; }
        }
      }
    }
  }
}

template <class Tag, int WIN, int WAVE>
__device__ void dt_wave(const typename Tag::S *__restrict__ x, const typename Tag::S *__restrict__ dy,
                        float *__restrict__ out, const KArgs &a, unsigned char *smem) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef DtCfg<Tag, WIN> G;
  constexpr int NPT = G::NPT, CW = G::CW, CWS = G::CWS, RP = G::RP, R = G::R;
  constexpr int K1 = G::K1, K2 = G::K2, NBT = G::NBT;
  constexpr PAssign<NPT> PA = make_passign<NPT>();
  constexpr int NP = PA.count[WAVE];

  S *Xt = reinterpret_cast<S *>(smem);
  S *Dt = Xt + G::BUF;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int g = lane >> 4;
  const int ln = lane & 15;
  const int64_t c = blockIdx.x / a.tiles_per_ch;
  const int64_t slab = blockIdx.x - c * a.tiles_per_ch;
  const int64_t s0 = slab * a.tile;
  const int64_t s1 = (s0 + a.tile < a.N) ? s0 + a.tile : a.N;

  f32x4 acc[NP > 0 ? NP : 1];
#pragma unroll
  for (int j = 0; j < NP; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // padded slots must read as zero: clear both buffers once
  {
    uint4 *t4 = reinterpret_cast<uint4 *>(smem);
    const int n16 = (2 * G::BUF * Tag::ES) / 16;
    for (int i = tid; i < n16; i += kThreads) t4[i] = make_uint4(0, 0, 0, 0);
  }
  __syncthreads();

  for (int64_t m0 = s0; m0 < s1; m0 += CW) {
    const int64_t m1 = (m0 + CW < s1) ? m0 + CW : s1;
    if (!(a.dense && m1 - m0 == CW) && m0 != s0) {
      uint4 *t4 = reinterpret_cast<uint4 *>(smem);
      const int n16 = (2 * G::BUF * Tag::ES) / 16;
      for (int i = tid; i < n16; i += kThreads) t4[i] = make_uint4(0, 0, 0, 0);
      __syncthreads();
    }
    dt_scatter<Tag, WIN>(a, c, m0, m1, reinterpret_cast<uintptr_t>(x), Xt, tid);
    dt_scatter<Tag, WIN>(a, c, m0, m1, reinterpret_cast<uintptr_t>(dy), Dt, tid);
    __syncthreads();

    if constexpr (Tag::W16) {
      Frag bf[NPT];
#pragma unroll
      for (int po = 0; po < NPT; ++po)
        bf[po] = *reinterpret_cast<const Frag *>(&Dt[(16 * po + ln) * CWS + 8 * g]);
#pragma unroll
      for (int pi = 0; pi < NPT; ++pi) {
        const Frag af = *reinterpret_cast<const Frag *>(&Xt[(16 * pi + ln) * CWS + 8 * g]);
#pragma unroll
        for (int j = 0; j < NP; ++j) {
          const int po = pi - (PA.list[WAVE][j] - (NPT - 1));
          if (po >= 0 && po < NPT) acc[j] = mma<Tag>(af, bf[po], acc[j]);
        }
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < CW / 4; ++ks) {
        float bf[NPT];
#pragma unroll
        for (int po = 0; po < NPT; ++po) bf[po] = Dt[(16 * po + ln) * CWS + 4 * ks + g];
#pragma unroll
        for (int pi = 0; pi < NPT; ++pi) {
          const float af = Xt[(16 * pi + ln) * CWS + 4 * ks + g];
#pragma unroll
          for (int j = 0; j < NP; ++j) {
            const int po = pi - (PA.list[WAVE][j] - (NPT - 1));
            if (po >= 0 && po < NPT) acc[j] = mma<Tag>(af, bf[po], acc[j]);
          }
        }
      }
    }
    __syncthreads();
  }

  // ---- diagonal binning, fixed order
  float *scr = reinterpret_cast<float *>(smem) + WAVE * 16 * 17;
  float *binsum = reinterpret_cast<float *>(smem) + kWaves * 16 * 17;
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    const int pidx = PA.list[WAVE][j];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) scr[(4 * g + rr) * 17 + ln] = acc[j][rr];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int bin = lane; bin < NBT; bin += 64) {
      const int da = bin / K1 - (R - 1);  // input sub-row minus output sub-row
      const int dw = bin - (bin / K1) * K1 - (WIN - 1);
      float s = 0.f;
      for (int ra = 0; ra < R; ++ra) {
        const int rb = ra - da;
        if (rb < 0 || rb >= R) continue;
        for (int xo = 0; xo < WIN; ++xo) {
          const int xi = xo + dw;
          if (xi < 0 || xi >= WIN) continue;
          s += scr[(ra * RP + xi) * 17 + rb * RP + xo];
        }
      }
      binsum[pidx * NBT + bin] = s;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  __syncthreads();
  for (int k = tid; k < K2; k += kThreads) {
    const int dhi = k / K1;
    const int dwi = k - dhi * K1;
    const int dh = dhi - (WIN - 1);
    float s = 0.f;
    for (int P = -(NPT - 1); P <= NPT - 1; ++P) {
      const int da = dh - P * R;
      if (da < -(R - 1) || da > R - 1) continue;
      s += binsum[(P + NPT - 1) * NBT + (da + R - 1) * K1 + dwi];
    }
    out[(slab * a.C + c) * K2 + k] = s;
  }
}

template <class Tag, int WIN>
__global__ __launch_bounds__(kThreads) void wbmm_dt_kernel(const typename Tag::S *__restrict__ x,
                                                           const typename Tag::S *__restrict__ dy,
                                                           float *__restrict__ out, KArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  switch (threadIdx.x >> 6) {
    case 0: dt_wave<Tag, WIN, 0>(x, dy, out, a, smem); break;
    case 1: dt_wave<Tag, WIN, 1>(x, dy, out, a, smem); break;
    case 2: dt_wave<Tag, WIN, 2>(x, dy, out, a, smem); break;
    default: dt_wave<Tag, WIN, 3>(x, dy, out, a, smem); break;
  }
}

// Sum of the per-slab partials in slab order: dt[i] = sum_s ws[s][i].
template <class Tag>
__global__ __launch_bounds__(kThreads) void wbmm_dt_reduce_kernel(const float *__restrict__ ws,
                                                                  float *__restrict__ dt,
                                                                  int64_t slabs, int64_t len) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= len) return;
  float s = 0.f;
  for (int64_t k = 0; k < slabs; ++k) s += ws[k * len + i];
  dt[i] = s;
}

// ============================================================ host side

static int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }

static KArgs make_args(const Geom &g) {
  KArgs a;
  a.B = g.B; a.C = g.C; a.H = g.H; a.W = g.W;
  a.NH = g.NH; a.NW = g.NW; a.N = g.N;
  a.tile = 0; a.tiles_per_ch = 0;
  a.dense = (g.H % g.w == 0) && (g.W % g.w == 0);
  return a;
}

static constexpr size_t kLdsBudget = 64 * 1024;

template <class Tag, int WIN>
static int64_t pick_fwd_tile(const Geom &g) {
  int64_t tile = rp_of(WIN) == 8 ? 128 : 64;
  if (!Tag::W16) tile = rp_of(WIN) == 8 ? 64 : 32;
  while (tile > 16 && fwd_lds_bytes<Tag, WIN>(tile) > kLdsBudget) tile /= 2;
  // keep enough workgroups to cover 256 compute units several times over
  while (tile > (Tag::W16 ? 64 : 16) && g.C * cdiv64(g.N, tile) < 1024) tile /= 2;
  return tile;
}

template <class Tag, int WIN>
static hipError_t run_forward(const void *x, const void *t, void *y, const Geom &g, bool rev,
                              hipStream_t st) {
  typedef typename Tag::S S;
  KArgs a = make_args(g);
  a.tile = pick_fwd_tile<Tag, WIN>(g);
  a.tiles_per_ch = cdiv64(g.N, a.tile);
  const int64_t grid = g.C * a.tiles_per_ch;
  const size_t lds = fwd_lds_bytes<Tag, WIN>(a.tile);
  if (rev)
    wbmm_fwd_kernel<Tag, WIN, true><<<dim3((unsigned)grid), dim3(kThreads), lds, st>>>(
        (const S *)x, (const S *)t, (S *)y, a);
  else
    wbmm_fwd_kernel<Tag, WIN, false><<<dim3((unsigned)grid), dim3(kThreads), lds, st>>>(
        (const S *)x, (const S *)t, (S *)y, a);
  return hipGetLastError();
}

template <class Tag, int WIN>
static DtPlan plan_dt(const Geom &g) {
  typedef DtCfg<Tag, WIN> G;
  DtPlan p;
  const int64_t chunks = cdiv64(g.N, G::CW);
  int64_t slabs = cdiv64(1024, g.C);
  if (slabs > chunks) slabs = chunks;
  if (slabs < 1) slabs = 1;
  p.slab_windows = cdiv64(cdiv64(g.N, slabs), G::CW) * G::CW;
  p.slabs = cdiv64(g.N, p.slab_windows);
  return p;
}

template <class Tag, int WIN>
static hipError_t run_dtable(const void *x, const void *dy, float *dt, void *ws, const Geom &g,
                             hipStream_t st) {
  typedef typename Tag::S S;
  typedef DtCfg<Tag, WIN> G;
  KArgs a = make_args(g);
  const DtPlan p = plan_dt<Tag, WIN>(g);
  a.tile = p.slab_windows;
  a.tiles_per_ch = p.slabs;
  float *out = p.slabs > 1 ? (float *)ws : dt;
  const size_t lds = dt_lds_bytes<Tag, WIN>();
  wbmm_dt_kernel<Tag, WIN><<<dim3((unsigned)(g.C * p.slabs)), dim3(kThreads), lds, st>>>(
      (const S *)x, (const S *)dy, out, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.slabs == 1) return e;
  const int64_t len = g.C * G::K2;
  wbmm_dt_reduce_kernel<Tag><<<dim3((unsigned)cdiv64(len, kThreads)), dim3(kThreads), 0, st>>>(
      (const float *)ws, dt, p.slabs, len);
  return hipGetLastError();
}

}  // namespace wbmm
