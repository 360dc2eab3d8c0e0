// WBMM kernels for gfx950 (MI355X, CDNA4): device code and per-shape host
// launchers.  Included by wbmm_inst.hip, which instantiates it for one dtype
// and a range of window sizes per translation unit.
//
// Operator (Alg. 1; eq. index_computation; eq. index_select; Theorem 3.2):
//   Y_window[j] = sum_i X_window[i] * T[c, I(i, j)],
//   I(i, j) = (h_i - h_j + w - 1)(2w - 1) + (w_i - w_j + w - 1)
// with i the input and j the output position inside one w x w window.
//
// Layout on chip
// --------------
// Window positions are "row padded": position (h, x) of a window sits at
// p = h * RP + x with RP = 8 (w <= 8) or 16 (w <= 16), columns x >= w and rows
// h >= w being zero.  A 16-wide tile of p is then one padded window row
// (RP = 16) or two (RP = 8).  M_c is block-Toeplitz (Theorem 3.2): the block
// linking input row h_i to output row h_j depends only on h_i - h_j.  So every
// matrix-core B fragment of M_c depends only on (2 * kstep - ntile), and a
// kernel needs 2S + NT - 2 distinct fragments (26 at w = 14) instead of M_c.
//
// Data movement
// -------------
// The unit of global traffic is one window row (w consecutive elements of an
// image row) or, where the windows tile the map, a 16-byte chunk of whole
// bands or whole images.  Rows land in window-major LDS tiles, already
// padded, so a matrix-core fragment of one window's positions is one 16-byte
// LDS read; the table gradient reads the transposed fragments (positions x
// windows) with the transposing 16-bit LDS reads.  Where the windows tile the
// map with a power-of-two count per row ("fixed-offset rows"), a row's offset
// inside its 16-window sub-tile depends only on its place there, so copies
// need no per-row index arithmetic.
//
// Forward / backward-input: one workgroup = (channel, tile of windows), four
// waves, each running 16-window sub-tiles.  The table T[c] and its Toeplitz
// blocks TB[dh][x_out][x_in] go to LDS (zero blocks padded around them so
// that fragment reads need no range check), and products run through
// v_mfma_f32_16x16x32_{bf16,f16} (v_mfma_f32_16x16x4_f32 for float32); 16-bit
// maps that the windows tile take the image-layout kernel (the sub-tile is
// copied in image layout with 16-byte accesses and the window fragments are
// gathered from it).  Results are rounded once and go back through LDS.  The
// input gradient is the same kernel with the table read back to front, since
// M_c^T is the matrix of the reversed table.
//
// Table gradient: K = windows.  The 16x16 block pair (input tile pi, output
// tile po) only matters through pi - po, so all pairs with equal pi - po
// share one accumulator (27 16x16 fp32 tiles at w = 14), split across four
// waves.  Diagonal sums of the tiles give dT.  A channel split into slabs
// writes one partial table per slab; a second kernel adds the partials in
// slab order, so the result is bitwise reproducible.
//
// Fused backward: x and dy are read once for both gradients.  With
// fixed-offset rows and no more channels than compute units (or, in rounds,
// a last round at least half full), one 16-wave workgroup per channel (or
// slab) streams the channel's stages through LDS:
// four waves accumulate the table gradient while eight compute the input
// gradient of the same stage (the former then store the previous stage's dX
// rows), and four copy waves bring the next stages in, with one workgroup
// barrier per stage.  Otherwise a
// four-wave workgroup per (channel, slab) runs the same products in turn.
// The hierarchical form (global window 2 wl plus local wl sub-windows) adds
// local-block products to the forward and input gradient and splits the
// table-gradient accumulators by row halves to bin both tables in one pass.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <initializer_list>

#include "wbmm_internal.h"

namespace wbmm {

typedef unsigned short u16;
typedef u16 u16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
// dword-aligned 16-byte vector (global rows are only 4-byte aligned)
typedef uint32_t u32x4a __attribute__((ext_vector_type(4))) __attribute__((aligned(4)));

constexpr int kThreads = 256;  // 4 waves of 64
constexpr int kWaves = 4;

__host__ __device__ constexpr int rp_of(int w) { return w <= 8 ? 8 : 16; }
__host__ __device__ constexpr int rup(int a, int b) { return (a + b - 1) / b * b; }
__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }

// ----------------------------------------------------------------- dtypes

struct TagF32 {
  typedef float S;     // storage
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

// Two float32 values rounded once (nearest even) and packed into a dword,
// the first in the low half.
template <class Tag> __device__ inline uint32_t pack2(float a, float b);
template <> __device__ inline uint32_t pack2<TagBF16>(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}
template <> __device__ inline uint32_t pack2<TagF16>(float a, float b) {
  const f16x2 v = {(_Float16)a, (_Float16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// One stored 16-bit value as float32 (exact).
template <class Tag> __device__ inline float to_f32(u16 v);
template <> __device__ inline float to_f32<TagBF16>(u16 v) { return __builtin_bit_cast(float, (uint32_t)v << 16); }
template <> __device__ inline float to_f32<TagF16>(u16 v) { return (float)__builtin_bit_cast(_Float16, v); }

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

// floor(v / d) for 0 <= v, d < 2^24 from a float reciprocal, corrected.
__device__ inline int fdiv(int v, int d, float inv) {
  int q = (int)((float)v * inv);
  if (q * d > v) --q;
  else if ((q + 1) * d <= v) ++q;
  return q;
}

// v / d for 0 <= v < 2^22 and d >= 1, from inv = 1 / d rounded to float, with
// no correction step: (v + 1/2) / d lies at least 1 / (2d) from an integer,
// and the two roundings move the product by less than (v + 1/2) / d * 2^-23,
// which is below that distance, so truncating the product gives the quotient.
__device__ __attribute__((always_inline)) inline int fdiv_small(int v, float inv) {
  return (int)(((float)v + 0.5f) * inv);
}

// ------------------------------------------------------------- geometry

struct KArgs {
  int64_t B, C, H, W;
  int64_t numel;       // elements of one [B,C,H,W] tensor
  int NH, NW;
  int64_t N;           // windows per channel, B * NH * NW
  int tile;            // windows per workgroup tile (forward) / per slab (dtable)
  int tiles_per_ch;    // workgroups per channel
  float inv_nw, inv_nhw;
  // Fixed-offset rows (gradient kernels): when tiled is set, windows tile the
  // map, every window row is whole and starts on a dword, and a 16-window
  // sub-tile (16-aligned) is whole bands of one image or whole images, so a
  // row's byte offset from its sub-tile's first element depends only on its
  // place in the sub-tile.
  int tiled;
  int lgnw;            // log2(NW)
  int lgw;             // log2(windows per piece of a sub-tile): 4 inside one image, else log2(NH * NW)
  int BE;              // elements of one band (w * W)
  int WPI;             // windows per image
  int64_t chw;         // elements between images of one channel (C * H * W)
  // Channel-stream runs (more channels than compute units): workgroup r
  // streams the stages [r run, (r + 1) run) of all channels' stages taken in
  // order (nstc per channel); 0: one workgroup per (channel, slab).
  int run;
  int nstc;
};

// Fourth word of a raw buffer resource (stride 0, byte offsets): 32-bit data
// format, so that loads return the bytes as stored and offsets at or past the
// record count read as zero.
constexpr int kBufWord3 = 0x00020000;

// A window row: element offset (from the tensor base) of its first element,
// number of columns inside the image (0: the row lies outside the image or the
// window does not exist) and how it moves:
//   kDword: whole row, dword-aligned, whole dwords;
//   kShift: whole 16-bit row that starts in the middle of a dword: the
//           enclosing aligned dwords are read and shifted by 16 bits (every
//           dword read holds at least one element of the tensor);
//   kElem:  element by element (rows cut by the image edge).
enum RowMode { kNone = 0, kDword = 1, kShift = 2, kElem = 3 };

template <int WIN, int ES>
struct Row {
  int64_t eoff;
  int cols;
  int mode;
  int odd;  // kShift: the row starts at the upper half of a dword
};

template <int WIN, int ES>
__device__ __attribute__((always_inline)) inline Row<WIN, ES> row_of(const KArgs &a, const void *base, int64_t c, int64_t n, int hi) {
  Row<WIN, ES> r;
  r.eoff = 0;
  r.cols = 0;
  r.mode = kNone;
  r.odd = 0;
  if (n >= a.N || hi >= WIN) return r;
  const int nhw = a.NH * a.NW;
  const int b = fdiv((int)n, nhw, a.inv_nhw);
  const int rem = (int)n - b * nhw;
  const int wy = fdiv(rem, a.NW, a.inv_nw);
  const int wx = rem - wy * a.NW;
  const int64_t h = (int64_t)wy * WIN + hi;
  if (h >= a.H) return r;
  const int64_t cw = a.W - (int64_t)wx * WIN;
  r.cols = cw < WIN ? (int)cw : WIN;
  r.eoff = (((int64_t)b * a.C + c) * a.H + h) * a.W + (int64_t)wx * WIN;
  r.mode = kElem;
  if (r.cols == WIN) {
    const uint64_t addr = reinterpret_cast<uintptr_t>(base) + (uint64_t)r.eoff * ES;
    if ((addr & 3u) == 0 && ((WIN * ES) & 3) == 0) {
      r.mode = kDword;
    } else if (ES == 2 && (WIN & 1)) {
      // (even windows are only misaligned for odd image widths: element path)
      r.odd = (int)((addr >> 1) & 1u);
      const int64_t first = r.eoff - r.odd;                 // first element read
      const int64_t last = first + 2 * (WIN / 2 + 1);       // one past the last
      if (first >= 0 && last <= a.numel) r.mode = kShift;
    }
  }
  return r;
}

// Fixed-offset rows: element offset of the first element of the 16-window
// sub-tile that starts at window m (a multiple of 16), and the byte offset of
// row hi of its window vv (0..15) from there.
__device__ __attribute__((always_inline)) inline int64_t tiled_sub_base(const KArgs &a, int64_t c, int64_t m) {
  const int mi = (int)m;
  const int img = mi / a.WPI;
  const int inw = mi - img * a.WPI;
  return (int64_t)img * a.chw + c * a.H * a.W + (int64_t)(inw >> a.lgnw) * a.BE;
}
template <int WIN, int ES>
__device__ __attribute__((always_inline)) inline uint32_t tiled_row_off(const KArgs &a, int vv, int hi) {
  const int nwm = (1 << a.lgnw) - 1, mw = (1 << a.lgw) - 1;
  return (uint32_t)(vv >> a.lgw) * (uint32_t)(a.chw * ES) +
         (uint32_t)((((vv & mw) >> a.lgnw) * a.BE + (vv & nwm) * WIN + hi * (int)a.W) * ES);
}

// Fixed-offset row hi of window m0 + vv (m0 a multiple of 16, vv < 16) as a
// whole dword-aligned row.
template <int WIN, int ES>
__device__ __attribute__((always_inline)) inline Row<WIN, ES> tiled_row(const KArgs &a, int64_t c, int64_t m0, int vv, int hi) {
  Row<WIN, ES> r;
  const int nwm = (1 << a.lgnw) - 1, mw = (1 << a.lgw) - 1;
  r.eoff = tiled_sub_base(a, c, m0) + (int64_t)(vv >> a.lgw) * a.chw +
           (int64_t)(((vv & mw) >> a.lgnw) * a.BE + (vv & nwm) * WIN + hi * (int)a.W);
  r.cols = WIN;
  r.mode = kDword;
  r.odd = 0;
  return r;
}

// Dwords of one padded row (RP elements) in registers.
template <int WIN, int ES>
struct RowData {
  static constexpr int RP = rp_of(WIN);
  static constexpr int ND = RP * ES / 4;  // dwords per padded row
  uint32_t d[ND];
};

// Load a window row: columns >= cols and padded columns read as zero.
template <int WIN, int ES>
__device__ __attribute__((always_inline)) inline void load_row(const void *base, const Row<WIN, ES> &r, RowData<WIN, ES> &o) {
  constexpr int ND = RowData<WIN, ES>::ND;
  constexpr int NDV = (WIN * ES) / 4;  // data dwords of a whole aligned row
#pragma unroll
  for (int i = 0; i < ND; ++i) o.d[i] = 0;
  if (r.mode == kNone) return;
  const char *p = reinterpret_cast<const char *>(base) + r.eoff * ES;
  if (r.mode == kDword) {
    const uint32_t *p4 = reinterpret_cast<const uint32_t *>(p);
#pragma unroll
    for (int i = 0; i + 4 <= NDV; i += 4) {
      const u32x4a v = *reinterpret_cast<const u32x4a *>(p4 + i);
      o.d[i] = v.x; o.d[i + 1] = v.y; o.d[i + 2] = v.z; o.d[i + 3] = v.w;
    }
#pragma unroll
    for (int i = NDV & ~3; i < NDV; ++i) o.d[i] = p4[i];
  } else if (ES == 2 && (WIN & 1) && r.mode == kShift) {
    constexpr int NL = WIN / 2 + 1;  // dwords read
    const uint32_t *p4 = reinterpret_cast<const uint32_t *>(p - 2 * r.odd);
    uint32_t in[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) in[i] = p4[i];
    const int sh = 16 * r.odd;
#pragma unroll
    for (int i = 0; i < (WIN + 1) / 2; ++i)
      o.d[i] = (uint32_t)((((uint64_t)(i + 1 < NL ? in[i + 1] : 0u) << 32) | in[i]) >> sh);
    if constexpr ((WIN & 1) != 0) o.d[WIN / 2] &= 0xffffu;
  } else {
    // branch-free: element x reads column min(x, cols - 1), which is inside
    // the row, and is then zeroed when x >= cols
    const int last = r.cols - 1;
#pragma unroll
    for (int x = 0; x < WIN; ++x) {
      const int xc = x < last ? x : last;
      if (ES == 4) {
        const uint32_t e = reinterpret_cast<const uint32_t *>(p)[xc];
        o.d[x] = x < r.cols ? e : 0u;
      } else {
        const uint32_t e = reinterpret_cast<const u16 *>(p)[xc];
        const uint32_t m = x < r.cols ? e : 0u;
        o.d[x >> 1] |= (x & 1) ? (m << 16) : m;
      }
    }
  }
}

// Store the first cols elements of a padded row held as dwords.
template <int WIN, int ES>
__device__ __attribute__((always_inline)) inline void store_row(void *base, const Row<WIN, ES> &r, const uint32_t *d) {
  constexpr int NDV = (WIN * ES) / 4;
  if (r.mode == kNone) return;
  char *p = reinterpret_cast<char *>(base) + r.eoff * ES;
  if (r.mode == kDword) {
    uint32_t *p4 = reinterpret_cast<uint32_t *>(p);
#pragma unroll
    for (int i = 0; i + 4 <= NDV; i += 4)
      *reinterpret_cast<u32x4a *>(p4 + i) = u32x4a{d[i], d[i + 1], d[i + 2], d[i + 3]};
#pragma unroll
    for (int i = NDV & ~3; i < NDV; ++i) p4[i] = d[i];
  } else if (ES == 2 && (WIN & 1) && r.mode == kShift) {
    u16 *p2 = reinterpret_cast<u16 *>(p);
    auto elem = [&](int x) -> uint32_t { return (x & 1) ? (d[x >> 1] >> 16) : (d[x >> 1] & 0xffffu); };
    if (r.odd) {
      // element 0 shares its dword with the previous element of the tensor
      p2[0] = (u16)elem(0);
#pragma unroll
      for (int x = 1; x + 1 < WIN; x += 2)
        *reinterpret_cast<uint32_t *>(p2 + x) = elem(x) | (elem(x + 1) << 16);
      if ((WIN - 1) & 1) p2[WIN - 1] = (u16)elem(WIN - 1);
    } else {
#pragma unroll
      for (int x = 0; x + 1 < WIN; x += 2)
        *reinterpret_cast<uint32_t *>(p2 + x) = elem(x) | (elem(x + 1) << 16);
      if (WIN & 1) p2[WIN - 1] = (u16)elem(WIN - 1);
    }
  } else {
#pragma unroll
    for (int x = 0; x < WIN; ++x) {
      if (x < r.cols) {
        if (ES == 4) reinterpret_cast<uint32_t *>(p)[x] = d[x];
        else reinterpret_cast<u16 *>(p)[x] = (u16)((x & 1) ? (d[x >> 1] >> 16) : (d[x >> 1] & 0xffffu));
      }
    }
  }
}

// ======================================================= forward kernel

template <class Tag, int WIN>
struct FwdCfg {
  static constexpr int RP = rp_of(WIN);
  static constexpr int PP = WIN * RP;                 // padded positions
  static constexpr int KP = rup(PP, Tag::KS);         // padded K
  static constexpr int KR = KP / RP;                  // padded rows per window
  static constexpr int S = KP / Tag::KS;              // K steps
  static constexpr int NT = cdiv(PP, 16);             // 16-wide output tiles
  static constexpr int NB = 2 * S + NT - 2;           // distinct B fragments (16-bit)
  // LDS row stride (elements) of the window-major tile, chosen so 16 lanes
  // reading one fragment each hit distinct banks.
  static constexpr int LDSW = Tag::W16 ? KP + 8 : KP + ((4 - KP) % 64 + 64) % 64;
  static constexpr int K1 = 2 * WIN - 1;
  static constexpr int K2 = K1 * K1;
  static constexpr int TS_LEN = rup(K2 + 9, 8);       // + the overrun of tb_chunk's dword reads
  // Toeplitz blocks TB[dh][x_out][x_in] for dh = -(w-1)..w-1, with zero
  // blocks beyond them for every dh a lane's B fragment can name (dh of
  // fragment q: q - (NT-1) + g/2 for 16-position rows, 2 (q - (NT-1)) + g -
  // x_out/8 for 8-position rows), so that the fragment reads need no range
  // check and their address is a per-lane base plus a constant
  static constexpr int DHMIN = RP == 16 ? -(NT - 1) : -2 * (NT - 1) - 1;
  static constexpr int DHMAX = RP == 16 ? 2 * S - 1 : 2 * (NB - NT) + 3;
  static constexpr int TBLO = -(WIN - 1) - DHMIN > 0 ? -(WIN - 1) - DHMIN : 0;  // zero blocks below
  static constexpr int TBHI = DHMAX - (WIN - 1) > 0 ? DHMAX - (WIN - 1) : 0;     // and above
  static constexpr int TB_LEN = Tag::W16 ? (TBLO + K1 + TBHI) * RP * RP : 0;
  // hierarchical form (WIN = 2 wl): the local table of the wl x wl
  // sub-windows and its Toeplitz blocks
  static constexpr int WL = WIN / 2;
  static constexpr int K1L = WL > 0 ? 2 * WL - 1 : 1;
  static constexpr int K2L = K1L * K1L;
  static constexpr int TSL_LEN = rup(K2L, 8);
  static constexpr int TBL_LEN = Tag::W16 ? K1L * RP * RP : 0;
};

// Rows of a window touched by the A operand of K step s and by output tile t
// (row-padded positions: a K step covers 32 / RP rows, a tile 16 / RP rows).
template <class Tag, int WIN>
__host__ __device__ constexpr bool fwd_rows_meet(int s, int t, bool same_half_only) {
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RK = Tag::KS / G::RP > 0 ? Tag::KS / G::RP : 1;  // rows per K step (16-bit)
  constexpr int RT = 16 / G::RP;                                 // rows per output tile
  for (int a = 0; a < RK; ++a)
    for (int b = 0; b < RT; ++b) {
      const int hi = RK * s + a, ho = RT * t + b;
      if (hi >= WIN || ho >= WIN) continue;
      if (same_half_only ? ((hi < G::WL) == (ho < G::WL)) : hi == ho) return true;
    }
  return false;
}

// The forward kernel runs four waves per workgroup.  Each wave owns a run of
// 16-window sub-tiles and pipelines them through one private LDS buffer: the
// rows of sub-tile j+1 are loaded into registers while sub-tile j is
// multiplied and its rows are stored, so reads and writes of the whole grid
// stay interleaved (a grid that reads everything first and writes everything
// afterwards moves data at about half the rate).
constexpr int kFwdWaves = 4;
constexpr int kFwdThreads = 64 * kFwdWaves;

template <class Tag, int WIN, bool HIER = false>
__host__ __device__ constexpr size_t fwd_lds_bytes() {
  typedef FwdCfg<Tag, WIN> G;
  return (size_t)kFwdWaves * 16 * G::LDSW * Tag::ES + (size_t)(G::TS_LEN + G::TB_LEN) * Tag::ES +
         (HIER ? (size_t)(G::TSL_LEN + G::TBL_LEN) * Tag::ES : 0);
}

// Workgroup index regrouped by die: the dispatcher deals workgroups to the
// eight dies in turn (workgroup b runs on die b mod 8), so with G a multiple
// of 8 workgroup b takes index (b mod 8) G/8 + b/8 and each die runs one
// consecutive block of indices: neighbouring channels, whose image planes
// share the 128-byte lines at their ends, then share that die's L2.
__device__ __attribute__((always_inline)) inline uint32_t die_major(uint32_t b, uint32_t G) {
  return (G & 7u) ? b : (b & 7u) * (G >> 3) + (b >> 3);
}

// Wave-level ordering of LDS accesses made by different lanes of one wave.
__device__ __attribute__((always_inline)) inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Row copies of one sub-tile (16 windows x KR padded rows) spread over the 64
// lanes of a wave; rows of one window are consecutive.
template <class Tag, int WIN>
struct SubRows {
  static constexpr int N = 16 * FwdCfg<Tag, WIN>::KR;
  static constexpr int PER_LANE = cdiv(N, 64);
  RowData<WIN, Tag::ES> rd[PER_LANE];
};

template <class Tag, int WIN, bool TILED>
__device__ __attribute__((always_inline)) inline void load_sub(const KArgs &a, const void *x, int64_t c, int64_t m0, int nwin, int lane,
                                SubRows<Tag, WIN> &o) {
  constexpr int KR = FwdCfg<Tag, WIN>::KR;
#pragma unroll
  for (int k = 0; k < SubRows<Tag, WIN>::PER_LANE; ++k) {
    const int q = lane + 64 * k;
    const int v = q / KR;
    const int hi = q - v * KR;
    Row<WIN, Tag::ES> r;
    r.cols = 0; r.eoff = 0; r.mode = kNone; r.odd = 0;
    if constexpr (TILED) {
      if (q < SubRows<Tag, WIN>::N && v < nwin && hi < WIN) r = tiled_row<WIN, Tag::ES>(a, c, m0, v, hi);
    } else if (q < SubRows<Tag, WIN>::N && v < nwin) {
      r = row_of<WIN, Tag::ES>(a, x, c, m0 + v, hi);
    }
    load_row<WIN, Tag::ES>(x, r, o.rd[k]);
  }
}

template <class Tag, int WIN>
__device__ __attribute__((always_inline)) inline void write_sub(unsigned char *buf, int lane, const SubRows<Tag, WIN> &o) {
  typedef FwdCfg<Tag, WIN> G;
  typedef RowData<WIN, Tag::ES> RD;
#pragma unroll
  for (int k = 0; k < SubRows<Tag, WIN>::PER_LANE; ++k) {
    const int q = lane + 64 * k;
    if (q >= SubRows<Tag, WIN>::N) continue;
    const int v = q / G::KR;
    const int hi = q - v * G::KR;
    uint32_t *l4 = reinterpret_cast<uint32_t *>(buf + (v * G::LDSW + hi * G::RP) * Tag::ES);
#pragma unroll
    for (int i = 0; i < RD::ND; i += 4)
      *reinterpret_cast<uint4 *>(l4 + i) = make_uint4(o.rd[k].d[i], o.rd[k].d[i + 1], o.rd[k].d[i + 2], o.rd[k].d[i + 3]);
  }
}

template <class Tag, int WIN, bool TILED>
__device__ __attribute__((always_inline)) inline void store_sub(const KArgs &a, void *y, int64_t c, int64_t m0, int nwin, int lane,
                                 const unsigned char *buf) {
  typedef FwdCfg<Tag, WIN> G;
  typedef RowData<WIN, Tag::ES> RD;
  for (int q = lane; q < 16 * WIN; q += 64) {
    const int v = q / WIN;
    const int hi = q - v * WIN;
    if (v >= nwin) break;
    const Row<WIN, Tag::ES> r = TILED ? tiled_row<WIN, Tag::ES>(a, c, m0, v, hi) : row_of<WIN, Tag::ES>(a, y, c, m0 + v, hi);
    if (r.mode == kNone) continue;
    const uint32_t *l4 = reinterpret_cast<const uint32_t *>(buf + (v * G::LDSW + hi * G::RP) * Tag::ES);
    uint32_t d[RD::ND];
#pragma unroll
    for (int i = 0; i < RD::ND; i += 4) {
      const uint4 u = *reinterpret_cast<const uint4 *>(l4 + i);
      d[i] = u.x; d[i + 1] = u.y; d[i + 2] = u.z; d[i + 3] = u.w;
    }
    store_row<WIN, Tag::ES>(y, r, d);
  }
}

// One 8-element chunk of a row of the Toeplitz blocks: table entries
// k0 + xi for xi = xi0 .. xi0 + 7, zero where xi >= WIN.  Read as five dwords
// of the table copy in LDS (4-byte aligned, padded past its end) and shifted
// by one element when k0 + xi0 is odd.
template <int WIN>
__device__ __attribute__((always_inline)) inline u16x8 tb_chunk(const u16 *Ts, int k0, int xi0) {
  const int kb = k0 + xi0;
  const uint32_t *p = reinterpret_cast<const uint32_t *>(Ts) + (kb >> 1);
  const uint32_t sh = (uint32_t)(kb & 1) * 16u;
  uint32_t d[5];
#pragma unroll
  for (int i = 0; i < 5; ++i) d[i] = p[i];
  uint32_t u[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t v = __builtin_amdgcn_alignbit(d[i + 1], d[i], sh);
    const int xa = xi0 + 2 * i;
    u[i] = xa >= WIN ? 0u : (xa + 1 >= WIN ? (v & 0xffffu) : v);
  }
  return __builtin_bit_cast(u16x8, make_uint4(u[0], u[1], u[2], u[3]));
}

// The table row of channel c (and the local table of the hierarchical form)
// held in registers between the loads and their copy to LDS, so that the
// loads can be issued before the bulk loads of the input rows instead of
// queueing behind them.
template <class Tag, int WIN, bool HIER, int NTH>
struct TabRegs {
  typedef FwdCfg<Tag, WIN> G;
  static constexpr int N = cdiv(G::K2, NTH);
  static constexpr int NL = HIER ? cdiv(G::K2L, NTH) : 1;
  typename Tag::S v[N];
  typename Tag::S vl[NL];
};

template <class Tag, int WIN, bool REV, bool HIER, int NTH>
__device__ __attribute__((always_inline)) inline void tab_load(const typename Tag::S *__restrict__ tab,
                                                                const typename Tag::S *__restrict__ tabl, int64_t c,
                                                                int tid, TabRegs<Tag, WIN, HIER, NTH> &tr) {
  typedef FwdCfg<Tag, WIN> G;
  constexpr int K2 = G::K2;
  const typename Tag::S *tc = tab + c * K2;
  // unconditional loads (the index clamped to the row): with no branch
  // around them, the wait for the table before its copy to LDS counts only
  // the loads issued before the input rows, not those rows too
#pragma unroll
  for (int i = 0; i < tr.N; ++i) {
    const int k0 = tid + i * NTH;
    const int k = k0 < K2 ? k0 : K2 - 1;
    tr.v[i] = tc[REV ? K2 - 1 - k : k];
  }
  if constexpr (HIER) {
    constexpr int K2L = G::K2L;
    const typename Tag::S *tl = tabl + c * K2L;
#pragma unroll
    for (int i = 0; i < tr.NL; ++i) {
      const int k0 = tid + i * NTH;
      const int k = k0 < K2L ? k0 : K2L - 1;
      tr.vl[i] = tl[REV ? K2L - 1 - k : k];
    }
  }
}

// The Toeplitz blocks of M_c (16-bit) from the table row in LDS: block
// TBLO + dh + (w-1) holds TB[dh][x_out][x_in], the pad blocks zero.  NTH
// threads take part; no barrier inside.
template <class Tag, int WIN, int NTH>
__device__ __attribute__((always_inline)) inline void build_tb(const typename Tag::S *Ts, typename Tag::S *TB, int tid) {
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RP = G::RP, K1 = G::K1, CPR = RP / 8;  // 8-element chunks per TB row
  constexpr int NCH = (G::TBLO + K1 + G::TBHI) * RP * CPR;
  for (int ch = tid; ch < NCH; ch += NTH) {
    const int row = ch / CPR;  // = block * RP + x_out
    const int xi0 = (ch - row * CPR) * 8;
    const int dhi = row / RP - G::TBLO;
    const int xo = row - (dhi + G::TBLO) * RP;
    u16x8 v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
    if (dhi >= 0 && dhi < K1 && xo < WIN) v = tb_chunk<WIN>(Ts, dhi * K1 - xo + WIN - 1, xi0);  // table index of x_in = 0
    *reinterpret_cast<u16x8 *>(&TB[row * RP + xi0]) = v;
  }
}

// The table row of channel c (read back to front for the input gradient)
// -> Ts with coalesced loads; for 16-bit, the Toeplitz blocks
// TB[dh][x_out][x_in] of M_c gathered from it.  The hierarchical form also
// stages the local table (-> Tsl) and, for 16-bit, its blocks
// TBL[dh][x_out][x_in], zero unless x_in and x_out lie in the same half of the
// window (the same local sub-window column).  Ends with a workgroup barrier.
template <class Tag, int WIN, bool REV, bool HIER = false, int NTH = kFwdThreads>
__device__ __attribute__((always_inline)) inline void fwd_tables(const TabRegs<Tag, WIN, HIER, NTH> &tr,
                                                                  typename Tag::S *Ts, typename Tag::S *TB,
                                                                  typename Tag::S *Tsl, typename Tag::S *TBL, int tid) {
  typedef typename Tag::S S;
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RP = G::RP, K1 = G::K1, K2 = G::K2;
#pragma unroll
  for (int i = 0; i < tr.N; ++i) {
    const int k = tid + i * NTH;
    if (k < K2) Ts[k] = tr.v[i];
  }
  if constexpr (HIER) {
    constexpr int K2L = G::K2L;
#pragma unroll
    for (int i = 0; i < tr.NL; ++i) {
      const int k = tid + i * NTH;
      if (k < K2L) Tsl[k] = tr.vl[i];
    }
  }
  if constexpr (Tag::W16) {
    __syncthreads();
    build_tb<Tag, WIN, NTH>(Ts, TB, tid);
    constexpr int CPR = RP / 8;  // 8-element chunks per TBL row
    if constexpr (HIER) {
      constexpr int WL = G::WL, K1L = G::K1L;
      constexpr int NCHL = K1L * RP * CPR;
      for (int ch = tid; ch < NCHL; ch += NTH) {
        const int row = ch / CPR;               // = dhl * RP + x_out
        const int xi0 = (ch - row * CPR) * 8;
        const int dhl = row / RP;
        const int xo = row - dhl * RP;
        u16x8 v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
        if (xo < WIN) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int xi = xi0 + e;
            const bool same = xi < WIN && (xi < WL) == (xo < WL);
            const int k = dhl * K1L + (same ? xi - xo + WL - 1 : 0);
            const u16 t = Tsl[k];
            v[e] = same ? t : (u16)0;
          }
        }
        *reinterpret_cast<u16x8 *>(&TBL[row * RP + xi0]) = v;
      }
    }
  }
  __syncthreads();
}

// B fragment q (= 2 * kstep - ntile + NT - 1) of M_c for lane (g, ln), from
// the Toeplitz blocks.
template <class Tag, int WIN>
__device__ __attribute__((always_inline)) inline typename Tag::Frag fwd_bfrag(const typename Tag::S *TB, int q,
                                                                               int g, int ln) {
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RP = G::RP, NT = G::NT;
  const int d0 = q - (NT - 1);
  int dh, xi0;
  if (RP == 16) { dh = d0 + (g >> 1); xi0 = 8 * (g & 1); }
  else { dh = 2 * d0 + g - (ln >> 3); xi0 = 0; }
  const int xo = ln & (RP - 1);
  return *reinterpret_cast<const typename Tag::Frag *>(&TB[((dh + G::TBLO + WIN - 1) * RP + xo) * RP + xi0]);
}

// Hierarchical form, 16-bit: the local-table fragment of K step s and output
// tile t for lane (g, ln) (zero where input and output rows lie in different
// halves of the window).
template <class Tag, int WIN>
__device__ __attribute__((always_inline)) inline typename Tag::Frag fwd_lfrag(const typename Tag::S *TBL, int s, int t,
                                                                               int g, int ln) {
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RP = G::RP, WL = G::WL;
  int hi, ho, xi0;
  if (RP == 16) { hi = 2 * s + (g >> 1); ho = t; xi0 = 8 * (g & 1); }
  else { hi = 4 * s + g; ho = 2 * t + (ln >> 3); xi0 = 0; }
  const int xo = ln & (RP - 1);
  const bool same = hi < WIN && ho < WIN && (hi < WL) == (ho < WL);
  const int dhl = same ? hi - ho + WL - 1 : 0;
  const typename Tag::Frag f = *reinterpret_cast<const typename Tag::Frag *>(&TBL[(dhl * RP + xo) * RP + xi0]);
  return same ? f : typename Tag::Frag{0, 0, 0, 0, 0, 0, 0, 0};
}

template <class Tag, int WIN, bool REV, bool HIER = false, bool TILED = false>
__global__ __launch_bounds__(kFwdThreads, 3) void wbmm_fwd_kernel(const typename Tag::S *__restrict__ x,
                                                                  const typename Tag::S *__restrict__ tab,
                                                                  const typename Tag::S *__restrict__ tabl,
                                                                  typename Tag::S *__restrict__ y, KArgs a) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RP = G::RP, LDSW = G::LDSW, K1 = G::K1;
  static_assert(!HIER || WIN % 2 == 0, "the hierarchical form needs an even window");
  static_assert(LDSW % 4 == 0, "8- and 16-byte result writes");

  extern __shared__ __align__(16) unsigned char smem[];
  S *Ts = reinterpret_cast<S *>(smem + kFwdWaves * 16 * LDSW * Tag::ES);
  S *TB = Ts + G::TS_LEN;
  S *Tsl = TB + G::TB_LEN;  // hierarchical form only
  S *TBL = Tsl + G::TSL_LEN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  unsigned char *buf = smem + wave * 16 * LDSW * Tag::ES;  // this wave's sub-tile
  S *rowp = reinterpret_cast<S *>(buf);

  const uint32_t bid = die_major(blockIdx.x, gridDim.x);
  const int64_t c = bid / a.tiles_per_ch;
  const int64_t n0 = (int64_t)(bid - c * a.tiles_per_ch) * a.tile;
  const int nwin = (int)((n0 + a.tile <= a.N) ? a.tile : a.N - n0);
  const int spw = a.tile / (16 * kFwdWaves);  // sub-tiles per wave
  const int first = wave * spw;               // this wave's first sub-tile
  int nsub = (nwin - first * 16 + 15) / 16;   // its sub-tiles holding windows
  nsub = nsub < 0 ? 0 : (nsub > spw ? spw : nsub);

  // ---- 1. first sub-tile's rows in flight; the table (Toeplitz blocks of
  //         M_c for 16-bit, the table itself for float32) -> LDS
  TabRegs<Tag, WIN, HIER, kFwdThreads> tr;
  tab_load<Tag, WIN, REV, HIER, kFwdThreads>(tab, tabl, c, tid, tr);
  SubRows<Tag, WIN> nxt;
  if (nsub > 0) load_sub<Tag, WIN, TILED>(a, x, c, n0 + first * 16, nwin - first * 16, lane, nxt);
  fwd_tables<Tag, WIN, REV, HIER>(tr, Ts, TB, Tsl, TBL, tid);

  const int g = lane >> 4;   // lane group
  const int ln = lane & 15;  // row (A) / column (B, C) inside a 16x16 tile
  if constexpr (Tag::W16) {
    constexpr int S_ = G::S, NT = G::NT, NB = G::NB;
    auto load_bf = [&](int q) -> Frag { return fwd_bfrag<Tag, WIN>(TB, q, g, ln); };
    // ---- 3. pipeline over this wave's sub-tiles
    for (int j = 0; j < nsub; ++j) {
      const int64_t m0 = n0 + (first + j) * 16;
      const int mw = nwin - (first + j) * 16;  // windows left from m0
      write_sub<Tag, WIN>(buf, lane, nxt);
      if (j + 1 < nsub) load_sub<Tag, WIN, TILED>(a, x, c, m0 + 16, mw - 16, lane, nxt);
      Frag af[S_];
#pragma unroll
      for (int s = 0; s < S_; ++s)
        af[s] = *reinterpret_cast<const Frag *>(&rowp[ln * LDSW + s * 32 + 8 * g]);
      // The products are taken as (M^T X^T): the table fragment is the A
      // operand and the window-major fragment the B operand (the same
      // registers serve both roles), so a lane's four results are four
      // consecutive positions of one window and go to LDS as one 8-byte write.
      S *outq = rowp + ln * LDSW + 4 * g;
      // Output tiles t and t+1 use the even and the odd fragments: two
      // independent accumulation chains.  Walking t upwards, fragment q is
      // first needed at t = max(0, NT-1-q) (same parity) and last at
      // 2(S-1) + NT-1-q: it is read from LDS when first needed, so only about
      // 2S fragments are live at once.
      Frag bf[NB];
#pragma unroll
      for (int t0 = 0; t0 < NT; t0 += 2) {
#pragma unroll
        for (int q = 0; q < NB; ++q) {
          const int tf = NT - 1 - q;  // smallest t with this parity using q
          const int first_t = tf >= 0 ? tf : (((-tf) & 1) ? 1 : 0);
          if (first_t == t0 || first_t == t0 + 1) bf[q] = load_bf(q);
        }
        f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < S_; ++s) {
          acc0 = mma<Tag>(bf[2 * s - t0 + NT - 1], af[s], acc0);
          if (t0 + 1 < NT) acc1 = mma<Tag>(bf[2 * s - t0 - 1 + NT - 1], af[s], acc1);
          if constexpr (HIER) {
            // local sub-window blocks
            if (fwd_rows_meet<Tag, WIN>(s, t0, true)) acc0 = mma<Tag>(fwd_lfrag<Tag, WIN>(TBL, s, t0, g, ln), af[s], acc0);
            if (t0 + 1 < NT && fwd_rows_meet<Tag, WIN>(s, t0 + 1, true))
              acc1 = mma<Tag>(fwd_lfrag<Tag, WIN>(TBL, s, t0 + 1, g, ln), af[s], acc1);
          }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int t = t0 + h;
          if (t >= NT) continue;
          f32x4 acc = h ? acc1 : acc0;
          uint2 *o2 = reinterpret_cast<uint2 *>(outq + 16 * t);
          if constexpr (HIER) {
            // the two identity shortcuts: + 2 x at the output's own position,
            // read before the result overwrites it (pads hold zero)
            const uint2 xv = *o2;
            acc[0] += 2.f * to_f32<Tag>((u16)(xv.x & 0xffffu));
            acc[1] += 2.f * to_f32<Tag>((u16)(xv.x >> 16));
            acc[2] += 2.f * to_f32<Tag>((u16)(xv.y & 0xffffu));
            acc[3] += 2.f * to_f32<Tag>((u16)(xv.y >> 16));
          }
          *o2 = uint2{pack2<Tag>(acc[0], acc[1]), pack2<Tag>(acc[2], acc[3])};
        }
        // small windows: the window rows of output tiles t0 and t0+1 are
        // final; storing them now overlaps the stores with the products of
        // the next tiles (large windows store the sub-tile at the end, which
        // keeps their registers within three waves per SIMD)
        if constexpr (RP == 8) {
          wave_lds_sync();
          constexpr int RPT = 16 / RP;  // window rows per output tile
          const int v = lane & 15;
          const int hr = t0 * RPT + (lane >> 4);
          if ((lane >> 4) < 2 * RPT && hr < WIN && v < mw) {
            const Row<WIN, Tag::ES> r =
                TILED ? tiled_row<WIN, Tag::ES>(a, c, m0, v, hr) : row_of<WIN, Tag::ES>(a, y, c, m0 + v, hr);
            if (r.mode != kNone) {
              const uint32_t *l4 = reinterpret_cast<const uint32_t *>(buf + (v * LDSW + hr * RP) * Tag::ES);
              uint32_t dd[RowData<WIN, Tag::ES>::ND];
#pragma unroll
              for (int i = 0; i < RowData<WIN, Tag::ES>::ND; i += 4) {
                const uint4 u4 = *reinterpret_cast<const uint4 *>(l4 + i);
                dd[i] = u4.x; dd[i + 1] = u4.y; dd[i + 2] = u4.z; dd[i + 3] = u4.w;
              }
              store_row<WIN, Tag::ES>(y, r, dd);
            }
          }
        }
      }
      if constexpr (RP != 8) store_sub<Tag, WIN, TILED>(a, y, c, m0, mw, lane, buf);
    }
  } else {
    constexpr int S_ = G::S, NT = G::NT;
    for (int j = 0; j < nsub; ++j) {
      const int64_t m0 = n0 + (first + j) * 16;
      const int mw = nwin - (first + j) * 16;
      write_sub<Tag, WIN>(buf, lane, nxt);
      if (j + 1 < nsub) load_sub<Tag, WIN, TILED>(a, x, c, m0 + 16, mw - 16, lane, nxt);
      float af[S_];
#pragma unroll
      for (int s = 0; s < S_; ++s) af[s] = rowp[ln * LDSW + 4 * s + g];
      // (M^T X^T) as in the 16-bit path: four consecutive positions per lane
      float4 *outq = reinterpret_cast<float4 *>(rowp + ln * LDSW + 4 * g);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        const int pn = 16 * t + ln;
        const int ho = pn / RP, xo = pn % RP;
#pragma unroll
        for (int s = 0; s < S_; ++s) {
          const int k = 4 * s + g;
          const int hi = k / RP, xi = k % RP;
          const int dh = hi - ho;
          float bv = 0.f;
          if (xo < WIN && xi < WIN && dh >= -(WIN - 1) && dh <= WIN - 1)
            bv = Ts[(dh + WIN - 1) * K1 + xi - xo + WIN - 1];
          if constexpr (HIER) {
            // local sub-window entry and the two identity shortcuts
            constexpr int WL = G::WL, K1L = G::K1L;
            if (xo < WIN && xi < WIN && hi < WIN && ho < WIN && (hi < WL) == (ho < WL) && (xi < WL) == (xo < WL))
              bv += Tsl[(dh + WL - 1) * K1L + xi - xo + WL - 1];
            if (hi == ho && xi == xo && xi < WIN && hi < WIN) bv += 2.f;
          }
          acc = mma<Tag>(bv, af[s], acc);
        }
        outq[4 * t] = float4{acc[0], acc[1], acc[2], acc[3]};
      }
      store_sub<Tag, WIN, TILED>(a, y, c, m0, mw, lane, buf);
    }
  }
}

// ------------------------------------------------ forward, image layout
// 16-bit windows on maps that the windows tile, with NW (windows per band
// row) a power of two and a 16-window sub-tile that is either a run of whole
// bands inside one image (NH * NW a multiple of 16) or a run of whole images
// (NH * NW divides 16).  A band is w contiguous image rows and the bands of
// one image are contiguous, so a sub-tile is at most a few contiguous pieces
// of memory: it moves with 16-byte loads and stores at consecutive addresses,
// keeps its image layout in LDS, and the per-lane addressing is fixed for the
// whole launch.  The products are those of the row kernel (same fragments,
// same order); A operands are read as dwords and realigned by 16 bits where a
// window row starts at an odd element, and results are written back into the
// image copy (pads never), whose finished rows are stored while the next
// output tiles are multiplied.
struct ImgArgs {
  int64_t chw;    // elements between consecutive images of a channel (C*H*W)
  int64_t hw;     // elements of one image (H*W)
  int W;          // image width
  int BE;         // elements of one band (w * W)
  int lgnw;       // log2(NW)
  int NH;         // bands per image
  int WPI;        // windows per image (NH * NW)
  int whole;      // 1: a sub-tile is 16 / WPI whole images
  int SEGC;       // 16-byte chunks per contiguous piece (an image, or the sub-tile)
  float inv_segc; // 1 / SEGC when whole, else 0
  int CPR;        // chunks per band in the rows of one output-tile pair
  float inv_cpr;  // 1 / CPR
  float inv_nh;   // 1 / NH
  uint32_t gap;   // bytes from the end of one piece to the start of the next (2 chw - 16 SEGC; 0 unless whole)
  int pair_store; // 1: rows are stored per output-tile pair, else per sub-tile
};

template <int WIN>
struct ImgCfg {
  static constexpr int ELEMS = 16 * WIN * WIN;              // elements of one sub-tile
  static constexpr int CH = ELEMS / 8;                      // its 16-byte chunks
  static constexpr int KC = cdiv(CH, 64);                   // chunks per lane
  static constexpr int DUMMY = ELEMS + 8;                   // element that takes masked writes
  static constexpr int BUF_BYTES = rup((ELEMS + 16) * 2, 16);  // + read overrun and dummy slot
  static constexpr int RPP = rp_of(WIN) == 8 ? 4 : 2;       // window rows per output-tile pair
};

template <class Tag, int WIN, bool HIER = false>
__host__ __device__ constexpr size_t fwd_img_lds_bytes() {
  typedef FwdCfg<Tag, WIN> G;
  return (size_t)kFwdWaves * ImgCfg<WIN>::BUF_BYTES + (size_t)(G::TS_LEN + G::TB_LEN) * Tag::ES +
         (HIER ? (size_t)(G::TSL_LEN + G::TBL_LEN) * Tag::ES : 0);
}

// Byte offset of chunk q of a sub-tile from the sub-tile's first element
// (pieces of a sub-tile lie within 2^31 bytes of each other; the host checks
// it); 0x7fffffff past the sub-tile's last chunk, unless INSIDE (q < nch
// known).  Offsets of the chunks of missing pieces (a partial last sub-tile)
// are at least nseg * chw * 2.  inv_segc is 0 for a one-piece sub-tile, so
// seg is 0 there.
template <bool INSIDE>
__device__ __attribute__((always_inline)) inline uint32_t img_chunk(const ImgArgs &ia, int q, int nch) {
  const int seg = fdiv_small(q, ia.inv_segc);  // q < 2^22
  const uint32_t off = 16u * (uint32_t)q + (uint32_t)seg * ia.gap;
  return (INSIDE || q < nch) ? off : 0x7fffffffu;
}

// HIER: the hierarchical form (WIN = 2 wl, local table tabl): the local
// sub-window blocks are extra products where input and output rows lie in
// the same half of the window, and the two identity shortcuts add 2 x in
// float32 before the single rounding.
template <class Tag, int WIN, bool REV, bool HIER = false>
__global__ __launch_bounds__(kFwdThreads, 3) void wbmm_fwd_img_kernel(const typename Tag::S *__restrict__ x,
                                                                      const typename Tag::S *__restrict__ tab,
                                                                      const typename Tag::S *__restrict__ tabl,
                                                                      typename Tag::S *__restrict__ y, KArgs a,
                                                                      ImgArgs ia) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef FwdCfg<Tag, WIN> G;
  typedef ImgCfg<WIN> IC;
  static_assert(Tag::W16, "image layout: 16-bit");
  static_assert(!HIER || WIN % 2 == 0, "the hierarchical form needs an even window");
  constexpr int RP = G::RP, S_ = G::S, NT = G::NT, NB = G::NB, KC = IC::KC, RPP = IC::RPP;

  extern __shared__ __align__(16) unsigned char smem[];
  S *Ts = reinterpret_cast<S *>(smem + kFwdWaves * IC::BUF_BYTES);
  S *TB = Ts + G::TS_LEN;
  S *Tsl = TB + G::TB_LEN;  // hierarchical form only
  S *TBL = Tsl + G::TSL_LEN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: the sub-tile bases go to scalar registers
  u16 *raw = reinterpret_cast<u16 *>(smem + wave * IC::BUF_BYTES);  // this wave's sub-tile, image layout
  const uint32_t *raw32 = reinterpret_cast<const uint32_t *>(raw);

  const uint32_t bid = die_major(blockIdx.x, gridDim.x);
  const int64_t c = bid / a.tiles_per_ch;
  const int64_t n0 = (int64_t)(bid - c * a.tiles_per_ch) * a.tile;
  const int nwin = (int)((n0 + a.tile <= a.N) ? a.tile : a.N - n0);
  const int spw = a.tile / (16 * kFwdWaves);
  const int first = wave * spw;
  int nsub = (nwin - first * 16 + 15) / 16;
  nsub = nsub < 0 ? 0 : (nsub > spw ? spw : nsub);

  // per-lane addressing, fixed for the launch (the chunk offsets are
  // recomputed where used rather than held in registers)
  auto chunk_off = [&](int k) -> uint32_t {
    int l = lane;
    asm volatile("" : "+v"(l));
    // (k is a constant of the unrolled loops: chunks of the first CH / 64
    // rounds lie inside the sub-tile)
    return 64 * (k + 1) <= IC::CH ? img_chunk<true>(ia, l + 64 * k, IC::CH) : img_chunk<false>(ia, l + 64 * k, IC::CH);
  };
  const int g = lane >> 4;
  const int ln = lane & 15;
  const int nwm = (1 << ia.lgnw) - 1;
  const int abase = (ln >> ia.lgnw) * ia.BE + (ln & nwm) * WIN;  // window ln of the sub-tile in LDS
  // store task of this lane per output-tile pair: band jj, chunk i of its rows
  const int sjj = fdiv_small(lane, ia.inv_cpr);
  const int si = lane - sjj * ia.CPR;
  const int sseg = ia.whole ? fdiv_small(sjj, ia.inv_nh) : 0;
  const uint32_t soff = (uint32_t)sseg * (uint32_t)(2 * ia.chw) + 2u * (uint32_t)((sjj - sseg * ia.NH) * ia.BE + 8 * si);
  const int sloff = sjj * ia.BE + 8 * si;

  // element offset of the first element of sub-tile m0, the byte bound of
  // its chunk offsets and its band count
  auto sub_base = [&](int64_t m0, uint32_t &lim, int &nb) -> int64_t {
    const int mi = (int)m0;
    const int img = mi / ia.WPI;
    const int inw = mi - img * ia.WPI;
    const int64_t left = a.N - m0;
    const int nw = left < 16 ? (int)left : 16;
    lim = ia.whole ? (uint32_t)(nw / ia.WPI) * (uint32_t)(2 * ia.chw) : 0x7fffffffu;
    nb = nw >> ia.lgnw;
    return (int64_t)img * ia.chw + c * ia.hw + (int64_t)(inw >> ia.lgnw) * ia.BE;
  };
  // sub-tile m0 into v, zero past its end (none at all unless any): buffer
  // loads over the sub-tile's byte range, whose range check returns zero for
  // the chunks beyond it without touching memory, so no lane is masked and
  // the waits on these loads are counted exactly (chunk offsets are below
  // 2^31; the host checks it)
  auto load = [&](int64_t m0, bool any, uint4 (&v)[KC]) {
    uint32_t lim;
    int nb;
    const int64_t base = sub_base(any ? m0 : n0, lim, nb);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<S *>(x + base), 0, any ? (int)lim : 0, kBufWord3);
#pragma unroll
    for (int k = 0; k < KC; ++k)
      v[k] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)chunk_off(k), 0, 0));
  };

  // the table loads go first and the input rows right behind them; the
  // table's copy to LDS and the Toeplitz blocks are built while the rows are
  // in flight
  TabRegs<Tag, WIN, HIER, kFwdThreads> tr;
  tab_load<Tag, WIN, REV, HIER, kFwdThreads>(tab, tabl, c, tid, tr);
  uint4 nxt[KC];
  load(n0 + first * 16, nsub > 0, nxt);
  fwd_tables<Tag, WIN, REV, HIER>(tr, Ts, TB, Tsl, TBL, tid);

  for (int j = 0; j < nsub; ++j) {
    const int64_t m0 = n0 + (first + j) * 16;
    uint32_t lim;
    int nb;
    char *dst = reinterpret_cast<char *>(y + sub_base(m0, lim, nb));
    wave_lds_sync();
#pragma unroll
    for (int k = 0; k < KC; ++k) {
      const int q = lane + 64 * k;
      if (q < IC::CH) *reinterpret_cast<uint4 *>(raw + 8 * q) = nxt[k];
    }
    if (j + 1 < nsub) load(m0 + 16, true, nxt);
    wave_lds_sync();
    // LDS addresses derived from ab are recomputed per sub-tile rather than
    // held in registers across the loop
    int ab = abase;
    asm volatile("" : "+v"(ab));
    // B operand of K step s (the window-major fragment): window ln, 8
    // consecutive positions of one window row, read as dwords from its image
    // copy and shifted by one element when the row starts at an odd element
    Frag af[S_];
#pragma unroll
    for (int s = 0; s < S_; ++s) {
      const int r = RP == 8 ? 4 * s + g : 2 * s + (g >> 1);  // window row
      const int x0 = RP == 8 ? 0 : 8 * (g & 1);              // first column
      const bool rok = r < WIN;
      const int e0 = ab + (rok ? r : 0) * ia.W + x0;
      const uint32_t *p = raw32 + (e0 >> 1);
      // (an even window tiles an even image width, so its rows start at
      // even elements: no shift)
      const uint32_t sh = (WIN & 1) ? (uint32_t)(e0 & 1) * 16u : 0u;
      uint32_t d[5];
#pragma unroll
      for (int i = 0; i < 5; ++i) d[i] = p[i];
      uint32_t u[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t v = __builtin_amdgcn_alignbit(d[i + 1], d[i], sh);
        // columns x0 + 2i, x0 + 2i + 1 beyond the window are zero pads
        const int xa = x0 + 2 * i;
        v = xa >= WIN ? 0u : (xa + 1 >= WIN ? (v & 0xffffu) : v);
        u[i] = rok ? v : 0u;
      }
      af[s] = __builtin_bit_cast(Frag, make_uint4(u[0], u[1], u[2], u[3]));
    }
    // stores rows [r0, r1) of every band of the sub-tile
    auto store_rows = [&](int r0, int r1) {
      const int cpr = (r1 - r0) * ia.W / 8;
      if (si < cpr && sjj < nb) {
        const uint4 val = *reinterpret_cast<const uint4 *>(raw + sloff + r0 * ia.W);
        *reinterpret_cast<uint4 *>(dst + soff + 2u * (uint32_t)(r0 * ia.W)) = val;
      }
    };
    // output tiles per step: a pair, or one in the hierarchical form (whose
    // local fragments leave no registers for a second accumulator chain);
    // each tile takes the same products in the same order either way
    constexpr int TS = HIER ? 1 : 2;
    // 16-position rows and an even window: output tile t is window row t,
    // so each of the lane's two result dwords moves down one image row per
    // tile (byte offsets in raw, advanced per tile); one whose columns lie
    // past the window stays on the dummy element
    constexpr bool STEP = RP == 16 && (WIN & 1) == 0;
    uint32_t pa = 0, pb = 0, sa = 0, sb = 0;
    if constexpr (STEP) {
      const int xo0 = 4 * g;
      const bool va = xo0 < WIN, vb = xo0 + 2 < WIN;
      pa = 2u * (uint32_t)(va ? ab + xo0 : IC::DUMMY);
      pb = 2u * (uint32_t)(vb ? ab + xo0 + 2 : IC::DUMMY);
      sa = va ? 2u * (uint32_t)ia.W : 0u;
      sb = vb ? 2u * (uint32_t)ia.W : 0u;
    }
    Frag bf[NB];
#pragma unroll
    for (int t0 = 0; t0 < NT; t0 += TS) {
#pragma unroll
      for (int q = 0; q < NB; ++q) {
        const int tf = NT - 1 - q;
        const int first_t = tf >= 0 ? tf : (((-tf) & 1) ? 1 : 0);
        if (first_t == t0 || (TS == 2 && first_t == t0 + 1)) bf[q] = fwd_bfrag<Tag, WIN>(TB, q, g, ln);
      }
      f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < S_; ++s) {
        acc0 = mma<Tag>(bf[2 * s - t0 + NT - 1], af[s], acc0);
        if (TS == 2 && t0 + 1 < NT) acc1 = mma<Tag>(bf[2 * s - t0 - 1 + NT - 1], af[s], acc1);
        if constexpr (HIER) {
          // local sub-window blocks
          if (fwd_rows_meet<Tag, WIN>(s, t0, true)) acc0 = mma<Tag>(fwd_lfrag<Tag, WIN>(TBL, s, t0, g, ln), af[s], acc0);
          if (TS == 2 && t0 + 1 < NT && fwd_rows_meet<Tag, WIN>(s, t0 + 1, true))
            acc1 = mma<Tag>(fwd_lfrag<Tag, WIN>(TBL, s, t0 + 1, g, ln), af[s], acc1);
        }
      }
      // results (M^T X^T): window ln, positions 16 t + 4 g .. + 3, i.e. one
      // window row ho, columns xo0 .. xo0 + 3; columns and rows beyond the
      // window go to the dummy element
#pragma unroll
      for (int h = 0; h < TS; ++h) {
        const int t = t0 + h;
        if (t >= NT) continue;
        const f32x4 acc = h ? acc1 : acc0;
        const int ho = RP == 8 ? 2 * t + (g >> 1) : t;
        const int xo0 = RP == 8 ? 4 * (g & 1) : 4 * g;
        const int o = ab + (ho < WIN ? ho : 0) * ia.W + xo0;
        if constexpr (STEP) {
          uint32_t *wa = reinterpret_cast<uint32_t *>(reinterpret_cast<unsigned char *>(raw) + pa);
          uint32_t *wb = reinterpret_cast<uint32_t *>(reinterpret_cast<unsigned char *>(raw) + pb);
          f32x4 r = acc;
          if constexpr (HIER) {
            // the two identity shortcuts: + 2 x at the output's own
            // position, read before the result overwrites it
            const uint32_t xa = *wa, xb = *wb;
            r[0] += 2.f * to_f32<Tag>((u16)(xa & 0xffffu));
            r[1] += 2.f * to_f32<Tag>((u16)(xa >> 16));
            r[2] += 2.f * to_f32<Tag>((u16)(xb & 0xffffu));
            r[3] += 2.f * to_f32<Tag>((u16)(xb >> 16));
          }
          *wa = pack2<Tag>(r[0], r[1]);
          *wb = pack2<Tag>(r[2], r[3]);
          pa += sa;
          pb += sb;
        } else if constexpr ((WIN & 1) == 0) {
          // even windows: every window row starts at an even element
          uint32_t *o32 = reinterpret_cast<uint32_t *>(raw);
          const int da = (ho < WIN && xo0 < WIN) ? o : IC::DUMMY;
          const int db = (ho < WIN && xo0 + 2 < WIN) ? o + 2 : IC::DUMMY;
          f32x4 r = acc;
          if constexpr (HIER) {
            // the two identity shortcuts: + 2 x at the output's own
            // position, read before the result overwrites it
            const uint32_t xa = o32[da >> 1], xb = o32[db >> 1];
            r[0] += 2.f * to_f32<Tag>((u16)(xa & 0xffffu));
            r[1] += 2.f * to_f32<Tag>((u16)(xa >> 16));
            r[2] += 2.f * to_f32<Tag>((u16)(xb & 0xffffu));
            r[3] += 2.f * to_f32<Tag>((u16)(xb >> 16));
          }
          o32[da >> 1] = pack2<Tag>(r[0], r[1]);
          o32[db >> 1] = pack2<Tag>(r[2], r[3]);
        } else {
          const uint32_t lo = pack2<Tag>(acc[0], acc[1]);
          const uint32_t hi = pack2<Tag>(acc[2], acc[3]);
          const u16 vals[4] = {(u16)(lo & 0xffffu), (u16)(lo >> 16), (u16)(hi & 0xffffu), (u16)(hi >> 16)};
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) raw[(ho < WIN && xo0 + rr < WIN) ? o + rr : IC::DUMMY] = vals[rr];
        }
      }
      // rows are stored per output-tile pair, once both tiles are written
      if (ia.pair_store && (TS == 2 || (t0 & 1) || t0 + 1 >= NT)) {
        wave_lds_sync();
        const int r0 = RPP * (t0 / 2);
        const int r1 = r0 + RPP < WIN ? r0 + RPP : WIN;
        if (r0 < WIN) store_rows(r0, r1);
      }
    }
    if (!ia.pair_store) {
      wave_lds_sync();
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        const uint32_t off = chunk_off(k);
        if (off < lim) *reinterpret_cast<uint4 *>(dst + off) = *reinterpret_cast<const uint4 *>(raw + 8 * (lane + 64 * k));
      }
    }
  }
}

// ===================================================== table gradient

template <class Tag, int WIN>
struct DtCfg {
  static constexpr int RP = rp_of(WIN);
  static constexpr int PP = WIN * RP;
  static constexpr int NPT = cdiv(PP, 16);        // 16-position tiles
  static constexpr int KR = cdiv(NPT * 16, RP);   // rows per staged window
  static constexpr int R = 16 / RP;               // window rows per tile
  static constexpr int CW = Tag::W16 ? 32 : 16;   // windows per LDS stage
  // window-major staging, as in the forward, with a row pitch (elements) that
  // keeps the fragment reads free of bank conflicts: 16-bit transposing reads
  // of 4 windows x 16 positions; float32 reads of 4 windows x 16 positions
  static constexpr int LDSW = Tag::W16 ? NPT * 16 + 8 : NPT * 16 + ((16 - NPT * 16) % 64 + 64) % 64;
  static constexpr int BUF = CW * LDSW * Tag::ES;  // bytes per operand buffer
  static constexpr int NACC = 2 * NPT - 1;        // accumulators: pi - po
  static constexpr int K1 = 2 * WIN - 1;
  static constexpr int K2 = K1 * K1;
  static constexpr int NBT = (2 * R - 1) * K1;    // bins per accumulator tile
  static constexpr int ROWS = 2 * CW * KR;        // row copies per stage (x and dy)
  static constexpr int RPT = cdiv(ROWS, kThreads);  // row copies per thread
};

// Staging of the fused backward: the table gradient's stages, with enough
// padded rows (zero beyond the window) for both readers of the tile: the
// input-gradient products (K over KP positions) and the table-gradient tiles
// (NPT * 16 positions); the forward's row pitch when it holds them.
// LDS: [x stage][dy stage][table row][Toeplitz blocks (16-bit)].
template <class Tag, int WIN>
struct BwdCfg {
  typedef DtCfg<Tag, WIN> T;
  typedef FwdCfg<Tag, WIN> F;
  static constexpr int RP = T::RP, NPT = T::NPT, R = T::R, CW = T::CW;
  static constexpr int NACC = T::NACC, K1 = T::K1, K2 = T::K2, NBT = T::NBT;
  static constexpr int KR = F::KR > T::KR ? F::KR : T::KR;
  static constexpr int LDSW = F::LDSW >= KR * RP ? F::LDSW : T::LDSW;
  static constexpr int BUF = CW * LDSW * Tag::ES;
  static constexpr int ROWS = 2 * CW * KR;
  static constexpr int RPT = cdiv(ROWS, kThreads);
  static constexpr int SUBS = CW / 16;            // input-gradient sub-tiles per stage
  static constexpr int WPS = kWaves / SUBS;       // waves per sub-tile
  static constexpr int TS_OFF = 2 * BUF;
  static constexpr int TB_OFF = TS_OFF + rup(F::TS_LEN * Tag::ES, 16);
  static constexpr int TAB_END = TB_OFF + F::TB_LEN * Tag::ES;
  static_assert(KR * RP <= LDSW && NPT * 16 <= LDSW, "staged rows must fit the pitch");
};

// Accumulator tiles are split among the waves in contiguous ranges of
// P = pi - po (tile P carries NPT - |P| block products per K step), the
// ranges chosen to balance that work.  With a contiguous range, the B
// fragment of output tile po is live only while pi runs over po + [lo, hi].
struct PRange {
  int lo[kWaves];
  int hi[kWaves];
};

template <int NPT>
__host__ __device__ constexpr PRange make_prange() {
  constexpr int n = 2 * NPT - 1;  // P = -(NPT-1) .. NPT-1
  int work[n] = {};
  for (int i = 0; i < n; ++i) {
    const int P = i - (NPT - 1);
    work[i] = NPT - (P < 0 ? -P : P);
  }
  int pre[n + 1] = {};
  for (int i = 0; i < n; ++i) pre[i + 1] = pre[i] + work[i];
  // cut points 0 <= c1 <= c2 <= c3 <= n minimising the largest share
  int best = 1 << 30, b1 = 0, b2 = 0, b3 = 0;
  for (int c1 = 0; c1 <= n; ++c1)
    for (int c2 = c1; c2 <= n; ++c2)
      for (int c3 = c2; c3 <= n; ++c3) {
        int m = pre[c1];
        if (pre[c2] - pre[c1] > m) m = pre[c2] - pre[c1];
        if (pre[c3] - pre[c2] > m) m = pre[c3] - pre[c2];
        if (pre[n] - pre[c3] > m) m = pre[n] - pre[c3];
        if (m < best) { best = m; b1 = c1; b2 = c2; b3 = c3; }
      }
  PRange r{};
  const int cut[kWaves + 1] = {0, b1, b2, b3, n};
  for (int w = 0; w < kWaves; ++w) {
    r.lo[w] = cut[w] - (NPT - 1);
    r.hi[w] = cut[w + 1] - 1 - (NPT - 1);  // hi < lo: the wave owns nothing
  }
  return r;
}

// Largest number of accumulator tiles a wave owns.
template <int NPT>
__host__ __device__ constexpr int max_tiles_per_wave() {
  constexpr PRange r = make_prange<NPT>();
  int m = 1;
  for (int w = 0; w < kWaves; ++w)
    if (r.hi[w] - r.lo[w] + 1 > m) m = r.hi[w] - r.lo[w] + 1;
  return m;
}

// The accumulator tiles of one wave: P = lo .. lo + np - 1.
template <int NPT, int WAVE>
struct PSpan {
  static constexpr PRange PR = make_prange<NPT>();
  static constexpr int lo = PR.lo[WAVE];
  static constexpr int np = PR.hi[WAVE] - PR.lo[WAVE] + 1;  // may be 0
  static constexpr int hi = lo + np - 1;
  static constexpr int na = np > 0 ? np : 1;                // array length
};

template <class G>
__host__ __device__ constexpr size_t bins_lds_bytes() {
  return (size_t)(kWaves * max_tiles_per_wave<G::NPT>() * 272 + G::NACC * G::NBT) * 4;
}

template <class Tag, int WIN>
__host__ __device__ constexpr size_t dt_lds_bytes() {
  typedef DtCfg<Tag, WIN> G;
  const size_t ops = 2 * (size_t)G::BUF;
  const size_t bins = bins_lds_bytes<G>();
  return ops > bins ? ops : bins;
}

template <class Tag, int WIN>
__host__ __device__ constexpr size_t bwd_lds_bytes() {
  typedef BwdCfg<Tag, WIN> G;
  const size_t ops = (size_t)G::TAB_END;
  const size_t bins = bins_lds_bytes<G>();
  return ops > bins ? ops : bins;
}

// Row copies of one stage: task q covers tensor (q / (CW * KR)), window
// (q / KR) % CW of the stage and padded row q % KR (rows >= w are zero).
// Fixed-offset rows take another mapping: copy k covers tensor k / SUBS and
// sub-tile k % SUBS (SUBS = CW / 16), thread tid its window tid / KR and
// padded row tid % KR, so that every copy instruction has one base address.
template <class G>
__host__ __device__ constexpr int tiled_rpt() { return 2 * (G::CW / 16); }

template <class Tag, int WIN, class G>
struct Stage {
  static constexpr int N = G::RPT > tiled_rpt<G>() ? G::RPT : tiled_rpt<G>();
  RowData<WIN, Tag::ES> rd[N];
};

template <class Tag, int WIN, class G, bool TILED>
__device__ __attribute__((always_inline)) inline void stage_load(const KArgs &a, const void *x, const void *dy,
                                                                  int64_t c, int64_t m0, int64_t m1, int tid,
                                                                  Stage<Tag, WIN, G> &st) {
  if constexpr (TILED) {
    // fixed-offset rows: whole and dword-aligned; one base address per copy
    constexpr int NDV = (WIN * Tag::ES) / 4, SUBS = G::CW / 16;
    typedef typename Tag::S S;
    const int vv = tid / G::KR;
    const int hi = tid - vv * G::KR;
    const uint32_t off = tiled_row_off<WIN, Tag::ES>(a, vv & 15, hi);
#pragma unroll
    for (int k = 0; k < tiled_rpt<G>(); ++k) {
      const int tens = k / SUBS, sub = k % SUBS;
#pragma unroll
      for (int i = 0; i < RowData<WIN, Tag::ES>::ND; ++i) st.rd[k].d[i] = 0;
      const int64_t ms = m0 + 16 * sub;
      if (vv < 16 && hi < WIN && ms + vv < m1) {
        const S *src = tens ? reinterpret_cast<const S *>(dy) : reinterpret_cast<const S *>(x);
        const uint32_t *p4 = reinterpret_cast<const uint32_t *>(
            reinterpret_cast<const char *>(src + tiled_sub_base(a, c, ms)) + off);
#pragma unroll
        for (int i = 0; i + 4 <= NDV; i += 4) {
          const u32x4a u = *reinterpret_cast<const u32x4a *>(p4 + i);
          st.rd[k].d[i] = u.x; st.rd[k].d[i + 1] = u.y; st.rd[k].d[i + 2] = u.z; st.rd[k].d[i + 3] = u.w;
        }
#pragma unroll
        for (int i = NDV & ~3; i < NDV; ++i) st.rd[k].d[i] = p4[i];
      }
    }
    return;
  }
#pragma unroll
  for (int k = 0; k < G::RPT; ++k) {
    const int q = tid + k * kThreads;
    const int tens = q / (G::CW * G::KR);
    const int rem = q - tens * (G::CW * G::KR);
    const int v = rem / G::KR;
    const int hi = rem - v * G::KR;
    const void *src = tens ? dy : x;
    Row<WIN, Tag::ES> r;
    r.cols = 0; r.eoff = 0; r.mode = kNone; r.odd = 0;
    if (q < G::ROWS && m0 + v < m1) r = row_of<WIN, Tag::ES>(a, src, c, m0 + v, hi);
    load_row<WIN, Tag::ES>(src, r, st.rd[k]);
  }
}

// Write a loaded stage window-major (padded rows, as in the forward tile).
template <class Tag, int WIN, class G, bool TILED>
__device__ __attribute__((always_inline)) inline void stage_write(unsigned char *smem, int tid,
                                                                   const Stage<Tag, WIN, G> &st) {
  typedef RowData<WIN, Tag::ES> RD;
  if constexpr (TILED) {
    constexpr int SUBS = G::CW / 16;
    const int vv = tid / G::KR;
    const int hi = tid - vv * G::KR;
    if (vv < 16) {
#pragma unroll
      for (int k = 0; k < tiled_rpt<G>(); ++k) {
        const int tens = k / SUBS, sub = k % SUBS;
        uint32_t *l4 = reinterpret_cast<uint32_t *>(smem + tens * G::BUF +
                                                    ((16 * sub + vv) * G::LDSW + hi * G::RP) * Tag::ES);
#pragma unroll
        for (int i = 0; i < RD::ND; i += 4)
          *reinterpret_cast<uint4 *>(l4 + i) = make_uint4(st.rd[k].d[i], st.rd[k].d[i + 1], st.rd[k].d[i + 2], st.rd[k].d[i + 3]);
      }
    }
    return;
  }
#pragma unroll
  for (int k = 0; k < G::RPT; ++k) {
    const int q = tid + k * kThreads;
    if (q >= G::ROWS) continue;
    const int tens = q / (G::CW * G::KR);
    const int rem = q - tens * (G::CW * G::KR);
    const int v = rem / G::KR;
    const int hi = rem - v * G::KR;
    uint32_t *l4 = reinterpret_cast<uint32_t *>(smem + tens * G::BUF + (v * G::LDSW + hi * G::RP) * Tag::ES);
#pragma unroll
    for (int i = 0; i < RD::ND; i += 4)
      *reinterpret_cast<uint4 *>(l4 + i) = make_uint4(st.rd[k].d[i], st.rd[k].d[i + 1], st.rd[k].d[i + 2], st.rd[k].d[i + 3]);
  }
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Matrix-core fragment of a position-major view of a window-major stage
// (16-bit): lane (g, i) receives the 8 values of positions 16 * pt + i for
// windows 8g .. 8g + 7, by two transposing LDS reads.  Within a 16-lane group
// the transposing read hands lane i the i-th column of the 4 x 16 block whose
// row r is the 4-element chunks of lanes 4r .. 4r + 3; lane 4r + q points at
// window 8g + r (+4), positions 16 * pt + 4q .. + 3.
template <int LDSW>
__device__ __attribute__((always_inline)) inline u16x8 dt_frag16(const unsigned char *buf, int pt, int lane) {
  const int g = lane >> 4;
  const int i = lane & 15;
  const int r = i >> 2, q = i & 3;
  // K index 8 g + 4 h + r (h: first or second read) takes window
  // 8 g + 2 r + h: the same permutation of the stage's windows for both
  // operands leaves X^T dY unchanged, and with it the eight windows that one
  // read cycle serves (lanes of g and g + 1) fall in distinct LDS banks (64
  // banks for reads) at a row pitch of 232 elements (w = 14); the identity
  // order put windows r and r + 8 ... on the same banks
  const int e0 = (8 * g + 2 * r) * LDSW + 16 * pt + 4 * q;
  lds_i16x4 *p0 = (lds_i16x4 *)(buf + 2 * e0);
  lds_i16x4 *p1 = (lds_i16x4 *)(buf + 2 * (e0 + LDSW));
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p0);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(p1);
  return __builtin_bit_cast(u16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// This wave's share of X^T dY for one stage (K = the stage's windows).  With
// HL > 0 (hierarchical form, local window HL, one window row per tile) the
// products of tile pairs whose rows lie in the same half of the window go to
// accl instead of acc: acc + accl is the global table's tile, accl alone
// holds every pair of the local table (the same products, none added).
template <class Tag, class G, int WAVE, int HL>
__device__ __attribute__((always_inline)) inline void dt_products_split(const unsigned char *Xt,
                                                                         const unsigned char *Dt,
                                                                         f32x4 (&acc)[PSpan<G::NPT, WAVE>::na],
                                                                         f32x4 (&accl)[PSpan<G::NPT, WAVE>::na],
                                                                         int lane) {
  static_assert(HL == 0 || G::R == 1, "local halves need one window row per tile");
  typedef typename Tag::Frag Frag;
  typedef PSpan<G::NPT, WAVE> SP;
  constexpr int NPT = G::NPT, CW = G::CW;
  constexpr int PLO = SP::lo, NP = SP::np, PHI = SP::hi;
  const int g = lane >> 4;
  const int ln = lane & 15;
  if constexpr (NP > 0) {
    if constexpr (Tag::W16) {
      Frag bf[NPT];
#pragma unroll
      for (int pi = 0; pi < NPT; ++pi) {
        // B fragments first needed at this pi: po with max(0, po + PLO) == pi
#pragma unroll
        for (int po = 0; po < NPT; ++po) {
          const bool used = po + PHI >= 0 && po + PLO <= NPT - 1;
          if (used && (po + PLO > 0 ? po + PLO : 0) == pi) bf[po] = dt_frag16<G::LDSW>(Dt, po, lane);
        }
        const Frag af = dt_frag16<G::LDSW>(Xt, pi, lane);
#pragma unroll
        for (int j = 0; j < NP; ++j) {
          const int po = pi - (PLO + j);
          if (po >= 0 && po < NPT) {
            if (HL > 0 && (pi < HL) == (po < HL)) accl[j] = mma<Tag>(af, bf[po], accl[j]);
            else acc[j] = mma<Tag>(af, bf[po], acc[j]);
          }
        }
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < CW / 4; ++ks) {
        float bf[NPT];
#pragma unroll
        for (int pi = 0; pi < NPT; ++pi) {
#pragma unroll
          for (int po = 0; po < NPT; ++po) {
            const bool used = po + PHI >= 0 && po + PLO <= NPT - 1;
            if (used && (po + PLO > 0 ? po + PLO : 0) == pi)
              bf[po] = reinterpret_cast<const float *>(Dt)[(4 * ks + g) * G::LDSW + 16 * po + ln];
          }
          const float af = reinterpret_cast<const float *>(Xt)[(4 * ks + g) * G::LDSW + 16 * pi + ln];
#pragma unroll
          for (int j = 0; j < NP; ++j) {
            const int po = pi - (PLO + j);
            if (po >= 0 && po < NPT) {
              if (HL > 0 && (pi < HL) == (po < HL)) accl[j] = mma<Tag>(af, bf[po], accl[j]);
              else acc[j] = mma<Tag>(af, bf[po], acc[j]);
            }
          }
        }
      }
    }
  }
}

template <class Tag, class G, int WAVE>
__device__ __attribute__((always_inline)) inline void dt_products(const unsigned char *Xt, const unsigned char *Dt,
                                                                   f32x4 (&acc)[PSpan<G::NPT, WAVE>::na], int lane) {
  dt_products_split<Tag, G, WAVE, 0>(Xt, Dt, acc, acc, lane);
}

// Diagonal binning of one wave's accumulator tiles, in two halves: the
// tiles go to this wave's scratch (scr) and the bins are summed from it into
// binsum.  No workgroup barrier inside; the halves are separated by a wave
// barrier (dt_bin) or by anything that orders the wave's LDS accesses.
template <class G>
__host__ __device__ constexpr int bin_tiles_per_wave() { return max_tiles_per_wave<G::NPT>(); }
constexpr int kBinTile = 272;  // floats per tile (16 rows of 17, or of 16 for one-row tiles)

template <class Tag, int WIN, class G, int WAVE>
__device__ __attribute__((always_inline)) inline void dt_bin_write(const f32x4 (&acc)[PSpan<G::NPT, WAVE>::na],
                                                                    float *scr) {
  typedef PSpan<G::NPT, WAVE> SP;
  constexpr int R = G::R, NP = SP::np, TSTR = kBinTile;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int ln = lane & 15;
  if constexpr (R == 1) {
    // One window row per tile (RP = 16): a bin is one diagonal dw = xi - xo
    // of the 16 x 16 tile.  The tile is written skewed, element (xi, xo) at
    // column (xo - xi) mod 16 of row xi, so that column s holds diagonal -s
    // in rows 0 .. 15-s and diagonal 16-s in the rows below; a lane sums one
    // column of one tile, top to bottom (the order of the general path).
    // Pad positions (xi or xo >= WIN) are written as zero.  Row xi is
    // stored at row 4 (xi / 4) + (xi + xi / 4) % 4 (pitch 16), so that the
    // four 16-lane groups of a write (xi = 4 g + rr) fall on four different
    // 16-bank groups.
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int xi = 4 * g + rr;
      float *row = scr + (4 * g + ((rr + g) & 3)) * 16 + ((ln - xi) & 15);
      const bool ok = xi < WIN && ln < WIN;
#pragma unroll
      for (int j = 0; j < NP; ++j) row[j * TSTR] = ok ? acc[j][rr] : 0.f;
    }
  } else {
#pragma unroll
    for (int j = 0; j < NP; ++j) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) scr[j * TSTR + (4 * g + rr) * 17 + ln] = acc[j][rr];
    }
  }
}

template <class Tag, int WIN, class G, int WAVE>
__device__ __attribute__((always_inline)) inline void dt_bin_sum(const float *scr, float *binsum) {
  typedef PSpan<G::NPT, WAVE> SP;
  constexpr int NPT = G::NPT, RP = G::RP, R = G::R;
  constexpr int K1 = G::K1, NBT = G::NBT;
  constexpr int PLO = SP::lo, NP = SP::np, TSTR = kBinTile;
  const int lane = threadIdx.x & 63;
  if constexpr (R == 1) {
    const int s = lane & 15;
#pragma unroll
    for (int it = 0; it < cdiv(NP * 16, 64); ++it) {
      const int j = (lane >> 4) + 4 * it;
      if (j < NP) {
        const float *col = scr + j * TSTR + s;
        float lo = 0.f, hi = 0.f;
#pragma unroll
        for (int xi = 0; xi < 16; ++xi) {
          const float v = col[((xi & ~3) + ((xi + (xi >> 2)) & 3)) * 16];
          const bool upper = xi + s <= 15;
          lo += upper ? v : 0.f;
          hi += upper ? 0.f : v;
        }
        float *bp = binsum + (PLO + j + NPT - 1) * NBT + WIN - 1;
        if (s <= WIN - 1) bp[-s] = lo;
        if (s >= 1 && 16 - s <= WIN - 1) bp[16 - s] = hi;
      }
    }
  } else {
#pragma unroll
    for (int it = 0; it < cdiv(NP * NBT, 64); ++it) {
      const int b2 = lane + 64 * it;
      if (b2 < NP * NBT) {
        const int j = b2 / NBT;
        const int bin = b2 - j * NBT;
        const int da = bin / K1 - (R - 1);  // input sub-row minus output sub-row
        const int dw = bin - (bin / K1) * K1 - (WIN - 1);
        const float *t = scr + j * TSTR;
        float sum = 0.f;
#pragma unroll
        for (int ra = 0; ra < R; ++ra) {
          const int rb = ra - da;
          const bool rok = rb >= 0 && rb < R;
#pragma unroll
          for (int xo = 0; xo < WIN; ++xo) {
            const int xi = xo + dw;
            const bool ok = rok && xi >= 0 && xi < WIN;
            const float v = t[ok ? (ra * RP + xi) * 17 + rb * RP + xo : 0];
            sum += ok ? v : 0.f;
          }
        }
        binsum[(PLO + j + NPT - 1) * NBT + bin] = sum;
      }
    }
  }
}

// dt_bin_sum for one window row per tile (bin index = table index, stored
// straight to the table gradient out), its tile loop kept rolled: called
// between the stages of the channel-stream runs, where the unrolled loop's
// loads in flight would take registers the stages need.  The same sums in
// the same order.
template <class Tag, int WIN, class G, int WAVE>
__device__ __attribute__((always_inline)) inline void dt_bin_sum_rows(const float *scr, float *out) {
  typedef PSpan<G::NPT, WAVE> SP;
  static_assert(G::R == 1, "one window row per tile");
  constexpr int NPT = G::NPT, NBT = G::NBT, PLO = SP::lo, NP = SP::np, TSTR = kBinTile;
  const int lane = threadIdx.x & 63;
  const int s = lane & 15;
#pragma unroll 1
  for (int it = 0; it < cdiv(NP * 16, 64); ++it) {
    const int j = (lane >> 4) + 4 * it;
    if (j < NP) {
      const float *col = scr + j * TSTR + s;
      float lo = 0.f, hi = 0.f;
#pragma unroll
      for (int xi = 0; xi < 16; ++xi) {
        const float v = col[((xi & ~3) + ((xi + (xi >> 2)) & 3)) * 16];
        const bool upper = xi + s <= 15;
        lo += upper ? v : 0.f;
        hi += upper ? 0.f : v;
      }
      float *bp = out + (PLO + j + NPT - 1) * NBT + WIN - 1;
      if (s <= WIN - 1) bp[-s] = lo;
      if (s >= 1 && 16 - s <= WIN - 1) bp[16 - s] = hi;
    }
  }
}

// Diagonal binning of one wave's accumulator tiles into the bins at the
// end of the scratch (LDS of the stages); no workgroup barrier inside.
// Every tile of the wave goes to LDS at once; bin (da, dw) of tile P sums
// the elements (ra*RP + xo + dw, rb*RP + xo) with ra - rb = da over xo, in a
// fixed order.
template <class Tag, int WIN, class G, int WAVE>
__device__ __attribute__((always_inline)) inline void dt_bin(const f32x4 (&acc)[PSpan<G::NPT, WAVE>::na],
                                                              unsigned char *smem) {
  constexpr int NPM = bin_tiles_per_wave<G>();
  float *scr = reinterpret_cast<float *>(smem) + WAVE * NPM * kBinTile;
  float *binsum = reinterpret_cast<float *>(smem) + kWaves * NPM * kBinTile;
  dt_bin_write<Tag, WIN, G, WAVE>(acc, scr);
  wave_lds_sync();
  dt_bin_sum<Tag, WIN, G, WAVE>(scr, binsum);
}

// The bins of the four table-gradient waves' tiles (already written to the
// scratch by dt_bin_write) summed by all NTH threads of the workgroup: task
// (wave, tile, column) for one-row tiles, (wave, tile, bin) otherwise, each
// summed as dt_bin_sum sums it.
template <class Tag, int WIN, class G, int NTH>
__device__ __attribute__((always_inline)) inline void dt_bin_sum_all(const float *scr0, float *binsum, int tid) {
  constexpr int NPT = G::NPT, RP = G::RP, R = G::R, K1 = G::K1, NBT = G::NBT;
  constexpr int NPM = bin_tiles_per_wave<G>(), TSTR = kBinTile;
  constexpr int TPT = R == 1 ? 16 : NBT;  // tasks per tile
  constexpr int NP0 = PSpan<NPT, 0>::np, NP1 = PSpan<NPT, 1>::np, NP2 = PSpan<NPT, 2>::np, NP3 = PSpan<NPT, 3>::np;
  constexpr int E0 = NP0 * TPT, E1 = E0 + NP1 * TPT, E2 = E1 + NP2 * TPT, E3 = E2 + NP3 * TPT;
  for (int t = tid; t < E3; t += NTH) {
    int W, r, plo;
    if (t < E0) { W = 0; r = t; plo = PSpan<NPT, 0>::lo; }
    else if (t < E1) { W = 1; r = t - E0; plo = PSpan<NPT, 1>::lo; }
    else if (t < E2) { W = 2; r = t - E1; plo = PSpan<NPT, 2>::lo; }
    else { W = 3; r = t - E2; plo = PSpan<NPT, 3>::lo; }
    const int j = r / TPT;
    const int q = r - j * TPT;
    const float *tile = scr0 + (W * NPM + j) * TSTR;
    if constexpr (R == 1) {
      const int s = q;
      const float *col = tile + s;
      float lo = 0.f, hi = 0.f;
#pragma unroll
      for (int xi = 0; xi < 16; ++xi) {
        const float v = col[((xi & ~3) + ((xi + (xi >> 2)) & 3)) * 16];
        const bool upper = xi + s <= 15;
        lo += upper ? v : 0.f;
        hi += upper ? 0.f : v;
      }
      float *bp = binsum + (plo + j + NPT - 1) * NBT + WIN - 1;
      if (s <= WIN - 1) bp[-s] = lo;
      if (s >= 1 && 16 - s <= WIN - 1) bp[16 - s] = hi;
    } else {
      const int bin = q;
      const int da = bin / K1 - (R - 1);
      const int dw = bin - (bin / K1) * K1 - (WIN - 1);
      float sum = 0.f;
#pragma unroll
      for (int ra = 0; ra < R; ++ra) {
        const int rb = ra - da;
        const bool rok = rb >= 0 && rb < R;
#pragma unroll
        for (int xo = 0; xo < WIN; ++xo) {
          const int xi = xo + dw;
          const bool ok = rok && xi >= 0 && xi < WIN;
          const float v = tile[ok ? (ra * RP + xi) * 17 + rb * RP + xo : 0];
          sum += ok ? v : 0.f;
        }
      }
      binsum[(plo + j + NPT - 1) * NBT + bin] = sum;
    }
  }
}

// Hierarchical form: the local table's bins from the same-half accumulator
// tiles of the four table-gradient waves (written to the scratch by
// dt_bin_write; one window row per tile).  Bin (P, dwl), P = hi - ho and
// dwl = xi - xo, sums the elements (xi, xo) of tile P with both columns in
// the same half of the window, xo ascending; one task per bin.
template <class G, int HL, int NTH>
__device__ __attribute__((always_inline)) inline void dt_bin_sum_local(const float *scr0, float *binl, int tid) {
  static_assert(G::R == 1, "one window row per tile");
  constexpr int WIN = G::NPT, K1L = 2 * HL - 1, NPM = bin_tiles_per_wave<G>();
  constexpr PRange PR = make_prange<G::NPT>();
  for (int t = tid; t < K1L * K1L; t += NTH) {
    const int P = t / K1L - (HL - 1);
    const int dw = t - (t / K1L) * K1L - (HL - 1);
    int W = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w)
      if (P >= PR.lo[w] && P <= PR.hi[w]) W = w;
    int lo = PR.lo[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w)
      if (W == w) lo = PR.lo[w];
    const float *tile = scr0 + (W * NPM + (P - lo)) * kBinTile;
    float sum = 0.f;
#pragma unroll
    for (int xo = 0; xo < WIN; ++xo) {
      const int xi = xo + dw;
      const bool ok = xi >= 0 && xi < WIN && (xi < HL) == (xo < HL);
      const int xs = ok ? xi : 0;
      // element (xi, xo) of the skewed tile: row 4 (xi / 4) + (xi + xi / 4) % 4,
      // column (xo - xi) mod 16
      const float v = tile[((xs & ~3) + ((xs + (xs >> 2)) & 3)) * 16 + ((xo - xs) & 15)];
      sum += ok ? v : 0.f;
    }
    binl[t] = sum;
  }
}

// Hierarchical form: both table gradients of the slab from their bins (one
// window row per tile: bin k of either table is its entry k), written as the
// tables (one slab per channel) or as this slab's partial sums, which the
// sum kernel adds in slab order once this kernel has finished.
template <class G, int HL, int NTH>
__device__ __attribute__((always_inline)) inline void dt_reduce_hier(const float *bing, const float *binl,
                                                                      float *__restrict__ dtg, float *__restrict__ dtl,
                                                                      float *__restrict__ partg,
                                                                      float *__restrict__ partl, const KArgs &a,
                                                                      int64_t c, int64_t slab) {
  static_assert(G::R == 1, "one window row per tile");
  constexpr int K2 = G::K2, K2L = (2 * HL - 1) * (2 * HL - 1), KT = K2 + K2L;
  const int tid = threadIdx.x;
  const bool single = a.tiles_per_ch == 1;
  float *og = single ? dtg + c * K2 : partg + (slab * a.C + c) * K2;
  float *ol = single ? dtl + c * K2L : partl + (slab * a.C + c) * K2L;
  for (int k = tid; k < KT; k += NTH) {
    if (k >= K2) ol[k - K2] = binl[k - K2];
    else og[k] = bing[k];
  }
}

// This slab's table gradient from the bins (a fixed-order combine), written
// as the table gradient (one slab per channel) or as the slab's partial sums,
// which the sum kernel adds in slab order once this kernel has finished.
// NTH threads take part; starts after a workgroup barrier that follows the
// binning.
template <class Tag, int WIN, class G, int NTH>
__device__ __attribute__((always_inline)) inline void dt_reduce(unsigned char *smem, float *__restrict__ dt,
                                                                 float *__restrict__ part, const KArgs &a, int64_t c,
                                                                 int64_t slab) {
  constexpr int NPT = G::NPT, R = G::R;
  constexpr int K1 = G::K1, K2 = G::K2, NBT = G::NBT;
  constexpr int NPM = max_tiles_per_wave<NPT>();
  const int tid = threadIdx.x;
  const float *binsum = reinterpret_cast<const float *>(smem) + kWaves * NPM * 272;
  float *out = a.tiles_per_ch == 1 ? dt + c * K2 : part + (slab * a.C + c) * K2;
  // combine the (P, sub-row offset) bins of each offset (dh, dw) in a fixed
  // order
  for (int k = tid; k < K2; k += NTH) {
    float s = 0.f;
    if constexpr (R == 1) {
      // one window row per tile: offset dh has the single bin of P = dh,
      // stored at index k
      s = binsum[k];
    } else {
      const int dhi = k / K1;
      const int dwi = k - dhi * K1;
      const int dh = dhi - (WIN - 1);
      // the tiles P with |dh - P R| <= R - 1 (at most two), in increasing P
      // floor(dh / R) .. floor((dh + R - 1) / R), numerators made positive
      const int plo = (dh + R * WIN) / R - WIN;
      const int phi = (dh + R - 1 + R * WIN) / R - WIN;
      for (int P = plo; P <= phi; ++P) {
        if (P < -(NPT - 1) || P > NPT - 1) continue;
        s += binsum[(P + NPT - 1) * NBT + (dh - P * R + R - 1) * K1 + dwi];
      }
    }
    out[k] = s;
  }
}

// Table gradient of the workgroup's slab from the accumulators: diagonal
// bins, then the slab's dT (or its partial sums).  Starts with a workgroup
// barrier (the bins reuse the LDS of the stages).
template <class Tag, int WIN, class G, int WAVE>
__device__ __attribute__((always_inline)) inline void dt_finish(const f32x4 (&acc)[PSpan<G::NPT, WAVE>::na],
                                                                 unsigned char *smem, float *__restrict__ dt,
                                                                 float *__restrict__ part, const KArgs &a, int64_t c,
                                                                 int64_t slab) {
  __syncthreads();
  dt_bin<Tag, WIN, G, WAVE>(acc, smem);
  __syncthreads();
  dt_reduce<Tag, WIN, G, kThreads>(smem, dt, part, a, c, slab);
}

template <class Tag, int WIN, int WAVE, bool TILED>
__device__ __attribute__((always_inline)) void dt_wave(const typename Tag::S *__restrict__ x, const typename Tag::S *__restrict__ dy,
                        float *__restrict__ dt, float *__restrict__ part, const KArgs &a,
                        unsigned char *smem) {
  typedef DtCfg<Tag, WIN> G;
  typedef PSpan<G::NPT, WAVE> SP;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const uint32_t bid = die_major(blockIdx.x, gridDim.x);
  const int64_t c = bid / a.tiles_per_ch;
  const int64_t slab = bid - c * a.tiles_per_ch;
  const int64_t s0 = slab * a.tile;
  const int64_t s1 = (s0 + a.tile < a.N) ? s0 + a.tile : a.N;

  f32x4 acc[SP::na];
#pragma unroll
  for (int j = 0; j < SP::na; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  Stage<Tag, WIN, G> st;
  stage_load<Tag, WIN, G, TILED>(a, x, dy, c, s0, s1, tid, st);
  for (int64_t m0 = s0; m0 < s1; m0 += G::CW) {
    if (m0 != s0) __syncthreads();  // previous stage consumed
    stage_write<Tag, WIN, G, TILED>(smem, tid, st);
    __syncthreads();
    if (m0 + G::CW < s1) stage_load<Tag, WIN, G, TILED>(a, x, dy, c, m0 + G::CW, s1, tid, st);
    dt_products<Tag, G, WAVE>(smem, smem + G::BUF, acc, lane);
  }
  dt_finish<Tag, WIN, G, WAVE>(acc, smem, dt, part, a, c, slab);
}

template <class Tag, int WIN, bool TILED>
__global__ __launch_bounds__(kThreads, 3) void wbmm_dt_kernel(const typename Tag::S *__restrict__ x,
                                                              const typename Tag::S *__restrict__ dy,
                                                              float *__restrict__ dt, float *__restrict__ part,
                                                              KArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  switch (threadIdx.x >> 6) {
    case 0: dt_wave<Tag, WIN, 0, TILED>(x, dy, dt, part, a, smem); break;
    case 1: dt_wave<Tag, WIN, 1, TILED>(x, dy, dt, part, a, smem); break;
    case 2: dt_wave<Tag, WIN, 2, TILED>(x, dy, dt, part, a, smem); break;
    default: dt_wave<Tag, WIN, 3, TILED>(x, dy, dt, part, a, smem); break;
  }
}

// ===================================================== fused backward

// Input-gradient products of one stage: dX = dY M^T per window, i.e. the
// forward products with the reversed table.  The wave takes sub-tile
// WAVE % SUBS of the stage and the output tiles [T0, T1) of its part; K runs
// outermost (all its output tiles accumulate at once), each tile's sum over
// K in the forward's order.  The rounded results go to Obuf (window-major,
// the x stage, no longer read).
// Input-gradient work of wave WAVE of NDX: sub-tile SUB of the stage,
// output tiles [T0, T1); 16-bit B fragments q = 2 s - t + NT - 1 of its
// steps and tiles run over [QLO, QLO + NQ).
template <class Tag, int WIN, int WAVE, int NDX>
struct DxSplit {
  typedef BwdCfg<Tag, WIN> G;
  typedef FwdCfg<Tag, WIN> F;
  static constexpr int NT = F::NT, S_ = F::S;
  static constexpr int WPS = NDX / G::SUBS;  // waves per sub-tile
  static constexpr int SUB = WAVE % G::SUBS, PART = WAVE / G::SUBS;
  static constexpr int T0 = PART * NT / WPS, T1 = (PART + 1) * NT / WPS, NTW = T1 - T0;
  static constexpr int QLO = NT - T1;
  static constexpr int NQ = NTW > 0 ? 2 * S_ - 2 + NTW : 1;
};

// HL > 0: the hierarchical form's input gradient (WIN = 2 HL; Tsl / TBL hold
// the reversed local table and its blocks): per K step the local-block
// product follows the global one, and 2 dY is added before the rounding, as
// in the forward kernels, so the result equals theirs bit for bit.  PRE:
// the wave's 16-bit B fragments come preloaded in bfw (the table does not
// change between stages) instead of being read from TB.
template <class Tag, int WIN, int WAVE, int NDX = kWaves, int HL = 0, bool PRE = false>
__device__ __attribute__((always_inline)) inline void dx_products(
    const unsigned char *Dbuf, unsigned char *Obuf, const typename Tag::S *Ts, const typename Tag::S *TB, int lane,
    const typename Tag::S *Tsl = nullptr, const typename Tag::S *TBL = nullptr,
    const typename Tag::Frag (*bfw)[DxSplit<Tag, WIN, WAVE, NDX>::NQ] = nullptr) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef BwdCfg<Tag, WIN> G;
  typedef FwdCfg<Tag, WIN> F;
  constexpr int RP = G::RP, LDSW = G::LDSW, NT = F::NT, S_ = F::S, K1 = G::K1;
  constexpr int WPS = NDX / G::SUBS;  // waves per sub-tile
  constexpr int SUB = WAVE % G::SUBS, PART = WAVE / G::SUBS;
  constexpr int T0 = PART * NT / WPS, T1 = (PART + 1) * NT / WPS, NTW = T1 - T0;
  const int g = lane >> 4;
  const int ln = lane & 15;
  const S *rowp = reinterpret_cast<const S *>(Dbuf) + SUB * 16 * LDSW;
  S *outp = reinterpret_cast<S *>(Obuf) + (SUB * 16 + 4 * g) * LDSW + ln;
  if constexpr (NTW > 0) {
    f32x4 acc[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (Tag::W16) {
      constexpr int NB = F::NB;
      auto load_bf = [&](int q) -> Frag {
        const int d0 = q - (NT - 1);
        int dh, xi0;
        if (RP == 16) { dh = d0 + (g >> 1); xi0 = 8 * (g & 1); }
        else { dh = 2 * d0 + g - (ln >> 3); xi0 = 0; }
        const int xo = ln & (RP - 1);
        return *reinterpret_cast<const Frag *>(&TB[((dh + F::TBLO + WIN - 1) * RP + xo) * RP + xi0]);
      };
      // fragment q = 2s - t + NT - 1 serves steps s with T0 <= t < T1; it is
      // read from LDS at the first of them (or preloaded)
      constexpr int QLO = DxSplit<Tag, WIN, WAVE, NDX>::QLO, NQ = DxSplit<Tag, WIN, WAVE, NDX>::NQ;
      Frag bf[NB];
      if constexpr (PRE) {
#pragma unroll
        for (int i = 0; i < NQ; ++i) bf[QLO + i] = (*bfw)[i];
      }
#pragma unroll
      for (int s = 0; s < S_; ++s) {
        if constexpr (!PRE) {
#pragma unroll
          for (int q = 0; q < NB; ++q) {
            const int lo = 2 * s + NT - T1, hi = 2 * s + NT - 1 - T0;  // fragments of step s
            const bool first = s == 0 ? true : !(q >= lo - 2 && q <= hi - 2);
            if (q >= lo && q <= hi && first) bf[q] = load_bf(q);
          }
        }
        const Frag af = *reinterpret_cast<const Frag *>(&rowp[ln * LDSW + s * 32 + 8 * g]);
        // operands swapped (the product is (dY M^T)^T): a lane's four
        // results are consecutive positions of one window, as in the forward
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          acc[j] = mma<Tag>(bf[2 * s - (T0 + j) + NT - 1], af, acc[j]);
          if constexpr (HL > 0) {
            if (fwd_rows_meet<Tag, WIN>(s, T0 + j, true))
              acc[j] = mma<Tag>(fwd_lfrag<Tag, WIN>(TBL, s, T0 + j, g, ln), af, acc[j]);
          }
        }
      }
      // window ln, positions 16 t + 4 g .. + 3: one 8-byte write per tile
      S *outw = reinterpret_cast<S *>(Obuf) + (SUB * 16 + ln) * LDSW + 4 * g;
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const int t = T0 + j;
        if constexpr (HL > 0) {
          // the two identity shortcuts: + 2 dY at the output's own position
          const uint2 yv = *reinterpret_cast<const uint2 *>(&rowp[ln * LDSW + 16 * t + 4 * g]);
          acc[j][0] += 2.f * to_f32<Tag>((u16)(yv.x & 0xffffu));
          acc[j][1] += 2.f * to_f32<Tag>((u16)(yv.x >> 16));
          acc[j][2] += 2.f * to_f32<Tag>((u16)(yv.y & 0xffffu));
          acc[j][3] += 2.f * to_f32<Tag>((u16)(yv.y >> 16));
        }
        *reinterpret_cast<uint2 *>(outw + 16 * t) = uint2{pack2<Tag>(acc[j][0], acc[j][1]), pack2<Tag>(acc[j][2], acc[j][3])};
      }
    } else {
#pragma unroll
      for (int s = 0; s < S_; ++s) {
        const float af = rowp[ln * LDSW + 4 * s + g];
        const int k = 4 * s + g;
        const int hi = k / RP, xi = k % RP;
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          const int pn = 16 * (T0 + j) + ln;
          const int ho = pn / RP, xo = pn % RP;
          const int dh = hi - ho;
          float bv = 0.f;
          if (xo < WIN && xi < WIN && dh >= -(WIN - 1) && dh <= WIN - 1)
            bv = Ts[(dh + WIN - 1) * K1 + xi - xo + WIN - 1];
          if constexpr (HL > 0) {
            // local sub-window entry and the two identity shortcuts
            constexpr int K1L = 2 * HL - 1;
            if (xo < WIN && xi < WIN && hi < WIN && ho < WIN && (hi < HL) == (ho < HL) && (xi < HL) == (xo < HL))
              bv += Tsl[(dh + HL - 1) * K1L + xi - xo + HL - 1];
            if (hi == ho && xi == xo && xi < WIN && hi < WIN) bv += 2.f;
          }
          acc[j] = mma<Tag>(af, bv, acc[j]);
        }
      }
#pragma unroll
      for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) outp[rr * LDSW + 16 * (T0 + j)] = acc[j][rr];
    }
  }
}

// Store the stage's input-gradient rows (window-major in Obuf).
template <class Tag, int WIN, bool TILED>
__device__ __attribute__((always_inline)) inline void dx_store(const KArgs &a, void *dx, int64_t c, int64_t m0,
                                                                int64_t m1, int tid, const unsigned char *Obuf) {
  typedef BwdCfg<Tag, WIN> G;
  typedef RowData<WIN, Tag::ES> RD;
  if constexpr (TILED) {
    constexpr int NDV = (WIN * Tag::ES) / 4, SUBS = G::CW / 16;
    typedef typename Tag::S S;
    const int vv = tid / WIN;
    const int hi = tid - vv * WIN;
    const uint32_t off = tiled_row_off<WIN, Tag::ES>(a, vv & 15, hi);
#pragma unroll
    for (int sub = 0; sub < SUBS; ++sub) {
      const int64_t ms = m0 + 16 * sub;
      if (vv < 16 && ms + vv < m1) {
        const uint32_t *l4 = reinterpret_cast<const uint32_t *>(Obuf + ((16 * sub + vv) * G::LDSW + hi * G::RP) * Tag::ES);
        uint32_t *p4 = reinterpret_cast<uint32_t *>(reinterpret_cast<char *>(reinterpret_cast<S *>(dx) + tiled_sub_base(a, c, ms)) + off);
        // the padded row in 16-byte reads (it spans whole 16-byte chunks)
        constexpr int NDR = (NDV + 3) & ~3;
        uint32_t d[NDR];
#pragma unroll
        for (int i = 0; i < NDR; i += 4) {
          const uint4 u = *reinterpret_cast<const uint4 *>(l4 + i);
          d[i] = u.x; d[i + 1] = u.y; d[i + 2] = u.z; d[i + 3] = u.w;
        }
#pragma unroll
        for (int i = 0; i + 4 <= NDV; i += 4) *reinterpret_cast<u32x4a *>(p4 + i) = u32x4a{d[i], d[i + 1], d[i + 2], d[i + 3]};
#pragma unroll
        for (int i = NDV & ~3; i < NDV; ++i) p4[i] = d[i];
      }
    }
    return;
  }
  for (int q = tid; q < G::CW * WIN; q += kThreads) {
    const int v = q / WIN;
    const int hi = q - v * WIN;
    if (m0 + v >= m1) break;
    const Row<WIN, Tag::ES> r = row_of<WIN, Tag::ES>(a, dx, c, m0 + v, hi);
    if (r.mode == kNone) continue;
    const uint32_t *l4 = reinterpret_cast<const uint32_t *>(Obuf + (v * G::LDSW + hi * G::RP) * Tag::ES);
    uint32_t d[RD::ND];
#pragma unroll
    for (int i = 0; i < RD::ND; i += 4) {
      const uint4 u = *reinterpret_cast<const uint4 *>(l4 + i);
      d[i] = u.x; d[i + 1] = u.y; d[i + 2] = u.z; d[i + 3] = u.w;
    }
    store_row<WIN, Tag::ES>(dx, r, d);
  }
}

// One workgroup = (channel, slab of windows), as the table gradient.  Per
// stage: the x and dy rows land window-major; the waves accumulate their
// share of X^T dY; after a barrier the x tile is free and receives the
// input-gradient results computed from the dy tile, which are then stored
// as rows.  dY is read once for both gradients.
template <class Tag, int WIN, int WAVE, bool TILED>
__device__ __attribute__((always_inline)) void bwd_wave(const typename Tag::S *__restrict__ x,
                                                        const typename Tag::S *__restrict__ dy,
                                                        const typename Tag::S *__restrict__ tab,
                                                        typename Tag::S *__restrict__ dx, float *__restrict__ dt,
                                                        float *__restrict__ part, const KArgs &a,
                                                        unsigned char *smem) {
  typedef typename Tag::S S;
  typedef BwdCfg<Tag, WIN> G;
  typedef PSpan<G::NPT, WAVE> SP;
  constexpr int RP = G::RP, K1 = G::K1, K2 = G::K2;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const uint32_t bid = die_major(blockIdx.x, gridDim.x);
  const int64_t c = bid / a.tiles_per_ch;
  const int64_t slab = bid - c * a.tiles_per_ch;
  const int64_t s0 = slab * a.tile;
  const int64_t s1 = (s0 + a.tile < a.N) ? s0 + a.tile : a.N;
  unsigned char *Xt = smem;
  unsigned char *Dt = smem + G::BUF;

  f32x4 acc[SP::na];
#pragma unroll
  for (int j = 0; j < SP::na; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the reversed table row and the first stage in flight (the table first,
  // ahead of the bulk loads); the table row and (16-bit) its Toeplitz
  // blocks -> LDS
  TabRegs<Tag, WIN, false, kThreads> tr;
  tab_load<Tag, WIN, true, false, kThreads>(tab, nullptr, c, tid, tr);
  Stage<Tag, WIN, G> st;
  stage_load<Tag, WIN, G, TILED>(a, x, dy, c, s0, s1, tid, st);
  {
    S *Ts = reinterpret_cast<S *>(smem + G::TS_OFF);
#pragma unroll
    for (int i = 0; i < tr.N; ++i)
      if (tid + i * kThreads < K2) Ts[tid + i * kThreads] = tr.v[i];
    if constexpr (Tag::W16) {
      __syncthreads();
      S *TB = reinterpret_cast<S *>(smem + G::TB_OFF);
      build_tb<Tag, WIN, kThreads>(Ts, TB, tid);
    }
  }

  for (int64_t m0 = s0; m0 < s1; m0 += G::CW) {
    if (m0 != s0) __syncthreads();  // previous stage's rows stored
    stage_write<Tag, WIN, G, TILED>(smem, tid, st);
    __syncthreads();
    if (m0 + G::CW < s1) stage_load<Tag, WIN, G, TILED>(a, x, dy, c, m0 + G::CW, s1, tid, st);
    dt_products<Tag, G, WAVE>(Xt, Dt, acc, lane);
    __syncthreads();  // the x tile is no longer read
    dx_products<Tag, WIN, WAVE>(Dt, Xt, reinterpret_cast<const S *>(smem + G::TS_OFF),
                                reinterpret_cast<const S *>(smem + G::TB_OFF), lane);
    __syncthreads();
    dx_store<Tag, WIN, TILED>(a, dx, c, m0, s1, tid, Xt);
  }
  dt_finish<Tag, WIN, G, WAVE>(acc, smem, dt, part, a, c, slab);
}

template <class Tag, int WIN, bool TILED>
__global__ __launch_bounds__(kThreads, (TILED ? 3 : 2)) void wbmm_bwd_kernel(const typename Tag::S *__restrict__ x,
                                                               const typename Tag::S *__restrict__ dy,
                                                               const typename Tag::S *__restrict__ tab,
                                                               typename Tag::S *__restrict__ dx,
                                                               float *__restrict__ dt, float *__restrict__ part,
                                                               KArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  switch (threadIdx.x >> 6) {
    case 0: bwd_wave<Tag, WIN, 0, TILED>(x, dy, tab, dx, dt, part, a, smem); break;
    case 1: bwd_wave<Tag, WIN, 1, TILED>(x, dy, tab, dx, dt, part, a, smem); break;
    case 2: bwd_wave<Tag, WIN, 2, TILED>(x, dy, tab, dx, dt, part, a, smem); break;
    default: bwd_wave<Tag, WIN, 3, TILED>(x, dy, tab, dx, dt, part, a, smem); break;
  }
}

// ------------------------------------------ fused backward, channel stream
// Fixed-offset rows: one workgroup per (channel, slab) and at most one
// workgroup per compute unit at a time, streaming the
// slab's stages through double-buffered LDS (x and dy tiles, and the
// input-gradient results) with one workgroup barrier per stage.  Waves 0-3
// take the table-gradient products (the P ranges of the 4-wave kernel),
// waves 4-11 the input-gradient products (four waves per 16-window
// sub-tile).  The table-gradient waves, whose products end first, store the
// previous stage's dX rows.  The other copies -- the next stage into LDS, the
// stage after it into registers -- are made either by NCW dedicated copy
// waves (waves 12 .. 11 + NCW) while the twelve compute waves multiply, or,
// with NCW = 0, by the compute waves after their products; the last stage's
// dX rows go out from the input-gradient and copy waves (every wave with
// NCW = 0).  Products, bins and sums are those of wbmm_bwd_kernel, so the
// results are bitwise the same.
constexpr int kStreamCompute = 12;  // compute waves
constexpr int kStreamDt = 4;        // of which table-gradient waves

template <int NCW>
__host__ __device__ constexpr int stream_threads() { return 64 * (kStreamCompute + NCW); }

template <class Tag, int WIN>
struct StreamCfg {
  typedef BwdCfg<Tag, WIN> G;
  typedef FwdCfg<Tag, WIN> F;
  static constexpr int SUBS = G::SUBS;                     // 16-window sub-tiles per stage
  static constexpr int NCP = 2 * SUBS;                     // row copies: (tensor, sub-tile)
  static constexpr int RC = 16 * G::KR;                    // rows per copy
  static constexpr int STAGE = 2 * G::BUF;                 // x tile + dy tile
  static constexpr int O_OFF = 2 * STAGE;                  // two dX result buffers of G::BUF
  static constexpr int TS_OFF = O_OFF + 2 * G::BUF;
  static constexpr int TB_OFF = TS_OFF + rup(F::TS_LEN * Tag::ES, 16);
  static constexpr int END = TB_OFF + F::TB_LEN * Tag::ES;
  // hierarchical form: the local table row and its blocks after them
  static constexpr int TSL_OFF = rup(END, 16);
  static constexpr int TBL_OFF = TSL_OFF + rup(F::TSL_LEN * Tag::ES, 16);
  static constexpr int END_H = TBL_OFF + F::TBL_LEN * Tag::ES;
  // runs (one window row per tile, 16-bit): the second channel's table row
  // and blocks, then the table-gradient waves' bin scratch, after everything
  // else, when it fits in the 160 KB of LDS
  static constexpr int NPM = bin_tiles_per_wave<G>();
  static constexpr int TS2_OFF = rup(END, 16);
  static constexpr int TB2_OFF = TS2_OFF + rup(F::TS_LEN * Tag::ES, 16);
  static constexpr int SCR_OFF = TB2_OFF + F::TB_LEN * Tag::ES;
  static constexpr int END_R = SCR_OFF + kWaves * NPM * kBinTile * 4;
  static constexpr bool RUNS = Tag::W16 && G::R == 1 && END_R <= 160 * 1024;
  static_assert(bins_lds_bytes<G>() <= O_OFF, "bins must not reach the dX buffers");
};

// How NC copying waves split a stage's row copies: WPC waves per (tensor,
// sub-tile) copy, IT rows per thread of it.
template <class Tag, int WIN, int NC>
struct StreamCopy {
  typedef StreamCfg<Tag, WIN> SC;
  static constexpr int WPC = NC / SC::NCP;
  static constexpr int IT = cdiv(SC::RC, WPC * 64);
  static_assert(NC % SC::NCP == 0, "whole waves per copy");
};

template <class Tag, int WIN, bool HIER = false>
__host__ __device__ constexpr size_t stream_lds_bytes() {
  typedef StreamCfg<Tag, WIN> SC;
  return (size_t)(HIER ? SC::END_H : SC::RUNS ? SC::END_R : SC::END);
}

template <class Tag, int WIN, int NC>
struct StreamRows {
  RowData<WIN, Tag::ES> rd[StreamCopy<Tag, WIN, NC>::IT];
};

// Rows of copying wave cw's copy (tensor, sub-tile) of the stage at m0 ->
// registers (NC copying waves).
template <class Tag, int WIN, int NC>
__device__ __attribute__((always_inline)) inline void stream_load(const KArgs &a, const typename Tag::S *x,
                                                                   const typename Tag::S *dy, int64_t c, int64_t m0,
                                                                   int64_t m1, int cw, int lane,
                                                                   StreamRows<Tag, WIN, NC> &st) {
  typedef StreamCfg<Tag, WIN> SC;
  typedef StreamCopy<Tag, WIN, NC> CP;
  typedef BwdCfg<Tag, WIN> G;
  constexpr int NDV = (WIN * Tag::ES) / 4;
  const int cp = cw / CP::WPC;
  const int tens = cp / SC::SUBS, sub = cp % SC::SUBS;
  const int64_t ms = m0 + 16 * sub;
  const char *base = reinterpret_cast<const char *>((tens ? dy : x) + tiled_sub_base(a, c, ms));
#pragma unroll
  for (int k = 0; k < CP::IT; ++k) {
    const int t = (cw % CP::WPC) * 64 + lane + k * CP::WPC * 64;
    const int vv = t / G::KR;
    const int hi = t - vv * G::KR;
#pragma unroll
    for (int i = 0; i < RowData<WIN, Tag::ES>::ND; ++i) st.rd[k].d[i] = 0;
    if (t < SC::RC && hi < WIN && ms + vv < m1) {
      const uint32_t *p4 = reinterpret_cast<const uint32_t *>(base + tiled_row_off<WIN, Tag::ES>(a, vv, hi));
#pragma unroll
      for (int i = 0; i + 4 <= NDV; i += 4) {
        const u32x4a u = *reinterpret_cast<const u32x4a *>(p4 + i);
        st.rd[k].d[i] = u.x; st.rd[k].d[i + 1] = u.y; st.rd[k].d[i + 2] = u.z; st.rd[k].d[i + 3] = u.w;
      }
#pragma unroll
      for (int i = NDV & ~3; i < NDV; ++i) st.rd[k].d[i] = p4[i];
    }
  }
}

// The loaded rows -> window-major padded rows of one stage buffer.
template <class Tag, int WIN, int NC>
__device__ __attribute__((always_inline)) inline void stream_write(unsigned char *stage, int cw, int lane,
                                                                    const StreamRows<Tag, WIN, NC> &st) {
  typedef StreamCfg<Tag, WIN> SC;
  typedef StreamCopy<Tag, WIN, NC> CP;
  typedef BwdCfg<Tag, WIN> G;
  typedef RowData<WIN, Tag::ES> RD;
  const int cp = cw / CP::WPC;
  const int tens = cp / SC::SUBS, sub = cp % SC::SUBS;
#pragma unroll
  for (int k = 0; k < CP::IT; ++k) {
    const int t = (cw % CP::WPC) * 64 + lane + k * CP::WPC * 64;
    const int vv = t / G::KR;
    const int hi = t - vv * G::KR;
    if (t < SC::RC) {
      uint32_t *l4 = reinterpret_cast<uint32_t *>(stage + tens * G::BUF + ((16 * sub + vv) * G::LDSW + hi * G::RP) * Tag::ES);
#pragma unroll
      for (int i = 0; i < RD::ND; i += 4)
        *reinterpret_cast<uint4 *>(l4 + i) = make_uint4(st.rd[k].d[i], st.rd[k].d[i + 1], st.rd[k].d[i + 2], st.rd[k].d[i + 3]);
    }
  }
}

// The dX rows of the stage at m0 (window-major in Obuf) -> dx, by NCT
// copying threads (ct = this thread's index among them).
template <class Tag, int WIN, int NCT>
__device__ __attribute__((always_inline)) inline void stream_store(const KArgs &a, typename Tag::S *dx, int64_t c,
                                                                    int64_t m0, int64_t m1, int ct,
                                                                    const unsigned char *Obuf) {
  typedef BwdCfg<Tag, WIN> G;
  constexpr int NDV = (WIN * Tag::ES) / 4, RS = 16 * WIN;  // rows per sub-tile
#pragma unroll
  for (int k = 0; k < cdiv(G::SUBS * RS, NCT); ++k) {
    const int q = ct + k * NCT;
    const int sub = q / RS;
    const int r = q - sub * RS;
    const int vv = r / WIN;
    const int hi = r - vv * WIN;
    const int64_t ms = m0 + 16 * sub;
    if (q < G::SUBS * RS && ms + vv < m1) {
      const uint32_t *l4 = reinterpret_cast<const uint32_t *>(Obuf + ((16 * sub + vv) * G::LDSW + hi * G::RP) * Tag::ES);
      uint32_t *p4 = reinterpret_cast<uint32_t *>(reinterpret_cast<char *>(dx + tiled_sub_base(a, c, ms)) +
                                                  tiled_row_off<WIN, Tag::ES>(a, vv, hi));
      // the padded row in 16-byte reads (it spans whole 16-byte chunks)
      constexpr int NDR = (NDV + 3) & ~3;
      uint32_t d[NDR];
#pragma unroll
      for (int i = 0; i < NDR; i += 4) {
        const uint4 u = *reinterpret_cast<const uint4 *>(l4 + i);
        d[i] = u.x; d[i + 1] = u.y; d[i + 2] = u.z; d[i + 3] = u.w;
      }
#pragma unroll
      for (int i = 0; i + 4 <= NDV; i += 4) *reinterpret_cast<u32x4a *>(p4 + i) = u32x4a{d[i], d[i + 1], d[i + 2], d[i + 3]};
#pragma unroll
      for (int i = NDV & ~3; i < NDV; ++i) p4[i] = d[i];
    }
  }
}

// One wave of the stream kernel: DTW >= 0 is a table-gradient wave (its P
// range), else DXW >= 0 an input-gradient wave (idle but for the copies
// when DX is false: the table gradient alone, with the same stages, bins and
// sums as the fused pass), else a copy wave.  With NCW = 0 every wave copies
// (after its products); otherwise only the NCW copy waves do.
template <class Tag, int WIN, int DTW, int DXW, bool DX, int HL, int NCW, bool RUN>
__device__ __attribute__((always_inline)) void stream_wave(const typename Tag::S *__restrict__ x,
                                                           const typename Tag::S *__restrict__ dy,
                                                           const typename Tag::S *__restrict__ tab,
                                                           const typename Tag::S *__restrict__ tabl,
                                                           typename Tag::S *__restrict__ dx, float *__restrict__ dt,
                                                           float *__restrict__ part, const KArgs &a,
                                                           unsigned char *smem,
                                                           float *__restrict__ dtl, float *__restrict__ partl) {
  typedef typename Tag::S S;
  typedef StreamCfg<Tag, WIN> SC;
  typedef BwdCfg<Tag, WIN> G;
  typedef PSpan<G::NPT, (DTW >= 0 ? DTW : 0)> SP;
  constexpr int RP = G::RP, K1 = G::K1, K2 = G::K2, CW = G::CW;
  constexpr int NTH = stream_threads<NCW>();
  constexpr int NC = NCW > 0 ? NCW : kStreamCompute;    // copying waves
  constexpr bool COPY = NCW == 0 || (DTW < 0 && DXW < 0);  // this wave copies
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: copy addresses in scalar registers
  const int cw = NCW > 0 ? wave - kStreamCompute : wave;  // index among the copying waves
  const uint32_t bid = die_major(blockIdx.x, gridDim.x);
  // runs: stages g0 .. g0 + nst - 1 of all channels' stages (the host keeps
  // their count below 2^31, so 32-bit arithmetic); c is the run's first
  // channel.  Otherwise one (channel, slab).
  constexpr bool RUNS = RUN && HL == 0 && SC::RUNS;
  constexpr bool runs = RUNS;
  int64_t c, slab, s0, s1;
  uint32_t g0 = 0;
  int nst;
  if (runs) {
    g0 = bid * (uint32_t)a.run;
    const uint32_t tot = (uint32_t)a.C * (uint32_t)a.nstc;
    nst = (int)((g0 + (uint32_t)a.run < tot ? g0 + (uint32_t)a.run : tot) - g0);
    c = g0 / (uint32_t)a.nstc;
    slab = 0;
    s0 = 0;
    s1 = a.N;
  } else {
    c = bid / a.tiles_per_ch;
    slab = bid - c * a.tiles_per_ch;
    s0 = slab * a.tile;
    s1 = (s0 + a.tile < a.N) ? s0 + a.tile : a.N;
    nst = (int)((s1 - s0 + CW - 1) / CW);
  }
  // stage j of this workgroup: channel cj, first window mj
  auto locate = [&](int j, int64_t &cj, int64_t &mj) {
    if (runs) {
      const uint32_t gg = g0 + (uint32_t)j;
      const uint32_t cc = gg / (uint32_t)a.nstc;
      cj = cc;
      mj = (int64_t)(gg - cc * (uint32_t)a.nstc) * CW;
    } else {
      cj = c;
      mj = s0 + (int64_t)j * CW;
    }
  };
  // runs: the second channel reached (if any) takes the second table copy
  int64_t cl, ml;
  locate(nst - 1, cl, ml);
  const bool two = runs && cl > c;
  S *Ts = reinterpret_cast<S *>(smem + SC::TS_OFF);
  S *TB = reinterpret_cast<S *>(smem + SC::TB_OFF);
  S *Tsl = reinterpret_cast<S *>(smem + SC::TSL_OFF);  // hierarchical input gradient only
  S *TBL = reinterpret_cast<S *>(smem + SC::TBL_OFF);

  f32x4 acc[SP::na], accl[SP::na];
#pragma unroll
  for (int j = 0; j < SP::na; ++j) acc[j] = accl[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the reversed table row and stage 0 in flight (the table first, ahead
  // of the bulk loads); the table row and (16-bit) its Toeplitz blocks ->
  // LDS; stage 0 -> LDS buffer 0, stage 1 in flight
  constexpr bool HX = DX && HL > 0;  // hierarchical input gradient: both tables
  TabRegs<Tag, WIN, HX, NTH> tr, tr2;
  if constexpr (DX) {
    tab_load<Tag, WIN, true, HX, NTH>(tab, tabl, c, tid, tr);
    if constexpr (RUNS) tab_load<Tag, WIN, true, false, NTH>(tab, nullptr, two ? c + 1 : c, tid, tr2);
  }
  StreamRows<Tag, WIN, NC> st;
  int64_t cj, mj;
  locate(0, cj, mj);
  if constexpr (COPY) stream_load<Tag, WIN, NC>(a, x, dy, cj, mj, s1, cw, lane, st);
  if constexpr (HX) {
    fwd_tables<Tag, WIN, true, true, NTH>(tr, Ts, TB, Tsl, TBL, tid);
  } else if constexpr (DX) {
    S *Ts2 = reinterpret_cast<S *>(smem + SC::TS2_OFF);
    S *TB2 = reinterpret_cast<S *>(smem + SC::TB2_OFF);
#pragma unroll
    for (int i = 0; i < tr.N; ++i)
      if (tid + i * NTH < K2) {
        Ts[tid + i * NTH] = tr.v[i];
        if constexpr (RUNS) {
          if (two) Ts2[tid + i * NTH] = tr2.v[i];
        }
      }
    __syncthreads();
    if constexpr (Tag::W16) {
      build_tb<Tag, WIN, NTH>(Ts, TB, tid);
      if constexpr (RUNS) {
        if (two) build_tb<Tag, WIN, NTH>(Ts2, TB2, tid);
      }
    }
  }
  if constexpr (COPY) {
    stream_write<Tag, WIN, NC>(smem, cw, lane, st);
    if (nst > 1) {
      locate(1, cj, mj);
      stream_load<Tag, WIN, NC>(a, x, dy, cj, mj, s1, cw, lane, st);
    }
  }
  __syncthreads();

  // the input-gradient waves' 16-bit B fragments, read once: the table is
  // the same for every stage
  constexpr int DXI = DXW >= 0 ? DXW : 0;
  constexpr bool PRE = DX && DXW >= 0 && Tag::W16;
  typedef DxSplit<Tag, WIN, DXI, kStreamCompute - kStreamDt> DS;
  typename Tag::Frag bfw[DS::NQ];
  if constexpr (PRE) {
    const int g = lane >> 4, ln = lane & 15;
#pragma unroll
    for (int i = 0; i < DS::NQ; ++i) bfw[i] = fwd_bfrag<Tag, WIN>(TB, DS::QLO + i, g, ln);
  }

  // runs: the table-gradient waves' tiles of channel cx binned (into scratch
  // of their own) and stored as that channel's partial: the first of its two
  // (slot 0) when this run holds the channel's first stage, else the second;
  // a channel whole in this run also zeroes its second.  The sum kernel adds
  // the two.
  auto run_bin = [&](int64_t cx) {
    if constexpr (RUNS && DTW >= 0) {
      float *mine = reinterpret_cast<float *>(smem + SC::SCR_OFF) + DTW * SC::NPM * kBinTile;
      const int64_t first = cx * a.nstc;
      const int slot = first >= (int64_t)g0 ? 0 : 1;
      wave_lds_sync();
      dt_bin_write<Tag, WIN, G, DTW>(acc, mine);
      wave_lds_sync();
      dt_bin_sum_rows<Tag, WIN, G, DTW>(mine, part + ((int64_t)slot * a.C + cx) * K2);
      if (slot == 0 && first + a.nstc <= (int64_t)g0 + nst) {
        float *z = part + (a.C + cx) * K2;
#pragma unroll
        for (int j = 0; j < SP::np; ++j)
          for (int q = lane; q < K1; q += 64) z[(SP::lo + j + G::NPT - 1) * K1 + q] = 0.f;
      }
#pragma unroll
      for (int j = 0; j < SP::na; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };

  // runs: channel and stage within it of this stage (cs, ls) and of the
  // previous one (cp, lp), advanced without divisions
  uint32_t cs = (uint32_t)c, ls = 0, cp = 0, lp = 0;
  if constexpr (RUNS) ls = g0 - cs * (uint32_t)a.nstc;
  auto stage = [&](int s) {
    const int64_t m0 = RUNS ? (int64_t)ls * CW : s0 + (int64_t)s * CW;
    const int64_t mprev = RUNS ? (int64_t)lp * CW : m0 - CW;
    unsigned char *cur = smem + (s & 1) * SC::STAGE;
    unsigned char *obuf = smem + SC::O_OFF + (s & 1) * G::BUF;
    // this stage's products
    if constexpr (DTW >= 0) {
      dt_products_split<Tag, G, DTW, HL>(cur, cur + G::BUF, acc, accl, lane);
    } else if constexpr (DX && DXW >= 0) {
      dx_products<Tag, WIN, DXW, kStreamCompute - kStreamDt, (HX ? HL : 0), PRE>(cur + G::BUF, obuf, Ts, TB, lane,
                                                                                  Tsl, TBL, &bfw);
    }
    // the next stage into the other buffer (free since the last barrier),
    // the one after it in flight, the previous stage's dX rows out
    if constexpr (COPY) {
      if (s + 1 < nst) stream_write<Tag, WIN, NC>(smem + ((s + 1) & 1) * SC::STAGE, cw, lane, st);
      if (s + 2 < nst) {
        uint32_t cn = cs, ln = ls;
        if constexpr (RUNS) {
          ln += 2;
          if (ln >= (uint32_t)a.nstc) { ln -= (uint32_t)a.nstc; ++cn; }
          if (ln >= (uint32_t)a.nstc) { ln -= (uint32_t)a.nstc; ++cn; }
        }
        stream_load<Tag, WIN, NC>(a, x, dy, RUNS ? (int64_t)cn : c, RUNS ? (int64_t)ln * CW : m0 + 2 * CW, s1, cw,
                                  lane, st);
      }
    }
    // the table-gradient waves (whose products end first) store the previous
    // stage's dX rows
    if constexpr (DX && DTW >= 0) {
      if (s > 0)
        stream_store<Tag, WIN, kStreamDt * 64>(a, dx, RUNS ? (int64_t)cp : c, mprev, s1, DTW * 64 + lane,
                                               smem + SC::O_OFF + ((s - 1) & 1) * G::BUF);
    }
    __syncthreads();
    if constexpr (RUNS) {
      cp = cs;
      lp = ls;
      if (++ls == (uint32_t)a.nstc) {
        ls = 0;
        ++cs;
      }
    }
  };
  if constexpr (RUNS) {
    // the first channel's stages; where the run reaches a second channel,
    // the first one's table gradient out and the input-gradient fragments
    // from the second table's blocks, then the second channel's stages (the
    // binning outside the stage loop, whose registers it would take)
    const int sw = two ? (int)((uint32_t)(c + 1) * (uint32_t)a.nstc - g0) : nst;
    for (int s = 0; s < sw; ++s) stage(s);
    if (two) {
      run_bin(c);
      if constexpr (PRE) {
        const S *TB2 = reinterpret_cast<const S *>(smem + SC::TB2_OFF);
        const int g = lane >> 4, ln = lane & 15;
#pragma unroll
        for (int i = 0; i < DS::NQ; ++i) bfw[i] = fwd_bfrag<Tag, WIN>(TB2, DS::QLO + i, g, ln);
      }
      for (int s = sw; s < nst; ++s) stage(s);
    }
  } else {
    for (int s = 0; s < nst; ++s) stage(s);
  }
  // the last stage's dX rows out while the table-gradient waves bin their
  // tiles (the bins lie below the dX buffers)
  if constexpr (DX && NCW > 0) {
    // the input-gradient waves (idle here) and the copy waves together
    if constexpr (DTW < 0)
      stream_store<Tag, WIN, (kStreamCompute - kStreamDt + NCW) * 64>(
          a, dx, cl, ml, s1, (wave - kStreamDt) * 64 + lane, smem + SC::O_OFF + ((nst - 1) & 1) * G::BUF);
  } else if constexpr (DX && COPY) {
    stream_store<Tag, WIN, NC * 64>(a, dx, cl, ml, s1, cw * 64 + lane, smem + SC::O_OFF + ((nst - 1) & 1) * G::BUF);
  }
  if constexpr (RUNS) {
    // runs: the last channel's table gradient, binned by each table-gradient
    // wave on its own (no workgroup barrier)
    if (runs) {
      run_bin(cl);
      return;
    }
  }
  // the table-gradient waves' tiles to the scratch, then the bins summed by
  // all the waves
  constexpr int NPM = bin_tiles_per_wave<G>();
  float *scr = reinterpret_cast<float *>(smem);
  float *bing = scr + kWaves * NPM * kBinTile;
  if constexpr (HL > 0) {
    // hierarchical form: the global table's tiles are acc + accl, the local
    // table's the same-half tiles accl alone, binned after them in the same
    // scratch
    float *binl = bing + G::NACC * G::NBT;
    if constexpr (DTW >= 0) {
      f32x4 tot[SP::na];
#pragma unroll
      for (int j = 0; j < SP::na; ++j) {
        const int P = SP::lo + j;
        tot[j] = acc[j];
        if (P > -HL && P < HL) {
#pragma unroll
          for (int e = 0; e < 4; ++e) tot[j][e] += accl[j][e];
        }
      }
      dt_bin_write<Tag, WIN, G, DTW>(tot, scr + DTW * NPM * kBinTile);
    }
    __syncthreads();
    dt_bin_sum_all<Tag, WIN, G, NTH>(scr, bing, tid);
    __syncthreads();
    if constexpr (DTW >= 0) dt_bin_write<Tag, WIN, G, DTW>(accl, scr + DTW * NPM * kBinTile);
    __syncthreads();
    dt_bin_sum_local<G, HL, NTH>(scr, binl, tid);
    __syncthreads();
    dt_reduce_hier<G, HL, NTH>(bing, binl, dt, dtl, part, partl, a, c, slab);
  } else {
    if constexpr (DTW >= 0) dt_bin_write<Tag, WIN, G, DTW>(acc, scr + DTW * NPM * kBinTile);
    __syncthreads();
    dt_bin_sum_all<Tag, WIN, G, NTH>(scr, bing, tid);
    __syncthreads();
    dt_reduce<Tag, WIN, G, NTH>(smem, dt, part, a, c, slab);
  }
}

// HL > 0: the hierarchical form (global window WIN, local window
// HL = WIN / 2): both table gradients from one pass, and with DX the input
// gradient of the fused matrix (tables tab and tabl, read back to front).
// NCW: dedicated copy waves (0 or 4).  RUN: runs of stages over all
// channels (a.run, a.nstc) instead of one (channel, slab) per workgroup.
template <class Tag, int WIN, bool DX, int HL = 0, int NCW = 0, bool RUN = false>
__global__ __launch_bounds__(stream_threads<NCW>(), (kStreamCompute + NCW) / 4) void wbmm_bwd_stream_kernel(
    const typename Tag::S *__restrict__ x, const typename Tag::S *__restrict__ dy,
    const typename Tag::S *__restrict__ tab, typename Tag::S *__restrict__ dx, float *__restrict__ dt,
    float *__restrict__ part, KArgs a, float *__restrict__ dtl,
    float *__restrict__ partl, const typename Tag::S *__restrict__ tabl) {
  static_assert(HL == 0 || 2 * HL == WIN, "hierarchical form: WIN = 2 HL");
  static_assert(HL == 0 || bins_lds_bytes<BwdCfg<Tag, WIN>>() + (size_t)(2 * HL - 1) * (2 * HL - 1) * 4 <=
                               (size_t)StreamCfg<Tag, WIN>::O_OFF,
                "both tables' bins within the stage buffers");
  static_assert(NCW == 0 || NCW == 4, "copy waves: none or one per SIMD");
  extern __shared__ __align__(16) unsigned char smem[];
#define WBMM_SW(D, X) stream_wave<Tag, WIN, D, X, DX, HL, NCW, RUN>(x, dy, tab, tabl, dx, dt, part, a, smem, dtl, partl)
  switch (threadIdx.x >> 6) {
    case 0: WBMM_SW(0, -1); break;
    case 1: WBMM_SW(1, -1); break;
    case 2: WBMM_SW(2, -1); break;
    case 3: WBMM_SW(3, -1); break;
    case 4: WBMM_SW(-1, 0); break;
    case 5: WBMM_SW(-1, 1); break;
    case 6: WBMM_SW(-1, 2); break;
    case 7: WBMM_SW(-1, 3); break;
    case 8: WBMM_SW(-1, 4); break;
    case 9: WBMM_SW(-1, 5); break;
    case 10: WBMM_SW(-1, 6); break;
    case 11: WBMM_SW(-1, 7); break;
    default:
      if constexpr (NCW > 0) WBMM_SW(-1, -1);
      break;
  }
#undef WBMM_SW
}

// ============================================================ host side

// Dedicated copy waves of the (plain) channel-stream kernel.
constexpr int kCopyWaves = 4;

static int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Compute units of the current device (cached per device; 0 if unknown).
static int compute_units() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

static KArgs make_args(const Geom &g) {
  KArgs a;
  a.B = g.B; a.C = g.C; a.H = g.H; a.W = g.W;
  a.numel = g.B * g.C * g.H * g.W;
  a.NH = (int)g.NH; a.NW = (int)g.NW; a.N = g.N;
  a.tile = 0; a.tiles_per_ch = 0;
  a.inv_nw = 1.0f / (float)g.NW;
  a.inv_nhw = 1.0f / (float)(g.NH * g.NW);
  a.tiled = 0;
  a.lgnw = 0; a.lgw = 0; a.BE = 0; a.WPI = 1; a.chw = 0;
  a.run = 0; a.nstc = 0;
  return a;
}

// Fixed-offset rows for the gradient kernels (see KArgs): windows tile the
// map, NW a power of two, a 16-window sub-tile is whole bands of one image or
// whole images (within 2^31 bytes), rows dword-aligned (float32, or an even
// window) in every tensor the kernel moves.
template <int WIN, int ES>
static void set_tiled(const Geom &g, KArgs &a, std::initializer_list<const void *> ptrs) {
  a.tiled = 0;
  if (g.H % WIN != 0 || g.W % WIN != 0 || g.NW > 16 || (g.NW & (g.NW - 1)) != 0) return;
  if (ES == 2 && (WIN & 1)) return;
  for (const void *p : ptrs)
    if ((reinterpret_cast<uintptr_t>(p) & 3) != 0) return;
  const int64_t wpi = g.NH * g.NW;
  const bool inside = wpi % 16 == 0, whole = !inside && 16 % wpi == 0;
  if (!inside && !whole) return;
  const int64_t chw = g.C * g.H * g.W;
  if (16 * chw * ES >= ((int64_t)1 << 31) && whole) return;
  if ((int64_t)WIN * g.W * 16 * ES >= ((int64_t)1 << 31)) return;
  int lg = 0;
  while ((1 << lg) < g.NW) ++lg;
  int lw = 0;
  while ((1 << lw) < wpi) ++lw;
  a.tiled = 1;
  a.lgnw = lg;
  a.lgw = inside ? 4 : lw;
  a.BE = (int)(WIN * g.W);
  a.WPI = (int)wpi;
  a.chw = chw;
}

// Windows per forward workgroup: kFwdWaves waves x sub-tiles per wave x 16.
// More sub-tiles per wave pipeline better; small problems keep enough
// workgroups to cover the 256 compute units.
template <class Tag, int WIN>
static int pick_fwd_tile(const Geom &g) {
  int spw = rp_of(WIN) == 8 ? 4 : 2;
  while (spw > 1 && g.C * cdiv64(g.N, 16 * kFwdWaves * spw) < 1024) spw /= 2;
  return 16 * kFwdWaves * spw;
}

// Whether a 16-bit forward can take the image-layout kernel, and its
// geometry: windows tile the map, NW is a power of two, a 16-window sub-tile
// is whole bands of one image or whole images, every piece starts on a 16-byte
// boundary (both tensors 16-byte aligned).
template <int WIN>
static bool img_layout(const Geom &g, const void *x, const void *y, ImgArgs &ia) {
  if (g.H % WIN != 0 || g.W % WIN != 0 || g.NW > 16 || (g.NW & (g.NW - 1)) != 0) return false;
  if ((reinterpret_cast<uintptr_t>(x) & 15) != 0 || (reinterpret_cast<uintptr_t>(y) & 15) != 0) return false;
  const int64_t wpi = g.NH * g.NW, be = (int64_t)WIN * g.W, hw = g.H * g.W;
  const bool inside = wpi % 16 == 0;        // sub-tile = bands of one image
  const bool whole = !inside && 16 % wpi == 0;  // sub-tile = whole images
  if (!inside && !whole) return false;
  if (inside ? be % 8 != 0 : hw % 8 != 0) return false;
  // chunk offsets inside a sub-tile are 32-bit byte offsets
  if (whole && 2 * (16 / wpi) * g.C * hw >= ((int64_t)1 << 31)) return false;
  constexpr int RPP = ImgCfg<WIN>::RPP;
  ia.chw = g.C * hw;
  ia.hw = hw;
  ia.W = (int)g.W;
  ia.BE = (int)be;
  int lg = 0;
  while ((1 << lg) < g.NW) ++lg;
  ia.lgnw = lg;
  ia.NH = (int)g.NH;
  ia.WPI = (int)wpi;
  ia.whole = whole ? 1 : 0;
  ia.SEGC = whole ? (int)(hw / 8) : ImgCfg<WIN>::CH;
  ia.inv_segc = whole ? 1.0f / (float)ia.SEGC : 0.0f;  // one piece: chunk q is at 16 q
  ia.pair_store = (RPP * g.W) % 8 == 0 && ((WIN % RPP) * g.W) % 8 == 0 && be % 8 == 0;
  ia.CPR = ia.pair_store ? (int)(RPP * g.W / 8) : 1;
  ia.inv_cpr = 1.0f / (float)ia.CPR;
  ia.inv_nh = 1.0f / (float)ia.NH;
  ia.gap = whole ? (uint32_t)(2 * ia.chw - 16 * (int64_t)ia.SEGC) : 0u;
  return true;
}

template <class Tag, int WIN>
static hipError_t run_forward(const void *x, const void *t, void *y, const Geom &g, bool rev,
                              hipStream_t st) {
  typedef typename Tag::S S;
  KArgs a = make_args(g);
  a.tile = pick_fwd_tile<Tag, WIN>(g);
  a.tiles_per_ch = (int)cdiv64(g.N, a.tile);
  const dim3 grid((unsigned)(g.C * a.tiles_per_ch));
  if constexpr (Tag::W16) {
    ImgArgs ia;
    if (img_layout<WIN>(g, x, y, ia)) {
      constexpr size_t ilds = fwd_img_lds_bytes<Tag, WIN>();
      static_assert(ilds <= 65536, "workgroup LDS above 64 KB");
      if (rev)
        wbmm_fwd_img_kernel<Tag, WIN, true><<<grid, dim3(kFwdThreads), ilds, st>>>((const S *)x, (const S *)t, nullptr,
                                                                                  (S *)y, a, ia);
      else
        wbmm_fwd_img_kernel<Tag, WIN, false><<<grid, dim3(kFwdThreads), ilds, st>>>((const S *)x, (const S *)t, nullptr,
                                                                                   (S *)y, a, ia);
      return hipGetLastError();
    }
  }
  constexpr size_t lds = fwd_lds_bytes<Tag, WIN>();
  // float32 windows of 13 and more take up to 70 KB (LDS is reached with ds
  // instructions only)
  static_assert(lds <= 160 * 1024, "workgroup LDS above the 160 KB of a compute unit");
  if constexpr (Tag::ES == 4 || WIN % 2 == 0) {
    set_tiled<WIN, Tag::ES>(g, a, {x, y});
    if (a.tiled) {
      if (rev)
        wbmm_fwd_kernel<Tag, WIN, true, false, true><<<grid, dim3(kFwdThreads), lds, st>>>((const S *)x, (const S *)t, nullptr,
                                                                                          (S *)y, a);
      else
        wbmm_fwd_kernel<Tag, WIN, false, false, true><<<grid, dim3(kFwdThreads), lds, st>>>((const S *)x, (const S *)t, nullptr,
                                                                                           (S *)y, a);
      return hipGetLastError();
    }
  }
  if (rev)
    wbmm_fwd_kernel<Tag, WIN, true><<<grid, dim3(kFwdThreads), lds, st>>>((const S *)x, (const S *)t, nullptr, (S *)y, a);
  else
    wbmm_fwd_kernel<Tag, WIN, false><<<grid, dim3(kFwdThreads), lds, st>>>((const S *)x, (const S *)t, nullptr, (S *)y, a);
  return hipGetLastError();
}

// Hierarchical form, window WIN = 2 wl: y = x M_fused per window (both tables
// read back to front for the input gradient).
template <class Tag, int WIN>
static hipError_t run_hier_forward(const void *x, const void *tg, const void *tl, void *y, const Geom &g, bool rev,
                                   hipStream_t st) {
  if constexpr (WIN % 2 != 0) {
    return hipErrorInvalidValue;
  } else {
    typedef typename Tag::S S;
    KArgs a = make_args(g);
    a.tile = pick_fwd_tile<Tag, WIN>(g);
    a.tiles_per_ch = (int)cdiv64(g.N, a.tile);
    const dim3 grid((unsigned)(g.C * a.tiles_per_ch));
    if constexpr (Tag::W16) {
      ImgArgs ia;
      if (img_layout<WIN>(g, x, y, ia)) {
        constexpr size_t ilds = fwd_img_lds_bytes<Tag, WIN, true>();
        static_assert(ilds <= 65536, "workgroup LDS above 64 KB");
        if (rev)
          wbmm_fwd_img_kernel<Tag, WIN, true, true><<<grid, dim3(kFwdThreads), ilds, st>>>(
              (const S *)x, (const S *)tg, (const S *)tl, (S *)y, a, ia);
        else
          wbmm_fwd_img_kernel<Tag, WIN, false, true><<<grid, dim3(kFwdThreads), ilds, st>>>(
              (const S *)x, (const S *)tg, (const S *)tl, (S *)y, a, ia);
        return hipGetLastError();
      }
    }
    constexpr size_t lds = fwd_lds_bytes<Tag, WIN, true>();
    static_assert(lds <= 160 * 1024, "workgroup LDS above the 160 KB of a compute unit");
    if (rev)
      wbmm_fwd_kernel<Tag, WIN, true, true><<<grid, dim3(kFwdThreads), lds, st>>>((const S *)x, (const S *)tg,
                                                                                  (const S *)tl, (S *)y, a);
    else
      wbmm_fwd_kernel<Tag, WIN, false, true><<<grid, dim3(kFwdThreads), lds, st>>>((const S *)x, (const S *)tg,
                                                                                   (const S *)tl, (S *)y, a);
    return hipGetLastError();
  }
}

template <class Tag, int WIN>
static DtPlan plan_dt(const Geom &g) {
  typedef DtCfg<Tag, WIN> G;
  DtPlan p;
  const int64_t stages = cdiv64(g.N, G::CW);
  int64_t slabs = cdiv64(1024, g.C);
  if (slabs > stages) slabs = stages;
  if (slabs < 1) slabs = 1;
  p.slab_windows = cdiv64(cdiv64(g.N, slabs), G::CW) * G::CW;
  p.slabs = cdiv64(g.N, p.slab_windows);
  return p;
}


// Launch plan of the channel-stream kernel (fixed-offset rows): one
// workgroup per (channel, slab), at most one per compute unit at a time; with
// more channels than compute units, one slab per channel in rounds (see
// below).  Its slabs never outnumber those of plan_dt, which sizes the
// workspace.
template <class Tag, int WIN>
static bool stream_runs(const Geom &g, KArgs &b, int ncu) {
  typedef BwdCfg<Tag, WIN> G;
  if constexpr (!StreamCfg<Tag, WIN>::RUNS) {
    (void)g; (void)b; (void)ncu;
    return false;
  } else {
    const int64_t nstc = cdiv64(g.N, G::CW), tot = g.C * nstc;
    if (tot >= ((int64_t)1 << 31)) return false;
    const int64_t L = cdiv64(tot, ncu);
    // every channel within at most two runs, every run over at most two
    // channels
    for (int64_t c = 0; c < g.C; ++c)
      if ((c * nstc + nstc - 1) / L - (c * nstc) / L > 1) return false;
    for (int64_t r = 0; r * L < tot; ++r) {
      const int64_t e = ((r + 1) * L < tot ? (r + 1) * L : tot) - 1;
      if (e / nstc - (r * L) / nstc > 1) return false;
    }
    b.run = (int)L;
    b.nstc = (int)nstc;
    b.tile = 0;
    b.tiles_per_ch = 0;
    return true;
  }
}

// Workgroups of a channel-stream launch planned by stream_plan, and the
// partial tables per channel the sum kernel adds (1: none).
static int64_t stream_grid(const Geom &g, const KArgs &b) {
  return b.run > 0 ? cdiv64(g.C * (int64_t)b.nstc, b.run) : g.C * b.tiles_per_ch;
}
static int64_t stream_parts(const KArgs &b) { return b.run > 0 ? 2 : b.tiles_per_ch; }

template <class Tag, int WIN>
static bool stream_plan(const Geom &g, KArgs &b, bool rounds = false, int64_t ws_slabs = 0) {
  typedef BwdCfg<Tag, WIN> G;
  const int ncu = compute_units();
  b.run = 0;
  b.nstc = 0;
  if (!b.tiled || ncu <= 0) return false;
  if (g.C > ncu) {
    // more channels than compute units (where the caller allows it): whole
    // channels in rounds of one workgroup per compute unit when the last
    // round fills at least half the chip; else runs of consecutive stages
    // over all channels, one per compute unit, when they apply and the
    // workspace holds two partial tables per channel (measured: runs and
    // their sum launch lose to a half-full last round, and beat the
    // four-wave kernels)
    if (!rounds) return false;
    const int64_t rem = g.C % ncu;
    if (rem != 0 && rem < ncu / 2) return ws_slabs >= 2 && stream_runs<Tag, WIN>(g, b, ncu);
  }
  const int64_t stages = cdiv64(g.N, G::CW);
  int64_t slabs = ncu / g.C;
  if (slabs > stages) slabs = stages;
  if (slabs < 1) slabs = 1;
  b.tile = (int)(cdiv64(cdiv64(g.N, slabs), G::CW) * G::CW);
  b.tiles_per_ch = (int)cdiv64(g.N, b.tile);
  return true;
}

template <int WIN>
constexpr int64_t table_len() { return (int64_t)(2 * WIN - 1) * (2 * WIN - 1); }

// After a launch: its error, else (several slabs per channel) the launch of
// the kernel that sums the slab partials into the table gradient(s).
static hipError_t sum_slabs(const float *part, float *dt, int64_t n, const float *part2, float *dt2, int64_t n2,
                            int64_t slabs, hipStream_t st) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || slabs <= 1) return e;
  return launch_dt_sum(part, dt, n, part2, dt2, n2, (int)slabs, st);
}

template <class Tag, int WIN>
static hipError_t run_dtable(const void *x, const void *dy, float *dt, void *ws, const Geom &g,
                             hipStream_t st) {
  typedef typename Tag::S S;
  KArgs a = make_args(g);
  const DtPlan p = plan_dt<Tag, WIN>(g);
  a.tile = (int)p.slab_windows;
  a.tiles_per_ch = (int)p.slabs;
  set_tiled<WIN, Tag::ES>(g, a, {x, dy});
  if constexpr (Tag::ES == 4 || WIN % 2 == 0) {
    KArgs b = a;
    if (stream_plan<Tag, WIN>(g, b, true, p.slabs)) {
      // the same stages, bins and sums as the fused pass
      float *spart = stream_parts(b) > 1 ? (float *)ws : nullptr;
      constexpr size_t slds = stream_lds_bytes<Tag, WIN>();
      // (no input-gradient products: the eight idle waves copy as well)
      bool launched = false;
      if constexpr (StreamCfg<Tag, WIN>::RUNS) {
        if (b.run > 0) {
          wbmm_bwd_stream_kernel<Tag, WIN, false, 0, 0, true><<<dim3((unsigned)stream_grid(g, b)),
                                                                 dim3(stream_threads<0>()), slds, st>>>(
              (const S *)x, (const S *)dy, nullptr, nullptr, dt, spart, b, nullptr, nullptr, nullptr);
          launched = true;
        }
      }
      if (!launched)
        wbmm_bwd_stream_kernel<Tag, WIN, false, 0, 0><<<dim3((unsigned)stream_grid(g, b)),
                                                        dim3(stream_threads<0>()), slds, st>>>(
            (const S *)x, (const S *)dy, nullptr, nullptr, dt, spart, b, nullptr, nullptr, nullptr);
      return sum_slabs(spart, dt, g.C * table_len<WIN>(), nullptr, nullptr, 0, stream_parts(b), st);
    }
  }
  float *part = p.slabs > 1 ? (float *)ws : nullptr;
  constexpr size_t lds = dt_lds_bytes<Tag, WIN>();
  static_assert(lds <= 65536, "workgroup LDS above 64 KB");
  const dim3 grid((unsigned)(g.C * p.slabs));
  if constexpr (Tag::ES == 4 || WIN % 2 == 0) {
    if (a.tiled) {
      wbmm_dt_kernel<Tag, WIN, true><<<grid, dim3(kThreads), lds, st>>>((const S *)x, (const S *)dy, dt, part, a);
      return sum_slabs(part, dt, g.C * table_len<WIN>(), nullptr, nullptr, 0, p.slabs, st);
    }
  }
  wbmm_dt_kernel<Tag, WIN, false><<<grid, dim3(kThreads), lds, st>>>((const S *)x, (const S *)dy, dt, part, a);
  return sum_slabs(part, dt, g.C * table_len<WIN>(), nullptr, nullptr, 0, p.slabs, st);
}

template <class Tag, int WIN>
static hipError_t run_backward(const void *x, const void *dy, const void *t, void *dx, float *dt, void *ws,
                               const Geom &g, hipStream_t st) {
  typedef typename Tag::S S;
  KArgs a = make_args(g);
  const DtPlan p = plan_dt<Tag, WIN>(g);
  a.tile = (int)p.slab_windows;
  a.tiles_per_ch = (int)p.slabs;
  set_tiled<WIN, Tag::ES>(g, a, {x, dy, dx});
  if constexpr (Tag::ES == 4 || WIN % 2 == 0) {
    KArgs b = a;
    if (stream_plan<Tag, WIN>(g, b, true, p.slabs)) {
      float *spart = stream_parts(b) > 1 ? (float *)ws : nullptr;
      constexpr size_t slds = stream_lds_bytes<Tag, WIN>();
      static_assert(slds <= 160 * 1024, "workgroup LDS above the 160 KB of a compute unit");
      bool launched = false;
      if constexpr (StreamCfg<Tag, WIN>::RUNS) {
        if (b.run > 0) {
          wbmm_bwd_stream_kernel<Tag, WIN, true, 0, kCopyWaves, true><<<dim3((unsigned)stream_grid(g, b)),
                                                                         dim3(stream_threads<kCopyWaves>()), slds, st>>>(
              (const S *)x, (const S *)dy, (const S *)t, (S *)dx, dt, spart, b, nullptr, nullptr, nullptr);
          launched = true;
        }
      }
      if (!launched)
        wbmm_bwd_stream_kernel<Tag, WIN, true, 0, kCopyWaves><<<dim3((unsigned)stream_grid(g, b)),
                                                                dim3(stream_threads<kCopyWaves>()), slds, st>>>(
            (const S *)x, (const S *)dy, (const S *)t, (S *)dx, dt, spart, b, nullptr, nullptr, nullptr);
      return sum_slabs(spart, dt, g.C * table_len<WIN>(), nullptr, nullptr, 0, stream_parts(b), st);
    }
  }
  float *part = p.slabs > 1 ? (float *)ws : nullptr;
  constexpr size_t lds = bwd_lds_bytes<Tag, WIN>();
  static_assert(lds <= 65536, "workgroup LDS above 64 KB");
  const dim3 grid((unsigned)(g.C * p.slabs));
  if constexpr (Tag::ES == 4 || WIN % 2 == 0) {
    if (a.tiled) {
      wbmm_bwd_kernel<Tag, WIN, true><<<grid, dim3(kThreads), lds, st>>>((const S *)x, (const S *)dy, (const S *)t,
                                                                         (S *)dx, dt, part, a);
      return sum_slabs(part, dt, g.C * table_len<WIN>(), nullptr, nullptr, 0, p.slabs, st);
    }
  }
  wbmm_bwd_kernel<Tag, WIN, false><<<grid, dim3(kThreads), lds, st>>>((const S *)x, (const S *)dy, (const S *)t,
                                                                      (S *)dx, dt, part, a);
  return sum_slabs(part, dt, g.C * table_len<WIN>(), nullptr, nullptr, 0, p.slabs, st);
}

// Hierarchical form (global window WIN = 2 wl): one channel-stream pass when
// it applies (one window row per tile, fixed-offset rows, no more channels
// than compute units, and the workspace holds both tables' partials): both
// table gradients, and with dx the input gradient too; *done tells whether
// it ran.
template <class Tag, int WIN>
static hipError_t run_hier_stream(const void *x, const void *dy, const void *tg, const void *tl, void *dx, float *dtg,
                                  float *dtl, void *ws, size_t ws_bytes, const Geom &g, hipStream_t st, bool *done) {
  *done = false;
  if constexpr (WIN % 2 == 0 && rp_of(WIN) == 16) {
    typedef typename Tag::S S;
    constexpr int WL = WIN / 2;
    constexpr int64_t K2 = (2 * WIN - 1) * (2 * WIN - 1), K2L = (2 * WL - 1) * (2 * WL - 1);
    KArgs a = make_args(g);
    const DtPlan p = plan_dt<Tag, WIN>(g);
    a.tile = (int)p.slab_windows;
    a.tiles_per_ch = (int)p.slabs;
    if (dx) set_tiled<WIN, Tag::ES>(g, a, {x, dy, dx});
    else set_tiled<WIN, Tag::ES>(g, a, {x, dy});
    KArgs b = a;
    if (!stream_plan<Tag, WIN>(g, b)) return hipSuccess;
    float *partg = nullptr, *partl = nullptr;
    if (b.tiles_per_ch > 1) {
      const size_t need = (size_t)b.tiles_per_ch * (size_t)g.C * (size_t)(K2 + K2L) * 4;
      if (ws == nullptr || need > ws_bytes) return hipSuccess;
      partg = (float *)ws;
      partl = partg + (size_t)b.tiles_per_ch * (size_t)g.C * (size_t)K2;
    }
    const dim3 grid((unsigned)(g.C * b.tiles_per_ch));
    if (dx) {
      constexpr size_t slds = stream_lds_bytes<Tag, WIN, true>();
      static_assert(slds <= 160 * 1024, "workgroup LDS above the 160 KB of a compute unit");
      wbmm_bwd_stream_kernel<Tag, WIN, true, WL><<<grid, dim3(stream_threads<0>()), slds, st>>>(
          (const S *)x, (const S *)dy, (const S *)tg, (S *)dx, dtg, partg, b, dtl, partl, (const S *)tl);
    } else {
      constexpr size_t slds = stream_lds_bytes<Tag, WIN>();
      wbmm_bwd_stream_kernel<Tag, WIN, false, WL><<<grid, dim3(stream_threads<0>()), slds, st>>>(
          (const S *)x, (const S *)dy, nullptr, nullptr, dtg, partg, b, dtl, partl, nullptr);
    }
    *done = true;
    return sum_slabs(partg, dtg, g.C * K2, partl, dtl, g.C * K2L, b.tiles_per_ch, st);
  } else {
    (void)x; (void)dy; (void)tg; (void)tl; (void)dx; (void)dtg; (void)dtl; (void)ws; (void)ws_bytes; (void)g;
    (void)st;
    return hipSuccess;
  }
}

}  // namespace wbmm
