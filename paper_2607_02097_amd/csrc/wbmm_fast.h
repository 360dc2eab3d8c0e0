// Fast-path WBMM kernels (included by wbmm_kernels.h).
//
// Window bands (w image rows of one (b, c) plane, contiguous in NCHW) are
// copied raw into LDS with aligned 16-byte global loads, each band into its
// own LDS slot at the same offset modulo 16 as in global memory.  The window
// view is taken at matrix-fragment time: a lane gathers the 8 elements of its
// fragment with 16-bit LDS reads, masked to zero outside the window (padded
// columns and rows, positions outside the image, windows past the end).  No
// zero fill, no per-element address decoding on the copy path.
#pragma once

namespace wbmm {

struct FArgs {
  int64_t B, C, H, W;
  int64_t NH, NW;
  int64_t nbands;       // B * NH bands per channel
  int bpt;              // bands per LDS stage
  int tiles_per_ch;     // workgroups per channel
  int stages;           // LDS stages per workgroup (table gradient)
  int bstride;          // LDS bytes per band slot, multiple of 16
  float inv_nw, inv_nh, inv_cps;
};

// floor(v / d) for 0 <= v, d < 2^24 from a float reciprocal, corrected.
__device__ inline int fdiv(int v, int d, float inv) {
  int q = (int)((float)v * inv);
  if (q * d > v) --q;
  else if ((q + 1) * d <= v) ++q;
  return q;
}

// Geometry of band bi of channel c: byte offset of its first element from the
// tensor base, number of image rows it holds, and its byte length.
template <int WIN, int ES>
__device__ inline void band_geom(const FArgs &a, int64_t c, int64_t bi, int64_t &boff, int &rows,
                                 int &blen) {
  const int64_t b = fdiv((int)bi, (int)a.NH, a.inv_nh);
  const int64_t wy = bi - b * a.NH;
  const int64_t r64 = a.H - wy * WIN;
  rows = r64 < WIN ? (int)r64 : WIN;
  boff = (((b * a.C + c) * a.H + wy * WIN) * a.W) * ES;
  blen = rows * (int)a.W * ES;
}

__device__ inline int addr_mis(const void *base, int64_t boff) {
  return (int)((reinterpret_cast<uintptr_t>(base) + (uint64_t)boff) & 15u);
}

// Raw copy of bands [bi0, bi0 + nb) of channel c into LDS slots.  binfo[j]
// receives (misalignment, rows) of band j.  Chunk slots past a band's end are
// skipped; chunks crossing the band's edge load only the band's elements.
template <int WIN, int ES>
__device__ inline void stage_bands(const void *src, char *lds, int2 *binfo, const FArgs &a,
                                   int64_t c, int64_t bi0, int nb, int tid) {
  constexpr int VE = 16 / ES;
  const int cps = a.bstride >> 4;
  const int total = nb * cps;
  constexpr int U = 8;
  for (int s0 = tid; s0 < total; s0 += kThreads * U) {
    uint4 v[U];
    int dst[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      dst[k] = -1;
      const int slot = s0 + k * kThreads;
      if (slot >= total) continue;
      const int j = fdiv(slot, cps, a.inv_cps);
      const int ci = slot - j * cps;
      int64_t boff;
      int rows, blen;
      band_geom<WIN, ES>(a, c, bi0 + j, boff, rows, blen);
      const int mis = addr_mis(src, boff);
      if (ci == 0) binfo[j] = make_int2(mis, rows);
      const int lo = ci * 16 - mis;  // band byte offset of the chunk start
      if (lo >= blen) continue;
      const char *p = reinterpret_cast<const char *>(src) + (boff + lo);
      dst[k] = j * a.bstride + ci * 16;
      if (lo >= 0 && lo + 16 <= blen) {
        v[k] = *reinterpret_cast<const uint4 *>(p);
      } else {
        uint32_t w4[4] = {0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < VE; ++u) {
          const int bo = lo + u * ES;
          if (bo >= 0 && bo < blen) {
            uint32_t e;
            if (ES == 4) e = *reinterpret_cast<const uint32_t *>(p + u * ES);
            else e = *reinterpret_cast<const u16 *>(p + u * ES);
            if (ES == 4) w4[u] = e;
            else w4[u >> 1] |= (u & 1) ? (e << 16) : e;
          }
        }
        v[k] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k)
      if (dst[k] >= 0) *reinterpret_cast<uint4 *>(lds + dst[k]) = v[k];
  }
}

// Copy bands back from LDS to global (same geometry, the destination may sit
// at another offset modulo 16 than the source the slots were filled from).
template <int WIN, int ES>
__device__ inline void unstage_bands(void *dstp, const char *lds, const int2 *binfo, const FArgs &a,
                                     int64_t c, int64_t bi0, int nb, int tid) {
  constexpr int VE = 16 / ES;
  const int cps = a.bstride >> 4;
  const int total = nb * cps;
  for (int slot = tid; slot < total; slot += kThreads) {
    const int j = fdiv(slot, cps, a.inv_cps);
    const int ci = slot - j * cps;
    int64_t boff;
    int rows, blen;
    band_geom<WIN, ES>(a, c, bi0 + j, boff, rows, blen);
    const int mis = addr_mis(dstp, boff);
    const int lo = ci * 16 - mis;
    if (lo >= blen) continue;
    char *p = reinterpret_cast<char *>(dstp) + (boff + lo);
    const int smis = binfo[j].x;                 // where the band starts in its slot
    const char *q = lds + j * a.bstride + smis + lo;  // LDS bytes for p[0..16)
    if (lo >= 0 && lo + 16 <= blen) {
      uint4 v;
      if (smis == mis) {
        v = *reinterpret_cast<const uint4 *>(q);
      } else if (((smis - mis) & 3) == 0) {
        const uint32_t *q4 = reinterpret_cast<const uint32_t *>(q);
        v = make_uint4(q4[0], q4[1], q4[2], q4[3]);
      } else {
        const u16 *q2 = reinterpret_cast<const u16 *>(q);
        v = make_uint4(q2[0] | ((uint32_t)q2[1] << 16), q2[2] | ((uint32_t)q2[3] << 16),
                       q2[4] | ((uint32_t)q2[5] << 16), q2[6] | ((uint32_t)q2[7] << 16));
      }
      *reinterpret_cast<uint4 *>(p) = v;
    } else {
#pragma unroll
      for (int u = 0; u < VE; ++u) {
        const int bo = lo + u * ES;
        if (bo >= 0 && bo < blen) {
          if (ES == 4) *reinterpret_cast<uint32_t *>(p + u * ES) = *reinterpret_cast<const uint32_t *>(q + u * ES);
          else *reinterpret_cast<u16 *>(p + u * ES) = *reinterpret_cast<const u16 *>(q + u * ES);
        }
      }
    }
  }
}

// Per-window view into the staged bands: LDS byte offset of the window's
// element (0, 0) and the number of valid rows / columns (0 if no window).
struct WinRef {
  int base;
  int rows;
  int cols;
};

template <int WIN, int ES>
__device__ inline WinRef win_ref(const FArgs &a, const int2 *binfo, int v, int nwin) {
  WinRef r;
  if (v >= nwin) {
    r.base = 0; r.rows = 0; r.cols = 0;
    return r;
  }
  const int nw = (int)a.NW;
  const int j = fdiv(v, nw, a.inv_nw);
  const int wx = v - j * nw;
  const int2 bi = binfo[j];
  const int c64 = (int)a.W - wx * WIN;
  r.base = j * a.bstride + bi.x + wx * WIN * ES;
  r.rows = bi.y;
  r.cols = c64 < WIN ? c64 : WIN;
  return r;
}

// ======================================================== fast forward

template <class Tag, int WIN>
__host__ __device__ constexpr size_t fwdf_lds_bytes(int bpt, int bstride) {
  typedef FwdCfg<Tag, WIN> G;
  return (size_t)bpt * bstride + 64 + (size_t)bpt * sizeof(int2) +
         (size_t)(G::TS_LEN + G::TB_LEN) * Tag::ES + 16;
}

template <class Tag, int WIN, bool REV>
__global__ __launch_bounds__(kThreads) void wbmm_fwd_fast_kernel(const typename Tag::S *__restrict__ x,
                                                                 const typename Tag::S *__restrict__ tab,
                                                                 typename Tag::S *__restrict__ y, FArgs a) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef FwdCfg<Tag, WIN> G;
  constexpr int RP = G::RP, K1 = G::K1, K2 = G::K2, ES = Tag::ES;

  extern __shared__ __align__(16) unsigned char smem[];
  char *bands = reinterpret_cast<char *>(smem);
  int2 *binfo = reinterpret_cast<int2 *>(bands + a.bpt * a.bstride + 64);
  S *Ts = reinterpret_cast<S *>(
      reinterpret_cast<char *>(binfo) + ((a.bpt * sizeof(int2) + 15) & ~(size_t)15));
  S *TB = Ts + G::TS_LEN;
  const S *lds_e = reinterpret_cast<const S *>(bands);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t c = blockIdx.x / a.tiles_per_ch;
  const int64_t tix = blockIdx.x - c * a.tiles_per_ch;
  const int64_t bi0 = tix * a.bpt;
  const int nb = (int)((bi0 + a.bpt <= a.nbands) ? a.bpt : a.nbands - bi0);
  const int nwin = nb * (int)a.NW;

  // ---- stage: table, bands
  for (int k = tid; k < K2; k += kThreads) Ts[k] = tab[c * K2 + (REV ? K2 - 1 - k : k)];
  stage_bands<WIN, ES>(x, bands, binfo, a, c, bi0, nb, tid);
  __syncthreads();

  const int g = lane >> 4;
  const int ln = lane & 15;
  const int Wi = (int)a.W;
  const int nsub = (nwin + 15) >> 4;

  if constexpr (Tag::W16) {
    constexpr int S_ = G::S, NT = G::NT, NB = G::NB;
    // Toeplitz blocks of M_c: TB[dh][x_out][x_in]
    for (int i = tid; i < G::TB_LEN; i += kThreads) {
      const int dhi = i / (RP * RP);
      const int rem = i - dhi * RP * RP;
      const int xo = rem / RP;
      const int xi = rem - xo * RP;
      TB[i] = (xo < WIN && xi < WIN) ? Ts[dhi * K1 + xi - xo + WIN - 1] : (S)0;
    }
    __syncthreads();
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
    for (int sub = wave; sub < nsub; sub += kWaves) {
      // A fragments: window (sub*16 + ln), positions 32s + 8g .. + 7
      const WinRef wa = win_ref<WIN, ES>(a, binfo, sub * 16 + ln, nwin);
      Frag af[S_];
#pragma unroll
      for (int s = 0; s < S_; ++s) {
        const int k0 = 32 * s + 8 * g;
        const int hi = k0 / RP, xi0 = k0 % RP;
        Frag f = Frag{0, 0, 0, 0, 0, 0, 0, 0};
        if (hi < wa.rows) {
          const int e0 = (wa.base >> 1) + hi * Wi + xi0;
#pragma unroll
          for (int e = 0; e < 8; ++e) f[e] = (xi0 + e < wa.cols) ? lds_e[e0 + e] : (u16)0;
        }
        af[s] = f;
      }
      WinRef wc[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) wc[r] = win_ref<WIN, ES>(a, binfo, sub * 16 + 4 * g + r, nwin);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < S_; ++s) acc = mma<Tag>(af[s], bf[2 * s - t + NT - 1], acc);
        const int p = 16 * t + ln;
        const int ho = p / RP, xo = p % RP;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (ho < wc[r].rows && xo < wc[r].cols)
            reinterpret_cast<S *>(bands)[(wc[r].base >> 1) + ho * Wi + xo] = from_f32<Tag>(acc[r]);
      }
    }
  } else {
    constexpr int S_ = G::S, NT = G::NT;
    for (int sub = wave; sub < nsub; sub += kWaves) {
      const WinRef wa = win_ref<WIN, ES>(a, binfo, sub * 16 + ln, nwin);
      float af[S_];
#pragma unroll
      for (int s = 0; s < S_; ++s) {
        const int k = 4 * s + g;
        const int hi = k / RP, xi = k % RP;
        af[s] = (hi < wa.rows && xi < wa.cols) ? lds_e[(wa.base >> 2) + hi * Wi + xi] : 0.f;
      }
      WinRef wc[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) wc[r] = win_ref<WIN, ES>(a, binfo, sub * 16 + 4 * g + r, nwin);
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
          acc = mma<Tag>(af[s], bv, acc);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (ho < wc[r].rows && xo < wc[r].cols)
            reinterpret_cast<S *>(bands)[(wc[r].base >> 2) + ho * Wi + xo] = acc[r];
      }
    }
  }
  __syncthreads();
  unstage_bands<WIN, ES>(y, bands, binfo, a, c, bi0, nb, tid);
}

// =================================================== fast table gradient

template <class Tag, int WIN>
__host__ __device__ constexpr size_t dtf_lds_bytes(int bpt, int bstride) {
  typedef DtCfg<Tag, WIN> G;
  const size_t ops = 2 * ((size_t)bpt * bstride + 64) + 2 * (size_t)bpt * sizeof(int2) + 32;
  const size_t bins = (size_t)(kWaves * 16 * 17 + G::NACC * G::NBT) * 4;
  return ops > bins ? ops : bins;
}

template <class Tag, int WIN, int WAVE>
__device__ void dtf_wave(const typename Tag::S *__restrict__ x, const typename Tag::S *__restrict__ dy,
                         float *__restrict__ out, const FArgs &a, unsigned char *smem) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef DtCfg<Tag, WIN> G;
  constexpr int NPT = G::NPT, RP = G::RP, R = G::R, ES = Tag::ES;
  constexpr int K1 = G::K1, K2 = G::K2, NBT = G::NBT;
  constexpr PAssign<NPT> PA = make_passign<NPT>();
  constexpr int NP = PA.count[WAVE];

  const int slot_bytes = a.bpt * a.bstride + 64;
  char *xb = reinterpret_cast<char *>(smem);
  char *db = xb + slot_bytes;
  int2 *xinfo = reinterpret_cast<int2 *>(db + slot_bytes);
  int2 *dinfo = xinfo + a.bpt;
  const S *xe = reinterpret_cast<const S *>(xb);
  const S *de = reinterpret_cast<const S *>(db);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int g = lane >> 4;
  const int ln = lane & 15;
  const int Wi = (int)a.W;
  const int64_t c = blockIdx.x / a.tiles_per_ch;
  const int64_t slab = blockIdx.x - c * a.tiles_per_ch;

  f32x4 acc[NP > 0 ? NP : 1];
#pragma unroll
  for (int j = 0; j < NP; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // position offsets (in elements, relative to a window's (0,0)) of this
  // lane's fragment row/column in every 16-position tile, and their validity
  for (int st = 0; st < a.stages; ++st) {
    const int64_t bi0 = (slab * a.stages + st) * a.bpt;
    if (bi0 >= a.nbands) break;
    const int nb = (int)((bi0 + a.bpt <= a.nbands) ? a.bpt : a.nbands - bi0);
    const int nwin = nb * (int)a.NW;
    if (st > 0) __syncthreads();
    stage_bands<WIN, ES>(x, xb, xinfo, a, c, bi0, nb, tid);
    stage_bands<WIN, ES>(dy, db, dinfo, a, c, bi0, nb, tid);
    __syncthreads();

    for (int k0 = 0; k0 < nwin; k0 += 32) {
      // the 8 windows whose values this lane contributes to each fragment
      int xbase[8], dbase[8], rows[8], cols[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int v = k0 + (Tag::W16 ? 8 * g + e : 4 * e + g);
        const WinRef wx = win_ref<WIN, ES>(a, xinfo, v, nwin);
        const WinRef wd = win_ref<WIN, ES>(a, dinfo, v, nwin);
        xbase[e] = wx.base / ES;
        dbase[e] = wd.base / ES;
        rows[e] = wx.rows;
        cols[e] = wx.cols;
      }
      if constexpr (Tag::W16) {
        Frag bf[NPT];
#pragma unroll
        for (int po = 0; po < NPT; ++po) {
          const int p = 16 * po + ln;
          const int hi = p / RP, xi = p % RP;
          const int off = hi * Wi + xi;
          Frag f;
#pragma unroll
          for (int e = 0; e < 8; ++e) f[e] = (hi < rows[e] && xi < cols[e]) ? de[dbase[e] + off] : (u16)0;
          bf[po] = f;
        }
#pragma unroll
        for (int pi = 0; pi < NPT; ++pi) {
          const int p = 16 * pi + ln;
          const int hi = p / RP, xi = p % RP;
          const int off = hi * Wi + xi;
          Frag af;
#pragma unroll
          for (int e = 0; e < 8; ++e) af[e] = (hi < rows[e] && xi < cols[e]) ? xe[xbase[e] + off] : (u16)0;
#pragma unroll
          for (int j = 0; j < NP; ++j) {
            const int po = pi - (PA.list[WAVE][j] - (NPT - 1));
            if (po >= 0 && po < NPT) acc[j] = mma<Tag>(af, bf[po], acc[j]);
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float bf[NPT];
#pragma unroll
          for (int po = 0; po < NPT; ++po) {
            const int p = 16 * po + ln;
            const int hi = p / RP, xi = p % RP;
            bf[po] = (hi < rows[e] && xi < cols[e]) ? de[dbase[e] + hi * Wi + xi] : 0.f;
          }
#pragma unroll
          for (int pi = 0; pi < NPT; ++pi) {
            const int p = 16 * pi + ln;
            const int hi = p / RP, xi = p % RP;
            const float af = (hi < rows[e] && xi < cols[e]) ? xe[xbase[e] + hi * Wi + xi] : 0.f;
#pragma unroll
            for (int j = 0; j < NP; ++j) {
              const int po = pi - (PA.list[WAVE][j] - (NPT - 1));
              if (po >= 0 && po < NPT) acc[j] = mma<Tag>(af, bf[po], acc[j]);
            }
          }
        }
      }
    }
  }
  __syncthreads();

  // ---- diagonal binning, fixed order (same as the generic kernel)
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
      const int da = bin / K1 - (R - 1);
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
__global__ __launch_bounds__(kThreads) void wbmm_dt_fast_kernel(const typename Tag::S *__restrict__ x,
                                                                const typename Tag::S *__restrict__ dy,
                                                                float *__restrict__ out, FArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  switch (threadIdx.x >> 6) {
    case 0: dtf_wave<Tag, WIN, 0>(x, dy, out, a, smem); break;
    case 1: dtf_wave<Tag, WIN, 1>(x, dy, out, a, smem); break;
    case 2: dtf_wave<Tag, WIN, 2>(x, dy, out, a, smem); break;
    default: dtf_wave<Tag, WIN, 3>(x, dy, out, a, smem); break;
  }
}

}  // namespace wbmm
