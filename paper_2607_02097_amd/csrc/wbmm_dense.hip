// Cached-matrix (dense) form of WBMM for any window w_h x w_w with
// d = w_h w_w <= 256 (Alg. 1 with the matrix built once, eq. index_select):
//   build:    M_c[i, j] = T[c, I(i, j)]                    (matrix per channel)
//   forward:  Y_window = X_window M_c, or X_window M_c^T   (input gradient)
//   gradient: dM_c = sum over windows of X_window^T dY_window   (float32)
//   bin:      dT[c, k] = sum of dM_c[i, j] over I(i, j) = k (fixed order)
// Positions are row-major inside a window, p = h * w_w + x.  M is an
// arbitrary dense matrix here (the table form's Toeplitz structure is not
// used), so rectangular windows, fused matrices and any cached M share one
// path.  The kernels are generic over the window (runtime sizes) and
// instantiated once per dtype.
#include "wbmm_kernels.h"

namespace wbmm {

constexpr int kDenseMaxD = 256;

template <class Tag>
struct DenseCfg {
  static constexpr int WAVES = Tag::W16 ? 4 : 2;       // 16 windows per wave
  static constexpr int TW = 16 * WAVES;                // windows per workgroup
  static constexpr int NC = Tag::W16 ? 32 : 16;        // output positions per chunk
  static constexpr int KMAX = kDenseMaxD;              // padded K bound
  static constexpr int LDSX = Tag::W16 ? KMAX + 8 : KMAX + 4;  // row pitch (elements)
  static constexpr int OW = NC + (Tag::W16 ? 8 : 4);   // output tile pitch
  static constexpr int SMAX = KMAX / Tag::KS;          // K steps bound
  static constexpr size_t LDS = (size_t)(TW + NC) * LDSX * Tag::ES + (size_t)TW * OW * Tag::ES;
  static_assert(LDS <= 65536, "dense workgroup above 64 KB of LDS");
};

struct DenseArgs {
  int64_t B, C, H, W;
  int wh, ww, d, kp;  // kp: d padded to the matrix-core K step
  int NH, NW;
  int64_t N;          // windows per channel
  int tiles_per_ch;
};

// Element offset of window position p of window n (channel c), or -1 when
// the position lies in the zero padding.
__device__ __attribute__((always_inline)) inline int64_t dense_offset(const DenseArgs &a, int64_t c, int64_t n, int p) {
  const int64_t nhw = (int64_t)a.NH * a.NW;
  const int64_t b = n / nhw;
  const int64_t r = n - b * nhw;
  const int64_t wy = r / a.NW, wx = r - wy * a.NW;
  const int h = p / a.ww, x = p - (p / a.ww) * a.ww;
  const int64_t gh = wy * a.wh + h, gw = wx * a.ww + x;
  if (gh >= a.H || gw >= a.W) return -1;
  return ((b * a.C + c) * a.H + gh) * a.W + gw;
}

// M_c[i, j] = T[c, I(i, j)], i the input and j the output position.
template <class Tag>
__global__ __launch_bounds__(256) void dense_build_kernel(const typename Tag::S *__restrict__ t,
                                                          typename Tag::S *__restrict__ m, int64_t C, int wh,
                                                          int ww) {
  const int d = wh * ww;
  const int64_t k1 = 2 * ww - 1, k2 = (int64_t)(2 * wh - 1) * k1;
  const int64_t total = C * d * d;
  for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t c = e / ((int64_t)d * d);
    const int r = (int)(e - c * d * d);
    const int i = r / d, j = r - (r / d) * d;
    const int hi = i / ww, xi = i - hi * ww, ho = j / ww, xo = j - ho * ww;
    m[e] = t[c * k2 + (hi - ho + wh - 1) * k1 + (xi - xo + ww - 1)];
  }
}

// Y = X M (TRANS: X M^T) per window.  One workgroup = (channel, TW windows);
// the windows' rows land window-major in LDS, each wave keeps the A
// fragments of its 16 windows in registers, and the output positions run in
// chunks of NC: the chunk's columns of M (stored output-major, so that a B
// fragment is one 16-byte read) are staged, multiplied, and the results
// stored.
template <class Tag, bool TRANS>
__global__ __launch_bounds__(256) void dense_fwd_kernel(const typename Tag::S *__restrict__ x,
                                                        const typename Tag::S *__restrict__ m,
                                                        typename Tag::S *__restrict__ y, DenseArgs a) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef DenseCfg<Tag> G;
  constexpr int NT_ = G::NC / 16;
  extern __shared__ __align__(16) unsigned char smem[];
  S *Xt = reinterpret_cast<S *>(smem);
  S *Mt = Xt + G::TW * G::LDSX;
  S *Ot = Mt + G::NC * G::LDSX;

  const int tid = threadIdx.x;
  const int nthr = 64 * G::WAVES;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, ln = lane & 15;
  const int64_t c = blockIdx.x / a.tiles_per_ch;
  const int64_t n0 = (int64_t)(blockIdx.x - c * a.tiles_per_ch) * G::TW;
  const int d = a.d, kp = a.kp;
  const S *mc = m + c * (int64_t)d * d;

  // ---- the windows' rows, window-major (zero beyond d and in the padding)
  for (int e = tid; e < G::TW * kp; e += nthr) {
    const int v = e / kp, p = e - (e / kp) * kp;
    S val = (S)0;
    if (p < d && n0 + v < a.N) {
      const int64_t o = dense_offset(a, c, n0 + v, p);
      if (o >= 0) val = x[o];
    }
    Xt[v * G::LDSX + p] = val;
  }
  __syncthreads();
  const int S_ = kp / Tag::KS;
  Frag af[G::SMAX];
  if constexpr (Tag::W16) {
#pragma unroll
    for (int s = 0; s < G::SMAX; ++s)
      if (s < S_) af[s] = *reinterpret_cast<const Frag *>(&Xt[(16 * wave + ln) * G::LDSX + 32 * s + 8 * g]);
  } else {
#pragma unroll
    for (int s = 0; s < G::SMAX; ++s)
      if (s < S_) af[s] = Xt[(16 * wave + ln) * G::LDSX + 4 * s + g];
  }

  for (int j0 = 0; j0 < d; j0 += G::NC) {
    // ---- columns j0 .. j0+NC of M (rows of M^T), output-major
    if (!TRANS) {
      for (int e = tid; e < G::NC * kp; e += nthr) {
        const int k = e / G::NC, nn = e - (e / G::NC) * G::NC;
        Mt[nn * G::LDSX + k] = (k < d && j0 + nn < d) ? mc[(int64_t)k * d + j0 + nn] : (S)0;
      }
    } else {
      for (int e = tid; e < G::NC * kp; e += nthr) {
        const int nn = e / kp, k = e - (e / kp) * kp;
        Mt[nn * G::LDSX + k] = (k < d && j0 + nn < d) ? mc[(int64_t)(j0 + nn) * d + k] : (S)0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NT_; ++t) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      if constexpr (Tag::W16) {
#pragma unroll
        for (int s = 0; s < G::SMAX; ++s)
          if (s < S_)
            acc = mma<Tag>(af[s], *reinterpret_cast<const Frag *>(&Mt[(16 * t + ln) * G::LDSX + 32 * s + 8 * g]), acc);
        const uint32_t lo = pack2<Tag>(acc[0], acc[1]), hi = pack2<Tag>(acc[2], acc[3]);
        S *o = Ot + (16 * wave + 4 * g) * G::OW + 16 * t + ln;
        o[0] = (S)(lo & 0xffffu);
        o[G::OW] = (S)(lo >> 16);
        o[2 * G::OW] = (S)(hi & 0xffffu);
        o[3 * G::OW] = (S)(hi >> 16);
      } else {
#pragma unroll
        for (int s = 0; s < G::SMAX; ++s)
          if (s < S_) acc = mma<Tag>(af[s], Mt[(16 * t + ln) * G::LDSX + 4 * s + g], acc);
        S *o = Ot + (16 * wave + 4 * g) * G::OW + 16 * t + ln;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r * G::OW] = acc[r];
      }
    }
    __syncthreads();
    for (int e = tid; e < G::TW * G::NC; e += nthr) {
      const int v = e / G::NC, nn = e - (e / G::NC) * G::NC;
      if (j0 + nn < d && n0 + v < a.N) {
        const int64_t o = dense_offset(a, c, n0 + v, j0 + nn);
        if (o >= 0) y[o] = Ot[v * G::OW + nn];
      }
    }
    __syncthreads();
  }
}

// dM_c = sum over windows of X^T dY (float32).  One workgroup = (channel,
// 64 x 64 block of dM); K = the channel's windows, in stages of 32 (16-bit)
// or 16 (float32) windows staged window-major; each wave owns one 16-row
// strip of the block (four 16 x 16 accumulators).
template <class Tag>
struct DenseDmCfg {
  static constexpr int CW = Tag::W16 ? 32 : 16;
  static constexpr int BP = 64;                                        // block side
  static constexpr int LDSP = Tag::W16 ? BP + 8 : BP + 16;             // pitch (elements)
  static constexpr size_t LDS = (size_t)2 * CW * LDSP * Tag::ES;
};

template <class Tag>
__global__ __launch_bounds__(256) void dense_dm_kernel(const typename Tag::S *__restrict__ x,
                                                       const typename Tag::S *__restrict__ dy,
                                                       float *__restrict__ dm, DenseArgs a, int nblk) {
  typedef typename Tag::S S;
  typedef typename Tag::Frag Frag;
  typedef DenseDmCfg<Tag> G;
  extern __shared__ __align__(16) unsigned char smem[];
  S *Xs = reinterpret_cast<S *>(smem);
  S *Gs = Xs + G::CW * G::LDSP;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, ln = lane & 15;
  const int64_t c = blockIdx.x / (nblk * nblk);
  const int blk = (int)(blockIdx.x - c * nblk * nblk);
  const int i0 = (blk / nblk) * G::BP, j0 = (blk - (blk / nblk) * nblk) * G::BP;
  const int d = a.d;

  f32x4 acc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int64_t n0 = 0; n0 < a.N; n0 += G::CW) {
    __syncthreads();  // previous stage consumed
    for (int e = tid; e < 2 * G::CW * G::BP; e += 256) {
      const int tens = e / (G::CW * G::BP);
      const int r = e - tens * (G::CW * G::BP);
      const int v = r / G::BP, pp = r - (r / G::BP) * G::BP;
      const int p = (tens ? j0 : i0) + pp;
      S val = (S)0;
      if (p < d && n0 + v < a.N) {
        const int64_t o = dense_offset(a, c, n0 + v, p);
        if (o >= 0) val = (tens ? dy : x)[o];
      }
      (tens ? Gs : Xs)[v * G::LDSP + pp] = val;
    }
    __syncthreads();
    if constexpr (Tag::W16) {
      const Frag af = dt_frag16<G::LDSP>(reinterpret_cast<const unsigned char *>(Xs), wave, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        acc[q] = mma<Tag>(af, dt_frag16<G::LDSP>(reinterpret_cast<const unsigned char *>(Gs), q, lane), acc[q]);
    } else {
#pragma unroll
      for (int ks = 0; ks < G::CW / 4; ++ks) {
        const float af = Xs[(4 * ks + g) * G::LDSP + 16 * wave + ln];
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = mma<Tag>(af, Gs[(4 * ks + g) * G::LDSP + 16 * q + ln], acc[q]);
      }
    }
  }
  float *mc = dm + c * (int64_t)d * d;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int j = j0 + 16 * q + ln;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 16 * wave + 4 * g + r;
      if (i < d && j < d) mc[(int64_t)i * d + j] = acc[q][r];
    }
  }
}

// dT[c, k] = sum over the pairs (i, j) with I(i, j) = k of dM_c[i, j], in a
// fixed order (output rows, then columns).
__global__ __launch_bounds__(256) void dense_bin_kernel(const float *__restrict__ dm, float *__restrict__ dt,
                                                        int64_t C, int wh, int ww) {
  const int d = wh * ww;
  const int k1 = 2 * ww - 1, k2 = (2 * wh - 1) * k1;
  const int64_t e = blockIdx.x * 256LL + threadIdx.x;
  if (e >= C * k2) return;
  const int64_t c = e / k2;
  const int k = (int)(e - c * k2);
  const int dh = k / k1 - (wh - 1), dw = k - (k / k1) * k1 - (ww - 1);
  const float *mc = dm + c * (int64_t)d * d;
  float s = 0.f;
  for (int ho = dh < 0 ? -dh : 0; ho < (dh > 0 ? wh - dh : wh); ++ho)
    for (int xo = dw < 0 ? -dw : 0; xo < (dw > 0 ? ww - dw : ww); ++xo)
      s += mc[(int64_t)((ho + dh) * ww + xo + dw) * d + ho * ww + xo];
  dt[e] = s;
}

// ------------------------------------------------------------ launchers

static DenseArgs dense_args(const Geom &g, int wh, int ww, int ks) {
  DenseArgs a;
  a.B = g.B; a.C = g.C; a.H = g.H; a.W = g.W;
  a.wh = wh; a.ww = ww; a.d = wh * ww;
  a.kp = (a.d + ks - 1) / ks * ks;
  a.NH = (int)((g.H + wh - 1) / wh);
  a.NW = (int)((g.W + ww - 1) / ww);
  a.N = g.B * (int64_t)a.NH * a.NW;
  a.tiles_per_ch = 0;
  return a;
}

template <class Tag>
static hipError_t run_dense_build(const void *t, void *m, int64_t C, int wh, int ww, hipStream_t st) {
  const int64_t total = C * (int64_t)(wh * ww) * (wh * ww);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  dense_build_kernel<Tag><<<dim3((unsigned)blocks), dim3(256), 0, st>>>((const typename Tag::S *)t,
                                                                         (typename Tag::S *)m, C, wh, ww);
  return hipGetLastError();
}

template <class Tag>
static hipError_t run_dense_fwd(const void *x, const void *m, void *y, const Geom &g, int wh, int ww, bool trans,
                                hipStream_t st) {
  typedef DenseCfg<Tag> G;
  DenseArgs a = dense_args(g, wh, ww, Tag::KS);
  a.tiles_per_ch = (int)((a.N + G::TW - 1) / G::TW);
  const dim3 grid((unsigned)(g.C * a.tiles_per_ch)), block(64 * G::WAVES);
  typedef typename Tag::S S;
  if (trans)
    dense_fwd_kernel<Tag, true><<<grid, block, G::LDS, st>>>((const S *)x, (const S *)m, (S *)y, a);
  else
    dense_fwd_kernel<Tag, false><<<grid, block, G::LDS, st>>>((const S *)x, (const S *)m, (S *)y, a);
  return hipGetLastError();
}

template <class Tag>
static hipError_t run_dense_dm(const void *x, const void *dy, float *dm, const Geom &g, int wh, int ww,
                               hipStream_t st) {
  typedef DenseDmCfg<Tag> G;
  DenseArgs a = dense_args(g, wh, ww, Tag::KS);
  const int nblk = (a.d + G::BP - 1) / G::BP;
  typedef typename Tag::S S;
  dense_dm_kernel<Tag><<<dim3((unsigned)(g.C * nblk * nblk)), dim3(256), G::LDS, st>>>(
      (const S *)x, (const S *)dy, dm, a, nblk);
  return hipGetLastError();
}

hipError_t launch_dense_build(Dt dt, const void *t, void *m, int64_t C, int wh, int ww, hipStream_t st) {
  switch (dt) {
    case Dt::F32: return run_dense_build<TagF32>(t, m, C, wh, ww, st);
    case Dt::BF16: return run_dense_build<TagBF16>(t, m, C, wh, ww, st);
    case Dt::F16: return run_dense_build<TagF16>(t, m, C, wh, ww, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_dense_forward(Dt dt, const void *x, const void *m, void *y, const Geom &g, int wh, int ww,
                                bool trans, hipStream_t st) {
  switch (dt) {
    case Dt::F32: return run_dense_fwd<TagF32>(x, m, y, g, wh, ww, trans, st);
    case Dt::BF16: return run_dense_fwd<TagBF16>(x, m, y, g, wh, ww, trans, st);
    case Dt::F16: return run_dense_fwd<TagF16>(x, m, y, g, wh, ww, trans, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_dense_backward_matrix(Dt dt, const void *x, const void *dy, float *dm, const Geom &g, int wh,
                                        int ww, hipStream_t st) {
  switch (dt) {
    case Dt::F32: return run_dense_dm<TagF32>(x, dy, dm, g, wh, ww, st);
    case Dt::BF16: return run_dense_dm<TagBF16>(x, dy, dm, g, wh, ww, st);
    case Dt::F16: return run_dense_dm<TagF16>(x, dy, dm, g, wh, ww, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_dense_bin(const float *dm, float *dt, int64_t C, int wh, int ww, hipStream_t st) {
  const int64_t total = C * (int64_t)(2 * wh - 1) * (2 * ww - 1);
  dense_bin_kernel<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st>>>(dm, dt, C, wh, ww);
  return hipGetLastError();
}

}  // namespace wbmm
