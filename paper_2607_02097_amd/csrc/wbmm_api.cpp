// C-ABI front end of the WBMM library: argument validation, status codes and
// dispatch to the HIP kernels.  Every check runs on the host before any GPU
// work is enqueued; nothing here allocates, prints or aborts.
#include "wbmm.h"

#include <stdint.h>
#include <string.h>

#include "wbmm_internal.h"

namespace {

using wbmm::Dt;
using wbmm::Geom;

size_t elem_size(wbmm_dtype d) {
  switch (d) {
    case WBMM_F32: return 4;
    case WBMM_BF16: return 2;
    case WBMM_F16: return 2;
  }
  return 0;
}

bool valid_dtype(int d) { return d == WBMM_F32 || d == WBMM_BF16 || d == WBMM_F16; }

// Overflow-checked product of non-negative int64 values.
bool mul_ok(int64_t a, int64_t b, int64_t *out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > INT64_MAX / a) return false;
  *out = a * b;
  return true;
}

// Validates the shape and fills g.  Returns WBMM_OK, INVALID_ARG or
// UNSUPPORTED; bytes receives the size of one [B,C,H,W] tensor.
wbmm_status check_shape(int64_t B, int64_t C, int64_t H, int64_t W, int w, wbmm_dtype dtype,
                        Geom *g, int64_t *bytes) {
  if (!valid_dtype((int)dtype)) return WBMM_ERR_UNSUPPORTED;
  if (B <= 0 || C <= 0 || H <= 0 || W <= 0 || w <= 0) return WBMM_ERR_INVALID_ARG;
  if (w < wbmm::kMinWindow || w > wbmm::kMaxWindow) return WBMM_ERR_UNSUPPORTED;
  int64_t bc, hw, n, b;
  if (!mul_ok(B, C, &bc) || !mul_ok(H, W, &hw) || !mul_ok(bc, hw, &n) ||
      !mul_ok(n, (int64_t)elem_size(dtype), &b))
    return WBMM_ERR_INVALID_ARG;
  g->B = B; g->C = C; g->H = H; g->W = W; g->w = w;
  g->NH = (H + w - 1) / w;
  g->NW = (W + w - 1) / w;
  int64_t nwin;
  if (!mul_ok(B, g->NH * g->NW, &nwin)) return WBMM_ERR_INVALID_ARG;
  g->N = nwin;
  // Kernel-side limits: window indices per channel are split with a float
  // reciprocal (exact below 2^24) and the grid is one-dimensional.
  if (g->N >= (int64_t)1 << 24) return WBMM_ERR_UNSUPPORTED;
  if (C * g->N > (int64_t)UINT32_MAX) return WBMM_ERR_UNSUPPORTED;
  *bytes = b;
  return WBMM_OK;
}

bool overlap(const void *a, int64_t an, const void *b, int64_t bn) {
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return pa < pb + (uintptr_t)bn && pb < pa + (uintptr_t)an;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

wbmm_status from_hip(hipError_t e) { return e == hipSuccess ? WBMM_OK : WBMM_ERR_HIP; }

wbmm_status forward_like(const void *in, const void *table, void *out, int64_t B, int64_t C,
                         int64_t H, int64_t W, int w, wbmm_dtype dtype, void *stream, bool rev) {
  Geom g;
  int64_t bytes = 0;
  wbmm_status s = check_shape(B, C, H, W, w, dtype, &g, &bytes);
  if (s != WBMM_OK) return s;
  if (!in || !table || !out) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  if (!aligned(in, es) || !aligned(table, es) || !aligned(out, es)) return WBMM_ERR_INVALID_ARG;
  const int64_t tbytes = C * (int64_t)(2 * w - 1) * (2 * w - 1) * (int64_t)es;
  if (overlap(in, bytes, out, bytes) || overlap(table, tbytes, out, bytes)) return WBMM_ERR_INVALID_ARG;
  return from_hip(wbmm::launch_forward((Dt)dtype, in, table, out, g, rev, (hipStream_t)stream));
}

}  // namespace

namespace wbmm {

wbmm_status check_backward_args(const void *x, const void *dy, const void *table, const void *dx,
                                const float *dtable, int64_t B, int64_t C, int64_t H, int64_t W, int w,
                                wbmm_dtype dtype, Geom *g, int64_t *bytes) {
  wbmm_status s = check_shape(B, C, H, W, w, dtype, g, bytes);
  if (s != WBMM_OK) return s;
  if (!x || !dy || !table || !dx || !dtable) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(dy, es) || !aligned(table, es) || !aligned(dx, es) || !aligned(dtable, 4))
    return WBMM_ERR_INVALID_ARG;
  const int64_t k2 = (int64_t)(2 * w - 1) * (2 * w - 1);
  const int64_t tbytes = C * k2 * (int64_t)es;  // table
  const int64_t gbytes = C * k2 * 4;            // dtable
  const int64_t n = *bytes;
  // outputs overlap neither inputs nor each other
  if (overlap(dx, n, x, n) || overlap(dx, n, dy, n) || overlap(dx, n, table, tbytes) || overlap(dx, n, dtable, gbytes) ||
      overlap(dtable, gbytes, x, n) || overlap(dtable, gbytes, dy, n) || overlap(dtable, gbytes, table, tbytes))
    return WBMM_ERR_INVALID_ARG;
  return WBMM_OK;
}

}  // namespace wbmm

extern "C" {

wbmm_status wbmm_forward(const void *x, const void *table, void *y, int64_t B, int64_t C, int64_t H,
                         int64_t W, int w, wbmm_dtype dtype, void *stream) {
  return forward_like(x, table, y, B, C, H, W, w, dtype, stream, false);
}

wbmm_status wbmm_backward_input(const void *dy, const void *table, void *dx, int64_t B, int64_t C,
                                int64_t H, int64_t W, int w, wbmm_dtype dtype, void *stream) {
  return forward_like(dy, table, dx, B, C, H, W, w, dtype, stream, true);
}

size_t wbmm_backward_table_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W, int w,
                                           wbmm_dtype dtype) {
  Geom g;
  int64_t bytes = 0;
  if (check_shape(B, C, H, W, w, dtype, &g, &bytes) != WBMM_OK) return 0;
  return wbmm::dtable_workspace_bytes((Dt)dtype, g);
}

wbmm_status wbmm_backward_table(const void *x, const void *dy, float *dtable, void *workspace,
                                size_t workspace_bytes, int64_t B, int64_t C, int64_t H, int64_t W,
                                int w, wbmm_dtype dtype, void *stream) {
  Geom g;
  int64_t bytes = 0;
  wbmm_status s = check_shape(B, C, H, W, w, dtype, &g, &bytes);
  if (s != WBMM_OK) return s;
  if (!x || !dy || !dtable) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(dy, es) || !aligned(dtable, 4)) return WBMM_ERR_INVALID_ARG;
  const int64_t tbytes = C * (int64_t)(2 * w - 1) * (2 * w - 1) * 4;
  if (overlap(x, bytes, dtable, tbytes) || overlap(dy, bytes, dtable, tbytes)) return WBMM_ERR_INVALID_ARG;
  const size_t need = wbmm::dtable_workspace_bytes((Dt)dtype, g);
  if (need > 0) {
    if (!workspace || workspace_bytes < need || !aligned(workspace, 4)) return WBMM_ERR_INVALID_ARG;
    if (overlap(workspace, (int64_t)need, dtable, tbytes) || overlap(workspace, (int64_t)need, x, bytes) ||
        overlap(workspace, (int64_t)need, dy, bytes))
      return WBMM_ERR_INVALID_ARG;
  }
  return from_hip(wbmm::launch_dtable((Dt)dtype, x, dy, dtable, workspace, g, (hipStream_t)stream));
}

size_t wbmm_backward_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W, int w,
                                     wbmm_dtype dtype) {
  return wbmm_backward_table_workspace_bytes(B, C, H, W, w, dtype);
}

wbmm_status wbmm_backward(const void *x, const void *dy, const void *table, void *dx, float *dtable,
                          void *workspace, size_t workspace_bytes, int64_t B, int64_t C, int64_t H,
                          int64_t W, int w, wbmm_dtype dtype, void *stream) {
  Geom g;
  int64_t bytes = 0;
  wbmm_status s = wbmm::check_backward_args(x, dy, table, dx, dtable, B, C, H, W, w, dtype, &g, &bytes);
  if (s != WBMM_OK) return s;
  const size_t es = elem_size(dtype);
  const int64_t k2 = (int64_t)(2 * w - 1) * (2 * w - 1);
  const int64_t tbytes = C * k2 * (int64_t)es;  // table
  const int64_t gbytes = C * k2 * 4;            // dtable
  const size_t need = wbmm::dtable_workspace_bytes((Dt)dtype, g);
  if (need > 0) {
    if (!workspace || workspace_bytes < need || !aligned(workspace, 4)) return WBMM_ERR_INVALID_ARG;
    if (overlap(workspace, (int64_t)need, dtable, gbytes) || overlap(workspace, (int64_t)need, dx, bytes) ||
        overlap(workspace, (int64_t)need, x, bytes) || overlap(workspace, (int64_t)need, dy, bytes) ||
        overlap(workspace, (int64_t)need, table, tbytes))
      return WBMM_ERR_INVALID_ARG;
  }
  return from_hip(wbmm::launch_backward((Dt)dtype, x, dy, table, dx, dtable, workspace, g, (hipStream_t)stream));
}

// ---- hierarchical (global + local) form: global window 2 wl, local wl

static wbmm_status hier_shapes(int64_t B, int64_t C, int64_t H, int64_t W, int wl, wbmm_dtype dtype, Geom *gg,
                               Geom *gl, int64_t *bytes) {
  if (!valid_dtype((int)dtype)) return WBMM_ERR_UNSUPPORTED;
  if (wl <= 0) return WBMM_ERR_INVALID_ARG;
  if (2 * wl > wbmm::kMaxWindow) return WBMM_ERR_UNSUPPORTED;
  wbmm_status s = check_shape(B, C, H, W, 2 * wl, dtype, gg, bytes);
  if (s != WBMM_OK) return s;
  return check_shape(B, C, H, W, wl, dtype, gl, bytes);
}

static wbmm_status hier_forward_like(const void *in, const void *tg, const void *tl, void *out, int64_t B, int64_t C,
                                     int64_t H, int64_t W, int wl, wbmm_dtype dtype, void *stream, bool rev) {
  Geom gg, gl;
  int64_t bytes = 0;
  wbmm_status s = hier_shapes(B, C, H, W, wl, dtype, &gg, &gl, &bytes);
  if (s != WBMM_OK) return s;
  if (!in || !tg || !tl || !out) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  if (!aligned(in, es) || !aligned(tg, es) || !aligned(tl, es) || !aligned(out, es)) return WBMM_ERR_INVALID_ARG;
  const int64_t kg = (int64_t)(4 * wl - 1) * (4 * wl - 1), kl = (int64_t)(2 * wl - 1) * (2 * wl - 1);
  if (overlap(in, bytes, out, bytes) || overlap(tg, C * kg * (int64_t)es, out, bytes) ||
      overlap(tl, C * kl * (int64_t)es, out, bytes))
    return WBMM_ERR_INVALID_ARG;
  return from_hip(wbmm::launch_hier_forward((Dt)dtype, in, tg, tl, out, gg, rev, (hipStream_t)stream));
}

wbmm_status wbmm_hier_forward(const void *x, const void *table_g, const void *table_l, void *y, int64_t B,
                              int64_t C, int64_t H, int64_t W, int wl, wbmm_dtype dtype, void *stream) {
  return hier_forward_like(x, table_g, table_l, y, B, C, H, W, wl, dtype, stream, false);
}

wbmm_status wbmm_hier_backward_input(const void *dy, const void *table_g, const void *table_l, void *dx, int64_t B,
                                     int64_t C, int64_t H, int64_t W, int wl, wbmm_dtype dtype, void *stream) {
  return hier_forward_like(dy, table_g, table_l, dx, B, C, H, W, wl, dtype, stream, true);
}

size_t wbmm_hier_backward_workspace_bytes(int64_t B, int64_t C, int64_t H, int64_t W, int wl, wbmm_dtype dtype) {
  Geom gg, gl;
  int64_t bytes = 0;
  if (hier_shapes(B, C, H, W, wl, dtype, &gg, &gl, &bytes) != WBMM_OK) return 0;
  const size_t a = wbmm::dtable_workspace_bytes((Dt)dtype, gg), b = wbmm::dtable_workspace_bytes((Dt)dtype, gl);
  size_t need = a > b ? a : b;
  // one pass over both tables: both tables' partials, for at most the
  // slabs of the global table's plan
  const wbmm::DtPlan p = wbmm::plan_dtable((Dt)dtype, gg);
  if (p.slabs > 1) {
    const int64_t kg = (int64_t)(4 * wl - 1) * (4 * wl - 1), kl = (int64_t)(2 * wl - 1) * (2 * wl - 1);
    const size_t both = (size_t)p.slabs * (size_t)C * (size_t)(kg + kl) * 4;
    if (both > need) need = both;
  }
  return need;
}

wbmm_status wbmm_hier_backward(const void *x, const void *dy, const void *table_g, const void *table_l, void *dx,
                               float *dtable_g, float *dtable_l, void *workspace, size_t workspace_bytes, int64_t B,
                               int64_t C, int64_t H, int64_t W, int wl, wbmm_dtype dtype, void *stream) {
  Geom gg, gl;
  int64_t bytes = 0;
  wbmm_status s = hier_shapes(B, C, H, W, wl, dtype, &gg, &gl, &bytes);
  if (s != WBMM_OK) return s;
  if (!x || !dy || !table_g || !table_l || !dx || !dtable_g || !dtable_l) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(dy, es) || !aligned(table_g, es) || !aligned(table_l, es) || !aligned(dx, es) ||
      !aligned(dtable_g, 4) || !aligned(dtable_l, 4))
    return WBMM_ERR_INVALID_ARG;
  const int64_t kg = (int64_t)(4 * wl - 1) * (4 * wl - 1), kl = (int64_t)(2 * wl - 1) * (2 * wl - 1);
  struct Buf { const void *p; int64_t n; };
  const Buf ins[] = {{x, bytes}, {dy, bytes}, {table_g, C * kg * (int64_t)es}, {table_l, C * kl * (int64_t)es}};
  const Buf outs[] = {{dx, bytes}, {dtable_g, C * kg * 4}, {dtable_l, C * kl * 4}};
  for (const Buf &o : outs) {
    for (const Buf &i : ins)
      if (overlap(o.p, o.n, i.p, i.n)) return WBMM_ERR_INVALID_ARG;
    for (const Buf &o2 : outs)
      if (&o2 != &o && overlap(o.p, o.n, o2.p, o2.n)) return WBMM_ERR_INVALID_ARG;
  }
  const size_t need = wbmm_hier_backward_workspace_bytes(B, C, H, W, wl, dtype);
  if (need > 0) {
    if (!workspace || workspace_bytes < need || !aligned(workspace, 4)) return WBMM_ERR_INVALID_ARG;
    for (const Buf &b : ins)
      if (overlap(workspace, (int64_t)need, b.p, b.n)) return WBMM_ERR_INVALID_ARG;
    for (const Buf &b : outs)
      if (overlap(workspace, (int64_t)need, b.p, b.n)) return WBMM_ERR_INVALID_ARG;
  }
  hipStream_t st = (hipStream_t)stream;
  // one pass for all three gradients where it applies; else the input
  // gradient (the forward kernel, tables reversed), then both table
  // gradients in one pass or two launches
  bool done = false;
  hipError_t e = wbmm::launch_hier_stream((Dt)dtype, x, dy, table_g, table_l, dx, dtable_g, dtable_l, workspace,
                                          need, gg, st, &done);
  if (e != hipSuccess || done) return from_hip(e);
  e = wbmm::launch_hier_forward((Dt)dtype, dy, table_g, table_l, dx, gg, true, st);
  if (e == hipSuccess)
    e = wbmm::launch_hier_stream((Dt)dtype, x, dy, nullptr, nullptr, nullptr, dtable_g, dtable_l, workspace, need,
                                 gg, st, &done);
  if (e == hipSuccess && !done) {
    e = wbmm::launch_dtable((Dt)dtype, x, dy, dtable_g, workspace, gg, st);
    if (e == hipSuccess) e = wbmm::launch_dtable((Dt)dtype, x, dy, dtable_l, workspace, gl, st);
  }
  return from_hip(e);
}

// ---- cached-matrix (dense) form: any w_h x w_w window, d = w_h w_w <= 256

static wbmm_status dense_window(int wh, int ww) {
  if (wh <= 0 || ww <= 0) return WBMM_ERR_INVALID_ARG;
  if (wh > wbmm::kMaxWindow || ww > wbmm::kMaxWindow) return WBMM_ERR_UNSUPPORTED;
  return WBMM_OK;
}

// Shape check of a [B,C,H,W] tensor with w_h x w_w windows (Geom.w unused).
static wbmm_status dense_shape(int64_t B, int64_t C, int64_t H, int64_t W, int wh, int ww, wbmm_dtype dtype,
                               Geom *g, int64_t *bytes) {
  wbmm_status s = dense_window(wh, ww);
  if (s != WBMM_OK) return s;
  // the square check with the larger side validates sizes and products;
  // the window counts are then recomputed for w_h x w_w
  s = check_shape(B, C, H, W, wh > ww ? wh : ww, dtype, g, bytes);
  if (s != WBMM_OK) return s;
  g->NH = (H + wh - 1) / wh;
  g->NW = (W + ww - 1) / ww;
  int64_t n;
  if (!mul_ok(B, g->NH * g->NW, &n)) return WBMM_ERR_INVALID_ARG;
  g->N = n;
  if (n >= (int64_t)1 << 31 || C * n > (int64_t)UINT32_MAX) return WBMM_ERR_UNSUPPORTED;
  return WBMM_OK;
}

wbmm_status wbmm_build_matrix(const void *table, void *m, int64_t C, int wh, int ww, wbmm_dtype dtype,
                              void *stream) {
  if (!valid_dtype((int)dtype)) return WBMM_ERR_UNSUPPORTED;
  wbmm_status s = dense_window(wh, ww);
  if (s != WBMM_OK) return s;
  if (!table || !m || C <= 0) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  const int64_t d = (int64_t)wh * ww, k2 = (int64_t)(2 * wh - 1) * (2 * ww - 1);
  int64_t mbytes;
  if (!mul_ok(C, d * d * (int64_t)es, &mbytes)) return WBMM_ERR_INVALID_ARG;
  if (!aligned(table, es) || !aligned(m, es)) return WBMM_ERR_INVALID_ARG;
  if (overlap(table, C * k2 * (int64_t)es, m, mbytes)) return WBMM_ERR_INVALID_ARG;
  return from_hip(wbmm::launch_dense_build((Dt)dtype, table, m, C, wh, ww, (hipStream_t)stream));
}

static wbmm_status dense_forward_like(const void *in, const void *m, void *out, int64_t B, int64_t C, int64_t H,
                                      int64_t W, int wh, int ww, wbmm_dtype dtype, void *stream, bool trans) {
  Geom g;
  int64_t bytes = 0;
  wbmm_status s = dense_shape(B, C, H, W, wh, ww, dtype, &g, &bytes);
  if (s != WBMM_OK) return s;
  if (!in || !m || !out) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  if (!aligned(in, es) || !aligned(m, es) || !aligned(out, es)) return WBMM_ERR_INVALID_ARG;
  const int64_t d = (int64_t)wh * ww;
  if (overlap(in, bytes, out, bytes) || overlap(m, C * d * d * (int64_t)es, out, bytes)) return WBMM_ERR_INVALID_ARG;
  return from_hip(wbmm::launch_dense_forward((Dt)dtype, in, m, out, g, wh, ww, trans, (hipStream_t)stream));
}

wbmm_status wbmm_dense_forward(const void *x, const void *m, void *y, int64_t B, int64_t C, int64_t H, int64_t W,
                               int wh, int ww, wbmm_dtype dtype, void *stream) {
  return dense_forward_like(x, m, y, B, C, H, W, wh, ww, dtype, stream, false);
}

wbmm_status wbmm_dense_backward_input(const void *dy, const void *m, void *dx, int64_t B, int64_t C, int64_t H,
                                      int64_t W, int wh, int ww, wbmm_dtype dtype, void *stream) {
  return dense_forward_like(dy, m, dx, B, C, H, W, wh, ww, dtype, stream, true);
}

wbmm_status wbmm_dense_backward_matrix(const void *x, const void *dy, float *dm, int64_t B, int64_t C, int64_t H,
                                       int64_t W, int wh, int ww, wbmm_dtype dtype, void *stream) {
  Geom g;
  int64_t bytes = 0;
  wbmm_status s = dense_shape(B, C, H, W, wh, ww, dtype, &g, &bytes);
  if (s != WBMM_OK) return s;
  if (!x || !dy || !dm) return WBMM_ERR_INVALID_ARG;
  const size_t es = elem_size(dtype);
  if (!aligned(x, es) || !aligned(dy, es) || !aligned(dm, 4)) return WBMM_ERR_INVALID_ARG;
  const int64_t d = (int64_t)wh * ww;
  if (overlap(dm, C * d * d * 4, x, bytes) || overlap(dm, C * d * d * 4, dy, bytes)) return WBMM_ERR_INVALID_ARG;
  return from_hip(wbmm::launch_dense_backward_matrix((Dt)dtype, x, dy, dm, g, wh, ww, (hipStream_t)stream));
}

wbmm_status wbmm_bin_matrix(const float *dm, float *dtable, int64_t C, int wh, int ww, void *stream) {
  wbmm_status s = dense_window(wh, ww);
  if (s != WBMM_OK) return s;
  if (!dm || !dtable || C <= 0) return WBMM_ERR_INVALID_ARG;
  if (!aligned(dm, 4) || !aligned(dtable, 4)) return WBMM_ERR_INVALID_ARG;
  const int64_t d = (int64_t)wh * ww, k2 = (int64_t)(2 * wh - 1) * (2 * ww - 1);
  int64_t mb;
  if (!mul_ok(C, d * d * 4, &mb) || C * k2 > (int64_t)UINT32_MAX * 256) return WBMM_ERR_INVALID_ARG;
  if (overlap(dm, mb, dtable, C * k2 * 4)) return WBMM_ERR_INVALID_ARG;
  return from_hip(wbmm::launch_dense_bin(dm, dtable, C, wh, ww, (hipStream_t)stream));
}

const char *wbmm_status_string(wbmm_status s) {
  switch (s) {
    case WBMM_OK: return "WBMM_OK";
    case WBMM_ERR_INVALID_ARG: return "WBMM_ERR_INVALID_ARG: invalid argument";
    case WBMM_ERR_UNSUPPORTED: return "WBMM_ERR_UNSUPPORTED: unsupported window size or dtype";
    case WBMM_ERR_HIP: return "WBMM_ERR_HIP: HIP runtime error";
    case WBMM_ERR_SCRATCH: return "WBMM_ERR_SCRATCH: the shape needs more than the library's static scratch";
  }
  return "WBMM: unknown status";
}

wbmm_status wbmm_relative_index(int w, int32_t *out_host) {
  if (!out_host || w <= 0) return WBMM_ERR_INVALID_ARG;
  if (w > wbmm::kMaxWindow) return WBMM_ERR_UNSUPPORTED;
  const int d = w * w, k1 = 2 * w - 1;
  for (int i = 0; i < d; ++i)
    for (int j = 0; j < d; ++j)
      out_host[i * d + j] = (i / w - j / w + w - 1) * k1 + (i % w - j % w + w - 1);
  return WBMM_OK;
}

const char *wbmm_version(void) { return "0.1.0"; }

}  // extern "C"
