// Internal interface between the C-ABI front end (wbmm_api.cpp) and the HIP
// kernels (wbmm_kernels.h, instantiated by wbmm_inst.hip).  Not installed, not part of the ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "wbmm.h"

namespace wbmm {

enum class Dt { F32 = 0, BF16 = 1, F16 = 2 };

// Geometry of one call.  N is the number of windows per channel,
// N = B * NH * NW with NH = ceil(H / w), NW = ceil(W / w).
struct Geom {
  int64_t B, C, H, W;
  int w;
  int64_t NH, NW, N;
};

constexpr int kMinWindow = 1;
constexpr int kMaxWindow = 16;
// window sizes per instantiation unit (wbmm_inst.hip)
constexpr int kInstWindows = 4;

// Launch plan of the dtable pass: windows per slab and number of slabs; one
// workgroup per (channel, slab).  Slabs > 1 need a float32 workspace of
// slabs * C * (2w-1)^2 entries.
struct DtPlan {
  int64_t slab_windows;
  int64_t slabs;
};

DtPlan plan_dtable(Dt dt, const Geom &g);
size_t dtable_workspace_bytes(Dt dt, const Geom &g);

// Table gradients from per-slab partial sums (wbmm_reduce.hip): after the
// kernel that wrote them, on the same stream, dt[i] = sum over slabs s, in
// slab order, of part[s * n + i], for i < n; the same for part2 / dt2 / n2
// when n2 > 0 (the second table of the hierarchical form).
hipError_t launch_dt_sum(const float *part, float *dt, int64_t n, const float *part2, float *dt2, int64_t n2,
                         int slabs, hipStream_t stream);

// Host-side validation of wbmm_backward's tensor arguments (shape, pointers,
// alignment, overlaps; not the workspace); fills g and the bytes of one
// [B,C,H,W] tensor (wbmm_api.cpp).
wbmm_status check_backward_args(const void *x, const void *dy, const void *table, const void *dx,
                                const float *dtable, int64_t B, int64_t C, int64_t H, int64_t W, int w,
                                wbmm_dtype dtype, Geom *g, int64_t *bytes);

// Each returns hipSuccess or the error of the launch.
hipError_t launch_forward(Dt dt, const void *x, const void *table, void *y,
                          const Geom &g, bool reverse_table,
                          hipStream_t stream);
hipError_t launch_dtable(Dt dt, const void *x, const void *dy, float *dtable,
                         void *workspace, const Geom &g, hipStream_t stream);
hipError_t launch_backward(Dt dt, const void *x, const void *dy, const void *table,
                           void *dx, float *dtable, void *workspace, const Geom &g,
                           hipStream_t stream);
// Hierarchical form: g.w is the global window (2 wl).
hipError_t launch_hier_forward(Dt dt, const void *x, const void *table_g,
                               const void *table_l, void *y, const Geom &g,
                               bool reverse_tables, hipStream_t stream);
// Hierarchical form in one pass where that applies (*done): both table
// gradients, and the input gradient too when dx is not null; otherwise
// nothing is launched and *done is false.
hipError_t launch_hier_stream(Dt dt, const void *x, const void *dy, const void *table_g,
                              const void *table_l, void *dx, float *dtable_g, float *dtable_l,
                              void *workspace, size_t workspace_bytes, const Geom &g,
                              hipStream_t stream, bool *done);

// Cached-matrix (dense) form, any w_h x w_w window with d = w_h w_w <= 256
// (wbmm_dense.hip).  g.w is unused by these.
hipError_t launch_dense_build(Dt dt, const void *table, void *m, int64_t C, int wh, int ww,
                              hipStream_t stream);
hipError_t launch_dense_forward(Dt dt, const void *x, const void *m, void *y, const Geom &g,
                                int wh, int ww, bool transpose, hipStream_t stream);
hipError_t launch_dense_backward_matrix(Dt dt, const void *x, const void *dy, float *dm,
                                        const Geom &g, int wh, int ww, hipStream_t stream);
hipError_t launch_dense_bin(const float *dm, float *dtable, int64_t C, int wh, int ww,
                            hipStream_t stream);

// Per-(dtype, window) entry points, defined by the wbmm_inst.hip
// translation units and collected into tables by wbmm_dispatch.cpp.
typedef hipError_t (*FwdFn)(const void *, const void *, void *, const Geom &, bool, hipStream_t);
typedef hipError_t (*DtFn)(const void *, const void *, float *, void *, const Geom &, hipStream_t);
typedef DtPlan (*PlanFn)(const Geom &);
typedef hipError_t (*BwdFn)(const void *, const void *, const void *, void *, float *, void *, const Geom &,
                            hipStream_t);
typedef hipError_t (*HierFn)(const void *, const void *, const void *, void *, const Geom &, bool, hipStream_t);
typedef hipError_t (*HierStreamFn)(const void *, const void *, const void *, const void *, void *, float *,
                                   float *, void *, size_t, const Geom &, hipStream_t, bool *);
struct Entry {
  FwdFn fwd;
  DtFn dtable;
  PlanFn plan;
  BwdFn bwd;
  HierFn hier_fwd;
  HierStreamFn hier_stream;
};

}  // namespace wbmm
