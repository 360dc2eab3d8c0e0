// Dispatch of (dtype, window size) to the kernel instantiations compiled in
// the wbmm_inst.hip translation units.
#include <hip/hip_runtime.h>

#include "wbmm_internal.h"

namespace wbmm {

#define WBMM_TABLES(tag)                                                                  \
  extern Entry entries_##tag##_1[kInstWindows], entries_##tag##_5[kInstWindows],          \
      entries_##tag##_9[kInstWindows], entries_##tag##_13[kInstWindows];                 \
  static Entry *const tables_##tag[4] = {entries_##tag##_1, entries_##tag##_5, entries_##tag##_9, \
                                         entries_##tag##_13};
WBMM_TABLES(TagF32)
WBMM_TABLES(TagBF16)
WBMM_TABLES(TagF16)
#undef WBMM_TABLES

namespace {

const Entry *find(Dt dt, int w) {
  if (w < kMinWindow || w > kMaxWindow) return nullptr;
  const int u = (w - 1) / kInstWindows;
  const int k = (w - 1) % kInstWindows;
  switch (dt) {
    case Dt::F32: return &tables_TagF32[u][k];
    case Dt::BF16: return &tables_TagBF16[u][k];
    case Dt::F16: return &tables_TagF16[u][k];
  }
  return nullptr;
}

}  // namespace

hipError_t launch_forward(Dt dt, const void *x, const void *table, void *y, const Geom &g,
                          bool reverse_table, hipStream_t stream) {
  const Entry *e = find(dt, g.w);
  if (!e) return hipErrorInvalidValue;
  return e->fwd(x, table, y, g, reverse_table, stream);
}

hipError_t launch_dtable(Dt dt, const void *x, const void *dy, float *dtable, void *workspace,
                         const Geom &g, hipStream_t stream) {
  const Entry *e = find(dt, g.w);
  if (!e) return hipErrorInvalidValue;
  return e->dtable(x, dy, dtable, workspace, g, stream);
}

hipError_t launch_backward(Dt dt, const void *x, const void *dy, const void *table, void *dx, float *dtable,
                           void *workspace, const Geom &g, hipStream_t stream) {
  const Entry *e = find(dt, g.w);
  if (!e) return hipErrorInvalidValue;
  return e->bwd(x, dy, table, dx, dtable, workspace, g, stream);
}

hipError_t launch_hier_forward(Dt dt, const void *x, const void *table_g, const void *table_l, void *y,
                               const Geom &g, bool reverse_tables, hipStream_t stream) {
  const Entry *e = find(dt, g.w);
  if (!e) return hipErrorInvalidValue;
  return e->hier_fwd(x, table_g, table_l, y, g, reverse_tables, stream);
}

hipError_t launch_hier_stream(Dt dt, const void *x, const void *dy, const void *table_g, const void *table_l,
                              void *dx, float *dtable_g, float *dtable_l, void *workspace, size_t workspace_bytes,
                              const Geom &g, hipStream_t stream, bool *done) {
  *done = false;
  const Entry *e = find(dt, g.w);
  if (!e) return hipErrorInvalidValue;
  return e->hier_stream(x, dy, table_g, table_l, dx, dtable_g, dtable_l, workspace, workspace_bytes, g, stream,
                        done);
}

DtPlan plan_dtable(Dt dt, const Geom &g) {
  const Entry *e = find(dt, g.w);
  if (!e) return DtPlan{0, 0};
  return e->plan(g);
}

size_t dtable_workspace_bytes(Dt dt, const Geom &g) {
  const DtPlan p = plan_dtable(dt, g);
  if (p.slabs <= 1) return 0;
  const int64_t k1 = 2 * g.w - 1;
  return (size_t)p.slabs * (size_t)g.C * (size_t)(k1 * k1) * sizeof(float);
}

}  // namespace wbmm
