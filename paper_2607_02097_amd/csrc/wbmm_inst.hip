// One translation unit of kernel instantiations: dtype WBMM_INST_TAG
// (TagF32 / TagBF16 / TagF16) and window sizes WBMM_INST_LO..WBMM_INST_LO+3.
// The build compiles this file once per (dtype, window range) so the
// instantiations compile in parallel; wbmm_dispatch.cpp collects the tables.
#include "wbmm_kernels.h"

#ifndef WBMM_INST_TAG
#error "WBMM_INST_TAG must be defined by the build"
#endif
#ifndef WBMM_INST_LO
#error "WBMM_INST_LO must be defined by the build"
#endif

#define WBMM_CAT3(a, b, c) a##b##c
#define WBMM_TABLE_NAME(tag, lo) WBMM_CAT3(entries_, tag, _##lo)
#define WBMM_TABLE(tag, lo) WBMM_TABLE_NAME(tag, lo)

namespace wbmm {

#define WBMM_E(W_)                                                              \
  Entry{&run_forward<WBMM_INST_TAG, WBMM_INST_LO + W_>,                         \
        &run_dtable<WBMM_INST_TAG, WBMM_INST_LO + W_>,                          \
        &plan_dt<WBMM_INST_TAG, WBMM_INST_LO + W_>,                            \
        &run_backward<WBMM_INST_TAG, WBMM_INST_LO + W_>,                       \
        &run_hier_forward<WBMM_INST_TAG, WBMM_INST_LO + W_>,                   \
        &run_hier_stream<WBMM_INST_TAG, WBMM_INST_LO + W_>}

Entry WBMM_TABLE(WBMM_INST_TAG, WBMM_INST_LO)[kInstWindows] = {WBMM_E(0), WBMM_E(1), WBMM_E(2), WBMM_E(3)};

}  // namespace wbmm
