// Sum of the table gradient's per-slab partial sums.  When a channel's
// windows are split into several slabs (one workgroup each), every slab
// writes its partial table gradient; this kernel, launched after that kernel
// on the same stream, adds them in slab order, so the result is reproducible
// bit for bit and needs no synchronisation between workgroups.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wbmm_internal.h"

namespace wbmm {

namespace {

constexpr int kSumThreads = 256;

// Thread i < n: dt[i] = part[0 * n + i] + part[1 * n + i] + ... (slab order);
// threads n .. n + n2 - 1 do the same for the second table.
__global__ __launch_bounds__(kSumThreads) void wbmm_dt_sum_kernel(const float *__restrict__ part,
                                                                  float *__restrict__ dt, int64_t n,
                                                                  const float *__restrict__ part2,
                                                                  float *__restrict__ dt2, int64_t n2, int slabs) {
  int64_t i = (int64_t)blockIdx.x * kSumThreads + threadIdx.x;
  if (i >= n) {
    i -= n;
    if (i >= n2) return;
    part = part2;
    dt = dt2;
    n = n2;
  }
  // the loads of a group of slabs are issued before their sums, which keep
  // the slab order
  constexpr int SG = 8;
  float s = 0.f;
  for (int j0 = 0; j0 < slabs; j0 += SG) {
    float v[SG];
#pragma unroll
    for (int j = 0; j < SG; ++j) v[j] = j0 + j < slabs ? part[(int64_t)(j0 + j) * n + i] : 0.f;
#pragma unroll
    for (int j = 0; j < SG; ++j)
      if (j0 + j < slabs) s += v[j];
  }
  dt[i] = s;
}

}  // namespace

hipError_t launch_dt_sum(const float *part, float *dt, int64_t n, const float *part2, float *dt2, int64_t n2,
                         int slabs, hipStream_t stream) {
  const int64_t total = n + (n2 > 0 ? n2 : 0);
  if (total <= 0) return hipSuccess;
  const int64_t blocks = (total + kSumThreads - 1) / kSumThreads;
  wbmm_dt_sum_kernel<<<dim3((unsigned)blocks), dim3(kSumThreads), 0, stream>>>(part, dt, n, part2, dt2,
                                                                                n2 > 0 ? n2 : 0, slabs);
  return hipGetLastError();
}

}  // namespace wbmm
