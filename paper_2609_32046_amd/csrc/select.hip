// Per-unit top-k kernels (gfx950) running the radix select of
// select_impl.h, one workgroup per unit.
//
// select_kernel: 512 threads, keys held in registers for T <= 16384; two
// workgroups fit a CU, so up to 512 units are selected in one round.
//
// Longer rows re-read the scores from L2 on every digit pass.
#include "kernels.h"
#include "select_impl.h"

namespace cb {
namespace {

constexpr int kThreads = 512;
constexpr int kKeysPerThread = 32;

__global__ __launch_bounds__(kThreads) void select_kernel(const float* __restrict__ importance,
                                                          int64_t T64, int64_t keep64,
                                                          int32_t* __restrict__ idx) {
  __shared__ uint32_t work[SelectLds<kThreads>::kWords];
  const int T = (int)T64;
  const int keep = (int)keep64;
  const int u = blockIdx.x;
  select_unit<kThreads, kKeysPerThread>(importance + (size_t)u * T, T, keep,
                                        idx + (size_t)u * keep, work);
}

}  // namespace

hipError_t launch_select(const float* importance, int64_t units, int64_t T, int64_t keep,
                         int32_t* idx, hipStream_t s) {
  select_kernel<<<(unsigned)units, kThreads, 0, s>>>(importance, T, keep, idx);
  return hipGetLastError();
}

}  // namespace cb
