// Per-unit top-k kernels (gfx950) running the radix select of
// select_impl.h, one workgroup of 512 threads per unit.
//
// Rows of up to 512*KPT scores are staged once through LDS (dynamic shared
// memory, select_stage_words(T) words) and held in registers, KPT = 16 or
// 32 keys per thread, whichever is the smaller that covers the row.  Longer
// rows re-read the scores from L2 on every digit pass.
#include "kernels.h"
#include "select_impl.h"

namespace cb {
namespace {

constexpr int kThreads = 512;

template <int KPT>
__global__ __launch_bounds__(kThreads) void select_kernel(const float* __restrict__ importance,
                                                          int64_t T64, int64_t keep64,
                                                          int32_t* __restrict__ idx) {
  __shared__ __align__(16) uint32_t work[SelectLds<kThreads>::kWords];
  extern __shared__ uint32_t stage[];
  const int T = (int)T64;
  const int keep = (int)keep64;
  const int u = blockIdx.x;
  select_unit<kThreads, KPT>(importance + (size_t)u * T, T, keep, idx + (size_t)u * keep, work,
                             stage);
}

}  // namespace

hipError_t launch_select(const float* importance, int64_t units, int64_t T, int64_t keep,
                         int32_t* idx, hipStream_t s) {
  const int64_t per = (T + kThreads - 1) / kThreads;
  if (per <= 16) {
    const size_t lds = (size_t)select_stage_words(T) * 4;
    select_kernel<16><<<(unsigned)units, kThreads, lds, s>>>(importance, T, keep, idx);
  } else if (per <= 32) {
    const size_t lds = (size_t)select_stage_words(T) * 4;
    select_kernel<32><<<(unsigned)units, kThreads, lds, s>>>(importance, T, keep, idx);
  } else {
    select_kernel<32><<<(unsigned)units, kThreads, 0, s>>>(importance, T, keep, idx);
  }
  return hipGetLastError();
}

}  // namespace cb
