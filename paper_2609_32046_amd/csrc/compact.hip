// Row gather of the selected K and V rows into the compact cache (gfx950).
//
// Pure data movement: every selected row is read once and written once.
// Each lane moves 16 bytes, so a 256-byte bf16 row (D = 128) is one
// contiguous 256-byte access by 16 lanes and a wavefront moves four rows of K
// and four of V per iteration.  A grid-stride loop keeps the launch at a
// fixed size of resident waves; stores are non-temporal because the compact
// cache is not read again by this path.
#include "kernels.h"

namespace cb {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void compact_kernel(
    const unsigned char* __restrict__ k, const unsigned char* __restrict__ v,
    const int32_t* __restrict__ idx, unsigned char* __restrict__ k_out,
    unsigned char* __restrict__ v_out, int S, int LH, int64_t T, int row_bytes, int64_t keep,
    int64_t unit0, int64_t total_chunks) {
  const int lanes_per_row = row_bytes >> 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; gid < total_chunks;
       gid += stride) {
    const int64_t row = unit0 * keep + gid / lanes_per_row;   // selected row: u*keep + j
    const int c = (int)(gid % lanes_per_row);
    const int64_t u = row / keep;
    const int64_t j = row - u * keep;
    const int64_t t = idx[row];
    const int64_t s = u / LH, lg = u - s * LH;   // unit = s*(L*Hkv) + (l*Hkv + g)
    const size_t dst = ((size_t)(lg * S + s) * keep + j) * row_bytes + (size_t)c * 16;
    u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
    if (t >= 0 && t < T) {
      const size_t src = ((size_t)u * T + t) * row_bytes + (size_t)c * 16;
      kv = *reinterpret_cast<const u32x4*>(k + src);
      vv = *reinterpret_cast<const u32x4*>(v + src);
    }
    __builtin_nontemporal_store(kv, reinterpret_cast<u32x4*>(k_out + dst));
    __builtin_nontemporal_store(vv, reinterpret_cast<u32x4*>(v_out + dst));
  }
}

}  // namespace

hipError_t launch_compact(const void* k, const void* v, const int32_t* idx, int S, int L,
                          int Hkv, int64_t T, int row_bytes, int64_t keep, int64_t unit0,
                          int64_t nunits, void* k_out, void* v_out, hipStream_t s) {
  const int64_t total = nunits * keep * (row_bytes / 16);
  int64_t blocks = (total + 255) / 256;
  const int64_t cap = 256 * 32;   // 32 workgroups per CU is plenty to saturate HBM
  if (blocks > cap) blocks = cap;
  compact_kernel<<<(unsigned)blocks, 256, 0, s>>>(
      static_cast<const unsigned char*>(k), static_cast<const unsigned char*>(v), idx,
      static_cast<unsigned char*>(k_out), static_cast<unsigned char*>(v_out), S, L * Hkv, T,
      row_bytes, keep, unit0, total);
  return hipGetLastError();
}

}  // namespace cb
