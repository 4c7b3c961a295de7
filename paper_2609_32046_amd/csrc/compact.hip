// Row gather of the selected K and V rows into the compact cache (gfx950).
//
// Pure data movement: every selected row is read once and written once.
// Each lane moves 16 bytes, so a row of 128, 256 or 512 bytes is one
// contiguous access by 8, 16 or 32 lanes.  A workgroup takes a block of
// consecutive selected rows of one unit and moves kUnroll row groups per
// thread, with every index load, then every K and V load, issued before the
// first store, so that each lane keeps 2*kUnroll 16-byte reads in flight.
// Stores are non-temporal because the compact cache is not read again here.
// Units run last first: the score kernel ends on the last units, so their K
// rows are the likeliest to be still cached when the gather starts, and
// taking them first reads them before the gather's own traffic evicts them.
#include "kernels.h"

namespace cb {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

// Grid: nunits * blocks_per_unit workgroups; workgroup b covers selected rows
// [(b % blocks_per_unit) * rows_per_block, ...) of unit
// unit0 + nunits - 1 - b / blocks_per_unit.
__global__ __launch_bounds__(kThreads) void compact_kernel(
    const unsigned char* __restrict__ k, const unsigned char* __restrict__ v,
    const int32_t* __restrict__ idx, unsigned char* __restrict__ k_out,
    unsigned char* __restrict__ v_out, int S, int LH, int64_t T, int lane_shift, int64_t keep,
    int64_t unit0, int blocks_per_unit) {
  const int row_bytes = 16 << lane_shift;
  const int rows_per_pass = kThreads >> lane_shift;
  const int bq = (int)(blockIdx.x / (unsigned)blocks_per_unit);
  const int rb = (int)blockIdx.x - bq * blocks_per_unit;            // in [0, blocks_per_unit)
  const int ub = (int)(gridDim.x / (unsigned)blocks_per_unit) - 1 - bq;   // in [0, nunits)
  const int64_t u = unit0 + ub;
  const int64_t s = u / LH, lg = u - s * LH;   // unit = s*(L*Hkv) + (l*Hkv + g)
  const int c = threadIdx.x & ((1 << lane_shift) - 1);
  const int64_t j0 = (int64_t)rb * rows_per_pass * kUnroll + (threadIdx.x >> lane_shift);
  const int32_t* iu = idx + u * keep;
  const unsigned char* ku = k + (size_t)u * T * row_bytes + (size_t)c * 16;
  const unsigned char* vu = v + (size_t)u * T * row_bytes + (size_t)c * 16;
  const size_t out0 = (size_t)(lg * S + s) * keep * row_bytes + (size_t)c * 16;

  int64_t t[kUnroll];
  bool ok[kUnroll];
#pragma unroll
  for (int i = 0; i < kUnroll; ++i) {
    const int64_t j = j0 + (int64_t)i * rows_per_pass;
    t[i] = iu[j < keep ? j : keep - 1];
    ok[i] = j < keep && t[i] >= 0 && t[i] < T;
  }
  u32x4 kv[kUnroll], vv[kUnroll];
#pragma unroll
  for (int i = 0; i < kUnroll; ++i) {
    // Out-of-range entries read row 0 (valid memory) and store zeros.
    const size_t src = (size_t)(ok[i] ? t[i] : 0) * row_bytes;
    kv[i] = *reinterpret_cast<const u32x4*>(ku + src);
    vv[i] = *reinterpret_cast<const u32x4*>(vu + src);
  }
#pragma unroll
  for (int i = 0; i < kUnroll; ++i) {
    const int64_t j = j0 + (int64_t)i * rows_per_pass;
    if (j >= keep) continue;
    const u32x4 zero = {0, 0, 0, 0};
    const size_t dst = out0 + (size_t)j * row_bytes;
    __builtin_nontemporal_store(ok[i] ? kv[i] : zero, reinterpret_cast<u32x4*>(k_out + dst));
    __builtin_nontemporal_store(ok[i] ? vv[i] : zero, reinterpret_cast<u32x4*>(v_out + dst));
  }
}

}  // namespace

hipError_t launch_compact(const void* k, const void* v, const int32_t* idx, int S, int L,
                          int Hkv, int64_t T, int row_bytes, int64_t keep, int64_t unit0,
                          int64_t nunits, void* k_out, void* v_out, hipStream_t s) {
  int lane_shift = 0;
  while ((16 << lane_shift) < row_bytes) ++lane_shift;
  if ((16 << lane_shift) != row_bytes || (kThreads >> lane_shift) < 1) return hipErrorInvalidValue;
  const int64_t rows_per_block = (int64_t)(kThreads >> lane_shift) * kUnroll;
  const int64_t bpu = (keep + rows_per_block - 1) / rows_per_block;
  if (bpu > 0x7fffffff) return hipErrorInvalidValue;
  const int64_t max_units = 0x7fffffff / bpu;   // keep each grid within 2^31 - 1 workgroups
  // grids of at most max_units units, the last units' grid first
  for (int64_t g = (nunits + max_units - 1) / max_units - 1; g >= 0; --g) {
    const int64_t u0 = g * max_units;
    const int64_t n = nunits - u0 < max_units ? nunits - u0 : max_units;
    compact_kernel<<<(unsigned)(n * bpu), kThreads, 0, s>>>(
        static_cast<const unsigned char*>(k), static_cast<const unsigned char*>(v), idx,
        static_cast<unsigned char*>(k_out), static_cast<unsigned char*>(v_out), S, L * Hkv, T,
        lane_shift, keep, unit0 + u0, (int)bpu);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace cb
