// Internal interface between the C ABI (api.hip) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cb {

// Tokens per K tile staged through LDS by the score kernels.
constexpr int kTileTokens = 64;
// Query rows one wavefront holds (four 16-row MFMA blocks).
constexpr int kRowsPerWave = 64;
// Waves per score workgroup at most; rows beyond 512 form more row groups.
constexpr int kMaxWaves = 8;
constexpr int kRowsPerGroup = kRowsPerWave * kMaxWaves;
// Rows per unit (G*m) the score path accepts.
constexpr int kMaxRows = 1024;

// How cb_score splits one call into launches.  Units are processed in
// groups whose K slabs (about 64 MiB) fit comfortably in the 256 MB Infinity
// Cache together with the next group's, so that the second pass over K is
// served from it rather than from HBM while the next group's first pass
// streams in.
struct ScorePlan {
  int64_t T;
  int units, L, Hq, Hkv, G, m, R, D, dtype;
  int chunk_tokens;   // tokens per workgroup (multiple of kTileTokens)
  int chunks;         // ceil(T / chunk_tokens)
  int row_groups;     // ceil(R / kRowsPerGroup)
  int units_per_launch;
  float c2;           // scale * log2(e)
  // workspace carve-up (byte offsets)
  size_t off_partial, off_imp_partial, total_bytes;
};

struct ScoreArgs {
  const void* q;
  const void* k;
  float* importance;     // [U][T]
  float* row_lse;        // [U][R] or null
  float2* partial;       // [U][chunks][R]: per-chunk (max, sum) in log2 units
  float* imp_partial;    // [row_groups][U][T] when row_groups > 1
  int64_t T;
  int L, Hq, Hkv, G, m, R;
  int chunk_tokens, chunks, row_groups;
  int units_total;       // U: every unit of the call
  int unit0, nunits;     // units [unit0, unit0 + nunits) in this launch
  int items, per_xcd;    // work items and their XCD-contiguous mapping
  float c2;
};

bool make_score_plan(int L, int Hq, int Hkv, int D, int m, int S, int64_t T, int dtype,
                     float scale, ScorePlan* plan);

hipError_t launch_score_pass(const ScorePlan& p, const ScoreArgs& a, bool pass2, hipStream_t s);
hipError_t launch_rowgroup_sum(const ScorePlan& p, const ScoreArgs& a, hipStream_t s);

hipError_t launch_select(const float* importance, int64_t units, int64_t T, int64_t keep,
                         int32_t* idx, hipStream_t s);

// Gathers units [unit0, unit0 + nunits); idx points at the full [U][keep] array.
hipError_t launch_compact(const void* k, const void* v, const int32_t* idx, int S, int L,
                          int Hkv, int64_t T, int row_bytes, int64_t keep, int64_t unit0,
                          int64_t nunits, void* k_out, void* v_out, hipStream_t s);

}  // namespace cb
