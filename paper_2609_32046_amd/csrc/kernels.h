// Internal interface between the C ABI (api.hip) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cb {

// Longest sender sequence any call accepts: 32-bit position arithmetic in
// the kernels (loop bounds that step past T by up to 2^16) stays in range.
constexpr int64_t kMaxSeqLen = ((int64_t)1 << 31) - ((int64_t)1 << 16);
// Tokens per K tile staged through LDS by the score kernels.
constexpr int kTileTokens = 64;
// Query rows one wavefront holds by default (four 16-row MFMA blocks).
constexpr int kRowsPerWave = 64;
// Waves per score workgroup at most; rows beyond 8 waves' worth form more
// row groups.
constexpr int kMaxWaves = 8;
constexpr int kRowsPerGroup = kRowsPerWave * kMaxWaves;
// Rows per unit (G*m) the score path accepts.
constexpr int kMaxRows = 1024;
// Sender positions per score work item: the largest of kMaxChunkTokens,
// ..., kMinChunkTokens (powers of two) that still gives the resident
// workgroups more items of the first pass than there are workgroups; larger
// items spend less of their time filling and draining the K ring.
constexpr int kMinChunkTokens = 1024;
constexpr int kMaxChunkTokens = 4096;
// Stages of the persistent kernel's work list, in dependency order, each
// with chunks*row_groups items per unit:
//   P1   per-chunk row statistics (max, sum of exp2)
//   P2   column sums of the normalised weights
// Stage s of unit u sits in step u + lag[s] of the list; a step holds the
// items of every stage that has a unit there, in stage order.  Lags grow
// with the stage, so an item's dependencies always precede it in the list.
enum Stage : int { kStageP1 = 0, kStageP2 = 1 };
constexpr int kMaxStages = 2;
constexpr int kMaxSegments = 2 * kMaxStages + 1;

// The list is cut into segments of steps with a constant number of items
// per step, so that the device decodes an item index with a short scan.
struct WorkList {
  int nstages;
  int units;
  int per_unit[kMaxStages];
  int lag[kMaxStages];
  int nseg;
  int seg_step[kMaxSegments];       // first step of each segment
  int seg_size[kMaxSegments];       // items per step in the segment
  int64_t seg_item[kMaxSegments];   // first item of each segment
  int64_t items;                    // total
};

// Host-side construction: lags from the number of resident workgroups so
// that an item's dependencies have normally finished when it is dequeued.
void make_work_list(int units, int nstages, const int* per_unit, int resident, WorkList* wl);

// Shape of one call and the carve-up of its workspace.
//
// With `position` set the plan is for the position-level score: the query
// rows of a unit are ordered token-major, rho = r*Gp + h, with the group
// padded to Gp in {4, 8} heads (padding rows carry no weight), so that the
// heads of one query token sit in one lane (Gp = 4) or in a pair of lane
// groups (Gp = 8) of the MFMA output, and the second pass also accumulates
// the pooled per-token numerator of the correction.
// Selection of rows split over several workgroups, for fewer units than
// compute units: `parts` workgroups per unit, each holding part_len
// positions of the row in registers (the last part the rest), with
// kv 16-byte vectors per thread of 1024.  At most kSplitGroups workgroups in
// all, so that every part of every unit is resident at once (checked
// against the device at launch: select_split_fits).
constexpr int kSplitGroups = 256;
constexpr int kSplitCounterWords = 8;   // arrival counters per unit, zero at launch
struct SelectSplit {
  int parts;        // 1: no split (rows of up to 16384, or too many units)
  int kv;           // 4, 8 or 16
  int part_len;     // 4 * kv * 1024
  size_t data_words_per_unit;   // 4*parts*256 digit counts
};
struct ScorePlan {
  int64_t T;
  int units, L, Hq, Hkv, G, m, R, D, dtype, S;
  bool position;    // position-level variant
  int Gp;           // padded group (position variant), else G
  int Rp;           // rows the kernel iterates per unit: R, or Gp*m
  int chunks;       // ceil(T / kMinChunkTokens): the workspace holds this many
  int rb;           // 16-row MFMA blocks per wave: 4, or 5 (see make_score_plan)
  SelectSplit sel;  // split selection of the same units (cb_pipeline)
  size_t off_sel_counters;   // in words from the sync words' start
  size_t off_sel_data;       // in bytes
  int row_groups;   // ceil(Rp / (16 * rb * kMaxWaves))
  int waves;        // waves per workgroup
  float c2;         // scale * log2(e)
  size_t off_partial, off_imp_partial, off_numer_partial, off_sync, sync_words, total_bytes;
};

bool make_score_plan(int L, int Hq, int Hkv, int D, int m, int S, int64_t T, int dtype,
                     float scale, bool position, ScorePlan* plan);

// Power used by the numerator of the correction (position variant).
enum PowMode : int { kPowSquare = 0, kPowGeneral = 1, kPowMax = 2 };

// Device-side synchronisation words of one call (zeroed before the launch):
//   [0..1] work-queue head (64-bit), [2] error flag (kSyncError), [3] unused,
//   then done1[U*row_groups] (P1 items finished per unit and row group),
//   done2[U] (P2 items finished per unit).
constexpr int kSyncHeader = 4;
constexpr int kSyncError = 2;

struct PersistArgs {
  const void* q;
  const void* k;
  float* importance;     // [U][T]
  float* row_lse;        // [U][R] or null
  float2* partial;       // [U][chunks][Rp]: per-chunk (max, sum) of each row, log2 units
  float* imp_partial;    // [row_groups][U][T] when row_groups > 1
  // Position variant: per unit and position, the sum over query tokens r of
  // P^p * 2^kappa (or the maximum of P), where P is Pool_7 over positions of
  // the token's weight summed over the group's heads: [U][T], or
  // [row_groups][U][T] partials when row_groups > 1.
  float* numer;
  float* numer_partial;
  int pow_mode;          // PowMode
  float pow_p;           // p (kPowGeneral)
  float pow_kappa;       // log2 of the scale of each term (kPowGeneral)
  float sq_scale;        // 2^(kappa/2): terms are (P * sq_scale)^2 (kPowSquare)
  uint32_t* sync;
  int64_t T;
  int L, Hq, Hkv, G, m, R, S;
  int Gp, gshift, Rp;    // padded group, log2(Gp), rows per unit iterated
  int chunk_tokens;      // positions per score item
  int chunks, row_groups, units;   // chunks = ceil(T / chunk_tokens)
  float c2;
  uint32_t spin_limit;   // polls before a dependency wait gives up
  WorkList wl;
};

// Zeroes the synchronisation words and launches the persistent kernel on
// `s`; with row_groups > 1 the row-group partial sums are added into
// importance afterwards.
hipError_t launch_persistent(const ScorePlan& p, PersistArgs& a, hipStream_t s);
// Per element size (bytes) and head dimension; instantiated in score_*.hip.
template <int ESZ, int D>
hipError_t launch_score_d(const ScorePlan& p, PersistArgs& a, hipStream_t s);
template <int ESZ, int D>
hipError_t launch_position_d(const ScorePlan& p, PersistArgs& a, hipStream_t s);

// err (nullable): a device word that, when nonzero at kernel start, makes
// every unit write -1 indices instead of a selection (the score kernel's
// error flag when the two run in one call).
hipError_t launch_select(const float* importance, int64_t units, int64_t T, int64_t keep,
                         int32_t* idx, const uint32_t* err, hipStream_t s);

bool select_split_plan(int64_t units, int64_t T, SelectSplit* sp);
bool select_split_fits(const SelectSplit& sp, int64_t units);
// counters: units*kSplitCounterWords words, zero; data: units*data_words_per_unit;
// err: zero, raised (and read by every part) when a wait gives up, and
// also the score kernel's error word when the selection follows it.
hipError_t launch_select_split(const float* importance, int64_t units, int64_t T, int64_t keep,
                               int32_t* idx, const SelectSplit& sp, uint32_t* counters,
                               uint32_t* data, uint32_t* err, uint32_t spin_limit,
                               hipStream_t s);
hipError_t launch_clear_words(uint32_t* p, int64_t n, hipStream_t s);

// Gathers units [unit0, unit0 + nunits); idx points at the full [U][keep] array.
hipError_t launch_compact(const void* k, const void* v, const int32_t* idx, int S, int L,
                          int Hkv, int64_t T, int row_bytes, int64_t keep, int64_t unit0,
                          int64_t nunits, void* k_out, void* v_out, hipStream_t s);

}  // namespace cb
