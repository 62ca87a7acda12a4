// Internal declarations shared by the C-ABI host code and the HIP kernel files.
// Not part of the public ABI (include/batchmax.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "batchmax.h"
#include "bm_probe.h"
#include "bm_synth.h"

namespace bm {

// Prefill attention tiling (gfx950: 64-wide waves, 32x32 MFMA tiles).
// A workgroup has 4 waves; each wave owns 32 query rows of one query head, so a
// workgroup covers 128 / G consecutive block positions of one unit for all G
// heads of its group.  Keys stream through LDS in tiles of 64.
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerWave = 32;
constexpr int kKeyTile = 64;
constexpr int kMaxCap = 4096;          // cuts keep up to this many keys in registers
constexpr int kMaxCapAny = 1 << 16;    // slots per unit (larger cuts stream their keys)
constexpr int kMaxDecodeLen = 4097;    // entries one decode step attends to (LDS rows)
constexpr int kMaxBlock = 1024;

// Ranking key of a cut packed with the position into 64 bits, (key bits << 32
// | pos); every key is >= 0 (scores are sums of probabilities), so the integer
// order is (key ascending, pos ascending): the smallest key goes first and, on
// an exact tie, the older entry.
//   BM_RANK_AVE:    ave = score / (curr_id + 1 - pos), correctly rounded fp32
//   BM_RANK_SUM:    score
//   BM_RANK_RECENT: pos alone (the oldest entry goes first)
//   BM_RANK_TOVA:   last, the last processed query's weight
__device__ __forceinline__ uint64_t rank_key(int rule, float score, float last, int pos,
                                             int curr_id) {
  if (rule == BM_RANK_RECENT) return (uint64_t)(uint32_t)pos;
  const float k = rule == BM_RANK_SUM    ? score
                  : rule == BM_RANK_TOVA ? last
                                         : score / (float)(curr_id + 1 - pos);
  return ((uint64_t)__float_as_uint(k) << 32) | (uint32_t)pos;
}

inline int positions_per_wg(int group) { return kWaves * kRowsPerWave / group; }

// Workspace carve-up (all offsets 256-byte aligned).
struct Layout {
  int npt;              // prefill workgroups per unit for a full block
  size_t partial_off;   // float  [U][npt][cap]  per-workgroup score column sums
  size_t holes_off;     // int32  [U][cap]       evicted slots below kv_max, slot order
  size_t srcs_off;      // int32  [U][cap]       surviving slots at or above kv_max
  size_t mcount_off;    // int32  [U]            number of moves per unit
  size_t lastw_off;     // float  [U][cap]       last query's weights (TOVA key)
  size_t total;
};

Layout workspace_layout(const bm_dims& d);

struct PrefillArgs {
  const void* q;      // row t0 of [b, H, seq_ld, D]
  const void* kin;    // row t0 of [b, Hk, seq_ld, D]
  const void* vin;
  void* o;
  void* kc;           // cache [U, cap, D]
  void* vc;
  int32_t* pos;       // [U, cap]
  float* score;       // [U, cap]
  int32_t* len;       // [U]
  float* partial;     // [U, npt, cap]
  int64_t seq_ld;
  int n_heads, n_kv_heads, cap, len0, n_tok, t0, npt_used, npt_stride, units;
  int accumulate;     // 0: outputs only (no score sums; new entries get score 0)
  const int32_t* pad; // [b] left pad tokens per sample, or null
  float* lastw;       // [U, cap] weights of the block's last query, or null
  float scale_log2;   // sm_scale * log2(e)
};

struct EvictArgs {
  void* kc;
  void* vc;
  float* score;
  int32_t* pos;
  int32_t* len;
  int32_t* holes;
  int32_t* srcs;
  int32_t* mcount;
  int cap, n, kv_max, curr_id, units, head_dim, elem_bytes;
  int rule;           // bm_rank_rule
  float* lastw;       // [U, cap] last query's weights (moved with the entries), or null
};

struct DecodeArgs {
  const void* q;      // [b, H, seq_ld, D] row of this step
  const void* kin;    // [b, Hk, seq_ld, D]
  const void* vin;
  void* o;
  void* kc;
  void* vc;
  float* score;
  int32_t* pos;
  int32_t* len;
  int64_t seq_ld;
  int n_heads, n_kv_heads, cap, len0, kv_max, cur_pos, units;   // kv_max: the decode bound
  int rule;           // bm_rank_rule
  const int32_t* pad; // [b] left pad tokens per sample, or null
  float* lastw;       // [U, cap] this step's weights are written here, or null
  float scale_log2;
};

struct LongDecodeArgs {
  const void* q;      // [b, H, seq_ld, D] row of this step
  const void* kin;    // [b, Hk, seq_ld, D]
  const void* vin;
  void* o;
  void* kc;
  void* vc;
  float* score;
  int32_t* pos;
  int32_t* len;
  float* part;        // [U][nsplit][G][D + 2] chunk partials (o, m, l)
  int64_t seq_ld;
  int n_heads, n_kv_heads, cap, len0, cur_pos, units, nsplit;
  const int32_t* pad; // [b] left pad tokens per sample, or null
  float scale_log2;
};

struct SynthArgs {
  void* q;
  void* k;
  void* v;
  int b, n_heads, n_kv_heads, head_dim, dtype, layer, s, n_sinks, t0, n_rows;
  int64_t seq_ld;
  uint32_t seed, hh_threshold;
  float hh_scale, sink_scale, value_scale;
};

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int head_dim, int group,
                          hipStream_t stream);
hipError_t launch_score_reduce(const PrefillArgs& a, hipStream_t stream);
hipError_t launch_select(const EvictArgs& a, hipStream_t stream);
hipError_t launch_fold_cut(const PrefillArgs& pa, const EvictArgs& a, int pt_positions,
                           hipStream_t stream);
hipError_t launch_compact(const EvictArgs& a, int max_moves, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& a, int dtype, int head_dim, int group,
                         hipStream_t stream);
int long_decode_splits(int len0);
hipError_t launch_decode_long(const LongDecodeArgs& a, int dtype, int head_dim, int group,
                              hipStream_t stream);
hipError_t launch_reset(float* score, int32_t* len, size_t n_score, size_t n_len,
                        hipStream_t stream);
hipError_t launch_synth_qkv(const SynthArgs& a, hipStream_t stream);
hipError_t launch_philox(const uint32_t* in, uint32_t* out, int64_t n, hipStream_t stream);
hipError_t launch_probe_read(const void* src, size_t bytes, uint32_t* sink, int blocks, bool nt,
                             hipStream_t stream);
hipError_t launch_probe_mfma(int iters, float* sink, int blocks, hipStream_t stream);
// prefill timeline records (a BM_PREFILL_TIMELINE build; else hipErrorNotSupported)
bool timeline_enabled();
hipError_t read_timeline(uint64_t* dst, int n_records);

}  // namespace bm
