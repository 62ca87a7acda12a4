/*
 * batchmax.h -- C ABI of the MI355X (gfx950) Batch-Max P&D attention library.
 *
 * Batch-Max (arXiv 2412.05693) bounds the KV cache of every attention head of
 * every sample to |kv|-bar pairs during both prefill and decode (Sec. 3).
 * Prefill runs block by block (Sec. 3.1, Algorithm 1); each block's queries
 * attend causally to the bounded cache plus the block's own keys; every key
 * accumulates the attention probabilities it receives (sum_weights, Sec. 3.2);
 * the cache is then cut back to |kv|-bar by removing the entries with the
 * smallest average attention sum_weights / (curr_id + 1 - kv_ids) (Sec. 3.2),
 * the older entry first on an exact tie, and the survivors are compacted in
 * place.  Decode repeats this with one query position and one removal per step.
 *
 * Terms.  A *unit* is one (sample, KV head) pair; with grouped-query attention
 * its G = n_heads / n_kv_heads query heads share its cache and their
 * probabilities are summed into its scores.  Query head h reads KV head
 * h / G.  cap = kv_max + block slots are allocated per unit.
 *
 * Ownership.  The caller owns every device buffer (for example torch tensors)
 * and keeps them alive until the enqueued work has finished.  The library
 * never allocates or frees device memory and never synchronises a stream; all
 * device work is enqueued on the stream passed to each call.  bm_ctx is a small
 * host object (dimensions, borrowed pointers, the host copy of the cache length
 * and of the next position) created by bm_init or bm_resume and freed by
 * bm_destroy.  A context is not thread-safe; separate contexts are independent.
 *
 * Errors.  Every call returns a bm_status.  Argument, capacity and order checks
 * run on the host before anything is enqueued; on such an error the context
 * and the cache are untouched and bm_last_error() describes the problem.  A
 * failed kernel launch returns BM_ERR_HIP.  Faults inside kernels surface at
 * the caller's next synchronisation of the stream.  No C++ exception crosses
 * this boundary.
 *
 * Element types.  BM_F32: q, k, v, o and the K/V cache are float32.  BM_BF16:
 * they are bfloat16 with float32 accumulation.  Scores are always float32 and
 * positions int32.
 */
#ifndef BATCHMAX_H
#define BATCHMAX_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BM_ABI_VERSION 1

typedef enum bm_status {
  BM_OK = 0,
  BM_ERR_INVALID_ARG = 1,  /* null pointer, non-positive size, bad divisibility  */
  BM_ERR_UNSUPPORTED = 2,  /* a head_dim, dtype, group size or size not supported */
  BM_ERR_CAPACITY = 3,     /* the call would overflow the cap = kv_max+block slots */
  BM_ERR_ORDER = 4,        /* position or phase out of the schedule's order      */
  BM_ERR_HIP = 5           /* a HIP runtime call or kernel launch failed          */
} bm_status;

typedef enum bm_dtype { BM_F32 = 0, BM_BF16 = 1 } bm_dtype;

/* What a cut ranks by (bm_set_rank_rule); every rule removes the smallest
 * keys first and, on an exact tie, the older entry. */
typedef enum bm_rank_rule {
  BM_RANK_AVE = 0,    /* score / (curr_id + 1 - pos): the method (Sec. 3.2)        */
  BM_RANK_SUM = 1,    /* score alone: the cumulative rule Sec. 3.2 corrects        */
  BM_RANK_RECENT = 2, /* pos: keep the most recent pairs (Algorithm 3, the
                         extreme decoding-only comparator of Sec. 4)               */
  BM_RANK_TOVA = 3    /* the weight the last processed query gave each entry,
                         summed over the group's heads (TOVA, Sec. 2); needs
                         score accumulation on (its weights come from the same
                         pass), kept per entry in the workspace                    */
} bm_rank_rule;

/* Problem statement (Sec. 3 and Algorithm 1): batch b, padded prompt length
 * s (s-bar), cache bound kv_max (|kv|-bar), prefill block (the removal amount
 * p of Algorithm 1), decode steps max_gen, and the attention shape.
 * Supported: head_dim 64 or 128; group n_heads / n_kv_heads of 1, 2 or 4;
 * 1 <= block <= 1024; kv_max >= 1; kv_max + block <= 65536.  A cut of more
 * than 4096 live entries streams its keys from memory (slower).  A decode
 * step over more than 4097 entries computes the outputs only (split over key
 * chunks; the appended entry gets score 0): it needs score accumulation off
 * and no removal in that step, else BM_ERR_UNSUPPORTED. */
typedef struct bm_dims {
  int32_t b;
  int32_t s;
  int32_t kv_max;
  int32_t block;
  int32_t max_gen;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t dtype;     /* bm_dtype */
  float sm_scale;    /* softmax scale of q.k; 0 selects 1/sqrt(head_dim) */
} bm_dims;

/* The bounded cache, caller-owned device memory, all C-contiguous.
 *   k, v   [b, n_kv_heads, cap, head_dim]  element type of dims.dtype
 *   score  [b, n_kv_heads, cap]  float32   sum_weights of every entry
 *   pos    [b, n_kv_heads, cap]  int32     kv_ids (token position) of every entry
 *   len    [b, n_kv_heads]       int32     |kv|: entries 0..len-1 are live
 *   work   bm_workspace_bytes(dims) bytes of scratch (partial score sums,
 *          eviction lists); contents need not survive between calls.
 * Slot order inside a unit carries no meaning: every result depends only on
 * the set of live entries (Sec. 3.2 treats them as a set of position ids). */
typedef struct bm_cache {
  void* k;
  void* v;
  float* score;
  int32_t* pos;
  int32_t* len;
  void* work;
  size_t work_bytes;
} bm_cache;

typedef struct bm_ctx bm_ctx;

/* BM_ABI_VERSION of the loaded library. */
int bm_abi_version(void);

/* Text of the last non-OK status returned on this thread ("" if none). */
const char* bm_last_error(void);

/* cap = kv_max + block slots per unit; -1 if dims are invalid. */
int32_t bm_cache_slots(const bm_dims* dims);

/* Block positions one prefill attention workgroup covers (all G heads of a
 * unit): a block of n_tok tokens runs ceil(n_tok / this) workgroups per unit,
 * each writing one row of partial score sums per live slot it sees.  -1 if
 * dims are invalid. */
int32_t bm_prefill_positions_per_workgroup(const bm_dims* dims);

/* Bytes of bm_cache.work the calls need; 0 if dims are invalid. */
size_t bm_workspace_bytes(const bm_dims* dims);

/* Check dims alone (no device work).  BM_OK, BM_ERR_INVALID_ARG or
 * BM_ERR_UNSUPPORTED. */
int bm_validate_dims(const bm_dims* dims);

/* Start a new P&D run over `cache` (Algorithm 1 starts from an empty cache):
 * validates dims and pointers, creates the host context, and enqueues on
 * `stream` the zeroing of len and score.  Next expected prefill position: 0. */
int bm_init(const bm_dims* dims, const bm_cache* cache, hipStream_t stream, bm_ctx** out);

/* Bytes of the library's static device workspace (bm_init_static_workspace). */
#define BM_STATIC_WORKSPACE_BYTES (64u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid allocation): bm_init, except
 * that cache->work and cache->work_bytes are ignored and the context's
 * workspace is the library's own static device array of
 * BM_STATIC_WORKSPACE_BYTES, one per GPU (the current device's copy; it lives
 * until the process ends).  The caller still owns k, v, score, pos and len.
 * Nothing here or in later calls on the context allocates or frees memory.
 * Every context made this way on one GPU shares that array and it keeps what
 * the last call left in it (no call needs it cleared first): work enqueued by
 * two such contexts that can overlap on one GPU -- concurrent streams or
 * threads -- races and gives wrong results; work serialised on one stream is
 * fine.  The current device must be the one `stream` runs on.
 * BM_ERR_UNSUPPORTED if bm_workspace_bytes(dims) exceeds the static size
 * (checked before any HIP call); otherwise as bm_init. */
int bm_init_static_workspace(const bm_dims* dims, const bm_cache* cache, hipStream_t stream,
                             bm_ctx** out);

/* Create a context over a cache that already holds a valid state (for
 * example one restored from a snapshot): `len` live entries per unit (the same
 * for every unit) and `next_pos` the next position to process.  No device
 * work.  Phase: prefill while next_pos < s, decode afterwards. */
int bm_resume(const bm_dims* dims, const bm_cache* cache, int32_t len, int32_t next_pos,
              bm_ctx** out);

/* Prefill one block (Algorithm 1, processing step, Sec. 3.1; score update of
 * Sec. 3.2): the n_tok prompt tokens at positions t0 .. t0+n_tok-1 are
 * appended to every unit's cache (score 0, pos = position) and each of their
 * queries attends causally to the live entries plus the block's keys up to
 * its own position; outputs go to o and every entry's score grows by the
 * probabilities it received from all G query heads of the unit.  No removal.
 *   q, o  point at row t0 of [b, n_heads, seq_ld, head_dim] buffers
 *   k, v  point at row t0 of [b, n_kv_heads, seq_ld, head_dim] buffers
 *   seq_ld >= n_tok: rows between consecutive (sample, head) planes.
 * Order: t0 must equal the next expected position, 1 <= n_tok <= block,
 * t0 + n_tok <= s, and the cache must hold at most kv_max entries (evict first). */
int bm_prefill_block(bm_ctx* ctx, int32_t t0, int32_t n_tok, const void* q, const void* k,
                     const void* v, void* o, int32_t seq_ld, hipStream_t stream);

/* bm_prefill_block followed by bm_evict_compact(ctx, t0 + n_tok - 1): one
 * prefill block and its cut (Algorithm 1's step for the block), with the fold
 * of the block's score sums, the select and the compaction in one kernel (one
 * workgroup per unit) instead of three launches when the cache then holds at
 * most 4096 entries; beyond that the separate kernels run.  Same results,
 * checks and errors as the two calls (a cut that would rank by scores a block
 * did not add to returns BM_ERR_ORDER before anything is enqueued). */
int bm_prefill_block_cut(bm_ctx* ctx, int32_t t0, int32_t n_tok, const void* q, const void* k,
                         const void* v, void* o, int32_t seq_ld, hipStream_t stream);

/* Cut every unit back to kv_max entries (Algorithm 1 removal step; rule of
 * Sec. 3.2): rank entries by ave = score / (curr_id + 1 - pos) ascending (or
 * by the key bm_set_rank_rule chose), then by pos ascending, remove the first
 * len - kv_max, and fill the holes among slots 0..kv_max-1 with the survivors
 * from slots kv_max..len-1 (K row, V row, score, pos).  curr_id must be the
 * last processed position.  No-op when the cache holds at most kv_max
 * entries. */
int bm_evict_compact(bm_ctx* ctx, int32_t curr_id, hipStream_t stream);

/* One decode step at position `pos` (Algorithm 1 decode loop with one removal
 * per step): append the step's (k, v), let the G queries attend to all live
 * entries and the new one, add their probabilities to the scores, and, if the
 * cache then holds more than kv_max entries (the decode bound, see
 * bm_set_decode_bound), remove the one with the smallest (ave, pos) -- or the
 * chosen rule's key -- with curr_id = pos, in place: the new entry overwrites
 * the removed slot, or is dropped if it is itself the one removed.  The
 * schedule of bm_set_decode_removal can replace this removal.
 *   q, o  point at [b, n_heads, seq_ld, head_dim] row 0 (the step's row)
 *   k, v  point at [b, n_kv_heads, seq_ld, head_dim] row 0
 * Order: prefill finished (pos == s on the first step, then consecutive),
 * pos < s + max_gen, and the cache holds at most kv_max entries. */
int bm_decode_step(bm_ctx* ctx, int32_t pos, const void* q, const void* k, const void* v,
                   void* o, int32_t seq_ld, hipStream_t stream);

/* Choose the decode removal schedule (default p = 0).
 *   p = 0: each decode step appends its pair and, if the cache then holds more
 *          than kv_max entries, removes the one with the smallest (ave, pos)
 *          with curr_id = the step's position (one removal per step; the new
 *          entry itself can be the one removed).
 *   1 <= p <= kv_max: Algorithm 1's decoding loop taken literally -- when a
 *          step starts with a full cache (kv_max entries), p entries are
 *          removed first, ranked with curr_id = the last processed position;
 *          the step then appends without removal, so the cache stays within
 *          [kv_max - p, kv_max].
 * BM_ERR_INVALID_ARG for p outside [0, kv_max]. */
int bm_set_decode_removal(bm_ctx* ctx, int32_t p);

/* Choose the ranking key of every later cut (default BM_RANK_AVE), in
 * bm_evict_compact and in decode steps.  BM_ERR_INVALID_ARG for an unknown
 * rule. */
int bm_set_rank_rule(bm_ctx* ctx, int32_t rule);

/* Cache bound during decode (default kv_max; 1 <= bound <= kv_max, else
 * BM_ERR_INVALID_ARG).  Decode steps then use `bound` where the schedule
 * above says kv_max; a cache larger than `bound` at a decode step is first
 * cut to `bound` (p = 0) or to bound - p (p > 0), ranked with curr_id = the
 * last processed position.  Algorithm 3 (extreme decoding-only, Sec. 4):
 * kv_max >= s (nothing removed while prefilling), bound 2, p = 1,
 * BM_RANK_RECENT.  A decode step with p > bound returns BM_ERR_INVALID_ARG. */
int bm_set_decode_bound(bm_ctx* ctx, int32_t bound);

/* Left padding (Sec. 3): pad points at b int32 values on the device (caller-
 * owned, alive while work is enqueued), pad[j] = s - s_j, the number of pad
 * tokens in front of sample j's prompt; null (the default) means none.  Pad
 * tokens occupy positions 0 .. pad[j]-1 and are processed like any token, but
 * their keys are visible to no query (their scores stay 0, so every cut
 * removes them first) and a pad query attends to nothing: its output is 0
 * and it adds to no score.  Values below 0 count as 0.  Set it before the
 * first prefill block and keep it for the whole run (a context rebuilt with
 * bm_resume needs it again); 4-byte aligned, else BM_ERR_INVALID_ARG. */
int bm_set_left_padding(bm_ctx* ctx, const int32_t* pad);

/* Score accumulation during prefill (default on = 1).  Off (0): later
 * bm_prefill_block calls compute the attention outputs only (new entries get
 * score 0), the prefill of the full-cache and decoding-only comparators of
 * Sec. 4; decode steps still add their probabilities.  Once a block has run
 * without accumulation, a cut ranked by BM_RANK_AVE or BM_RANK_SUM returns
 * BM_ERR_ORDER (its scores would miss that block) until the context is
 * rebuilt. */
int bm_set_score_accumulation(bm_ctx* ctx, int32_t on);

/* Instrumentation (no effect on results): when `event` is not null, every
 * later bm_prefill_block and bm_prefill_block_cut records it on its stream
 * right after the block's attention kernel and before the launches that fold
 * the score sums (and, for bm_prefill_block_cut, cut and compact), so a caller
 * can time the attention and the cut separately with events on one stream.
 * The event is caller-owned and must stay valid while set; null turns the
 * hook off.  BM_ERR_INVALID_ARG for a null context; a failed record returns
 * BM_ERR_HIP from the prefill call. */
int bm_set_split_event(bm_ctx* ctx, hipEvent_t event);

/* Host copies of the uniform cache length and of the next expected position
 * (-1 for a null context). */
int32_t bm_ctx_len(const bm_ctx* ctx);
int32_t bm_ctx_next_pos(const bm_ctx* ctx);

/* Free the host context (the cache is not touched). */
void bm_destroy(bm_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* BATCHMAX_H */
