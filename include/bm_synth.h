/*
 * bm_synth.h -- synthetic Q/K/V for the layer-stack workload (part of
 * libbatchmax.so; not part of the paper's method).
 *
 * The 32-layer stack workload draws per-layer Q/K/V with no model weights; its
 * prompt inputs (3.2 GB per sample at s = 8192) cannot be held in memory, so
 * they are evaluated per block on the device from a counter-based generator:
 * Philox4x32-10 as defined by Salmon, Moraes, Dror and Shaw ("Parallel random
 * numbers: as easy as 1, 2, 3", SC 2011).  The host side of the test suite
 * evaluates the same function (paper_2412_05693_amd/synth.py), so checked
 * units reach the CPU oracle with exactly the values the device used.
 *
 * Element recipe.  One Philox call with counter (pos * d/2 + pair,
 * tensor << 8 | head, sample, layer) and key (seed, 0) gives the two elements
 * 2*pair and 2*pair + 1 of row `pos` of (tensor, head): each is the sum S of
 * four 16-bit halves of two output words (words 0-1, then 2-3), mapped to
 * z = ((float)S - 131070) * value_scale.  tensor: 0 = Q (head = query head),
 * 1 = K, 2 = V (head = KV head), 3 = heavy-hitter selector.  K rows at prompt
 * positions (pos < s) are multiplied by sink_scale when pos < n_sinks, else by
 * hh_scale when word 0 of the selector call (pos, 3 << 8, sample, layer) is
 * below hh_threshold.  bf16 outputs are rounded to nearest even.
 *
 * Errors: host-side argument checks return BM_ERR_INVALID_ARG (see
 * bm_last_error()); a failed launch returns BM_ERR_HIP.  Buffers are
 * caller-owned device memory; the work is enqueued on `stream`.
 */
#ifndef BM_SYNTH_H
#define BM_SYNTH_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct bm_synth {
  int32_t b;             /* samples                                        */
  int32_t n_heads;       /* query heads                                    */
  int32_t n_kv_heads;    /* KV heads                                       */
  int32_t head_dim;      /* twice a power of two                           */
  int32_t dtype;         /* bm_dtype: 0 float32, 1 bfloat16                */
  uint32_t seed;         /* key word 0                                     */
  int32_t layer;         /* counter word 3                                 */
  int32_t s;             /* prompt length: positions < s are prompt rows   */
  uint32_t hh_threshold; /* selector words below it mark heavy hitters     */
  float hh_scale;
  int32_t n_sinks;
  float sink_scale;
  float value_scale;     /* float32(sqrt(3) / sqrt(head_dim) / 65536)     */
} bm_synth;

/* Fill rows 0 .. n_rows-1 (positions t0 .. t0+n_rows-1) of
 *   q [b, n_heads, seq_ld, head_dim] and k, v [b, n_kv_heads, seq_ld, head_dim]
 * (element type of p->dtype; 4-byte aligned).  seq_ld >= n_rows, t0 >= 0. */
int bm_synth_qkv(const bm_synth* p, int32_t t0, int32_t n_rows, void* q, void* k, void* v,
                 int32_t seq_ld, hipStream_t stream);

/* Raw Philox4x32-10: for i < n, out[4i .. 4i+3] = philox(ctr = in[6i .. 6i+3],
 * key = in[6i+4 .. 6i+5]).  Device buffers of uint32. */
int bm_philox4x32_10(const uint32_t* in, uint32_t* out, int64_t n, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* BM_SYNTH_H */
