// Host side of the C ABI declared in include/batchmax.h: argument, capacity and
// order checks (all before any HIP call), the host copy of the schedule state,
// and kernel launches on the caller's stream.  No device allocation, no stream
// synchronisation, no exception crosses the boundary.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <new>
#include <string>

#include "bm_internal.h"

#define BM_EXPORT extern "C" __attribute__((visibility("default")))

struct bm_ctx {
  bm_dims dims;
  bm_cache cache;
  int group;
  int cap;
  int units;
  int elem_bytes;
  float sm_scale;
  bm::Layout lay;
  int32_t len;        // live entries per unit (the same for every unit)
  int32_t next_pos;   // next position the schedule expects
  int32_t last_pos;   // last processed position, -1 before the first
  int32_t p_dec;      // decode removal: 0 one per step after appending, p > 0 p at once when full
  int32_t kv_dec;     // cache bound during decode (<= kv_max)
  int32_t rule;       // bm_rank_rule of every cut
  bool accumulate;    // prefill adds probabilities to the scores
  bool scores_valid;  // no block has run without accumulation
  const int32_t* pad; // device [b] left pad tokens per sample, or null
  hipEvent_t split;   // recorded between a block's attention and its score/cut launches, or null
};

namespace {

thread_local std::string g_err;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return status;
}

int ok() {
  g_err.clear();
  return BM_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int check_dims(const bm_dims* d) {
  if (!d) return fail(BM_ERR_INVALID_ARG, "dims is null");
  if (d->b < 1 || d->s < 1 || d->kv_max < 1 || d->block < 1 || d->max_gen < 0 ||
      d->n_heads < 1 || d->n_kv_heads < 1 || d->head_dim < 1)
    return fail(BM_ERR_INVALID_ARG,
                "sizes must be positive (b=%d s=%d kv_max=%d block=%d max_gen=%d H=%d Hk=%d d=%d)",
                d->b, d->s, d->kv_max, d->block, d->max_gen, d->n_heads, d->n_kv_heads,
                d->head_dim);
  if (d->n_heads % d->n_kv_heads != 0)
    return fail(BM_ERR_INVALID_ARG, "n_heads (%d) is not a multiple of n_kv_heads (%d)",
                d->n_heads, d->n_kv_heads);
  if (!(d->sm_scale >= 0.0f) || !std::isfinite(d->sm_scale))
    return fail(BM_ERR_INVALID_ARG, "sm_scale must be finite and >= 0");
  if ((int64_t)d->s + d->max_gen > (1 << 30))
    return fail(BM_ERR_INVALID_ARG, "s + max_gen too large");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(BM_ERR_UNSUPPORTED, "head_dim %d unsupported (64 or 128)", d->head_dim);
  if (d->dtype != BM_F32 && d->dtype != BM_BF16)
    return fail(BM_ERR_UNSUPPORTED, "dtype %d unsupported", d->dtype);
  const int g = d->n_heads / d->n_kv_heads;
  if (g != 1 && g != 2 && g != 4)
    return fail(BM_ERR_UNSUPPORTED, "query heads per KV head %d unsupported (1, 2 or 4)", g);
  if (d->block > bm::kMaxBlock)
    return fail(BM_ERR_UNSUPPORTED, "block %d exceeds %d", d->block, bm::kMaxBlock);
  if ((int64_t)d->kv_max + d->block > bm::kMaxCapAny)
    return fail(BM_ERR_UNSUPPORTED, "kv_max + block = %lld exceeds %d",
                (long long)d->kv_max + d->block, bm::kMaxCapAny);
  if ((int64_t)d->b * d->n_kv_heads > (1 << 24))
    return fail(BM_ERR_UNSUPPORTED, "b * n_kv_heads too large");
  return BM_OK;
}

float eff_scale(const bm_dims& d) {
  return d.sm_scale > 0.0f ? d.sm_scale : 1.0f / std::sqrt((float)d.head_dim);
}

int hip_fail(hipError_t e, const char* what) {
  return fail(BM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

namespace bm {

Layout workspace_layout(const bm_dims& d) {
  Layout l;
  const int g = d.n_heads / d.n_kv_heads;
  const int pt = positions_per_wg(g);
  const size_t cap = (size_t)d.kv_max + d.block;
  const size_t units = (size_t)d.b * d.n_kv_heads;
  l.npt = (d.block + pt - 1) / pt;
  size_t off = 0;
  l.partial_off = off;
  off = align256(off + units * l.npt * cap * sizeof(float));
  l.holes_off = off;
  off = align256(off + units * cap * sizeof(int32_t));
  l.srcs_off = off;
  off = align256(off + units * cap * sizeof(int32_t));
  l.mcount_off = off;
  off = align256(off + units * sizeof(int32_t));
  l.lastw_off = off;
  off = align256(off + units * cap * sizeof(float));
  l.total = off;
  return l;
}

}  // namespace bm

BM_EXPORT int bm_abi_version(void) { return BM_ABI_VERSION; }

BM_EXPORT const char* bm_last_error(void) { return g_err.c_str(); }

BM_EXPORT int bm_validate_dims(const bm_dims* dims) {
  const int st = check_dims(dims);
  return st == BM_OK ? ok() : st;
}

BM_EXPORT int32_t bm_cache_slots(const bm_dims* dims) {
  if (check_dims(dims) != BM_OK) return -1;
  return dims->kv_max + dims->block;
}

BM_EXPORT int32_t bm_prefill_positions_per_workgroup(const bm_dims* dims) {
  if (check_dims(dims) != BM_OK) return -1;
  return bm::positions_per_wg(dims->n_heads / dims->n_kv_heads);
}

BM_EXPORT size_t bm_workspace_bytes(const bm_dims* dims) {
  if (check_dims(dims) != BM_OK) return 0;
  return bm::workspace_layout(*dims).total;
}

namespace {

int make_ctx(const bm_dims* dims, const bm_cache* cache, bm_ctx** out) {
  int st = check_dims(dims);
  if (st != BM_OK) return st;
  if (!cache || !out) return fail(BM_ERR_INVALID_ARG, "cache or out is null");
  if (!cache->k || !cache->v || !cache->score || !cache->pos || !cache->len || !cache->work)
    return fail(BM_ERR_INVALID_ARG, "a cache pointer is null");
  if (((uintptr_t)cache->k | (uintptr_t)cache->v | (uintptr_t)cache->work) & 15)
    return fail(BM_ERR_INVALID_ARG, "k, v and work must be 16-byte aligned");
  if (((uintptr_t)cache->score | (uintptr_t)cache->pos | (uintptr_t)cache->len) & 3)
    return fail(BM_ERR_INVALID_ARG, "score, pos and len must be 4-byte aligned");
  const bm::Layout lay = bm::workspace_layout(*dims);
  if (cache->work_bytes < lay.total)
    return fail(BM_ERR_INVALID_ARG, "work_bytes %zu < required %zu", cache->work_bytes, lay.total);
  bm_ctx* c = new (std::nothrow) bm_ctx;
  if (!c) return fail(BM_ERR_INVALID_ARG, "out of host memory");
  c->dims = *dims;
  c->cache = *cache;
  c->group = dims->n_heads / dims->n_kv_heads;
  c->cap = dims->kv_max + dims->block;
  c->units = dims->b * dims->n_kv_heads;
  c->elem_bytes = dims->dtype == BM_BF16 ? 2 : 4;
  c->sm_scale = eff_scale(*dims);
  c->lay = lay;
  c->len = 0;
  c->next_pos = 0;
  c->last_pos = -1;
  c->p_dec = 0;
  c->kv_dec = dims->kv_max;
  c->rule = BM_RANK_AVE;
  c->accumulate = true;
  c->scores_valid = true;
  c->pad = nullptr;
  c->split = nullptr;
  *out = c;
  return BM_OK;
}

char* work_at(const bm_ctx* c, size_t off) { return static_cast<char*>(c->cache.work) + off; }

}  // namespace

BM_EXPORT int bm_init(const bm_dims* dims, const bm_cache* cache, hipStream_t stream,
                      bm_ctx** out) {
  if (out) *out = nullptr;
  bm_ctx* c = nullptr;
  const int st = make_ctx(dims, cache, &c);
  if (st != BM_OK) return st;
  const size_t n_score = (size_t)c->units * c->cap;
  const hipError_t e = bm::launch_reset(cache->score, cache->len, n_score, (size_t)c->units, stream);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e, "reset launch");
  }
  *out = c;
  return ok();
}

// ---------------------------------------------------------------------------
// the library's own workspace for callers that cannot allocate device memory
// ---------------------------------------------------------------------------
namespace {

// Each GPU the library runs on holds its own copy of this array until the
// process ends.  In host code `scratch` names a host-side stand-in, not the
// device address: host code only ever uses the address hipGetSymbolAddress
// returns for the current device.
static __device__ __align__(256) char scratch[BM_STATIC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up once per
// device (with that device current) and kept.
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(BM_ERR_UNSUPPORTED, "device %d beyond the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(BM_ERR_HIP, "hipGetSymbolAddress(scratch) returned null");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return BM_OK;
}

}  // namespace

BM_EXPORT int bm_init_static_workspace(const bm_dims* dims, const bm_cache* cache,
                                       hipStream_t stream, bm_ctx** out) {
  if (out) *out = nullptr;
  int st = check_dims(dims);
  if (st != BM_OK) return st;
  if (!cache || !out) return fail(BM_ERR_INVALID_ARG, "cache or out is null");
  const size_t need = bm::workspace_layout(*dims).total;
  if (need > (size_t)BM_STATIC_WORKSPACE_BYTES)
    return fail(BM_ERR_UNSUPPORTED,
                "workspace of %zu bytes exceeds the static workspace of %zu bytes: use bm_init "
                "with a caller-allocated workspace",
                need, (size_t)BM_STATIC_WORKSPACE_BYTES);
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != BM_OK) return st;
  bm_cache c = *cache;
  c.work = ws;
  c.work_bytes = (size_t)BM_STATIC_WORKSPACE_BYTES;
  return bm_init(dims, &c, stream, out);
}

BM_EXPORT int bm_resume(const bm_dims* dims, const bm_cache* cache, int32_t len,
                        int32_t next_pos, bm_ctx** out) {
  if (out) *out = nullptr;
  bm_ctx* c = nullptr;
  const int st = make_ctx(dims, cache, &c);
  if (st != BM_OK) return st;
  if (len < 0 || len > c->cap || next_pos < 0 || next_pos > dims->s + dims->max_gen ||
      len > next_pos) {
    delete c;
    return fail(BM_ERR_INVALID_ARG, "resume state len=%d next_pos=%d is not reachable", len,
                next_pos);
  }
  c->len = len;
  c->next_pos = next_pos;
  c->last_pos = next_pos - 1;
  *out = c;
  return ok();
}

namespace {

int check_rule(const bm_ctx* ctx);
int cut_to(bm_ctx* ctx, int target, int32_t curr_id, hipStream_t stream);

// Checks of a prefill block (all on the host); fills the kernel arguments.
int prefill_args(bm_ctx* ctx, int32_t t0, int32_t n_tok, const void* q, const void* k,
                 const void* v, void* o, int32_t seq_ld, bm::PrefillArgs* out) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if (!q || !k || !v || !o) return fail(BM_ERR_INVALID_ARG, "q, k, v or o is null");
  if (n_tok < 1 || n_tok > ctx->dims.block)
    return fail(BM_ERR_INVALID_ARG, "n_tok %d outside [1, block=%d]", n_tok, ctx->dims.block);
  if (seq_ld < n_tok) return fail(BM_ERR_INVALID_ARG, "seq_ld %d < n_tok %d", seq_ld, n_tok);
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o) & 15)
    return fail(BM_ERR_INVALID_ARG, "q, k, v and o must be 16-byte aligned");
  if (t0 != ctx->next_pos)
    return fail(BM_ERR_ORDER, "prefill t0=%d but the next position is %d", t0, ctx->next_pos);
  if ((int64_t)t0 + n_tok > ctx->dims.s)
    return fail(BM_ERR_ORDER, "block [%d, %d) runs past the prompt length s=%d", t0, t0 + n_tok,
                ctx->dims.s);
  if (ctx->len > ctx->dims.kv_max)
    return fail(BM_ERR_ORDER, "cache holds %d > kv_max=%d entries: evict before the next block",
                ctx->len, ctx->dims.kv_max);
  if (ctx->len + n_tok > ctx->cap)
    return fail(BM_ERR_CAPACITY, "len %d + n_tok %d exceeds cap %d", ctx->len, n_tok, ctx->cap);

  bm::PrefillArgs& a = *out;
  a.q = q;
  a.kin = k;
  a.vin = v;
  a.o = o;
  a.kc = ctx->cache.k;
  a.vc = ctx->cache.v;
  a.pos = ctx->cache.pos;
  a.score = ctx->cache.score;
  a.len = ctx->cache.len;
  a.partial = reinterpret_cast<float*>(work_at(ctx, ctx->lay.partial_off));
  a.seq_ld = seq_ld;
  a.n_heads = ctx->dims.n_heads;
  a.n_kv_heads = ctx->dims.n_kv_heads;
  a.cap = ctx->cap;
  a.len0 = ctx->len;
  a.n_tok = n_tok;
  a.t0 = t0;
  const int ppw = bm::positions_per_wg(ctx->group);
  a.npt_used = (n_tok + ppw - 1) / ppw;
  a.npt_stride = ctx->lay.npt;
  a.units = ctx->units;
  a.accumulate = ctx->accumulate ? 1 : 0;
  a.pad = ctx->pad;
  a.lastw = ctx->rule == BM_RANK_TOVA ? reinterpret_cast<float*>(work_at(ctx, ctx->lay.lastw_off))
                                      : nullptr;
  a.scale_log2 = ctx->sm_scale * 1.4426950408889634f;
  return BM_OK;
}

void advance(bm_ctx* ctx, int32_t t0, int32_t n_tok) {
  ctx->len += n_tok;
  ctx->next_pos = t0 + n_tok;
  ctx->last_pos = t0 + n_tok - 1;
  if (!ctx->accumulate) ctx->scores_valid = false;
}

}  // namespace

BM_EXPORT int bm_prefill_block(bm_ctx* ctx, int32_t t0, int32_t n_tok, const void* q,
                               const void* k, const void* v, void* o, int32_t seq_ld,
                               hipStream_t stream) {
  bm::PrefillArgs a;
  const int st = prefill_args(ctx, t0, n_tok, q, k, v, o, seq_ld, &a);
  if (st != BM_OK) return st;
  hipError_t e = bm::launch_prefill(a, ctx->dims.dtype, ctx->dims.head_dim, ctx->group, stream);
  if (e != hipSuccess) return hip_fail(e, "prefill launch");
  if (ctx->split && (e = hipEventRecord(ctx->split, stream)) != hipSuccess)
    return hip_fail(e, "split event record");
  e = bm::launch_score_reduce(a, stream);
  if (e != hipSuccess) return hip_fail(e, "score reduce launch");
  advance(ctx, t0, n_tok);
  return ok();
}

BM_EXPORT int bm_prefill_block_cut(bm_ctx* ctx, int32_t t0, int32_t n_tok, const void* q,
                                   const void* k, const void* v, void* o, int32_t seq_ld,
                                   hipStream_t stream) {
  bm::PrefillArgs a;
  int st = prefill_args(ctx, t0, n_tok, q, k, v, o, seq_ld, &a);
  if (st != BM_OK) return st;
  const int n = ctx->len + n_tok;
  const bool cuts = n > ctx->dims.kv_max;
  if (cuts && (!ctx->scores_valid || !ctx->accumulate) && ctx->rule != BM_RANK_RECENT)
    return fail(BM_ERR_ORDER,
                "a block ran without score accumulation: only BM_RANK_RECENT can rank this cache");
  hipError_t e = bm::launch_prefill(a, ctx->dims.dtype, ctx->dims.head_dim, ctx->group, stream);
  if (e != hipSuccess) return hip_fail(e, "prefill launch");
  if (ctx->split && (e = hipEventRecord(ctx->split, stream)) != hipSuccess)
    return hip_fail(e, "split event record");
  if (n > bm::kMaxCap) {
    // too many entries for the one-workgroup cut: fold, then the two-kernel cut
    e = bm::launch_score_reduce(a, stream);
    if (e != hipSuccess) return hip_fail(e, "score reduce launch");
    advance(ctx, t0, n_tok);
    if (cuts) {
      st = cut_to(ctx, ctx->dims.kv_max, ctx->last_pos, stream);
      if (st != BM_OK) return st;
    }
    return ok();
  }
  bm::EvictArgs c;
  c.kc = ctx->cache.k;
  c.vc = ctx->cache.v;
  c.score = ctx->cache.score;
  c.pos = ctx->cache.pos;
  c.len = ctx->cache.len;
  c.holes = nullptr;
  c.srcs = nullptr;
  c.mcount = nullptr;
  c.cap = ctx->cap;
  c.n = n;
  c.kv_max = ctx->dims.kv_max;
  c.curr_id = t0 + n_tok - 1;
  c.units = ctx->units;
  c.head_dim = ctx->dims.head_dim;
  c.elem_bytes = ctx->elem_bytes;
  c.rule = ctx->rule;
  c.lastw = reinterpret_cast<float*>(work_at(ctx, ctx->lay.lastw_off));
  e = bm::launch_fold_cut(a, c, bm::positions_per_wg(ctx->group), stream);
  if (e != hipSuccess) return hip_fail(e, "fold-cut launch");
  advance(ctx, t0, n_tok);
  if (cuts) ctx->len = ctx->dims.kv_max;
  return ok();
}

namespace {

// A cut ranked by the scores needs every block's probabilities in them.
int check_rule(const bm_ctx* ctx) {
  if (!ctx->scores_valid && ctx->rule != BM_RANK_RECENT)
    return fail(BM_ERR_ORDER,
                "a block ran without score accumulation: only BM_RANK_RECENT can rank this cache");
  return BM_OK;
}

// Enqueue the cut of every unit from ctx->len down to `target` entries (select
// + compaction), ranked at curr_id.  Requires ctx->len > target; the caller has
// checked the rule.
int cut_to(bm_ctx* ctx, int target, int32_t curr_id, hipStream_t stream) {
  bm::EvictArgs a;
  a.kc = ctx->cache.k;
  a.vc = ctx->cache.v;
  a.score = ctx->cache.score;
  a.pos = ctx->cache.pos;
  a.len = ctx->cache.len;
  a.holes = reinterpret_cast<int32_t*>(work_at(ctx, ctx->lay.holes_off));
  a.srcs = reinterpret_cast<int32_t*>(work_at(ctx, ctx->lay.srcs_off));
  a.mcount = reinterpret_cast<int32_t*>(work_at(ctx, ctx->lay.mcount_off));
  a.cap = ctx->cap;
  a.n = ctx->len;
  a.kv_max = target;
  a.curr_id = curr_id;
  a.units = ctx->units;
  a.head_dim = ctx->dims.head_dim;
  a.elem_bytes = ctx->elem_bytes;
  a.rule = ctx->rule;
  a.lastw = reinterpret_cast<float*>(work_at(ctx, ctx->lay.lastw_off));
  hipError_t e = bm::launch_select(a, stream);
  if (e != hipSuccess) return hip_fail(e, "select launch");
  const int n_evict = ctx->len - target;
  const int max_moves = n_evict < target ? n_evict : target;
  if (max_moves > 0) {
    e = bm::launch_compact(a, max_moves, stream);
    if (e != hipSuccess) return hip_fail(e, "compact launch");
  }
  ctx->len = target;
  return BM_OK;
}

}  // namespace

BM_EXPORT int bm_evict_compact(bm_ctx* ctx, int32_t curr_id, hipStream_t stream) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if (curr_id != ctx->last_pos)
    return fail(BM_ERR_ORDER, "curr_id=%d but the last processed position is %d", curr_id,
                ctx->last_pos);
  if (ctx->len <= ctx->dims.kv_max) return ok();
  int st = check_rule(ctx);
  if (st != BM_OK) return st;
  st = cut_to(ctx, ctx->dims.kv_max, curr_id, stream);
  return st == BM_OK ? ok() : st;
}

BM_EXPORT int bm_set_rank_rule(bm_ctx* ctx, int32_t rule) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if (rule != BM_RANK_AVE && rule != BM_RANK_SUM && rule != BM_RANK_RECENT &&
      rule != BM_RANK_TOVA)
    return fail(BM_ERR_INVALID_ARG, "unknown ranking rule %d", rule);
  ctx->rule = rule;
  return ok();
}

BM_EXPORT int bm_set_decode_bound(bm_ctx* ctx, int32_t bound) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if (bound < 1 || bound > ctx->dims.kv_max)
    return fail(BM_ERR_INVALID_ARG, "decode bound %d outside [1, kv_max=%d]", bound,
                ctx->dims.kv_max);
  ctx->kv_dec = bound;
  return ok();
}

BM_EXPORT int bm_set_left_padding(bm_ctx* ctx, const int32_t* pad) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if ((uintptr_t)pad & 3) return fail(BM_ERR_INVALID_ARG, "pad must be 4-byte aligned");
  ctx->pad = pad;
  return ok();
}

BM_EXPORT int bm_set_split_event(bm_ctx* ctx, hipEvent_t event) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  ctx->split = event;
  return ok();
}

BM_EXPORT int bm_set_score_accumulation(bm_ctx* ctx, int32_t on) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if (on != 0 && on != 1) return fail(BM_ERR_INVALID_ARG, "score accumulation flag %d", on);
  ctx->accumulate = on != 0;
  return ok();
}

BM_EXPORT int bm_set_decode_removal(bm_ctx* ctx, int32_t p) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if (p < 0 || p > ctx->dims.kv_max)
    return fail(BM_ERR_INVALID_ARG, "decode removal p=%d outside [0, kv_max=%d]", p,
                ctx->dims.kv_max);
  ctx->p_dec = p;
  return ok();
}

BM_EXPORT int bm_decode_step(bm_ctx* ctx, int32_t pos, const void* q, const void* k,
                             const void* v, void* o, int32_t seq_ld, hipStream_t stream) {
  if (!ctx) return fail(BM_ERR_INVALID_ARG, "ctx is null");
  if (!q || !k || !v || !o) return fail(BM_ERR_INVALID_ARG, "q, k, v or o is null");
  if (seq_ld < 1) return fail(BM_ERR_INVALID_ARG, "seq_ld %d < 1", seq_ld);
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o) & 15)
    return fail(BM_ERR_INVALID_ARG, "q, k, v and o must be 16-byte aligned");
  if (pos != ctx->next_pos)
    return fail(BM_ERR_ORDER, "decode pos=%d but the next position is %d", pos, ctx->next_pos);
  if (pos < ctx->dims.s)
    return fail(BM_ERR_ORDER, "decode at pos=%d before the prompt (s=%d) is processed", pos,
                ctx->dims.s);
  if ((int64_t)pos >= (int64_t)ctx->dims.s + ctx->dims.max_gen)
    return fail(BM_ERR_ORDER, "decode pos=%d beyond s + max_gen = %d", pos,
                ctx->dims.s + ctx->dims.max_gen);
  if (ctx->len > ctx->dims.kv_max)
    return fail(BM_ERR_CAPACITY, "cache holds %d > kv_max=%d entries: evict after the last block",
                ctx->len, ctx->dims.kv_max);
  // The decode bound kd (kv_max unless set lower).  Algorithm 1's decoding loop
  // taken literally: a cache of kd entries or more first drops to kd - p_dec,
  // ranked at the last processed position, and the step then only appends.
  // With one removal per step a cache above kd is first cut to kd.
  const int kd = ctx->kv_dec;
  if (ctx->p_dec > kd)
    return fail(BM_ERR_INVALID_ARG, "decode removal p=%d exceeds the decode bound %d", ctx->p_dec,
                kd);
  int target = -1;
  if (ctx->p_dec > 0 && ctx->len >= kd) target = kd - ctx->p_dec;
  if (ctx->p_dec == 0 && ctx->len > kd) target = kd;
  const int len_att = target >= 0 ? target : ctx->len;   // cached entries the step attends to
  const bool removes = target >= 0 || (ctx->p_dec == 0 && len_att + 1 > kd);
  if (removes) {
    const int st = check_rule(ctx);
    if (st != BM_OK) return st;
  }
  if (len_att + 1 > bm::kMaxDecodeLen) {
    // outputs only, split over key chunks: the full-cache comparator
    if (ctx->accumulate || removes)
      return fail(BM_ERR_UNSUPPORTED,
                  "a decode step over %d > %d entries computes outputs only: it needs score "
                  "accumulation off and no removal",
                  len_att + 1, bm::kMaxDecodeLen);
    const int nsplit = bm::long_decode_splits(len_att);
    const size_t need = (size_t)ctx->units * nsplit * ctx->group * (ctx->dims.head_dim + 2);
    const size_t have = (size_t)ctx->units * ctx->lay.npt * ctx->cap;
    if (need > have)
      return fail(BM_ERR_UNSUPPORTED, "workspace too small for a %d-entry decode step",
                  len_att + 1);
    bm::LongDecodeArgs a;
    a.q = q;
    a.kin = k;
    a.vin = v;
    a.o = o;
    a.kc = ctx->cache.k;
    a.vc = ctx->cache.v;
    a.score = ctx->cache.score;
    a.pos = ctx->cache.pos;
    a.len = ctx->cache.len;
    a.part = reinterpret_cast<float*>(work_at(ctx, ctx->lay.partial_off));
    a.seq_ld = seq_ld;
    a.n_heads = ctx->dims.n_heads;
    a.n_kv_heads = ctx->dims.n_kv_heads;
    a.cap = ctx->cap;
    a.len0 = ctx->len;
    a.cur_pos = pos;
    a.units = ctx->units;
    a.nsplit = nsplit;
    a.pad = ctx->pad;
    a.scale_log2 = ctx->sm_scale * 1.4426950408889634f;
    const hipError_t e =
        bm::launch_decode_long(a, ctx->dims.dtype, ctx->dims.head_dim, ctx->group, stream);
    if (e != hipSuccess) return hip_fail(e, "long decode launch");
    ctx->len += 1;
    ctx->next_pos = pos + 1;
    ctx->last_pos = pos;
    return ok();
  }
  if (target >= 0) {
    const int st = cut_to(ctx, target, ctx->last_pos, stream);
    if (st != BM_OK) return st;
  }
  bm::DecodeArgs a;
  a.q = q;
  a.kin = k;
  a.vin = v;
  a.o = o;
  a.kc = ctx->cache.k;
  a.vc = ctx->cache.v;
  a.score = ctx->cache.score;
  a.pos = ctx->cache.pos;
  a.len = ctx->cache.len;
  a.seq_ld = seq_ld;
  a.n_heads = ctx->dims.n_heads;
  a.n_kv_heads = ctx->dims.n_kv_heads;
  a.cap = ctx->cap;
  a.len0 = ctx->len;
  a.kv_max = kd;
  a.cur_pos = pos;
  a.units = ctx->units;
  a.rule = ctx->rule;
  a.pad = ctx->pad;
  a.lastw = ctx->rule == BM_RANK_TOVA ? reinterpret_cast<float*>(work_at(ctx, ctx->lay.lastw_off))
                                      : nullptr;
  a.scale_log2 = ctx->sm_scale * 1.4426950408889634f;
  const hipError_t e =
      bm::launch_decode(a, ctx->dims.dtype, ctx->dims.head_dim, ctx->group, stream);
  if (e != hipSuccess) return hip_fail(e, "decode launch");
  if (ctx->len < kd) ctx->len += 1;
  ctx->next_pos = pos + 1;
  ctx->last_pos = pos;
  return ok();
}

BM_EXPORT int32_t bm_ctx_len(const bm_ctx* ctx) { return ctx ? ctx->len : -1; }

BM_EXPORT int32_t bm_ctx_next_pos(const bm_ctx* ctx) { return ctx ? ctx->next_pos : -1; }

BM_EXPORT void bm_destroy(bm_ctx* ctx) { delete ctx; }

// ---------------------------------------------------------------------------
// synthetic inputs of the layer stack (bm_synth.h)
// ---------------------------------------------------------------------------
BM_EXPORT int bm_synth_qkv(const bm_synth* p, int32_t t0, int32_t n_rows, void* q, void* k,
                           void* v, int32_t seq_ld, hipStream_t stream) {
  if (!p) return fail(BM_ERR_INVALID_ARG, "params are null");
  if (!q || !k || !v) return fail(BM_ERR_INVALID_ARG, "q, k or v is null");
  const int half = p->head_dim / 2;
  if (p->b < 1 || p->n_heads < 1 || p->n_kv_heads < 1 || p->head_dim < 2 || (p->head_dim & 1) ||
      (half & (half - 1)))
    return fail(BM_ERR_INVALID_ARG, "b, heads must be positive and head_dim / 2 a power of two");
  if (p->dtype != BM_F32 && p->dtype != BM_BF16)
    return fail(BM_ERR_INVALID_ARG, "dtype %d is neither BM_F32 nor BM_BF16", p->dtype);
  if (t0 < 0 || n_rows < 1 || seq_ld < n_rows)
    return fail(BM_ERR_INVALID_ARG, "t0=%d n_rows=%d seq_ld=%d", t0, n_rows, seq_ld);
  if ((int64_t)(t0 + n_rows) * (p->head_dim / 2) > 0xFFFFFFFFll)
    return fail(BM_ERR_INVALID_ARG, "positions beyond the 32-bit counter word");
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v) & 3)
    return fail(BM_ERR_INVALID_ARG, "q, k and v must be 4-byte aligned");
  bm::SynthArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.b = p->b;
  a.n_heads = p->n_heads;
  a.n_kv_heads = p->n_kv_heads;
  a.head_dim = p->head_dim;
  a.dtype = p->dtype;
  a.layer = p->layer;
  a.s = p->s;
  a.n_sinks = p->n_sinks;
  a.t0 = t0;
  a.n_rows = n_rows;
  a.seq_ld = seq_ld;
  a.seed = p->seed;
  a.hh_threshold = p->hh_threshold;
  a.hh_scale = p->hh_scale;
  a.sink_scale = p->sink_scale;
  a.value_scale = p->value_scale;
  const hipError_t e = bm::launch_synth_qkv(a, stream);
  if (e != hipSuccess) return hip_fail(e, "synth launch");
  return ok();
}

BM_EXPORT int bm_philox4x32_10(const uint32_t* in, uint32_t* out, int64_t n, hipStream_t stream) {
  if (!in || !out || n < 1) return fail(BM_ERR_INVALID_ARG, "in, out null or n < 1");
  const hipError_t e = bm::launch_philox(in, out, n, stream);
  if (e != hipSuccess) return hip_fail(e, "philox launch");
  return ok();
}

// ---------------------------------------------------------------------------
// roofline probes (bm_probe.h)
// ---------------------------------------------------------------------------
BM_EXPORT int bm_probe_stream_read(const void* src, size_t bytes, uint32_t* sink, int32_t blocks,
                                   int32_t nontemporal, hipStream_t stream) {
  if (!src || !sink || blocks < 1) return fail(BM_ERR_INVALID_ARG, "null pointer or blocks < 1");
  if (((uintptr_t)src & 15) || (bytes & 15) || bytes == 0)
    return fail(BM_ERR_INVALID_ARG, "src and bytes must be 16-byte multiples");
  const hipError_t e = bm::launch_probe_read(src, bytes, sink, blocks, nontemporal != 0, stream);
  if (e != hipSuccess) return hip_fail(e, "probe launch");
  return ok();
}

BM_EXPORT int bm_probe_mfma(int32_t iters, float* sink, int32_t blocks, hipStream_t stream) {
  if (!sink || blocks < 1 || iters < 1)
    return fail(BM_ERR_INVALID_ARG, "null sink, blocks < 1 or iters < 1");
  const hipError_t e = bm::launch_probe_mfma(iters, sink, blocks, stream);
  if (e != hipSuccess) return hip_fail(e, "probe launch");
  return ok();
}

BM_EXPORT int bm_prefill_timeline(uint64_t* dst, int32_t n_records) {
  if (!bm::timeline_enabled())
    return fail(BM_ERR_UNSUPPORTED, "this library was built without BM_PREFILL_TIMELINE");
  if (!dst || n_records < 1 || n_records > BM_TIMELINE_MAX_RECORDS)
    return fail(BM_ERR_INVALID_ARG, "null dst or n_records outside [1, %d]", BM_TIMELINE_MAX_RECORDS);
  const hipError_t e = bm::read_timeline(dst, n_records);
  if (e != hipSuccess) return hip_fail(e, "timeline copy");
  return ok();
}

// ---------------------------------------------------------------------------
// cache reset: a fill kernel rather than hipMemsetAsync, so the enqueued work
// is safe to record into a HIP graph
// ---------------------------------------------------------------------------
namespace bm {
namespace {
__global__ void reset_kernel(float* score, int32_t* len, size_t n_score, size_t n_len) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_score; i += stride)
    score[i] = 0.0f;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_len; i += stride) len[i] = 0;
}
}  // namespace

hipError_t launch_reset(float* score, int32_t* len, size_t n_score, size_t n_len,
                        hipStream_t stream) {
  size_t blocks = (n_score + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(reset_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, score, len,
                     n_score, n_len);
  return hipGetLastError();
}
}  // namespace bm
