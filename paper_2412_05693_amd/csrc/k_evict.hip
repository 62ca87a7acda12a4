// K2 + K3: cut every unit back to kv_max entries and compact in place.
//
// K2 (select_kernel), one workgroup per unit: every live entry j gets the
// ranking key of the chosen rule (by default Sec. 3.2's ave_j = score_j /
// (curr_id + 1 - pos_j) in IEEE float32 division) packed with its position into
// one 64-bit integer (rank_key): the integer order is (key ascending, pos
// ascending), so the smallest key goes first and, on an exact tie, the older
// entry.  An LDS radix select over 8-bit digits (at most 8 passes, fewer when
// curr_id needs fewer position digits or a pass already settles the cut) finds
// a threshold with exactly E keys at or below it (positions are unique, so the
// E smallest keys are well defined).  Up to kMaxCap keys stay in registers;
// larger caches recompute each key from the scores and positions in every
// pass.  Evicted slots below kv_max become holes, surviving slots at or above
// kv_max become sources; both lists are built in slot order with workgroup
// prefix counts, so the pairing is deterministic.
//
// K3 (compact_kernel), units x chunks of 32 moves: the i-th source moves into
// the i-th hole (K row, V row, score, pos), 16-byte coalesced copies.  Sources
// and holes are disjoint, so moves never overlap.
#include "bm_internal.h"

namespace bm {
namespace {

constexpr int kMaxPer = kMaxCap / 256;  // keys per thread held in registers

// exclusive prefix count of `flag` over the workgroup in thread order; returns
// the workgroup total through *total
__device__ __forceinline__ int block_excl_count(bool flag, int* s_wave, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t b = __ballot(flag);
  const int in_wave = __popcll(b & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
  if (lane == 0) s_wave[w] = __popcll(b);
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = s_wave[i];
    before += (i < w) ? c : 0;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return before + in_wave;
}

// The need-th smallest (1-based) of the keys key_of(i) of the entries
// tid + 256 i < n: a radix select over 8-bit digits (histograms in LDS, a
// 64-lane scan of the 256 bins).  Keys are unique (they hold the position), so
// exactly `need` keys are <= the result.  The low 32 bits of every key are the
// entry's position, which is at most curr_id: the digits of that word at and
// above bit pos_bits are zero in every key, so only the four digits of the high
// word and the position digits below pos_bits get a pass (the others would keep
// the prefix and `need` as they are).  The two 256-bin histograms alternate
// between the passes, so clearing the next one needs no barrier of its own: two
// barriers per pass.  When the bin that holds the need-th key holds exactly the
// `need` keys still wanted, every key of that bin is among the smallest: the
// select stops there and returns the bin's prefix with all lower bits set, which
// has the same keys at or below it as the need-th key itself.
template <typename KeyOf>
__device__ __forceinline__ uint64_t radix_kth(KeyOf key_of, int n_iter, int per, int n, int need,
                                              int pos_bits, uint32_t* hist, uint64_t* s_prefix,
                                              int* s_need) {
  const int tid = threadIdx.x;
  const int n_pos = (pos_bits + 7) >> 3;   // position digits that can be nonzero
  const int n_pass = 4 + n_pos;
  uint64_t prefix = 0;
  hist[tid] = 0;
  __syncthreads();
  // pass r: the digit at `shift`, histogram r & 1 (r counts only the passes run)
  for (int r = 0; r < n_pass; ++r) {
    const int shift = r < 4 ? 56 - 8 * r : 8 * (n_pass - 1 - r);
    const uint64_t himask = r == 0 ? 0ull : (~0ull << (shift + 8));
    uint32_t* h = hist + 256 * (r & 1);
#pragma unroll
    for (int i = 0; i < n_iter; ++i) {
      const int j = tid + 256 * i;
      if (i < per && j < n) {
        const uint64_t kk = key_of(i);
        if ((kk & himask) == prefix) atomicAdd(&h[(kk >> shift) & 255u], 1u);
      }
    }
    hist[256 * ((r + 1) & 1) + tid] = 0;   // the next pass's histogram
    __syncthreads();
    if (tid < 64) {
      const uint32_t h0 = h[4 * tid], h1 = h[4 * tid + 1], h2 = h[4 * tid + 2], h3 = h[4 * tid + 3];
      const uint32_t mine = h0 + h1 + h2 + h3;
      uint32_t incl = mine;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t o = __shfl_up(incl, off);
        if (tid >= off) incl += o;
      }
      uint32_t ex = incl - mine;
      const uint32_t hv[4] = {h0, h1, h2, h3};
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if ((int)ex < need && need <= (int)(ex + hv[b])) {
          const int rest = need - (int)ex;
          const bool whole = rest == (int)hv[b];   // the whole bin is wanted
          *s_prefix = prefix | ((uint64_t)(4 * tid + b) << shift) |
                      (whole ? (1ull << shift) - 1 : 0ull);
          *s_need = whole ? 0 : rest;
        }
        ex += hv[b];
      }
    }
    __syncthreads();
    prefix = *s_prefix;
    need = *s_need;
    if (need == 0) break;   // uniform: every thread read the same value
  }
  return prefix;
}

// bits that hold every position of a cut ranked at curr_id (positions <= curr_id)
__device__ __forceinline__ int position_bits(int curr_id) {
  return curr_id > 0 ? 32 - __clz(curr_id) : 0;
}

// The hole list (evicted slots below kv_max) and the source list (kept slots at
// or above kv_max), both in slot order, slot j = tid + 256 i for i < per <=
// kMaxPer.  Each wave counts its holes and sources of every i with ballots;
// the counts (holes in the low 16 bits, sources in the high) go through LDS
// once and one wave scans them, so the lists take two barriers whatever `per`
// is.  evicted(i): the entry in slot tid + 256 i is evicted (false past n);
// emit(is_hole, index, slot) stores one list entry.
template <typename Evicted, typename Emit>
__device__ __forceinline__ void build_lists(Evicted evicted, int n_iter, int per, int n, int kv_max,
                                            uint32_t* s_cnt, int* s_tot, Emit emit) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int i = 0; i < n_iter; ++i) {
    if (i < per) {
      const int j = tid + 256 * i;
      const bool live = j < n, ev = live && evicted(i);
      const uint64_t bh = __ballot(live && j < kv_max && ev);
      const uint64_t bs = __ballot(live && j >= kv_max && !ev);
      if (lane == 0) s_cnt[4 * i + w] = (uint32_t)__popcll(bh) | ((uint32_t)__popcll(bs) << 16);
    }
  }
  __syncthreads();
  if (tid < 64) {
    // exclusive prefix over (i, wave) in slot order; both fields stay below 2^16
    const uint32_t mine = tid < 4 * per ? s_cnt[tid] : 0u;
    uint32_t incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t o = __shfl_up(incl, off);
      if (tid >= off) incl += o;
    }
    if (tid < 4 * per) s_cnt[tid] = incl - mine;
    if (tid == 63) {
      s_tot[0] = (int)(incl & 0xFFFFu);
      s_tot[1] = (int)(incl >> 16);
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < n_iter; ++i) {
    if (i < per) {
      const int j = tid + 256 * i;
      const bool live = j < n, ev = live && evicted(i);
      const bool is_hole = live && j < kv_max && ev, is_src = live && j >= kv_max && !ev;
      const uint64_t bh = __ballot(is_hole), bs = __ballot(is_src);
      const uint32_t base = s_cnt[4 * i + w];
      if (is_hole) emit(true, (int)(base & 0xFFFFu) + __popcll(bh & below), j);
      if (is_src) emit(false, (int)(base >> 16) + __popcll(bs & below), j);
    }
  }
}

// KP: keys per thread held in registers (n <= 256 KP); KP = 0 streams the keys
// from memory in every pass (any n up to kMaxCapAny)
template <int KP>
__global__ void __launch_bounds__(256) select_kernel(EvictArgs a) {
  constexpr bool STREAM = KP == 0;
  __shared__ uint32_t hist[512];
  __shared__ uint64_t s_prefix;
  __shared__ int s_need;
  __shared__ int s_wave[4];
  __shared__ uint32_t s_cnt[4 * kMaxPer];
  __shared__ int s_tot[2];
  const int u = blockIdx.x;
  const int tid = threadIdx.x;
  const float* score = a.score + (int64_t)u * a.cap;
  const int32_t* pos = a.pos + (int64_t)u * a.cap;
  // TOVA's weights (any slot of the unit when the rule does not read them)
  const float* last = a.rule == BM_RANK_TOVA ? a.lastw + (int64_t)u * a.cap : score;
  const int per = (a.n + 255) / 256;
  constexpr int NK = STREAM ? 1 : KP;

  uint64_t key[NK];
  if constexpr (!STREAM) {
    // every load issued before any is used (indices clamped into range)
    float sv[KP], lv[KP];
    int pv[KP];
#pragma unroll
    for (int i = 0; i < KP; ++i) {
      const int jc = min(tid + 256 * i, a.n - 1);
      sv[i] = score[jc];
      lv[i] = last[jc];
      pv[i] = pos[jc];
    }
#pragma unroll
    for (int i = 0; i < KP; ++i) {
      const int j = tid + 256 * i;
      key[i] = (i < per && j < a.n) ? rank_key(a.rule, sv[i], lv[i], pv[i], a.curr_id) : ~0ull;
    }
  }
  // key of entry tid + 256 i (registers, or recomputed when streaming)
  auto key_of = [&](int i) __device__ -> uint64_t {
    if constexpr (STREAM) {
      const int j = tid + 256 * i;
      return j < a.n ? rank_key(a.rule, score[j], last[j], pos[j], a.curr_id) : ~0ull;
    } else {
      return key[i];
    }
  };
  const int n_iter = STREAM ? per : KP;
  const uint64_t thr = radix_kth(key_of, n_iter, per, a.n, a.n - a.kv_max, position_bits(a.curr_id),
                                 hist, &s_prefix, &s_need);   // exactly n - kv_max keys are <= thr

  // holes (evicted, slot < kv_max) and sources (kept, slot >= kv_max), slot order
  int32_t* holes = a.holes + (int64_t)u * a.cap;
  int32_t* srcs = a.srcs + (int64_t)u * a.cap;
  int hbase = 0, sbase = 0;
  if constexpr (STREAM) {
    // more than kMaxPer entries per thread: one workgroup count per 256 slots
    for (int i = 0; i < per; ++i) {
      const int j = tid + 256 * i;
      const bool live = j < a.n;
      const bool ev = live && key_of(i) <= thr;
      const bool is_hole = live && j < a.kv_max && ev;
      const bool is_src = live && j >= a.kv_max && !ev;
      int ht, stot;
      const int hr = block_excl_count(is_hole, s_wave, &ht);
      const int sr = block_excl_count(is_src, s_wave, &stot);
      if (is_hole) holes[hbase + hr] = j;
      if (is_src) srcs[sbase + sr] = j;
      hbase += ht;
      sbase += stot;
    }
  } else {
    build_lists([&](int i) { return key_of(i) <= thr; }, n_iter, per, a.n, a.kv_max, s_cnt, s_tot,
                [&](bool hole, int idx, int j) { (hole ? holes : srcs)[idx] = j; });
    hbase = s_tot[0];
    sbase = s_tot[1];
  }
  if (tid == 0) {
    a.mcount[u] = min(hbase, sbase);
    a.len[u] = a.kv_max;
  }
}

__global__ void __launch_bounds__(256) compact_kernel(EvictArgs a, int nchunks) {
  constexpr int kMoves = 32;
  const int u = blockIdx.x / nchunks;
  const int chunk = blockIdx.x - u * nchunks;
  const int m = a.mcount[u];
  const int m0 = chunk * kMoves;
  if (m0 >= m) return;
  const int32_t* holes = a.holes + (int64_t)u * a.cap;
  const int32_t* srcs = a.srcs + (int64_t)u * a.cap;
  const int row_bytes = a.head_dim * a.elem_bytes;
  const int cpr = row_bytes / 16;
  char* kc = static_cast<char*>(a.kc) + (int64_t)u * a.cap * row_bytes;
  char* vc = static_cast<char*>(a.vc) + (int64_t)u * a.cap * row_bytes;
  const int total = kMoves * 2 * cpr;
  for (int c = threadIdx.x; c < total; c += 256) {
    const int mv = c / (2 * cpr);
    const int rem = c - mv * 2 * cpr;
    const int mi = m0 + mv;
    if (mi >= m) continue;
    const int which = rem / cpr, cc = rem - which * cpr;
    char* base = which ? vc : kc;
    const int64_t src = (int64_t)srcs[mi] * row_bytes + cc * 16;
    const int64_t dst = (int64_t)holes[mi] * row_bytes + cc * 16;
    *reinterpret_cast<uint4*>(base + dst) = *reinterpret_cast<const uint4*>(base + src);
  }
  if (threadIdx.x < kMoves) {
    const int mi = m0 + threadIdx.x;
    if (mi < m) {
      const int s = srcs[mi], d = holes[mi];
      a.score[(int64_t)u * a.cap + d] = a.score[(int64_t)u * a.cap + s];
      a.pos[(int64_t)u * a.cap + d] = a.pos[(int64_t)u * a.cap + s];
      if (a.rule == BM_RANK_TOVA) a.lastw[(int64_t)u * a.cap + d] = a.lastw[(int64_t)u * a.cap + s];
    }
  }
}

// K7: the fold of K1's partial column sums, the cut and the compaction of one
// unit in one workgroup (the block's Algorithm 1 step in one launch instead of
// three).  The folded scores, the positions and TOVA's weights stay in LDS, the
// keys in registers; the hole and source lists are built in LDS; the moves copy
// K and V rows with 16-byte loads and stores.  Needs n <= kMaxCap.
// KP: keys per thread held in registers (n <= 256 KP)
template <int KP>
__global__ void __launch_bounds__(256) fold_cut_kernel(PrefillArgs pa, EvictArgs a,
                                                        int pt_positions) {
  __shared__ uint32_t hist[512];
  __shared__ uint64_t s_prefix;
  __shared__ int s_need;
  __shared__ uint32_t s_cnt[4 * kMaxPer];
  __shared__ int s_tot[2];
  // per-slot LDS arrays, n4 = n rounded up to 4 entries each (dynamic size)
  extern __shared__ __attribute__((aligned(16))) char k7_lds[];
  const int n = a.n;
  const int n4 = (n + 3) & ~3;
  float* sc = reinterpret_cast<float*>(k7_lds);
  int32_t* ps = reinterpret_cast<int32_t*>(sc + n4);
  float* lw = reinterpret_cast<float*>(ps + n4);
  int32_t* holes = reinterpret_cast<int32_t*>(lw + n4);
  int32_t* srcs = holes + n4;
  const int u = blockIdx.x;
  const int tid = threadIdx.x;
  const int per = (n + 255) / 256;
  float* score = a.score + (int64_t)u * a.cap;
  int32_t* pos = a.pos + (int64_t)u * a.cap;
  float* last = a.rule == BM_RANK_TOVA ? a.lastw + (int64_t)u * a.cap : nullptr;
  const float* part = pa.partial + (int64_t)u * pa.npt_stride * pa.cap;

  // 1. fold the partial sums (workgroup order, as score_reduce_kernel) and key.
  //    Four entries at a time, every load of a round is issued before any is
  //    used: addresses are clamped into range (an unused term reads a row the
  //    entry needs anyway) and unused terms are selected to zero, so no load
  //    sits behind a branch and the sums keep their order (adding +0 changes
  //    nothing: the sums are >= 0).
  constexpr int FK = KP < 4 ? KP : 4;   // entries per round
  constexpr int PTC = 8;                // partial rows per round
  static_assert(KP % FK == 0, "whole rounds");
  uint64_t key[KP];
  const int nlast = n - 1;
  const int npt_used = pa.accumulate ? pa.npt_used : 0;
#pragma unroll
  for (int i0 = 0; i0 < KP; i0 += FK) {
    if (i0 >= per) break;   // uniform across the workgroup
    float acc[FK], l[FK], sc0[FK];
    int p[FK], pt0[FK];
    float x[FK][PTC];
    // partial row of term c0 + c, clamped into the rows the entry has (or row
    // 0 of the workspace when nothing accumulates)
    auto load_terms = [&](int c0) {
#pragma unroll
      for (int f = 0; f < FK; ++f) {
        const int jc = min(tid + 256 * (i0 + f), nlast);
#pragma unroll
        for (int c = 0; c < PTC; ++c) {
          const int pt = min(max(c0 + c, pt0[f]), max(npt_used - 1, 0));
          x[f][c] = part[(int64_t)pt * pa.cap + jc];
        }
      }
    };
    auto add_terms = [&](int c0) {
#pragma unroll
      for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int c = 0; c < PTC; ++c) {
          const int pt = c0 + c;
          acc[f] += pt >= pt0[f] && pt < npt_used ? x[f][c] : 0.0f;
        }
    };
#pragma unroll
    for (int f = 0; f < FK; ++f) {
      const int jc = min(tid + 256 * (i0 + f), nlast);
      pt0[f] = jc < pa.len0 ? 0 : (jc - pa.len0) / pt_positions;
      sc0[f] = score[jc];
      p[f] = pos[jc];
      l[f] = last ? last[jc] : 0.0f;
    }
    load_terms(0);   // issued with the loads above, before any of them is used
#pragma unroll
    for (int f = 0; f < FK; ++f) {
      const int jc = min(tid + 256 * (i0 + f), nlast);
      acc[f] = jc < pa.len0 ? sc0[f] : 0.0f;
    }
    add_terms(0);
    for (int c0 = PTC; c0 < npt_used; c0 += PTC) {
      load_terms(c0);
      add_terms(c0);
    }
#pragma unroll
    for (int f = 0; f < FK; ++f) {
      const int i = i0 + f, j = tid + 256 * i;
      key[i] = ~0ull;
      if (i < per && j < n) {
        score[j] = acc[f];
        sc[j] = acc[f];
        ps[j] = p[f];
        lw[j] = l[f];
        key[i] = rank_key(a.rule, acc[f], l[f], p[f], a.curr_id);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < KP; ++i)
    if (i >= per) key[i] = ~0ull;
  if (n <= a.kv_max) {
    if (tid == 0) a.len[u] = n;
    return;
  }

  // 2. the cut: the (n - kv_max)-th smallest key, then holes and sources
  auto key_of = [&](int i) __device__ -> uint64_t { return key[i]; };
  const uint64_t thr = radix_kth(key_of, KP, per, n, n - a.kv_max, position_bits(a.curr_id), hist,
                                 &s_prefix, &s_need);
  build_lists([&](int i) { return key[i] <= thr; }, KP, per, n, a.kv_max, s_cnt, s_tot,
              [&](bool hole, int idx, int j) { (hole ? holes : srcs)[idx] = j; });
  const int hbase = s_tot[0], sbase = s_tot[1];
  __syncthreads();

  // 3. the moves: the i-th source into the i-th hole (disjoint slot ranges)
  const int m = min(hbase, sbase);
  const int row_bytes = a.head_dim * a.elem_bytes;
  const int cpr = row_bytes / 16;
  char* kc = static_cast<char*>(a.kc) + (int64_t)u * a.cap * row_bytes;
  char* vc = static_cast<char*>(a.vc) + (int64_t)u * a.cap * row_bytes;
  for (int c = tid; c < m * 2 * cpr; c += 256) {
    const int mv = c / (2 * cpr);
    const int rem = c - mv * 2 * cpr;
    const int which = rem / cpr, cc = rem - which * cpr;
    char* base = which ? vc : kc;
    const int64_t src = (int64_t)srcs[mv] * row_bytes + cc * 16;
    const int64_t dst = (int64_t)holes[mv] * row_bytes + cc * 16;
    *reinterpret_cast<uint4*>(base + dst) = *reinterpret_cast<const uint4*>(base + src);
  }
  for (int mv = tid; mv < m; mv += 256) {
    const int sj = srcs[mv], dj = holes[mv];
    score[dj] = sc[sj];
    pos[dj] = ps[sj];
    if (last) last[dj] = lw[sj];
  }
  if (tid == 0) a.len[u] = a.kv_max;
}

}  // namespace

hipError_t launch_fold_cut(const PrefillArgs& pa, const EvictArgs& a, int pt_positions,
                           hipStream_t stream) {
  if (a.n > kMaxCap) return hipErrorInvalidValue;
  const size_t lds = 5 * sizeof(int32_t) * (size_t)((a.n + 3) & ~3);
  if (a.n <= 256 * 3)
    hipLaunchKernelGGL(fold_cut_kernel<3>, dim3((unsigned)a.units), dim3(256), lds, stream, pa, a,
                       pt_positions);
  else if (a.n <= 256 * 4)
    hipLaunchKernelGGL(fold_cut_kernel<4>, dim3((unsigned)a.units), dim3(256), lds, stream, pa, a,
                       pt_positions);
  else
    hipLaunchKernelGGL(fold_cut_kernel<kMaxPer>, dim3((unsigned)a.units), dim3(256), lds, stream, pa,
                       a, pt_positions);
  return hipGetLastError();
}

hipError_t launch_select(const EvictArgs& a, hipStream_t stream) {
  if (a.n > kMaxCap)
    hipLaunchKernelGGL(select_kernel<0>, dim3((unsigned)a.units), dim3(256), 0, stream, a);
  else if (a.n <= 256 * 3)
    hipLaunchKernelGGL(select_kernel<3>, dim3((unsigned)a.units), dim3(256), 0, stream, a);
  else if (a.n <= 256 * 4)
    hipLaunchKernelGGL(select_kernel<4>, dim3((unsigned)a.units), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(select_kernel<kMaxPer>, dim3((unsigned)a.units), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_compact(const EvictArgs& a, int max_moves, hipStream_t stream) {
  if (max_moves <= 0) return hipSuccess;
  const int nchunks = (max_moves + 31) / 32;
  hipLaunchKernelGGL(compact_kernel, dim3((unsigned)(a.units * nchunks)), dim3(256), 0, stream,
                     a, nchunks);
  return hipGetLastError();
}

}  // namespace bm
