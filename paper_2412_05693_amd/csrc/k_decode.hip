// K4: one decode step per unit, fused: attention over the bounded cache plus
// the step's own KV pair, score update, ranking, one eviction, in-place write.
//
// Decode is bandwidth-bound (the paper notes it reloads the whole cache every
// step, Sec. 1): the kernel reads each cached K and V row exactly once.  One
// workgroup per unit (sample, KV head); L = len + 1 entries (len cached slots
// plus the step's pair, which sits in a virtual slot `len`).
//   1. logits z[g][j] = sm_scale * q_g . k_j for the G query heads, kept in LDS
//      (bf16: a 16x16x32 MFMA per 16 keys, K rows as the A operand straight
//      from global memory; f32: VALU dot products);
//   2. exact softmax per query head in LDS (max and sum; each use multiplies
//      by the reciprocal of the sum);
//   3. score_j += sum_g P[g][j] (the sum_weights update of Sec. 3.2), ranking
//      key of the chosen rule (by default ave = score / (pos_now + 1 - pos))
//      packed with pos into 64 bits, and a workgroup argmin (older entry first
//      on an exact tie);
//   4. o_g = sum_j p[g][j] v_j on VALU (exponentials summed, then scaled once
//      by the reciprocal), V rows read once, 16 bytes per lane (marked
//      non-temporal when the launch's cached K and V exceed the
//      device's last-level cache: they are not read again before the next
//      step has streamed the whole cache through; below that size the next
//      step finds them in the cache);
//   5. write back the scores; if the cache exceeds kv_max, the new pair takes
//      the slot of the removed entry (or is dropped if it is the one removed);
//      otherwise it is appended at slot len.
#include <type_traits>

#include "bm_internal.h"
#include "bm_lanes.h"

namespace bm {
namespace {

using lanes::add_xor;
using lanes::wave_max;
using lanes::wave_min_u64;
using lanes::wave_sum;

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr float kNegInf = -__builtin_huge_valf();

// probability = exp2(z - max) * (1 / sum), rounded once and never fused into
// the sum that uses it (the scores and the ranking see the same value a
// normalised copy in LDS would hold)
__device__ __forceinline__ float prob(float e, float inv) {
#pragma clang fp contract(off)
  return e * inv;
}

template <bool NT>
__device__ __forceinline__ u32x4 load_v(const void* p) {
  if constexpr (NT) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  } else {
    return *reinterpret_cast<const u32x4*>(p);
  }
}

template <bool BF16, int D, int G, bool NTV>
__global__ void __launch_bounds__(256) decode_kernel(DecodeArgs a) {
  using E = typename std::conditional<BF16, uint16_t, float>::type;
  constexpr int EPC = 16 / sizeof(E);       // elements per 16-byte chunk
  constexpr int CPR = D / EPC;              // 16-byte chunks per row
  extern __shared__ float dsm[];
  __shared__ uint64_t s_wkey[4];
  __shared__ int s_wslot[4];
  __shared__ float s_inv[4];      // 1 / softmax sum per query head

  const int u = blockIdx.x;
  const int bi = u / a.n_kv_heads, hk = u - (u / a.n_kv_heads) * a.n_kv_heads;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int len0 = a.len0;
  const int L = len0 + 1;
  const int Lp = (L + 3) & ~3;
  float* P = dsm;                 // [G][Lp] logits, then exp2(logit - max)
  float* sc = P + G * Lp;         // [Lp] scores (prefetched, then updated)
  float* red = sc + Lp;           // [4][G][D] partial outputs per wave
  int32_t* pos_s = reinterpret_cast<int32_t*>(red + 4 * G * D);   // [Lp] positions

  const E* kc = static_cast<const E*>(a.kc) + (int64_t)u * a.cap * D;
  const E* vc = static_cast<const E*>(a.vc) + (int64_t)u * a.cap * D;
  const int64_t plane = ((int64_t)bi * a.n_kv_heads + hk) * a.seq_ld;
  const E* knew = static_cast<const E*>(a.kin) + plane * D;
  const E* vnew = static_cast<const E*>(a.vin) + plane * D;
  const E* qbase = static_cast<const E*>(a.q) + ((int64_t)bi * a.n_heads + hk * G) * a.seq_ld * D;
  const float c2 = a.scale_log2;

  // Scores and positions (used from the softmax on): the first NSP per thread
  // are loaded into registers here and written to LDS after the logits, so
  // their latency hides behind the K loads; entries beyond 256 * NSP are
  // copied after the logits.
  constexpr int NSP = 4;
  const float* score_g = a.score + (int64_t)u * a.cap;
  const int32_t* pos_g = a.pos + (int64_t)u * a.cap;
  float sp_score[NSP];
  int32_t sp_pos[NSP];
#pragma unroll
  for (int r = 0; r < NSP; ++r) {
    const int j = min(tid + 256 * r, max(len0 - 1, 0));   // slot 0 exists even when empty
    sp_score[r] = score_g[j];
    sp_pos[r] = pos_g[j];
  }

  // ---------------- 1. logits ----------------
  if constexpr (BF16) {
    const int col = lane & 15, g4 = lane >> 4;
    bf16x8 qop[D / 32];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      // columns G..15 repeat the last head (their results are not stored)
      const int qc = min(col, G - 1);
      qop[ks] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(qbase + (int64_t)qc * a.seq_ld * D + 32 * ks + 8 * g4));
    }
    const int ngroups = (L + 15) / 16;
    // Keys past the last entry read the step's own key row (valid memory; their
    // logits are never stored).  With no branch around a load the compiler
    // can count the loads in flight and wait only for the group it multiplies
    // while the next group's rows are still arriving.
    auto k_rows = [&](int kg, u32x4 (&dst)[D / 32]) {
      const int key = kg * 16 + col;
      const E* src = key < len0 ? kc + (int64_t)key * D : knew;
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        dst[ks] = *reinterpret_cast<const u32x4*>(src + 32 * ks + 8 * g4);
    };
    auto logits = [&](int kg, const u32x4 (&src)[D / 32]) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, src[ks]), qop[ks],
                                                      acc, 0, 0, 0);
      if (col < G) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int kk = kg * 16 + 4 * g4 + j;
          if (kk < L) P[col * Lp + kk] = acc[j] * c2;
        }
      }
    };
    // KD register sets in turn, KD groups in flight (no copy between sets,
    // which would make the loop wait for a group still in flight)
    constexpr int KD = 2;
    u32x4 kr[KD][D / 32];
#pragma unroll
    for (int i = 0; i + 1 < KD; ++i) k_rows(w + 4 * i, kr[i]);
    for (int kg = w; kg < ngroups; kg += 4 * KD) {
#pragma unroll
      for (int i = 0; i < KD; ++i) {
        k_rows(kg + 4 * (i + KD - 1), kr[(i + KD - 1) % KD]);
        if (i == 0 || kg + 4 * i < ngroups) logits(kg + 4 * i, kr[i]);
      }
    }
  } else {
    constexpr int CH = D / 4;               // float4 chunks per row
    constexpr int NKL = 256 / CH;           // keys in flight per workgroup pass
    const int c = tid % CH, kl = tid / CH;
    float4 qr[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
      qr[g] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(qbase) +
                                               (int64_t)g * a.seq_ld * D + 4 * c);
    const int iters = (L + NKL - 1) / NKL;
    for (int it = 0; it < iters; ++it) {
      const int j = kl + it * NKL;
      const float* src = j < len0 ? reinterpret_cast<const float*>(kc) + (int64_t)j * D
                                  : (j == len0 ? reinterpret_cast<const float*>(knew) : nullptr);
      const float4 kv = src ? *reinterpret_cast<const float4*>(src + 4 * c) : make_float4(0, 0, 0, 0);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float part = qr[g].x * kv.x + qr[g].y * kv.y + qr[g].z * kv.z + qr[g].w * kv.w;
        part = lanes::group_sum<CH>(part);
        if (c == 0 && j < L) P[g * Lp + j] = part * c2;
      }
    }
  }
#pragma unroll
  for (int r = 0; r < NSP; ++r) {
    const int j = tid + 256 * r;
    if (j < L) {
      sc[j] = j < len0 ? sp_score[r] : 0.0f;
      pos_s[j] = j < len0 ? sp_pos[r] : a.cur_pos;
    }
  }
  for (int j = tid + 256 * NSP; j < L; j += 256) {
    sc[j] = j < len0 ? score_g[j] : 0.0f;
    pos_s[j] = j < len0 ? pos_g[j] : a.cur_pos;
  }
  __syncthreads();

  // first batch of V rows for phase 4, in flight during the softmax
  constexpr int NKL4 = 256 / CPR;
  constexpr int UNR = 8;   // V rows per thread in flight (and as many prefetched)
  const int c4 = tid % CPR, kl4 = tid / CPR;
  // rows past the last entry read the step's own V row (valid memory, never
  // used): unconditional loads, so only the batch being consumed is waited for
  auto v_row = [&](int j) -> u32x4 {
    const E* src = j < len0 ? vc + (int64_t)j * D : vnew;
    return load_v<NTV>(src + c4 * EPC);
  };
  u32x4 vw[UNR];
#pragma unroll
  for (int r = 0; r < UNR; ++r) vw[r] = v_row(kl4 + r * NKL4);

  // ---------------- 2. softmax per query head ----------------
  // P keeps exp2(z - max) and s_inv[g] = 1 / sum; each use forms the
  // probability with prob().  Left padding: pad entries (pos < pad) are
  // visible to no query.
  const int pad = a.pad ? max(0, a.pad[bi]) : 0;
  constexpr int NSM = 16;   // logits per lane held in registers when L <= 64 * NSM
  for (int g = w; g < G; g += 4) {
    float* pg = P + g * Lp;
    auto visible = [&](int j) { return j < L && !(pad > 0 && pos_s[min(j, L - 1)] < pad); };
    float m = kNegInf, s = 0.0f;
    if (L <= 64 * NSM) {
      // one read of the row with no branch around an LDS read (the pad test
      // is chosen once), so the reads are issued together
      float x[NSM];
      auto load_row = [&](auto padded) {
#pragma unroll
        for (int i = 0; i < NSM; ++i) {
          const int j = lane + 64 * i, jc = min(j, L - 1);
          const float z = pg[jc];
          bool vis = j < L;
          if constexpr (decltype(padded)::value) vis = vis && pos_s[jc] >= pad;
          x[i] = vis ? z : kNegInf;
        }
      };
      if (pad > 0)
        load_row(std::true_type{});
      else
        load_row(std::false_type{});
#pragma unroll
      for (int i = 0; i < NSM; ++i) m = fmaxf(m, x[i]);
      m = wave_max(m);
#pragma unroll
      for (int i = 0; i < NSM; ++i) {
        const int j = lane + 64 * i;
        const float e = __builtin_amdgcn_exp2f(x[i] - m);
        if (j < L) pg[j] = e;
        s += e;
      }
    } else {
      for (int j = lane; j < L; j += 64) m = fmaxf(m, visible(j) ? pg[j] : kNegInf);
      m = wave_max(m);
      for (int j = lane; j < L; j += 64) {
        const float e = __builtin_amdgcn_exp2f((visible(j) ? pg[j] : kNegInf) - m);
        pg[j] = e;
        s += e;
      }
    }
    s = wave_sum(s);
    if (lane == 0) s_inv[g] = 1.0f / s;
  }
  __syncthreads();

  // ---------------- 3. scores and ranking ----------------
  const bool evict = L > a.kv_max;
  {
    uint64_t best = ~0ull;
    int bslot = -1;
    for (int j = tid; j < L; j += 256) {
      float ps = 0.0f;
#pragma unroll
      for (int g = 0; g < G; ++g) ps += prob(P[g * Lp + j], s_inv[g]);
      const float s = sc[j] + ps;
      sc[j] = s;
      const uint64_t key = rank_key(a.rule, s, ps, pos_s[j], a.cur_pos);
      if (key < best) {
        best = key;
        bslot = j;
      }
    }
    // the wave's smallest key (unique: it carries the entry's position) and
    // the slot of the lane that holds it
    const uint64_t wmin = wave_min_u64(best);
    const uint64_t holders = __ballot(best == wmin);
    bslot = __builtin_amdgcn_readlane(bslot, (int)__builtin_ctzll(holders));
    best = wmin;
    if (lane == 0) {
      s_wkey[w] = best;
      s_wslot[w] = bslot;
    }
  }

  // ---------------- 4. outputs o_g = s_inv[g] * sum_j P[g][j] v_j ----------------
  static_assert(2 * CPR <= 256, "one thread per 16-byte chunk of the new K and V rows");
  u32x4 nrow;   // this thread's chunk of the step's own K or V row (write back)
  {
    constexpr int NKL = NKL4;
    const int c = c4;
    float acc[G][EPC];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[g][e] = 0.0f;
    for (int j0 = kl4; j0 < L; j0 += NKL * UNR) {
      // next batch in flight while this one is consumed
      u32x4 vn[UNR];
#pragma unroll
      for (int r = 0; r < UNR; ++r) vn[r] = v_row(j0 + (UNR + r) * NKL);
#pragma unroll
      for (int r = 0; r < UNR; ++r) {
        const int j = j0 + r * NKL;
        if (j >= L) break;
        float vf[EPC];
        if constexpr (BF16) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            vf[2 * e] = __uint_as_float(vw[r][e] << 16);
            vf[2 * e + 1] = __uint_as_float(vw[r][e] & 0xffff0000u);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) vf[e] = __uint_as_float(vw[r][e]);
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const float p = P[g * Lp + j];
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e]);
        }
      }
#pragma unroll
      for (int r = 0; r < UNR; ++r) vw[r] = vn[r];
    }
    // the new rows for the write back, loaded while the outputs are reduced
    {
      const int nc = min(tid, 2 * CPR - 1);
      nrow = *reinterpret_cast<const u32x4*>((nc >= CPR ? vnew : knew) + (nc % CPR) * EPC);
    }
    // reduce the lanes of a wave that share chunk c (lanes c, c + CPR, ...),
    // then across waves in LDS
    static_assert(CPR == 8 || CPR == 16 || CPR == 32, "16-byte chunks per row");
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        float x = acc[g][e];
        if constexpr (CPR <= 8) x = add_xor<8>(x);
        if constexpr (CPR <= 16) x = add_xor<16>(x);
        acc[g][e] = add_xor<32>(x);
      }
    if (lane < CPR) {
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < EPC; ++e) red[(w * G + g) * D + c * EPC + e] = acc[g][e];
    }
  }
  __syncthreads();

  // final outputs
  for (int idx = tid; idx < G * D; idx += 256) {
    const int g = idx / D, d = idx - g * D;
    const float x = (red[(0 * G + g) * D + d] + red[(1 * G + g) * D + d] +
                     red[(2 * G + g) * D + d] + red[(3 * G + g) * D + d]) * s_inv[g];
    E* o = static_cast<E*>(a.o) + (((int64_t)bi * a.n_heads + hk * G + g) * a.seq_ld) * D + d;
    if constexpr (BF16) {
      *o = __builtin_bit_cast(uint16_t, (__bf16)x);
    } else {
      *o = x;
    }
  }

  // ---------------- 5. write back ----------------
  int e_slot = -1;
  if (evict) {
    uint64_t best = s_wkey[0];
    e_slot = s_wslot[0];
#pragma unroll
    for (int i = 1; i < 4; ++i)
      if (s_wkey[i] < best) {
        best = s_wkey[i];
        e_slot = s_wslot[i];
      }
  }
  const int dst = evict ? e_slot : len0;          // slot that receives the new pair
  float* score = a.score + (int64_t)u * a.cap;
  for (int j = tid; j < len0; j += 256)
    if (j != dst) score[j] = sc[j];
  if (dst >= 0 && dst < len0 + (evict ? 0 : 1)) {
    E* kd = static_cast<E*>(a.kc) + ((int64_t)u * a.cap + dst) * D;
    E* vd = static_cast<E*>(a.vc) + ((int64_t)u * a.cap + dst) * D;
    if (tid < 2 * CPR) {
      const int which = tid / CPR, cc = tid - which * CPR;
      *reinterpret_cast<u32x4*>((which ? vd : kd) + cc * EPC) = nrow;
    }
    if (tid == 0) {
      score[dst] = sc[len0];
      a.pos[(int64_t)u * a.cap + dst] = a.cur_pos;
    }
  }
  if (a.lastw) {
    // this step's weights, summed over the group's heads: the TOVA key of the
    // next cut (the new pair's lands in its slot)
    float* lw = a.lastw + (int64_t)u * a.cap;
    for (int j = tid; j <= len0; j += 256) {
      const int slot = j < len0 ? j : dst;
      if ((j < len0 && j == dst) || slot < 0 || slot >= len0 + (evict ? 0 : 1)) continue;
      float ps = 0.0f;
#pragma unroll
      for (int g = 0; g < G; ++g) ps += prob(P[g * Lp + j], s_inv[g]);
      lw[slot] = ps;
    }
  }
  if (tid == 0) a.len[u] = evict ? len0 : len0 + 1;
}

// MI355X's last-level (Infinity) cache: 256 MiB
constexpr size_t kLastLevelCacheBytes = (size_t)256 << 20;

template <bool BF16, int D, int G>
hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  const int L = a.len0 + 1;
  const int Lp = (L + 3) & ~3;
  const size_t lds = sizeof(float) * ((size_t)G * Lp + Lp + 4 * G * D + Lp);
  const size_t kv_bytes = (size_t)a.units * 2 * a.len0 * D * (BF16 ? 2 : 4);
  if (kv_bytes > kLastLevelCacheBytes)
    hipLaunchKernelGGL((decode_kernel<BF16, D, G, true>), dim3((unsigned)a.units), dim3(256), lds,
                       stream, a);
  else
    hipLaunchKernelGGL((decode_kernel<BF16, D, G, false>), dim3((unsigned)a.units), dim3(256), lds,
                       stream, a);
  return hipGetLastError();
}

template <bool BF16, int D>
hipError_t launch_g(const DecodeArgs& a, int group, hipStream_t stream) {
  switch (group) {
    case 1: return launch_t<BF16, D, 1>(a, stream);
    case 2: return launch_t<BF16, D, 2>(a, stream);
    case 4: return launch_t<BF16, D, 4>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int dtype, int head_dim, int group,
                         hipStream_t stream) {
  if (dtype == BM_BF16) {
    if (head_dim == 128) return launch_g<true, 128>(a, group, stream);
    if (head_dim == 64) return launch_g<true, 64>(a, group, stream);
  } else if (dtype == BM_F32) {
    if (head_dim == 128) return launch_g<false, 128>(a, group, stream);
    if (head_dim == 64) return launch_g<false, 64>(a, group, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace bm
