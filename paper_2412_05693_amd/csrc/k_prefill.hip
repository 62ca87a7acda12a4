// K1: fused block-prefill attention with per-key score column sums, gfx950.
//
// One workgroup = one unit (sample, KV head) x one tile of 128/G block
// positions x all G query heads of the unit; wave w owns query head w % G and
// 32 consecutive positions.  For every query row the kernel computes the
// causal softmax attention over the unit's live cache entries plus the block's
// keys up to the row's own position (Sec. 3.1 block-wise prefill), writes the
// output, and adds the row's probabilities to a per-key partial sum (the
// sum_weights update of Sec. 3.2).  Per-workgroup partial sums land in the
// workspace; score_reduce_kernel folds them into the scores in a fixed order,
// so the result does not depend on scheduling.
//
// Exact column sums need every row's final softmax normaliser before any of
// its probabilities can be added to a key's sum.  The kernel therefore makes
// two sweeps over the key tiles:
//   sweep 1 (S^T = K Q^T orientation: one query per lane) -- online softmax,
//            O^T += V^T P^T on MFMA, final row max m and sum l;
//   sweep 2 (S = Q K^T orientation: one key per lane) -- recompute the logits,
//            P = exp2(z - m - log2 l) exactly, and sum over the rows held in
//            the lane's registers, so each lane ends with one key's column sum.
// Keys stream through LDS (double-buffered, one barrier per tile); V tiles are
// stored as 8-key groups transposed to [group][d][8] so one 16-byte LDS read
// yields an MFMA operand.  Keys of a 32-key sub-tile are stored in LDS row
// order kappa (bits 2 and 3 of the row swapped), which makes the register
// layout of the S^T accumulator coincide with the PV MFMA's B operand.
#include <type_traits>

#include "bm_internal.h"

namespace bm {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kPosInf = __builtin_huge_valf();

__device__ __forceinline__ int kappa(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 r = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, r);
}

// key index inside the 64-key tile held by accumulator register (i, j) of lane
// half h in S^T orientation, sub-tile st
__device__ __forceinline__ int st_key(int st, int i, int j, int h) {
  return 32 * st + 16 * (i >> 1) + 8 * h + 4 * (i & 1) + j;
}

template <bool BF16, int D>
struct Tile {
  // LDS row strides in elements (16-byte padding)
  static constexpr int kRow = BF16 ? D + 8 : D + 4;
  static constexpr int kKElems = kKeyTile * kRow;
  static constexpr int kGStride = D * 8 + 8;                    // bf16 V group stride
  static constexpr int kVElems = BF16 ? 8 * kGStride : kKeyTile * kRow;
  static constexpr int kQSteps = BF16 ? D / 16 : D / 2;         // MFMA K-steps over d
  static constexpr int kMT = D / 32;                             // 32-row M-tiles of O^T
  using elem_t = typename std::conditional<BF16, uint16_t, float>::type;
  using qfrag_t = typename std::conditional<BF16, bf16x8, float>::type;
  static constexpr int kKChunks = kKeyTile * D * (int)sizeof(elem_t) / 16 / kThreads;
  static constexpr int kVCombos = BF16 ? (8 * (D / 4) * 2) / kThreads : kKChunks;
};

template <bool BF16, int D>
struct SMem {
  using T = Tile<BF16, D>;
  typename T::elem_t k[2][T::kKElems];
  typename T::elem_t v[2][T::kVElems];
  float cs[2][kWaves][kKeyTile];
};

template <bool BF16, int D>
__device__ __forceinline__ f32x16 mfma_step(typename Tile<BF16, D>::qfrag_t a,
                                            typename Tile<BF16, D>::qfrag_t b, f32x16 c) {
  if constexpr (BF16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
}

// fragment of LDS row `row` of the K tile for K-step kk, lane half h
template <bool BF16, int D>
__device__ __forceinline__ typename Tile<BF16, D>::qfrag_t
k_frag(const typename Tile<BF16, D>::elem_t* ks, int row, int h, int kk) {
  using T = Tile<BF16, D>;
  if constexpr (BF16) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(ks + row * T::kRow + h * (D / 2) + 8 * kk);
    return __builtin_bit_cast(bf16x8, w);
  } else {
    return ks[row * T::kRow + h * (D / 2) + kk];
  }
}

struct Geo {
  int u, bi, hk, pt, w, lane, n, h, g, sub;
  int pbase;       // first block position (relative to t0) of the workgroup
  int row;         // this lane's query row (relative to t0) in S^T orientation
  bool qvalid;
  bool wave_active;
  int nkeys_wg;    // keys the workgroup touches: len0 + its last position + 1
  int nkeys_w;     // keys this wave's rows can see
};

template <int G>
__device__ __forceinline__ Geo make_geo(const PrefillArgs& a) {
  Geo s;
  const int lin = blockIdx.x;
  s.u = lin / a.npt_used;
  s.pt = lin - s.u * a.npt_used;
  s.bi = s.u / a.n_kv_heads;
  s.hk = s.u - s.bi * a.n_kv_heads;
  s.w = threadIdx.x >> 6;
  s.lane = threadIdx.x & 63;
  s.n = s.lane & 31;
  s.h = s.lane >> 5;
  s.g = s.w % G;
  s.sub = s.w / G;
  constexpr int PT = kWaves * kRowsPerWave / G;
  s.pbase = s.pt * PT;
  const int wrow0 = s.pbase + s.sub * kRowsPerWave;
  s.row = wrow0 + s.n;
  s.qvalid = s.row < a.n_tok;
  s.wave_active = wrow0 < a.n_tok;
  s.nkeys_wg = a.len0 + min(a.n_tok, s.pbase + PT);
  s.nkeys_w = a.len0 + min(a.n_tok, wrow0 + kRowsPerWave);
  return s;
}

// ---------------------------------------------------------------------------
// staging: global -> registers -> LDS
// ---------------------------------------------------------------------------
template <bool BF16, int D>
struct Stage {
  using T = Tile<BF16, D>;
  using E = typename T::elem_t;
  u32x4 kr[T::kKChunks];
  u32x2 vr[BF16 ? T::kVCombos * 4 : 1];
  u32x4 vf[BF16 ? 1 : T::kKChunks];

  __device__ __forceinline__ static const E* key_src(const PrefillArgs& a, const Geo& s,
                                                    const E* kc, const E* kin, int key) {
    if (key < a.len0) return kc + ((int64_t)s.u * a.cap + key) * D;
    if (key < s.nkeys_wg)
      return kin + (((int64_t)s.bi * a.n_kv_heads + s.hk) * a.seq_ld + (key - a.len0)) * D;
    return nullptr;
  }

  __device__ __forceinline__ void load_k(const PrefillArgs& a, const Geo& s, int tile_base) {
    const E* kc = static_cast<const E*>(a.kc);
    const E* kin = static_cast<const E*>(a.kin);
    constexpr int CPR = D * (int)sizeof(E) / 16;  // 16-byte chunks per row
#pragma unroll
    for (int i = 0; i < T::kKChunks; ++i) {
      const int c = threadIdx.x + kThreads * i;
      const int r = c / CPR, cc = c - r * CPR;
      const int key = tile_base + (r & ~31) + kappa(r & 31);
      const E* src = key_src(a, s, kc, kin, key);
      kr[i] = src ? *reinterpret_cast<const u32x4*>(src + cc * (16 / sizeof(E))) : u32x4{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store_k(E* ks) const {
    constexpr int CPR = D * (int)sizeof(E) / 16;
#pragma unroll
    for (int i = 0; i < T::kKChunks; ++i) {
      const int c = threadIdx.x + kThreads * i;
      const int r = c / CPR, cc = c - r * CPR;
      *reinterpret_cast<u32x4*>(ks + r * T::kRow + cc * (16 / sizeof(E))) = kr[i];
    }
  }

  __device__ __forceinline__ void load_v(const PrefillArgs& a, const Geo& s, int tile_base) {
    const E* vc = static_cast<const E*>(a.vc);
    const E* vin = static_cast<const E*>(a.vin);
    if constexpr (BF16) {
      // combo = (group of 8 keys, half of the group, 4 consecutive d)
#pragma unroll
      for (int i = 0; i < T::kVCombos; ++i) {
        const int c = threadIdx.x + kThreads * i;
        const int dq = c % (D / 4);
        const int rest = c / (D / 4);
        const int kh = rest & 1, grp = rest >> 1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = tile_base + 8 * grp + 4 * kh + e;
          const E* src = key_src(a, s, vc, vin, key);
          vr[4 * i + e] = src ? *reinterpret_cast<const u32x2*>(src + 4 * dq) : u32x2{0, 0};
        }
      }
    } else {
      constexpr int CPR = D * 4 / 16;
#pragma unroll
      for (int i = 0; i < T::kKChunks; ++i) {
        const int c = threadIdx.x + kThreads * i;
        const int r = c / CPR, cc = c - r * CPR;
        const E* src = key_src(a, s, vc, vin, tile_base + r);
        vf[i] = src ? *reinterpret_cast<const u32x4*>(src + cc * 4) : u32x4{0, 0, 0, 0};
      }
    }
  }
  __device__ __forceinline__ void store_v(E* vs) const {
    if constexpr (BF16) {
#pragma unroll
      for (int i = 0; i < T::kVCombos; ++i) {
        const int c = threadIdx.x + kThreads * i;
        const int dq = c % (D / 4);
        const int rest = c / (D / 4);
        const int kh = rest & 1, grp = rest >> 1;
        const u32x2 r0 = vr[4 * i + 0], r1 = vr[4 * i + 1], r2 = vr[4 * i + 2], r3 = vr[4 * i + 3];
        // transpose 4 keys x 4 d (bf16) into 4 d-rows of 4 keys
        u32x2 o0, o1, o2, o3;
        o0.x = (r0.x & 0xffffu) | (r1.x << 16);
        o0.y = (r2.x & 0xffffu) | (r3.x << 16);
        o1.x = (r0.x >> 16) | (r1.x & 0xffff0000u);
        o1.y = (r2.x >> 16) | (r3.x & 0xffff0000u);
        o2.x = (r0.y & 0xffffu) | (r1.y << 16);
        o2.y = (r2.y & 0xffffu) | (r3.y << 16);
        o3.x = (r0.y >> 16) | (r1.y & 0xffff0000u);
        o3.y = (r2.y >> 16) | (r3.y & 0xffff0000u);
        E* base = vs + grp * T::kGStride + (4 * dq) * 8 + 4 * kh;
        *reinterpret_cast<u32x2*>(base + 0 * 8) = o0;
        *reinterpret_cast<u32x2*>(base + 1 * 8) = o1;
        *reinterpret_cast<u32x2*>(base + 2 * 8) = o2;
        *reinterpret_cast<u32x2*>(base + 3 * 8) = o3;
      }
    } else {
      constexpr int CPR = D * 4 / 16;
#pragma unroll
      for (int i = 0; i < T::kKChunks; ++i) {
        const int c = threadIdx.x + kThreads * i;
        const int r = c / CPR, cc = c - r * CPR;
        *reinterpret_cast<u32x4*>(vs + r * T::kRow + cc * 4) = vf[i];
      }
    }
  }
};

template <bool BF16, int D, int G>
__global__ void __launch_bounds__(kThreads, (BF16 || D == 64) ? 2 : 1) prefill_attn_kernel(PrefillArgs a) {
  using T = Tile<BF16, D>;
  using E = typename T::elem_t;
  __shared__ SMem<BF16, D> sm;
  const Geo s = make_geo<G>(a);
  const int tid = threadIdx.x;

  // ---- append the workgroup's block rows to the cache tail (Sec. 3.2: new
  //      entries start with score 0; the score is written by score_reduce) ----
  {
    constexpr int PT = kWaves * kRowsPerWave / G;
    constexpr int CPR = D * (int)sizeof(E) / 16;
    const int r0 = s.pbase, r1 = min(a.n_tok, s.pbase + PT);
    const E* kin = static_cast<const E*>(a.kin);
    const E* vin = static_cast<const E*>(a.vin);
    E* kc = static_cast<E*>(a.kc);
    E* vc = static_cast<E*>(a.vc);
    const int64_t plane = ((int64_t)s.bi * a.n_kv_heads + s.hk) * a.seq_ld;
    for (int c = tid; c < (r1 - r0) * CPR; c += kThreads) {
      const int r = r0 + c / CPR, cc = c % CPR;
      const int64_t dst = ((int64_t)s.u * a.cap + a.len0 + r) * D + cc * (16 / sizeof(E));
      const int64_t src = (plane + r) * D + cc * (16 / sizeof(E));
      *reinterpret_cast<u32x4*>(kc + dst) = *reinterpret_cast<const u32x4*>(kin + src);
      *reinterpret_cast<u32x4*>(vc + dst) = *reinterpret_cast<const u32x4*>(vin + src);
    }
    for (int r = r0 + tid; r < r1; r += kThreads)
      a.pos[(int64_t)s.u * a.cap + a.len0 + r] = a.t0 + r;
  }

  // ---- query fragments: lane (n, h) holds row n, d-range [h*D/2, (h+1)*D/2) ----
  typename T::qfrag_t qf[T::kQSteps];
  {
    const int qh = s.hk * G + s.g;
    const E* q = static_cast<const E*>(a.q) +
                 (((int64_t)s.bi * a.n_heads + qh) * a.seq_ld + s.row) * D + s.h * (D / 2);
#pragma unroll
    for (int kk = 0; kk < T::kQSteps; ++kk) {
      if constexpr (BF16) {
        const u32x4 w = s.qvalid ? *reinterpret_cast<const u32x4*>(q + 8 * kk) : u32x4{0, 0, 0, 0};
        qf[kk] = __builtin_bit_cast(bf16x8, w);
      } else {
        qf[kk] = s.qvalid ? q[kk] : 0.0f;
      }
    }
  }

  const int ntiles = (s.nkeys_wg + kKeyTile - 1) / kKeyTile;
  const float c2 = a.scale_log2;
  // a row sees key slots j <= lim (cached slots, then block keys up to itself)
  const int lim = a.len0 + (s.qvalid ? s.row : a.n_tok - 1);

  // ======================= sweep 1: online softmax + PV =======================
  f32x16 oacc[T::kMT];
#pragma unroll
  for (int mt = 0; mt < T::kMT; ++mt) oacc[mt] = f32x16{};
  float m_run = kNegInf, l_run = 0.0f;

  Stage<BF16, D> stg;
  stg.load_k(a, s, 0);
  stg.load_v(a, s, 0);
  stg.store_k(sm.k[0]);
  stg.store_v(sm.v[0]);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int tile_base = t * kKeyTile;
    if (t + 1 < ntiles) {
      stg.load_k(a, s, tile_base + kKeyTile);
      stg.load_v(a, s, tile_base + kKeyTile);
    }
    if (s.wave_active && tile_base < s.nkeys_w) {
      const E* ks = sm.k[buf];
      const E* vs = sm.v[buf];
      f32x16 sacc[2];
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        sacc[st] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < T::kQSteps; ++kk)
          sacc[st] = mfma_step<BF16, D>(k_frag<BF16, D>(ks, st * 32 + s.n, s.h, kk), qf[kk], sacc[st]);
      }
      // mask, scale, tile max
      float tmax = kNegInf;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = tile_base + st_key(st, r >> 2, r & 3, s.h);
          const float x = key <= lim ? sacc[st][r] * c2 : kNegInf;
          sacc[st][r] = x;
          tmax = fmaxf(tmax, x);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      const float m_new = fmaxf(m_run, tmax);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float psum = 0.0f;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(sacc[st][r] - m_new);
          sacc[st][r] = p;
          psum += p;
        }
      l_run = l_run * alpha + psum;
      m_run = m_new;
      if (__ballot(alpha != 1.0f) != 0) {
#pragma unroll
        for (int mt = 0; mt < T::kMT; ++mt)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[mt][r] *= alpha;
      }
      // O^T += V^T P^T
      if constexpr (BF16) {
#pragma unroll
        for (int ks4 = 0; ks4 < 4; ++ks4) {
          const int st = ks4 >> 1, half = ks4 & 1;
          u32x4 pw;
          pw.x = pack_bf16x2(sacc[st][8 * half + 0], sacc[st][8 * half + 1]);
          pw.y = pack_bf16x2(sacc[st][8 * half + 2], sacc[st][8 * half + 3]);
          pw.z = pack_bf16x2(sacc[st][8 * half + 4], sacc[st][8 * half + 5]);
          pw.w = pack_bf16x2(sacc[st][8 * half + 6], sacc[st][8 * half + 7]);
          const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
          const E* vg = vs + (2 * ks4 + s.h) * T::kGStride;
#pragma unroll
          for (int mt = 0; mt < T::kMT; ++mt) {
            const u32x4 vw = *reinterpret_cast<const u32x4*>(vg + (32 * mt + s.n) * 8);
            oacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vw), pb,
                                                                oacc[mt], 0, 0, 0);
          }
        }
      } else {
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = st_key(st, r >> 2, r & 3, s.h);
#pragma unroll
            for (int mt = 0; mt < T::kMT; ++mt)
              oacc[mt] = __builtin_amdgcn_mfma_f32_32x32x2f32(vs[key * T::kRow + 32 * mt + s.n],
                                                              sacc[st][r], oacc[mt], 0, 0, 0);
          }
      }
    }
    if (t + 1 < ntiles) {
      stg.store_k(sm.k[buf ^ 1]);
      stg.store_v(sm.v[buf ^ 1]);
    }
    __syncthreads();
  }

  // ---- finish rows: normalise, store O, row log-sum-exp (log2 units) ----
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  float lse2 = kPosInf;
  if (s.wave_active) {
    const float inv = 1.0f / l_tot;
    lse2 = s.qvalid ? m_run + __builtin_amdgcn_logf(l_tot) : kPosInf;
    if (s.qvalid) {
      const int qh = s.hk * G + s.g;
      E* o = static_cast<E*>(a.o) + (((int64_t)s.bi * a.n_heads + qh) * a.seq_ld + s.row) * D;
#pragma unroll
      for (int mt = 0; mt < T::kMT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d0 = 32 * mt + 8 * i + 4 * s.h;
          const float x0 = oacc[mt][4 * i + 0] * inv, x1 = oacc[mt][4 * i + 1] * inv;
          const float x2 = oacc[mt][4 * i + 2] * inv, x3 = oacc[mt][4 * i + 3] * inv;
          if constexpr (BF16) {
            u32x2 w = {pack_bf16x2(x0, x1), pack_bf16x2(x2, x3)};
            *reinterpret_cast<u32x2*>(o + d0) = w;
          } else {
            *reinterpret_cast<float4*>(o + d0) = make_float4(x0, x1, x2, x3);
          }
        }
    }
  }

  // ======================= sweep 2: exact column sums ========================
  // S orientation: lane (n, h) holds key n of a 32-key sub-tile and rows
  // 8i + 4h + j of the wave's 32 rows in accumulator register 4i + j.
  float lse_r[16];
  int lim_r[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int rr = 8 * (r >> 2) + 4 * s.h + (r & 3);
    lse_r[r] = __shfl(lse2, rr);
    lim_r[r] = a.len0 + s.pbase + s.sub * kRowsPerWave + rr;
  }
  float* partial = a.partial + ((int64_t)s.u * a.npt_stride + s.pt) * a.cap;

  stg.load_k(a, s, 0);
  stg.store_k(sm.k[0]);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int tile_base = t * kKeyTile;
    if (t + 1 < ntiles) stg.load_k(a, s, tile_base + kKeyTile);
    if (s.wave_active && tile_base < s.nkeys_w) {
      const E* ks = sm.k[buf];
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        f32x16 acc = f32x16{};
#pragma unroll
        for (int kk = 0; kk < T::kQSteps; ++kk)
          acc = mfma_step<BF16, D>(qf[kk], k_frag<BF16, D>(ks, st * 32 + s.n, s.h, kk), acc);
        const int key = tile_base + 32 * st + kappa(s.n);
        float csum = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float x = key <= lim_r[r] ? acc[r] * c2 - lse_r[r] : kNegInf;
          csum += __builtin_amdgcn_exp2f(x);
        }
        csum += __shfl_xor(csum, 32);
        if (s.h == 0) sm.cs[buf][s.w][32 * st + kappa(s.n)] = csum;
      }
    } else if (s.lane < 32) {
      sm.cs[buf][s.w][s.lane] = 0.0f;
      sm.cs[buf][s.w][32 + s.lane] = 0.0f;
    }
    if (t + 1 < ntiles) stg.store_k(sm.k[buf ^ 1]);
    __syncthreads();
    if (tid < kKeyTile && tile_base + tid < s.nkeys_wg) {
      float acc = 0.0f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) acc += sm.cs[buf][w][tid];
      partial[tile_base + tid] = acc;
    }
  }
}

// Fold the per-workgroup partial column sums into the scores, in workgroup
// order: score[j] = (j < len0 ? score[j] : 0) + sum over workgroups that saw j.
__global__ void __launch_bounds__(256) score_reduce_kernel(PrefillArgs a, int pt_positions) {
  const int u = blockIdx.x;
  const int n = a.len0 + a.n_tok;
  const float* part = a.partial + (int64_t)u * a.npt_stride * a.cap;
  float* score = a.score + (int64_t)u * a.cap;
  for (int j = threadIdx.x; j < n; j += blockDim.x) {
    const int pt0 = j < a.len0 ? 0 : (j - a.len0) / pt_positions;
    float acc = j < a.len0 ? score[j] : 0.0f;
    for (int pt = pt0; pt < a.npt_used; ++pt) acc += part[(int64_t)pt * a.cap + j];
    score[j] = acc;
  }
  if (threadIdx.x == 0) a.len[u] = n;
}

template <bool BF16, int D, int G>
hipError_t launch_t(const PrefillArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)(a.units * a.npt_used));
  hipLaunchKernelGGL((prefill_attn_kernel<BF16, D, G>), grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <bool BF16, int D>
hipError_t launch_g(const PrefillArgs& a, int group, hipStream_t stream) {
  switch (group) {
    case 1: return launch_t<BF16, D, 1>(a, stream);
    case 2: return launch_t<BF16, D, 2>(a, stream);
    case 4: return launch_t<BF16, D, 4>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int head_dim, int group,
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

hipError_t launch_score_reduce(const PrefillArgs& a, hipStream_t stream) {
  const int group = a.n_heads / a.n_kv_heads;
  hipLaunchKernelGGL(score_reduce_kernel, dim3((unsigned)a.units), dim3(256), 0, stream, a,
                     positions_per_wg(group));
  return hipGetLastError();
}

}  // namespace bm
