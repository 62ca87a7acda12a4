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
// Both sweeps are software-pipelined: the MFMAs of tile t+1's logits are issued
// before tile t's softmax, so the matrix cores and the VALU work overlap within
// a wave.
//
// Key tiles hold 64 rows from one source: the unit's cache rows [0, len0) first,
// then the block's input rows.  Tiles are copied global -> LDS by buffer loads
// that write LDS directly (no staging registers); rows past a source's range
// come back as zeros.  LDS rows are padded (the DMA writes zeros into the
// padding slots), so the MFMA operand reads are free of bank conflicts and use
// base + immediate addressing.
// K rows of a 32-key sub-tile sit in LDS row order kappa (bits 2 and 3 of the
// row swapped), which makes the register layout of the S^T accumulator equal
// to the PV MFMA's B operand; V reaches the PV MFMA through gfx950's
// transposing LDS load (ds_read_b64_tr_b16).
#include <type_traits>

#include "bm_internal.h"

namespace bm {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __bf16 __attribute__((vector_size(8))) bf16v4;   // operand type of the LDS transpose read
typedef __attribute__((address_space(3))) bf16v4 lds_bf16v4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kPosInf = __builtin_huge_valf();
constexpr int kRsrcWord3 = 0x00020000;
constexpr float kRescaleLog2 = 8.0f;
// s_waitcnt with vmcnt(0) and the other counters left alone
constexpr int kWaitVm0 = 0x0F70;

// ---- prefill timeline (measurement builds: BM_PREFILL_TIMELINE) ----
// Thread 0 of each workgroup keeps the fields of include/bm_probe.h in
// registers and stores them at its end; in the ordinary build every use sits
// in an `if constexpr (kTimeline)` branch and nothing is emitted.
#ifdef BM_PREFILL_TIMELINE
constexpr bool kTimeline = true;
__device__ uint64_t g_timeline[(size_t)BM_TIMELINE_MAX_RECORDS * BM_TIMELINE_FIELDS];
__device__ __forceinline__ void timeline_store(int id, const uint64_t* tl) {
  if (threadIdx.x == 0 && id < BM_TIMELINE_MAX_RECORDS) {
#pragma unroll
    for (int i = 0; i < BM_TIMELINE_FIELDS; ++i) g_timeline[(size_t)id * BM_TIMELINE_FIELDS + i] = tl[i];
  }
}
#else
constexpr bool kTimeline = false;
__device__ __forceinline__ void timeline_store(int, const uint64_t*) {}
#endif
// the constant-rate real-time counter (read only in timeline builds)
__device__ __forceinline__ uint64_t tl_now() {
  if constexpr (kTimeline) return __builtin_amdgcn_s_memrealtime();
  return 0;
}

__device__ __forceinline__ int kappa(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// x of lane i combined with x of lane i ^ 32 through gfx950's cross-half swap
// (no LDS round trip); the swap returns the two values in the same order on
// both lanes, so both get bit-identical results
__device__ __forceinline__ float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
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
struct Cfg {
  using E = typename std::conditional<BF16, uint16_t, float>::type;
  using qfrag_t = typename std::conditional<BF16, bf16x8, float>::type;
  static constexpr int RB = D * (int)sizeof(E);          // bytes per K/V row
  static constexpr int CPR = RB / 16;                     // 16-byte chunks per row
  // LDS rows are padded by one (K) or two (V) 16-byte chunks: the MFMA operand
  // reads of K (16 lanes, 16 rows, one chunk each) and the transposing reads of
  // V (4 rows x 32 bytes per 16-lane group) then fall in distinct banks.
  static constexpr int KCP = CPR + 1, VCP = CPR + 2;     // chunks per padded row
  static constexpr int KSTRIDE = KCP * 16, VSTRIDE = VCP * 16;
  static constexpr int K_BYTES = kKeyTile * KSTRIDE, V_BYTES = kKeyTile * VSTRIDE;
  static constexpr int QSTEPS = BF16 ? D / 16 : D / 2;   // MFMA K-steps over d
  static constexpr int MT = D / 32;                       // 32-row M-tiles of O^T
};


template <bool BF16, int D>
__device__ __forceinline__ f32x16 mfma_step(typename Cfg<BF16, D>::qfrag_t a,
                                            typename Cfg<BF16, D>::qfrag_t b, f32x16 c) {
  if constexpr (BF16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
}

// fragment of LDS row `row` of a K tile for K-step kk, lane half h.  bf16:
// K-step kk contracts the 16-byte chunks 2 kk (lane half 0) and 2 kk + 1 (lane
// half 1) of d, so the two halves of a query row's load fall in one cache line
template <bool BF16, int D>
__device__ __forceinline__ typename Cfg<BF16, D>::qfrag_t k_frag(const char* ks, int row, int h,
                                                                 int kk) {
  using C = Cfg<BF16, D>;
  if constexpr (BF16) {
    const int b = (2 * kk + h) * 16;
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(ks + row * C::KSTRIDE + b));
  } else {
    const int b = (h * (D / 2) + kk) * 4;
    return *reinterpret_cast<const float*>(ks + row * C::KSTRIDE + b);
  }
}

struct Geo {
  int u, bi, hk, pt, w, lane, n, h, g, sub;
  int pbase;       // first block position (relative to t0) of the workgroup
  int wrow0;       // first query row (relative to t0) of this wave
  int row;         // this lane's query row (relative to t0) in S^T orientation
  int wlast;       // last real query row of this wave
  bool qvalid;
  bool wave_active;
  int in_rows;     // block rows the workgroup reads: min(n_tok, pbase + PT)
  int ntc, nt;     // cache tiles, all tiles
  int pad;         // left pad tokens of the sample (positions < pad are pads)
  bool qpad;       // this lane's query row is a pad token
};

template <int G, bool PAD>
__device__ __forceinline__ Geo make_geo(const PrefillArgs& a) {
  Geo s;
  // Workgroups are dispatched round-robin over the 8 XCDs (each with its own
  // L2).  Renumber them so that consecutive logical ids -- the workgroups of
  // one unit -- land on the same XCD and share that unit's K/V in its L2.
  const int nwg = gridDim.x, L = blockIdx.x;
  const int q8 = nwg >> 3, r8 = nwg & 7, xcd = L & 7;
  const int lin = xcd * q8 + min(xcd, r8) + (L >> 3);
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
  s.wrow0 = s.pbase + s.sub * kRowsPerWave;
  s.row = s.wrow0 + s.n;
  s.qvalid = s.row < a.n_tok;
  s.wave_active = s.wrow0 < a.n_tok;
  s.wlast = min(a.n_tok - 1, s.wrow0 + kRowsPerWave - 1);
  s.in_rows = min(a.n_tok, s.pbase + PT);
  s.ntc = (a.len0 + kKeyTile - 1) / kKeyTile;
  s.nt = s.ntc + (s.in_rows + kKeyTile - 1) / kKeyTile;
  s.pad = PAD ? max(0, a.pad[s.bi]) : 0;
  s.qpad = a.t0 + s.row < s.pad;
  return s;
}

// Where tile t comes from and which of its rows exist.
struct TileInfo {
  bool cache;      // rows from the unit's cache (else the block's input rows)
  int base;        // first source row of the tile
  int slot0;       // cache slot of the tile's row 0 (for the score sums)
  int valid;       // rows of the tile that exist
};

__device__ __forceinline__ TileInfo tile_info(const PrefillArgs& a, const Geo& s, int t) {
  TileInfo ti;
  ti.cache = t < s.ntc;
  ti.base = (ti.cache ? t : t - s.ntc) * kKeyTile;
  ti.slot0 = ti.cache ? ti.base : a.len0 + ti.base;
  ti.valid = min(kKeyTile, (ti.cache ? a.len0 : s.in_rows) - ti.base);
  return ti;
}

// does the wave see any key of tile t; does the tile need masking for it
__device__ __forceinline__ bool tile_active(const Geo& s, const TileInfo& ti) {
  return s.wave_active && (ti.cache || ti.base <= s.wlast);
}
__device__ __forceinline__ bool tile_masked(const Geo& s, const TileInfo& ti) {
  return ti.cache ? ti.valid < kKeyTile : ti.base + kKeyTile - 1 > s.wrow0;
}

// Tiles of K (rows in kappa order) and V are copied into LDS with buffer loads
// that write LDS directly; lane i of instruction j of wave w fills the 16-byte
// chunk (w * DMA_PER_WAVE + j) * 64 + i of the tile.  The buffer resource of a
// tile's source (cache rows [0, len0) or the block rows the workgroup reads) is
// built per tile from values forced into scalar registers, so the loads take
// it straight from SGPRs.
struct TileSrc {
  __amdgpu_buffer_rsrc_t rsrc;
};

// An out-of-range offset: the lane writes zeros (used for the padding slots).
constexpr int kOutOfRange = 0x7FFFFFF0;

// Copy one tile into padded LDS rows.  Slot g = 64 * seg + lane of the tile
// holds chunk g % CP of row g / CP; chunks >= CPR are padding.  K rows are
// stored in kappa order within each 32-row sub-tile.
template <bool BF16, int D, bool K>
__device__ __forceinline__ void dma_rows(char* dst, const TileSrc& src, const TileInfo& ti,
                                         const Geo& s) {
  using C = Cfg<BF16, D>;
  constexpr int CP = K ? C::KCP : C::VCP;   // also the number of 1 KB segments
#pragma unroll
  for (int j = 0; j < (CP + kWaves - 1) / kWaves; ++j) {
    const int seg = s.w + kWaves * j;
    if (seg < CP) {   // uniform per wave
      const int g = seg * 64 + s.lane;
      const int r = g / CP, c = g - r * CP;
      const int key = K ? (r & ~31) + kappa(r & 31) : r;
      const int off = c < C::CPR ? (ti.base + key) * C::RB + c * 16 : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(src.rsrc, (lds_void*)(dst + seg * 1024), 16, off, 0, 0, 0);
    }
  }
}

template <bool BF16, int D, int G, bool PAD>
__global__ void __launch_bounds__(kThreads, (BF16 || D == 64) ? 2 : 1) prefill_attn_kernel(PrefillArgs a) {
  // PAD: the launch has left padding (a separate instantiation, so the common
  // case carries none of its registers)
  using C = Cfg<BF16, D>;
  using E = typename C::E;
  constexpr int RB = C::RB;
  // separate arrays per buffer: with the ping-pong index known at compile time
  // the compiler can tell the tile being filled from the tile being read
  __shared__ __attribute__((aligned(1024))) char kb0[C::K_BYTES];
  __shared__ __attribute__((aligned(1024))) char kb1[C::K_BYTES];
  __shared__ __attribute__((aligned(1024))) char vb0[C::V_BYTES];
  __shared__ __attribute__((aligned(1024))) char vb1[C::V_BYTES];
  __shared__ float cs0[kWaves][kKeyTile];
  __shared__ float cs1[kWaves][kKeyTile];
  // positions of the cached keys of tile t in pk_ring[t % 3] (left padding
  // only): tile t's positions are read while tile t + 2's are being fetched
  __shared__ int32_t pk_ring[3][kKeyTile];
  // the block's last query's weights per wave (TOVA's key), double-buffered like cs
  __shared__ float lws0[kWaves][kKeyTile];
  __shared__ float lws1[kWaves][kKeyTile];
  uint64_t tl[BM_TIMELINE_FIELDS] = {};
  if constexpr (kTimeline) tl[BM_TL_ENTRY] = tl_now();
  const Geo s = make_geo<G, PAD>(a);
  const int tid = threadIdx.x;
  auto stamp = [&](int field) __device__ {
    if constexpr (kTimeline) tl[field] = tl_now();
  };
  auto timeline_end = [&]() __device__ {
    if constexpr (kTimeline) {
      tl[BM_TL_END] = tl_now();
      // HW_ID (all 32 bits) and, above it, XCC_ID (hardware registers 4 and 20)
      tl[BM_TL_HW_ID] = (uint64_t)__builtin_amdgcn_s_getreg(0xF804) |
                        ((uint64_t)__builtin_amdgcn_s_getreg(0xF814) << 32);
      tl[BM_TL_ITEM] = ((uint64_t)s.u << 32) | (uint32_t)s.pt;
      tl[BM_TL_TILES] = (uint64_t)s.nt;
      timeline_store(blockIdx.x, tl);
    }
  };
  // end of a tile: wait for this wave's copies, then for every wave
  auto wait_and_sync = [&](int f_wait, int f_barrier) __device__ {
    if constexpr (kTimeline) {
      const uint64_t a0 = tl_now();
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
      const uint64_t a1 = tl_now();
      __syncthreads();
      tl[f_wait] += a1 - a0;
      tl[f_barrier] += tl_now() - a1;
    } else {
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
      __syncthreads();
    }
  };

  constexpr int PT = kWaves * kRowsPerWave / G;   // block positions per workgroup

  // ---- append the workgroup's block rows to the cache tail (Sec. 3.2: new
  //      entries start with score 0; the score is written by score_reduce).
  //      The loads are issued here, with the query loads and the first tile
  //      copies behind them, and the stores follow the wait those need anyway,
  //      so the workgroup waits for memory once before its first tile. ----
  const int64_t plane = ((int64_t)s.bi * a.n_kv_heads + s.hk) * a.seq_ld;
  constexpr int NA = (PT * C::CPR + kThreads - 1) / kThreads;   // chunks per thread
  const int app_chunks = (s.in_rows - s.pbase) * C::CPR;
  u32x4 app_k[NA], app_v[NA];
  {
    const E* kin = static_cast<const E*>(a.kin);
    const E* vin = static_cast<const E*>(a.vin);
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int c = tid + i * kThreads;
      if (c < app_chunks) {
        const int r = s.pbase + c / C::CPR, cc = c % C::CPR;
        const int64_t src = (plane + r) * D + cc * (16 / sizeof(E));
        app_k[i] = *reinterpret_cast<const u32x4*>(kin + src);
        app_v[i] = *reinterpret_cast<const u32x4*>(vin + src);
      }
    }
  }
  auto append_store = [&]() __device__ {
    E* kc = static_cast<E*>(a.kc);
    E* vc = static_cast<E*>(a.vc);
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int c = tid + i * kThreads;
      if (c < app_chunks) {
        const int r = s.pbase + c / C::CPR, cc = c % C::CPR;
        const int64_t dst = ((int64_t)s.u * a.cap + a.len0 + r) * D + cc * (16 / sizeof(E));
        *reinterpret_cast<u32x4*>(kc + dst) = app_k[i];
        *reinterpret_cast<u32x4*>(vc + dst) = app_v[i];
      }
    }
    for (int r = s.pbase + tid; r < s.in_rows; r += kThreads)
      a.pos[(int64_t)s.u * a.cap + a.len0 + r] = a.t0 + r;
  };

  // ---- row sources of the tiles (out-of-range rows read as zero) ----
  const uint64_t kc_base = (uint64_t)(static_cast<const E*>(a.kc) + (int64_t)s.u * a.cap * D);
  const uint64_t vc_base = (uint64_t)(static_cast<const E*>(a.vc) + (int64_t)s.u * a.cap * D);
  const uint64_t ki_base = (uint64_t)(static_cast<const E*>(a.kin) + plane * D);
  const uint64_t vi_base = (uint64_t)(static_cast<const E*>(a.vin) + plane * D);
  auto tile_src = [&](const TileInfo& ti, bool kside) __device__ {
    const uint64_t p = ti.cache ? (kside ? kc_base : vc_base) : (kside ? ki_base : vi_base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
    const int nrec = __builtin_amdgcn_readfirstlane((ti.cache ? a.len0 : s.in_rows) * RB);
    TileSrc r;
    r.rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), 0, nrec, kRsrcWord3);
    return r;
  };
  const uint64_t pos_base = (uint64_t)(a.pos + (int64_t)s.u * a.cap);
  auto dma_k = [&](char* dst, const TileInfo& ti, int t) __device__ {
    dma_rows<BF16, D, true>(dst, tile_src(ti, true), ti, s);
    if (PAD && s.pad > 0 && ti.cache && s.w == 0) {
      // the tile's key positions, in key order, next to the K rows
      const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)pos_base);
      const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(pos_base >> 32));
      const int nrec = __builtin_amdgcn_readfirstlane(a.len0 * 4);
      const __amdgpu_buffer_rsrc_t r =
          __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), 0, nrec, kRsrcWord3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)pk_ring[t % 3], 4,
                                               (ti.base + s.lane) * 4, 0, 0, 0);
    }
  };
  // bit k set: key k of tile ti is a pad token (cache keys through the LDS copy
  // of their positions); uniform across the workgroup
  auto pad_bits = [&](const TileInfo& ti, const int32_t* pk) __device__ -> uint64_t {
    if (!PAD || s.pad == 0) return 0;
    if (ti.cache) return __ballot(pk[s.lane] < s.pad);
    const int n = min(max(s.pad - a.t0 - ti.base, 0), kKeyTile);
    return n >= 64 ? ~0ull : ((1ull << n) - 1);
  };
  auto dma_v = [&](char* dst, const TileInfo& ti) __device__ {
    dma_rows<BF16, D, false>(dst, tile_src(ti, false), ti, s);
  };

  // ---- query fragments: lane (n, h) holds row n; bf16: the d-chunks 2 kk + h
  //      (the order k_frag reads K in), fp32: d-range [h*D/2, (h+1)*D/2) ----
  typename C::qfrag_t qf[C::QSTEPS];
  {
    const int qh = s.hk * G + s.g;
    const E* q = static_cast<const E*>(a.q) +
                 (((int64_t)s.bi * a.n_heads + qh) * a.seq_ld + s.row) * D;
#pragma unroll
    for (int kk = 0; kk < C::QSTEPS; ++kk) {
      if constexpr (BF16) {
        const u32x4 w = s.qvalid ? *reinterpret_cast<const u32x4*>(q + 8 * (2 * kk + s.h))
                                 : u32x4{0, 0, 0, 0};
        qf[kk] = __builtin_bit_cast(bf16x8, w);
      } else {
        qf[kk] = s.qvalid ? q[s.h * (D / 2) + kk] : 0.0f;
      }
    }
  }

  stamp(BM_TL_QUERY_ISSUED);
  const int nt = s.nt;
  const float c2 = a.scale_log2;
  // the row this lane's causal mask uses (padding rows reuse the last real row)
  const int qrow = s.qvalid ? s.row : a.n_tok - 1;

  // logits of one tile: S^T (one query per lane) or S (one key per lane); the
  // K fragments of step kk + 1 are read while the MFMAs of step kk run
  auto qk_tile = [&](auto st_tag, const char* ks, f32x16* acc) __device__ {
    constexpr bool ST = decltype(st_tag)::value;
    acc[0] = f32x16{};
    acc[1] = f32x16{};
    typename C::qfrag_t kf[2][2];
    kf[0][0] = k_frag<BF16, D>(ks, s.n, s.h, 0);
    kf[0][1] = k_frag<BF16, D>(ks, 32 + s.n, s.h, 0);
#pragma unroll
    for (int kk = 0; kk < C::QSTEPS; ++kk) {
      if (kk + 1 < C::QSTEPS) {
        kf[(kk + 1) & 1][0] = k_frag<BF16, D>(ks, s.n, s.h, kk + 1);
        kf[(kk + 1) & 1][1] = k_frag<BF16, D>(ks, 32 + s.n, s.h, kk + 1);
      }
#pragma unroll
      for (int st = 0; st < 2; ++st)
        acc[st] = ST ? mfma_step<BF16, D>(kf[kk & 1][st], qf[kk], acc[st])
                     : mfma_step<BF16, D>(qf[kk], kf[kk & 1][st], acc[st]);
    }
    if constexpr (BF16) {
      // pin the order: the reads of step kk + 1 go out before the MFMAs of
      // step kk (left alone, the scheduler sinks each read to its MFMA)
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);   // DS reads
#pragma unroll
      for (int kk = 0; kk + 2 < C::QSTEPS; ++kk) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0); // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    }
  };
  auto qk_st = [&](const char* ks, f32x16* acc) __device__ { qk_tile(std::true_type{}, ks, acc); };
  auto qk_s = [&](const char* ks, f32x16* acc) __device__ { qk_tile(std::false_type{}, ks, acc); };

  // ======================= sweep 1: online softmax + PV =======================
  f32x16 oacc[C::MT];
#pragma unroll
  for (int mt = 0; mt < C::MT; ++mt) oacc[mt] = f32x16{};
  float m_run = kNegInf, l_run = 0.0f;

  // softmax of tile t (S^T in sacc) and O^T += V^T P^T
  // left padding: a real query row sees no pad key (a pad row keeps its causal
  // keys; its output and score contributions are dropped later).  The lane's
  // keys all have bit 3 equal to h, so the pad bits are shifted once.
  auto hide_pads = [&](f32x16* sacc, uint64_t padk) __device__ {
    const uint64_t hide = s.qpad ? 0 : (padk >> (8 * s.h));
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if ((hide >> st_key(st, r >> 2, r & 3, 0)) & 1) sacc[st][r] = kNegInf;
  };

  auto sweep1_tile = [&](auto mask_tag, f32x16* sacc, const char* vs, const TileInfo& ti) __device__ {
    constexpr bool MASK = decltype(mask_tag)::value;
    if constexpr (MASK) {
      // key k of the tile is visible iff k <= lim_k
      const int lim_k = ti.cache ? ti.valid - 1 : qrow - ti.base;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sacc[st][r] = st_key(st, r >> 2, r & 3, s.h) <= lim_k ? sacc[st][r] : kNegInf;
    }
    // tile max on the raw logits (the scale is positive), then one fma per exp2
    float tmax = kNegInf;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, sacc[st][r]);
    tmax = xhalf_max(tmax);
    // The reference m_run moves only when some row of the wave sees a logit
    // more than kRescaleLog2 above it: the probabilities stay below
    // 2^kRescaleLog2 (exact in fp32, fine in bf16) and the O rescale is rare.
    if (__ballot(tmax * c2 > m_run + kRescaleLog2) != 0) {
      const float m_new = fmaxf(m_run, tmax * c2);
      // (a padded row that has seen no key yet keeps m = -inf: nothing to scale)
      const float alpha = PAD && m_new == kNegInf ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
      m_run = m_new;
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[mt][r] *= alpha;
    }
    float psum = 0.0f;
    // with left padding a row's first tiles can be all pad keys: m_run is still
    // -inf there and every logit is -inf, so subtract 0 to get p = 0, not NaN
    // (without padding every row sees a key in its first tile)
    const float m_sub = PAD && m_run == kNegInf ? 0.0f : m_run;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[st][r], c2, -m_sub));
        sacc[st][r] = p;
        psum += p;
      }
    l_run += psum;
    if constexpr (BF16) {
      // A operand (V^T): lane (n, h) needs V[key][32 mt + n] for the 8 keys
      // 16 ks + 8 h + e of P's k-slots.  The LDS transpose load gives lane i of
      // a 16-lane group column i of the 4 x 16 block formed by the group's
      // lanes 4r..4r+3 (row r), so lane 4r + c points at V[key0 + r][d0 + 4c]
      // and receives V[key0 + 0..3][d0 + i].
      const int j16 = s.lane & 15, dhalf = (s.lane >> 4) & 1;
      const int vrow = 8 * s.h + (j16 >> 2);
      const int vb = (16 * dhalf + 4 * (j16 & 3)) * 2;
      // the 2 x MT transposing reads of K-step ks4 + 1 are issued before the
      // MFMAs of step ks4
      u32x4 vf[2][C::MT];
      auto vload = [&](int ks4, u32x4* dst) __device__ {
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) {
          const int r0 = 16 * ks4 + vrow, b = vb + 64 * mt;
          const bf16v4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16v4*)(vs + r0 * C::VSTRIDE + b));
          const bf16v4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16v4*)(vs + (r0 + 4) * C::VSTRIDE + b));
          const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
          dst[mt] = u32x4{l2.x, l2.y, h2.x, h2.y};
        }
      };
      vload(0, vf[0]);
#pragma unroll
      for (int ks4 = 0; ks4 < 4; ++ks4) {
        if (ks4 + 1 < 4) vload(ks4 + 1, vf[(ks4 + 1) & 1]);
        const int st = ks4 >> 1, half = ks4 & 1;
        u32x4 pw;
        pw.x = pack_bf16x2(sacc[st][8 * half + 0], sacc[st][8 * half + 1]);
        pw.y = pack_bf16x2(sacc[st][8 * half + 2], sacc[st][8 * half + 3]);
        pw.z = pack_bf16x2(sacc[st][8 * half + 4], sacc[st][8 * half + 5]);
        pw.w = pack_bf16x2(sacc[st][8 * half + 6], sacc[st][8 * half + 7]);
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
          oacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vf[ks4 & 1][mt]), pb,
                                                              oacc[mt], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = st_key(st, r >> 2, r & 3, s.h);
#pragma unroll
          for (int mt = 0; mt < C::MT; ++mt) {
            const float vv = *reinterpret_cast<const float*>(vs + key * C::VSTRIDE + (32 * mt + s.n) * 4);
            oacc[mt] = __builtin_amdgcn_mfma_f32_32x32x2f32(vv, sacc[st][r], oacc[mt], 0, 0, 0);
          }
        }
    }
  };

  // prologue: K(0), V(0), K(1) land in LDS; logits of tile 0
  dma_k(kb0, tile_info(a, s, 0), 0);
  dma_v(vb0, tile_info(a, s, 0));
  if (nt > 1) dma_k(kb1, tile_info(a, s, 1), 1);
  stamp(BM_TL_COPIES_ISSUED);
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  append_store();
  __syncthreads();
  stamp(BM_TL_FIRST_TILE);
  // logits ping-pong between two register sets; the loop is unrolled by two so
  // every buffer choice below is a compile-time constant
  f32x16 sa[2], sb[2];
  // sweep 2's first K tiles are fetched during sweep 1's last iteration (not
  // with left padding: that iteration still reads the position ring slots the
  // early copies would refill)
  const bool early_k2 = !PAD && a.accumulate;
  if (tile_active(s, tile_info(a, s, 0))) qk_st(kb0, sa);
  __syncthreads();   // every wave has read K(0) before iteration 0 refills its buffer
  // iteration t (parity P = t & 1): K(t+1) and V(t) are in LDS and `cur` holds
  // tile t's logits; K(t+2) and V(t+1) are fetched meanwhile
  auto sweep1_iter = [&](auto par, int t, f32x16* cur, f32x16* nxt) __device__ {
    constexpr int P = decltype(par)::value;
    char* k_fill = P == 0 ? kb0 : kb1;
    char* k_next = P == 0 ? kb1 : kb0;
    char* v_cur = P == 0 ? vb0 : vb1;
    char* v_fill = P == 0 ? vb1 : vb0;
    const int32_t* pk_cur = pk_ring[t % 3];       // positions of tile t
    const TileInfo ti = tile_info(a, s, t);
    const uint64_t issue0 = tl_now();
    if (t + 2 < nt) dma_k(k_fill, tile_info(a, s, t + 2), t + 2);
    if (t + 1 < nt) {
      const TileInfo tn = tile_info(a, s, t + 1);
      dma_v(v_fill, tn);
      if constexpr (kTimeline) tl[BM_TL_S1_COPY_ISSUE] += tl_now() - issue0;
      if (tile_active(s, tn)) qk_st(k_next, nxt);
    }
    if (early_k2 && t == nt - 1) {
      // both K buffers are free in the last iteration: fetch the first two K
      // tiles of sweep 2 now, so they land with this iteration's wait
      dma_k(kb0, tile_info(a, s, 0), 0);
      if (nt > 1) dma_k(kb1, tile_info(a, s, 1), 1);
    }
    if (tile_active(s, ti)) {
      if constexpr (PAD) {
        const uint64_t padk = pad_bits(ti, pk_cur);
        if (padk) hide_pads(cur, padk);
      }
      if (tile_masked(s, ti))
        sweep1_tile(std::true_type{}, cur, v_cur, ti);
      else
        sweep1_tile(std::false_type{}, cur, v_cur, ti);
    }
    wait_and_sync(BM_TL_S1_WAIT, BM_TL_S1_BARRIER);
  };
  for (int t = 0; t < nt; t += 2) {
    sweep1_iter(std::integral_constant<int, 0>{}, t, sa, sb);
    if (t + 1 < nt) sweep1_iter(std::integral_constant<int, 1>{}, t + 1, sb, sa);
  }
  stamp(BM_TL_SWEEP1_END);

  // ---- finish rows: normalise, store O, row log-sum-exp (log2 units) ----
  const float l_tot = xhalf_sum(l_run);
  float lse2 = kPosInf;
  if (s.wave_active) {
    const float inv = 1.0f / l_tot;
    lse2 = s.qvalid && !s.qpad ? m_run + __builtin_amdgcn_logf(l_tot) : kPosInf;
    // a pad row has no output (zeros)
    const float sc = s.qpad ? 0.0f : inv;
    if constexpr (BF16) {
      // The wave's 32 output rows are contiguous in memory (one head, 32
      // consecutive positions).  They go through LDS -- the V buffers are
      // idle once sweep 1 is over; each wave uses its own padded 32-row
      // region -- so the stores are whole 1 KB runs instead of 16 bytes per
      // row per instruction.
      constexpr int OSTRIDE = C::KSTRIDE;   // padded row: D * 2 + 16 bytes
      static_assert(kWaves == 4 && 2 * kRowsPerWave * OSTRIDE <= C::V_BYTES,
                    "two waves' rows per V buffer");
      char* ost = (s.w < 2 ? vb0 : vb1) + (s.w & 1) * (kRowsPerWave * OSTRIDE);
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d0 = 32 * mt + 8 * i + 4 * s.h;
          const u32x2 w = {pack_bf16x2(oacc[mt][4 * i + 0] * sc, oacc[mt][4 * i + 1] * sc),
                           pack_bf16x2(oacc[mt][4 * i + 2] * sc, oacc[mt][4 * i + 3] * sc)};
          *reinterpret_cast<u32x2*>(ost + s.n * OSTRIDE + d0 * 2) = w;
        }
      // the output row's address is computed here rather than kept from the
      // query load (which would hold two registers through both sweeps)
      int orow0 = s.wrow0, ohead = s.bi * a.n_heads + s.hk * G + s.g;
      asm volatile("" : "+v"(orow0), "+v"(ohead));
      char* o = reinterpret_cast<char*>(static_cast<E*>(a.o) + ((int64_t)ohead * a.seq_ld + orow0) * D);
      constexpr int RUNS = kRowsPerWave * RB / 1024;   // 1 KB runs per wave
      constexpr int RPR = 1024 / RB;                   // rows per run
#pragma unroll
      for (int j = 0; j < RUNS; ++j) {
        const int r = RPR * j + s.lane / (RB / 16), c = s.lane % (RB / 16);
        const u32x4 v = *reinterpret_cast<const u32x4*>(ost + r * OSTRIDE + c * 16);
        if (s.wrow0 + r < a.n_tok)
          *reinterpret_cast<u32x4*>(o + (int64_t)r * RB + c * 16) = v;
      }
    } else if (s.qvalid) {
      int orow = s.row, ohead = s.bi * a.n_heads + s.hk * G + s.g;
      asm volatile("" : "+v"(orow), "+v"(ohead));
      E* o = static_cast<E*>(a.o) + ((int64_t)ohead * a.seq_ld + orow) * D;
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d0 = 32 * mt + 8 * i + 4 * s.h;
          const float x0 = oacc[mt][4 * i + 0] * sc, x1 = oacc[mt][4 * i + 1] * sc;
          const float x2 = oacc[mt][4 * i + 2] * sc, x3 = oacc[mt][4 * i + 3] * sc;
          *reinterpret_cast<float4*>(o + d0) = make_float4(x0, x1, x2, x3);
        }
    }
  }

  // ======================= sweep 2: exact column sums ========================
  // (skipped when the caller asked for outputs only)
  stamp(BM_TL_OUTPUT_STORED);
  if (!a.accumulate) {
    timeline_end();
    return;
  }
  // S orientation: lane (n, h) holds key n of a 32-key sub-tile and rows
  // 8i + 4h + j of the wave's 32 rows in accumulator register 4i + j.
  float lse_r[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) lse_r[r] = __shfl(lse2, 8 * (r >> 2) + 4 * s.h + (r & 3));
  float* partial = a.partial + ((int64_t)s.u * a.npt_stride + s.pt) * a.cap;
  // TOVA: the workgroup holding the block's last row also keeps that row's
  // weights (summed over the heads) for every key; its waves for that row find
  // it in accumulator register ri of lane half hr
  const int last_row = a.n_tok - 1;
  const bool wg_last = a.lastw && s.pbase <= last_row && last_row < s.pbase + PT;
  const bool wave_last = wg_last && s.wrow0 <= last_row && last_row < s.wrow0 + kRowsPerWave;
  const int rl = last_row - s.wrow0;
  const int ri = 4 * (rl >> 3) + (rl & 3), hr = (rl >> 2) & 1;
  float lse_last = lse_r[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) lse_last = r == ri ? lse_r[r] : lse_last;

  auto sweep2_tile = [&](auto mask_tag, f32x16* acc, const TileInfo& ti, float (*cs)[kKeyTile]) __device__ {
    constexpr bool MASK = decltype(mask_tag)::value;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int key = 32 * st + kappa(s.n);
      float csum = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = fmaf(acc[st][r], c2, -lse_r[r]);
        if constexpr (MASK) {
          const int qr = s.wrow0 + 8 * (r >> 2) + 4 * s.h + (r & 3);
          const int lim_k = ti.cache ? ti.valid - 1 : qr - ti.base;
          x = key <= lim_k ? x : kNegInf;
        }
        csum += __builtin_amdgcn_exp2f(x);
      }
      csum = xhalf_sum(csum);
      if (s.h == 0) cs[s.w][key] = csum;
    }
  };

  // prologue: K(0), K(1) land in LDS (already there when sweep 1's last
  // iteration fetched them); logits of tile 0
  if (!early_k2) {
    dma_k(kb0, tile_info(a, s, 0), 0);
    if (nt > 1) dma_k(kb1, tile_info(a, s, 1), 1);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
  }
  if (tile_active(s, tile_info(a, s, 0))) qk_s(kb0, sa);
  __syncthreads();   // every wave has read K(0) before iteration 0 refills its buffer
  stamp(BM_TL_SWEEP2_START);
  // iteration t (parity P = t & 1): K(t+1) is in LDS and `cur` holds tile t's logits
  auto sweep2_iter = [&](auto par, int t, f32x16* cur, f32x16* nxt) __device__ {
    constexpr int P = decltype(par)::value;
    char* k_fill = P == 0 ? kb0 : kb1;
    char* k_next = P == 0 ? kb1 : kb0;
    float (*cs)[kKeyTile] = P == 0 ? cs0 : cs1;
    float (*lws)[kKeyTile] = P == 0 ? lws0 : lws1;
    const int32_t* pk_cur = pk_ring[t % 3];
    const TileInfo ti = tile_info(a, s, t);
    if (t + 2 < nt) dma_k(k_fill, tile_info(a, s, t + 2), t + 2);
    if (t + 1 < nt) {
      const TileInfo tn = tile_info(a, s, t + 1);
      if (tile_active(s, tn)) qk_s(k_next, nxt);
    }
    if (tile_active(s, ti)) {
      if (tile_masked(s, ti))
        sweep2_tile(std::true_type{}, cur, ti, cs);
      else
        sweep2_tile(std::false_type{}, cur, ti, cs);
      if constexpr (PAD) {
        // a pad key is visible to no real row (pad rows add nothing: lse = +inf)
        const uint64_t padk = pad_bits(ti, pk_cur);
        if (padk && s.h == 0) {
#pragma unroll
          for (int st = 0; st < 2; ++st) {
            const int key = 32 * st + kappa(s.n);
            if ((padk >> key) & 1) cs[s.w][key] = 0.0f;
          }
        }
      }
    } else if (s.lane < 32) {
      cs[s.w][s.lane] = 0.0f;
      cs[s.w][32 + s.lane] = 0.0f;
    }
    if (wg_last) {
      // the last row sees every key of the tile (pads aside)
      const uint64_t padk = PAD ? pad_bits(ti, pk_cur) : 0;
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int key = 32 * st + kappa(s.n);
        float v = 0.0f;
        if (wave_last && tile_active(s, ti)) {
          float z = cur[st][0];
#pragma unroll
          for (int r = 1; r < 16; ++r) z = r == ri ? cur[st][r] : z;
          v = s.h == hr ? __builtin_amdgcn_exp2f(fmaf(z, c2, -lse_last)) : 0.0f;
          v = xhalf_sum(v);
          if (PAD && ((padk >> key) & 1)) v = 0.0f;
        }
        if (s.h == 0) lws[s.w][key] = v;
      }
    }
    wait_and_sync(BM_TL_S2_WAIT, BM_TL_S2_BARRIER);
    if (tid < ti.valid) {
      float acc = 0.0f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) acc += cs[w][tid];
      partial[ti.slot0 + tid] = acc;
      if (wg_last) {
        float lw = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) lw += lws[w][tid];
        a.lastw[(int64_t)s.u * a.cap + ti.slot0 + tid] = lw;
      }
    }
  };
  for (int t = 0; t < nt; t += 2) {
    sweep2_iter(std::integral_constant<int, 0>{}, t, sa, sb);
    if (t + 1 < nt) sweep2_iter(std::integral_constant<int, 1>{}, t + 1, sb, sa);
  }
  timeline_end();
}

// Fold the per-workgroup partial column sums into the scores, in workgroup
// order: score[j] = (j < len0 ? score[j] : 0) + sum over workgroups that saw j
// (without accumulation: new entries get 0, older scores stay).
// Grid: (units, slot chunks of 256); every thread owns one slot.  The partial
// rows are read eight at a time, all eight loads issued before any is used:
// row indices are clamped into the rows the slot has and the terms outside
// them are selected to zero, so the sum keeps its order bit for bit.
__global__ void __launch_bounds__(256) score_reduce_kernel(PrefillArgs a, int pt_positions) {
  const int u = blockIdx.x;
  const int n = a.len0 + a.n_tok;
  const int j = blockIdx.y * 256 + threadIdx.x;
  if (j < n) {
    const float* part = a.partial + (int64_t)u * a.npt_stride * a.cap + j;
    float* score = a.score + (int64_t)u * a.cap;
    const int pt0 = j < a.len0 ? 0 : (j - a.len0) / pt_positions;
    const int last = a.npt_used - 1;
    float acc = j < a.len0 ? score[j] : 0.0f;
    if (a.accumulate) {
      for (int c0 = pt0 & ~7; c0 <= last; c0 += 8) {
        float x[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) x[c] = part[(int64_t)min(max(c0 + c, pt0), last) * a.cap];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int pt = c0 + c;
          acc += pt >= pt0 && pt <= last ? x[c] : 0.0f;
        }
      }
    }
    score[j] = acc;
  }
  if (blockIdx.y == 0 && threadIdx.x == 0) a.len[u] = n;
}

template <bool BF16, int D, int G>
hipError_t launch_t(const PrefillArgs& a, hipStream_t stream) {
  dim3 grid((unsigned)(a.units * a.npt_used));
  if (a.pad)
    hipLaunchKernelGGL((prefill_attn_kernel<BF16, D, G, true>), grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((prefill_attn_kernel<BF16, D, G, false>), grid, dim3(kThreads), 0, stream, a);
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

bool timeline_enabled() { return kTimeline; }

hipError_t read_timeline(uint64_t* dst, int n_records) {
#ifdef BM_PREFILL_TIMELINE
  return hipMemcpyFromSymbol(dst, HIP_SYMBOL(g_timeline),
                             (size_t)n_records * BM_TIMELINE_FIELDS * sizeof(uint64_t), 0,
                             hipMemcpyDeviceToHost);
#else
  (void)dst;
  (void)n_records;
  return hipErrorNotSupported;
#endif
}

hipError_t launch_score_reduce(const PrefillArgs& a, hipStream_t stream) {
  const int group = a.n_heads / a.n_kv_heads;
  const unsigned chunks = (unsigned)((a.len0 + a.n_tok + 255) / 256);
  hipLaunchKernelGGL(score_reduce_kernel, dim3((unsigned)a.units, chunks), dim3(256), 0, stream,
                     a, positions_per_wg(group));
  return hipGetLastError();
}

}  // namespace bm
