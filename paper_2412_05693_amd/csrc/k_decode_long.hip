// K6: one decode step over a long cache, outputs only (the full-cache
// comparator of Sec. 4, where nothing is ever removed and no scores are kept).
//
// K4 holds a step's probabilities for every cached entry in LDS, which bounds
// it to kMaxDecodeLen entries.  Past that the attention is split over chunks of
// kChunk keys (flash-decoding): decode_split_kernel, grid (units, chunks), gives
// each chunk's partial softmax -- its log2-domain maximum m, its sum l of
// exp2(z - m) and the unnormalised output o = sum exp2(z - m) v -- for all G
// query heads of the unit; decode_combine_kernel, one workgroup per unit, merges
// the chunks, o = sum_c 2^(m_c - M) o_c / sum_c 2^(m_c - M) l_c with M the
// largest m_c, writes the outputs and appends the step's pair to the cache
// (score 0, pos = the step's position).
//
// HBM-bound: K and V rows are read once, 16 bytes per lane; a wave load covers
// 64 / CPR whole rows (CPR 16-byte chunks per row), each row's dot products are
// finished with shuffles inside its CPR lanes; every lane issues four row
// loads together (whole 1 KB runs per wave instruction, few registers, so
// many workgroups per compute unit keep the loads in flight).
#include <type_traits>

#include "bm_internal.h"
#include "bm_lanes.h"

namespace bm {
namespace {

constexpr int kChunk = 512;   // keys per split workgroup
constexpr float kNegInf = -__builtin_huge_valf();

// one 16-byte chunk of a row as floats (8 bf16 or 4 float32 elements)
template <bool BF16>
__device__ __forceinline__ void unpack_chunk(const uint4 w, float* x) {
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
  if constexpr (BF16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(u[i] << 16);
      x[2 * i + 1] = __uint_as_float(u[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(u[i]);
  }
}

template <bool BF16, int D, int G>
__global__ void __launch_bounds__(256) decode_split_kernel(LongDecodeArgs a) {
  using E = typename std::conditional<BF16, uint16_t, float>::type;
  constexpr int EPC = 16 / sizeof(E);     // elements per 16-byte chunk
  constexpr int CPR = D / EPC;            // chunks per row
  constexpr int RPL = 64 / CPR;           // rows per wave load
  __shared__ float qs[G][D];              // q * scale * log2(e)
  __shared__ float z[G][kChunk];          // logits, then exp2(z - m)
  __shared__ float red[4][G][D];          // per-wave partial outputs
  __shared__ float s_m[G], s_l[G];

  const int u = blockIdx.x, c = blockIdx.y;
  const int bi = u / a.n_kv_heads, hk = u - bi * a.n_kv_heads;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int L = a.len0 + 1;
  const int j0 = c * kChunk;
  const int nj = min(kChunk, L - j0);
  const E* kc = static_cast<const E*>(a.kc) + (int64_t)u * a.cap * D;
  const E* vc = static_cast<const E*>(a.vc) + (int64_t)u * a.cap * D;
  const int64_t plane = ((int64_t)bi * a.n_kv_heads + hk) * a.seq_ld;
  const E* knew = static_cast<const E*>(a.kin) + plane * D;
  const E* vnew = static_cast<const E*>(a.vin) + plane * D;
  const E* qb = static_cast<const E*>(a.q) + ((int64_t)bi * a.n_heads + hk * G) * a.seq_ld * D;

  for (int i = tid; i < G * D; i += 256) {
    const int g = i / D, e = i - g * D;
    const E x = qb[(int64_t)g * a.seq_ld * D + e];
    float f;
    if constexpr (BF16) f = __uint_as_float((uint32_t)x << 16);
    else f = x;
    qs[g][e] = f * a.scale_log2;
  }
  __syncthreads();

  const int r_in = lane / CPR, ch = lane - r_in * CPR;
  // Every row load is unconditional: rows past the chunk's last entry read the
  // step's own row (valid memory; their results are never stored), so the
  // compiler can count the loads in flight and wait only for the rows in use.
  // A lane issues UL row loads together.
  constexpr int UL = 4;
  auto k_src = [&](int r) -> const E* { return j0 + r < a.len0 ? kc + (int64_t)(j0 + r) * D : knew; };
  auto v_src = [&](int r) -> const E* { return j0 + r < a.len0 ? vc + (int64_t)(j0 + r) * D : vnew; };
  // 1. logits: wave w takes row groups w, w + 4, ... of the chunk
  for (int base = w * RPL; base < nj; base += 4 * RPL * UL) {
    uint4 raw[UL];
#pragma unroll
    for (int i = 0; i < UL; ++i)
      raw[i] = *reinterpret_cast<const uint4*>(k_src(base + 4 * RPL * i + r_in) + ch * EPC);
#pragma unroll
    for (int i = 0; i < UL; ++i) {
      const int r = base + 4 * RPL * i + r_in;
      float x[EPC];
      unpack_chunk<BF16>(raw[i], x);
      float part[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        part[g] = 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) part[g] = fmaf(qs[g][ch * EPC + e], x[e], part[g]);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) part[g] = lanes::group_sum<CPR>(part[g]);
      if (ch == 0 && r < nj) {
#pragma unroll
        for (int g = 0; g < G; ++g) z[g][r] = part[g];
      }
    }
  }
  __syncthreads();
  // left padding: a pad entry (pos < pad) is visible to no query
  const int pad = a.pad ? max(0, a.pad[bi]) : 0;
  if (pad > 0) {
    for (int r = tid; r < nj; r += 256) {
      const int j = j0 + r;
      if (j < a.len0 && a.pos[(int64_t)u * a.cap + j] < pad) {
#pragma unroll
        for (int g = 0; g < G; ++g) z[g][r] = kNegInf;
      }
    }
    __syncthreads();
  }

  // 2. chunk maximum and exp2 sums, wave g < G handles head g
  if (w < G) {
    float m = kNegInf;
    for (int r = lane; r < nj; r += 64) m = fmaxf(m, z[w][r]);
    m = lanes::wave_max(m);
    float l = 0.0f;
    for (int r = lane; r < nj; r += 64) {
      // a chunk of pad entries only: no weight (m = -inf)
      const float p = m == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(z[w][r] - m);
      z[w][r] = p;
      l += p;
    }
    l = lanes::wave_sum(l);
    if (lane == 0) {
      s_m[w] = m;
      s_l[w] = l;
    }
  }
  __syncthreads();

  // 3. unnormalised outputs: lane (r_in, ch) accumulates elements ch*EPC.. of
  //    every head over its rows
  float acc[G][EPC];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[g][e] = 0.0f;
  for (int base = w * RPL; base < nj; base += 4 * RPL * UL) {
    uint4 raw[UL];
#pragma unroll
    for (int i = 0; i < UL; ++i)
      raw[i] = *reinterpret_cast<const uint4*>(v_src(base + 4 * RPL * i + r_in) + ch * EPC);
#pragma unroll
    for (int i = 0; i < UL; ++i) {
      // rows past the chunk's end weigh 0 (their V row is the step's own,
      // finite): no early exit, so the loads are not moved to their uses
      const int r = base + 4 * RPL * i + r_in;
      float x[EPC];
      unpack_chunk<BF16>(raw[i], x);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = r < nj ? z[g][min(r, nj - 1)] : 0.0f;
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[g][e] = fmaf(p, x[e], acc[g][e]);
      }
    }
  }
  // sum over the RPL rows of a wave load (lanes ch, ch + CPR, ...)
  static_assert(CPR == 8 || CPR == 16 || CPR == 32, "16-byte chunks per row");
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      float x = acc[g][e];
      if constexpr (CPR <= 8) x = lanes::add_xor<8>(x);
      if constexpr (CPR <= 16) x = lanes::add_xor<16>(x);
      acc[g][e] = lanes::add_xor<32>(x);
    }
  if (r_in == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPC; ++e) red[w][g][ch * EPC + e] = acc[g][e];
  }
  __syncthreads();

  // partial record of this chunk: [G][D + 2] floats (o, then m, l)
  float* out = a.part + ((int64_t)u * a.nsplit + c) * G * (D + 2);
  for (int i = tid; i < G * D; i += 256) {
    const int g = i / D, e = i - g * D;
    out[g * (D + 2) + e] = red[0][g][e] + red[1][g][e] + red[2][g][e] + red[3][g][e];
  }
  if (tid < G) {
    out[tid * (D + 2) + D] = s_m[tid];
    out[tid * (D + 2) + D + 1] = s_l[tid];
  }
}

template <bool BF16, int D, int G>
__global__ void __launch_bounds__(256) decode_combine_kernel(LongDecodeArgs a) {
  using E = typename std::conditional<BF16, uint16_t, float>::type;
  const int u = blockIdx.x;
  const int bi = u / a.n_kv_heads, hk = u - bi * a.n_kv_heads;
  const int tid = threadIdx.x;
  const float* part = a.part + (int64_t)u * a.nsplit * G * (D + 2);
  for (int i = tid; i < G * D; i += 256) {
    const int g = i / D, e = i - g * D;
    float M = kNegInf;
    for (int c = 0; c < a.nsplit; ++c) M = fmaxf(M, part[(c * G + g) * (D + 2) + D]);
    float num = 0.0f, den = 0.0f;
    for (int c = 0; c < a.nsplit; ++c) {
      const float* pc = part + (c * G + g) * (D + 2);
      const float f = pc[D] == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(pc[D] - M);
      num = fmaf(f, pc[e], num);
      den = fmaf(f, pc[D + 1], den);
    }
    const float x = num / den;
    E* o = static_cast<E*>(a.o) + (((int64_t)bi * a.n_heads + hk * G + g) * a.seq_ld) * D + e;
    if constexpr (BF16) {
      *reinterpret_cast<__bf16*>(o) = (__bf16)x;
    } else {
      *o = x;
    }
  }
  // append the step's pair at slot len0
  const int64_t plane = ((int64_t)bi * a.n_kv_heads + hk) * a.seq_ld;
  const E* knew = static_cast<const E*>(a.kin) + plane * D;
  const E* vnew = static_cast<const E*>(a.vin) + plane * D;
  E* kdst = static_cast<E*>(a.kc) + ((int64_t)u * a.cap + a.len0) * D;
  E* vdst = static_cast<E*>(a.vc) + ((int64_t)u * a.cap + a.len0) * D;
  for (int e = tid; e < D; e += 256) {
    kdst[e] = knew[e];
    vdst[e] = vnew[e];
  }
  if (tid == 0) {
    a.score[(int64_t)u * a.cap + a.len0] = 0.0f;
    a.pos[(int64_t)u * a.cap + a.len0] = a.cur_pos;
    a.len[u] = a.len0 + 1;
  }
}

template <bool BF16, int D, int G>
hipError_t launch_t(const LongDecodeArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((decode_split_kernel<BF16, D, G>), dim3((unsigned)a.units, (unsigned)a.nsplit),
                     dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_combine_kernel<BF16, D, G>), dim3((unsigned)a.units), dim3(256), 0,
                     stream, a);
  return hipGetLastError();
}

template <bool BF16, int D>
hipError_t launch_g(const LongDecodeArgs& a, int group, hipStream_t stream) {
  switch (group) {
    case 1: return launch_t<BF16, D, 1>(a, stream);
    case 2: return launch_t<BF16, D, 2>(a, stream);
    case 4: return launch_t<BF16, D, 4>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int long_decode_splits(int len0) { return (len0 + 1 + kChunk - 1) / kChunk; }

hipError_t launch_decode_long(const LongDecodeArgs& a, int dtype, int head_dim, int group,
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
