// K5: counter-based synthetic Q/K/V for the layer-stack workload.
//
// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011): ten rounds, each
// mapping (c0, c1, c2, c3) with the 64-bit products M0 * c0 = (hi0, lo0) and
// M1 * c2 = (hi1, lo1) to (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0), the key
// growing by the Weyl constants (W0, W1) between rounds.  One call yields two
// elements (Irwin-Hall sums of four 16-bit uniforms, see bm_synth.h); a thread
// owns one element pair, so every store is 4 or 8 contiguous bytes.
#include "bm_internal.h"

namespace bm {
namespace {

constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
constexpr int64_t kMaxGrid = 1 << 20;   // workgroups per launch (2^28 work-items)

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(kM0, c.x), lo0 = kM0 * c.x;
    const uint32_t hi1 = __umulhi(kM1, c.z), lo1 = kM1 * c.z;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += kW0;
    k1 += kW1;
  }
  return c;
}

__device__ __forceinline__ uint32_t ih4(uint32_t a, uint32_t b) {
  return (a & 0xFFFFu) + (a >> 16) + (b & 0xFFFFu) + (b >> 16);
}

// A virtual block covers 256 element pairs of one (sample, Q/K/V head) row
// range; workgroups stride over the virtual blocks, so a launch never needs
// more than kMaxGrid workgroups.  All index arithmetic is 32-bit (pairs per
// row is a power of two).
template <bool BF16>
__device__ __forceinline__ void synth_block(const SynthArgs& a, int chunks, int pshift, int blk) {
  const int P = 1 << pshift;                          // element pairs per row (d / 2)
  const int HT = a.n_heads + 2 * a.n_kv_heads;        // rows of Q, K, V heads
  const int chunk = blk % chunks;
  const int sh = blk / chunks;                        // sample * HT + ht
  const int ht = sh % HT, sample = sh / HT;
  const int local = chunk * 256 + threadIdx.x;
  const int r = local >> pshift, pair = local & (P - 1);
  if (r >= a.n_rows) return;   // past the last row of the range: no pair for this thread
  int tensor, head, nh;
  void* base;
  if (ht < a.n_heads) {
    tensor = 0; head = ht; nh = a.n_heads; base = a.q;
  } else if (ht < a.n_heads + a.n_kv_heads) {
    tensor = 1; head = ht - a.n_heads; nh = a.n_kv_heads; base = a.k;
  } else {
    tensor = 2; head = ht - a.n_heads - a.n_kv_heads; nh = a.n_kv_heads; base = a.v;
  }
  const uint32_t pos = (uint32_t)(a.t0 + r);
  const uint4 w = philox4x32_10(
      make_uint4(pos * (uint32_t)P + (uint32_t)pair, ((uint32_t)tensor << 8) | (uint32_t)head,
                 (uint32_t)sample, (uint32_t)a.layer),
      a.seed, 0u);
  float z0 = ((float)ih4(w.x, w.y) - 131070.0f) * a.value_scale;
  float z1 = ((float)ih4(w.z, w.w) - 131070.0f) * a.value_scale;
  if (tensor == 1 && (int)pos < a.s) {
    float f = 1.0f;
    if ((int)pos < a.n_sinks) {
      f = a.sink_scale;
    } else {
      const uint4 sel = philox4x32_10(make_uint4(pos, 3u << 8, (uint32_t)sample, (uint32_t)a.layer),
                                      a.seed, 0u);
      if (sel.x < a.hh_threshold) f = a.hh_scale;
    }
    z0 *= f;
    z1 *= f;
  }
  const int64_t off = (((int64_t)sample * nh + head) * a.seq_ld + r) * (2 * P) + 2 * pair;
  if constexpr (BF16) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
    *reinterpret_cast<bf16x2*>(static_cast<__bf16*>(base) + off) = bf16x2{(__bf16)z0, (__bf16)z1};
  } else {
    *reinterpret_cast<float2*>(static_cast<float*>(base) + off) = make_float2(z0, z1);
  }
}

template <bool BF16>
__global__ void __launch_bounds__(256) synth_qkv_kernel(SynthArgs a, int chunks, int pshift,
                                                        int blocks) {
  for (int blk = blockIdx.x; blk < blocks; blk += gridDim.x)
    synth_block<BF16>(a, chunks, pshift, blk);
}

__global__ void __launch_bounds__(256) philox_kernel(const uint32_t* in, uint32_t* out, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint32_t* x = in + 6 * i;
    const uint4 w = philox4x32_10(make_uint4(x[0], x[1], x[2], x[3]), x[4], x[5]);
    out[4 * i + 0] = w.x;
    out[4 * i + 1] = w.y;
    out[4 * i + 2] = w.z;
    out[4 * i + 3] = w.w;
  }
}

unsigned grid_for(int64_t items) {
  int64_t blocks = (items + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  return (unsigned)blocks;
}

}  // namespace

hipError_t launch_synth_qkv(const SynthArgs& a, hipStream_t stream) {
  int pshift = 0;
  while ((1 << pshift) < a.head_dim / 2) ++pshift;
  if ((1 << pshift) != a.head_dim / 2) return hipErrorInvalidValue;   // d / 2 a power of two
  const int64_t chunks = ((int64_t)a.n_rows * (a.head_dim / 2) + 255) / 256;
  const int64_t blocks = (int64_t)a.b * (a.n_heads + 2 * a.n_kv_heads) * chunks;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)(blocks < kMaxGrid ? blocks : kMaxGrid);
  if (a.dtype == BM_BF16)
    hipLaunchKernelGGL(synth_qkv_kernel<true>, dim3(grid), dim3(256), 0, stream, a, (int)chunks,
                       pshift, (int)blocks);
  else
    hipLaunchKernelGGL(synth_qkv_kernel<false>, dim3(grid), dim3(256), 0, stream, a, (int)chunks,
                       pshift, (int)blocks);
  return hipGetLastError();
}

hipError_t launch_philox(const uint32_t* in, uint32_t* out, int64_t n, hipStream_t stream) {
  hipLaunchKernelGGL(philox_kernel, dim3(grid_for(n)), dim3(256), 0, stream, in, out, n);
  return hipGetLastError();
}

}  // namespace bm
