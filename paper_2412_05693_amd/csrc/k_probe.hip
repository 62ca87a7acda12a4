// Roofline probes (include/bm_probe.h): a streaming read of device memory and
// an MFMA issue loop, to measure what the device sustains on the two resources
// the attention kernels are bounded by.  Measurement only.
#include "bm_internal.h"

namespace bm {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

template <bool NT>
__device__ __forceinline__ u32x4 load16(const u32x4* p) {
  if constexpr (NT) {
    return __builtin_nontemporal_load(p);
  } else {
    return *p;
  }
}

// grid-stride read, kReadRound 16-byte loads in flight per lane per round
// (eight: with fewer the read rate depends on the grid size)
constexpr int kReadRound = 8;
template <bool NT>
__global__ void __launch_bounds__(256) probe_read_kernel(const u32x4* src, size_t n16,
                                                         uint32_t* sink) {
  __shared__ uint32_t red[4];
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kReadRound - 1) * stride < n16; i += kReadRound * stride) {
    u32x4 v[kReadRound];
#pragma unroll
    for (int k = 0; k < kReadRound; ++k) v[k] = load16<NT>(src + i + k * stride);
#pragma unroll
    for (int k = 0; k < kReadRound; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  }
  for (; i < n16; i += stride) {
    const u32x4 a = load16<NT>(src + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

// four independent accumulator chains per wave; operands derived from the lane
// so nothing is constant-folded
__global__ void __launch_bounds__(256) probe_mfma_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (float)(lane + e));
    b[e] = (__bf16)(0.002f * (float)(lane - e));
  }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
  if (lane == 0) sink[blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

}  // namespace

hipError_t launch_probe_read(const void* src, size_t bytes, uint32_t* sink, int blocks, bool nt,
                             hipStream_t stream) {
  const u32x4* p = static_cast<const u32x4*>(src);
  if (nt)
    hipLaunchKernelGGL(probe_read_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, p,
                       bytes / 16, sink);
  else
    hipLaunchKernelGGL(probe_read_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, p,
                       bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_probe_mfma(int iters, float* sink, int blocks, hipStream_t stream) {
  hipLaunchKernelGGL(probe_mfma_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, iters, sink);
  return hipGetLastError();
}

}  // namespace bm
