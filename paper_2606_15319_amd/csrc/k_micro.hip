// Measurement kernels: what the matrix cores and HBM deliver on this GPU,
// measured the same way as the block's kernels, so every roofline fraction
// can be given against a measured peak as well as the published one.
//  - mfma_peak_kernel: each wave runs CHAINS independent accumulator chains
//    of one MFMA on register operands (no memory traffic in the loop), two
//    waves per SIMD as in the attention and GEMM kernels;
//  - copy_kernel: 16-byte streaming loads and stores, four in flight per
//    thread, reading and writing `bytes` each (a plain device copy);
//  - read_kernel: 16-byte loads, four in flight per thread, folded into one
//    word per workgroup (a read of `bytes`: the read bandwidth, and the cache
//    flush before a cold timing -- a buffer larger than L2 and the last-level
//    cache read through, which leaves them holding clean lines of it only);
//  - fill_kernel: 16-byte stores of one value.
#include "launch.h"

namespace ardit {

namespace {

constexpr int kMicroThreads = 256;
constexpr int kChains = 8;

typedef int i32x8 __attribute__((ext_vector_type(8)));

template <int DTYPE>
__global__ __launch_bounds__(kMicroThreads, 2) void mfma_peak_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  float sum = 0.f;
  if (DTYPE == 0) {
    bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = static_cast<__bf16>(static_cast<float>((lane + i) & 7) * 0.125f);
      b[i] = static_cast<__bf16>(static_cast<float>((lane * 3 + i) & 7) * 0.0625f);
    }
    f32x4 acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[c][v] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int c = 0; c < kChains; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[c], 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) sum += acc[c][v];
  } else {
    i32x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = 0x38383838 + ((lane + i) & 3);   // E4M3 codes near 0.5..1
      b[i] = 0x30303030 + ((lane * 3 + i) & 3);
    }
    f32x16 acc[kChains / 2];
#pragma unroll
    for (int c = 0; c < kChains / 2; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int c = 0; c < kChains / 2; ++c)
        acc[c] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc[c], 0, 0, 0, 127, 0,
                                                                 127);
    }
#pragma unroll
    for (int c = 0; c < kChains / 2; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) sum += acc[c][v];
  }
  sink[static_cast<size_t>(blockIdx.x) * kMicroThreads + threadIdx.x] = sum;
}

// Streaming (nontemporal) loads and stores: the fastest plain copy measured on
// MI355X at 1 GiB (5.4 TB/s read + write against 4.5 with cached accesses,
// over grids of 1024-16384 workgroups and 4 or 8 accesses in flight per
// thread), so the measured copy rate is the best a streaming kernel reaches.
__global__ __launch_bounds__(kMicroThreads) void copy_kernel(const u32x4* __restrict__ src,
                                                           u32x4* __restrict__ dst, size_t n16) {
  const size_t stride = static_cast<size_t>(gridDim.x) * kMicroThreads;
  size_t i = static_cast<size_t>(blockIdx.x) * kMicroThreads + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
  }
  for (; i < n16; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

__global__ __launch_bounds__(kMicroThreads) void fill_kernel(uint4* __restrict__ dst, size_t n16,
                                                           uint32_t value) {
  const size_t stride = static_cast<size_t>(gridDim.x) * kMicroThreads;
  const uint4 v = make_uint4(value, value, value, value);
  for (size_t i = static_cast<size_t>(blockIdx.x) * kMicroThreads + threadIdx.x; i < n16;
       i += stride)
    dst[i] = v;
}

__global__ __launch_bounds__(kMicroThreads) void read_kernel(const uint4* __restrict__ src,
                                                           size_t n16, uint32_t* sink) {
  const size_t stride = static_cast<size_t>(gridDim.x) * kMicroThreads;
  size_t i = static_cast<size_t>(blockIdx.x) * kMicroThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= a.x ^ a.w ^ b.y ^ b.z ^ c.x ^ c.w ^ d.y ^ d.z;
  }
  for (; i < n16; i += stride) acc ^= src[i].x;
  // one word per workgroup, written by the lane that ends the reduction
  __shared__ uint32_t red[kMicroThreads / 64];
  for (int m = 32; m >= 1; m >>= 1) acc ^= __shfl_xor(acc, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

int stream_grid(size_t n16) {
  // 32 workgroups per CU at most, fewer for small copies
  const size_t want = (n16 + kMicroThreads - 1) / kMicroThreads;
  const size_t cap = static_cast<size_t>(256) * 32;
  return static_cast<int>(want < cap ? (want > 0 ? want : 1) : cap);
}

}  // namespace

double micro_mfma_flops_per_wave_iter(int dtype) {
  // 16x16x32 bf16: 2 * 16 * 16 * 32; 32x32x64 fp8: 2 * 32 * 32 * 64
  return dtype == 0 ? kChains * 16384.0 : (kChains / 2) * 131072.0;
}

hipError_t launch_micro_mfma(hipStream_t st, int dtype, int workgroups, int iters, float* sink) {
  if (dtype == 0)
    hipLaunchKernelGGL(mfma_peak_kernel<0>, dim3(workgroups), dim3(kMicroThreads), 0, st, iters,
                       sink);
  else
    hipLaunchKernelGGL(mfma_peak_kernel<1>, dim3(workgroups), dim3(kMicroThreads), 0, st, iters,
                       sink);
  return hipGetLastError();
}

hipError_t launch_micro_copy(hipStream_t st, const void* src, void* dst, size_t bytes) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  hipLaunchKernelGGL(copy_kernel, dim3(stream_grid(n16)), dim3(kMicroThreads), 0, st,
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), n16);
  return hipGetLastError();
}

int micro_read_workgroups(size_t bytes) { return stream_grid(bytes / 16); }

hipError_t launch_micro_read(hipStream_t st, const void* src, size_t bytes, uint32_t* sink) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  hipLaunchKernelGGL(read_kernel, dim3(stream_grid(n16)), dim3(kMicroThreads), 0, st,
                     static_cast<const uint4*>(src), n16, sink);
  return hipGetLastError();
}

hipError_t launch_fill(hipStream_t st, void* dst, size_t bytes, uint32_t value) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, dim3(stream_grid(n16)), dim3(kMicroThreads), 0, st,
                     static_cast<uint4*>(dst), n16, value);
  return hipGetLastError();
}

}  // namespace ardit
