// Few-step sampler update between the denoising passes of a chunk: from the
// stack's velocity prediction v at x_tau, x0_hat = x_tau - tau v, re-noised
// for the next timestep as (1 - tau') x0_hat + tau' eps (AR-DiT generation,
// Section 2.1; S steps per chunk, Appendix A).  Streaming HBM work: three bf16
// reads and one bf16 write per element, fp32 arithmetic in between.
#include "launch.h"

namespace ardit {

namespace {

constexpr int kSamplerRowsPerGroup = 4;   // one wave per row

__global__ __launch_bounds__(256) void sampler_kernel(const bf16_t* __restrict__ x,
                                                      const bf16_t* __restrict__ v,
                                                      const bf16_t* __restrict__ eps,
                                                      bf16_t* out, SamplerArgs a) {
  const int row = blockIdx.x * kSamplerRowsPerGroup + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const int lane = threadIdx.x & 63;
  const int b = row / a.rows_per_stream;
  const float tau = a.tau[b];
  const float tn = a.tau_next[b];   // < 0: no further step, keep x0_hat
  const size_t base = static_cast<size_t>(row) * a.vec_per_row;
  const uint4* xr = reinterpret_cast<const uint4*>(x) + base;
  const uint4* vr = reinterpret_cast<const uint4*>(v) + base;
  uint4* orow = reinterpret_cast<uint4*>(out) + base;
  for (int j = lane; j < a.vec_per_row; j += kWave) {
    float xf[8], vf[8], r[8];
    unpack8(xr[j], xf);
    unpack8(vr[j], vf);
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = fmaf(-tau, vf[i], xf[i]);
    if (tn >= 0.f) {
      float ef[8];
      unpack8(reinterpret_cast<const uint4*>(eps)[base + j], ef);
      const float keep = 1.0f - tn;
#pragma unroll
      for (int i = 0; i < 8; ++i) r[i] = fmaf(keep, r[i], tn * ef[i]);
    }
    orow[j] = pack8(r);
  }
}

}  // namespace

hipError_t launch_sampler(hipStream_t st, const bf16_t* x, const bf16_t* v, const bf16_t* eps,
                          bf16_t* out, const SamplerArgs& a) {
  if (a.rows <= 0) return hipSuccess;
  const int groups = (a.rows + kSamplerRowsPerGroup - 1) / kSamplerRowsPerGroup;
  hipLaunchKernelGGL(sampler_kernel, dim3(groups), dim3(256), 0, st, x, v, eps, out, a);
  return hipGetLastError();
}

}  // namespace ardit
