// bf16 GEMM with fp32 accumulation on gfx950 MFMA, C = epilogue(A W^T).
//
// A [M][K] and W [N][K] are both K-contiguous (every projection of the block
// stores its weight [out][in]).  A 256-thread workgroup computes a 128x128
// tile; each of its four waves owns a 64x64 quarter as 2x2 blocks of
// v_mfma_f32_32x32x16_bf16.  K advances in steps of 64 through two LDS
// buffers: the global loads of step k+1 are issued before the MFMAs of step k
// and stored to the other buffer afterwards, one barrier per step.  LDS rows
// are padded to 72 elements (144 bytes) so the 16-byte fragment reads of
// consecutive rows fall on distinct banks.
//
// The MFMA computes C^T = W A^T: W rows feed the A operand and A rows the B
// operand, so each lane ends up owning one output row m and four groups of
// four consecutive columns n, which the epilogue writes as 8-byte stores
// after applying bias / GELU / gate * y + residual in fp32.
#include "launch.h"

namespace ardit {

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_LD = BK + 8;     // padded row, elements
constexpr int GROUP_M = 8;         // m-tiles per raster group (L2 reuse of W columns)

__device__ __forceinline__ bf16x8 lds_frag(const bf16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

template <typename T>
__device__ __forceinline__ void load4(const T* p, float* f);
template <>
__device__ __forceinline__ void load4<bf16_t>(const bf16_t* p, float* f) {
  const uint2 r = *reinterpret_cast<const uint2*>(p);
  f[0] = __uint_as_float(r.x << 16);
  f[1] = __uint_as_float(r.x & 0xffff0000u);
  f[2] = __uint_as_float(r.y << 16);
  f[3] = __uint_as_float(r.y & 0xffff0000u);
}
template <>
__device__ __forceinline__ void load4<float>(const float* p, float* f) {
  const float4 r = *reinterpret_cast<const float4*>(p);
  f[0] = r.x;
  f[1] = r.y;
  f[2] = r.z;
  f[3] = r.w;
}

__device__ __forceinline__ void store4(bf16_t* p, const float* y) {
  uint2 out;
  out.x = pack_bf16x2(y[0], y[1]);
  out.y = pack_bf16x2(y[2], y[3]);
  *reinterpret_cast<uint2*>(p) = out;
}
__device__ __forceinline__ void store4(float* p, const float* y) {
  *reinterpret_cast<float4*>(p) = make_float4(y[0], y[1], y[2], y[3]);
}

// ResT / OutT: element type of the residual input and of C (bf16 or fp32)
template <int EPI, typename ResT, typename OutT>
__global__ __launch_bounds__(256, 2) void gemm_kernel(const bf16_t* __restrict__ A, int lda,
                                                      const bf16_t* __restrict__ W, int ldw,
                                                      OutT* __restrict__ C, int ldc, int M,
                                                      int N, int K, const GemmEpiArgs ep,
                                                      int tiles_m, int tiles_n, int per_xcd) {
  __shared__ __attribute__((aligned(16))) bf16_t sA[2][BM * LDS_LD];
  __shared__ __attribute__((aligned(16))) bf16_t sW[2][BN * LDS_LD];

  // XCD-aware tile order: consecutive logical tiles land on one XCD (shared L2)
  const int p = blockIdx.x;
  const int L = (p % kNumXcd) * per_xcd + p / kNumXcd;
  if (L >= tiles_m * tiles_n) return;
  const int group = GROUP_M * tiles_n;
  const int g0 = (L / group) * GROUP_M;
  const int gm = min(tiles_m - g0, GROUP_M);
  const int tm = g0 + (L % group) % gm;
  const int tn = (L % group) / gm;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const int wm = wave >> 1, wn = wave & 1;

  // global -> register staging: 4 chunks of A and 4 of W per thread per step
  const bf16_t* a_src[4];
  const bf16_t* w_src[4];
  int st_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int r = c >> 3, kc = c & 7;
    const int am = min(tm * BM + r, M - 1);
    a_src[i] = A + static_cast<size_t>(am) * lda + kc * 8;
    w_src[i] = W + static_cast<size_t>(tn * BN + r) * ldw + kc * 8;
    st_off[i] = r * LDS_LD + kc * 8;
  }
  u32x4 ra[4], rw[4];

  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

  const int nk = K / BK;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = *reinterpret_cast<const u32x4*>(a_src[i]);
    rw[i] = *reinterpret_cast<const u32x4*>(w_src[i]);
    *reinterpret_cast<u32x4*>(&sA[0][st_off[i]]) = ra[i];
    *reinterpret_cast<u32x4*>(&sW[0][st_off[i]]) = rw[i];
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
      const int k0 = (kt + 1) * BK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = *reinterpret_cast<const u32x4*>(a_src[i] + k0);
        rw[i] = *reinterpret_cast<const u32x4*>(w_src[i] + k0);
      }
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 fw[2], fa[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        fw[nb] = lds_frag(&sW[buf][(64 * wn + 32 * nb + l32) * LDS_LD + 16 * ks + 8 * g]);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
        fa[mb] = lds_frag(&sA[buf][(64 * wm + 32 * mb + l32) * LDS_LD + 16 * ks + 8 * g]);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mb][nb] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[nb], fa[mb], acc[mb][nb], 0, 0, 0);
    }
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<u32x4*>(&sA[buf ^ 1][st_off[i]]) = ra[i];
        *reinterpret_cast<u32x4*>(&sW[buf ^ 1][st_off[i]]) = rw[i];
      }
    }
    __syncthreads();
  }

  // epilogue: lane owns row m, columns n0..n0+3 of each (mb, nb, jj)
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int m = tm * BM + 64 * wm + 32 * mb + l32;
    if (m >= M) continue;
    const int sidx = (EPI == kEpiBiasGateRes) ? m / ep.rows_per_stream : 0;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int n0 = tn * BN + 64 * wn + 32 * nb + 8 * jj + 4 * g;
        float y[4];
        const uint2 bb = *reinterpret_cast<const uint2*>(ep.bias + n0);
        const float bias[4] = {__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xffff0000u),
                               __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xffff0000u)};
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = acc[mb][nb][4 * jj + e] + bias[e];
        if (EPI == kEpiBiasGelu) {
#pragma unroll
          for (int e = 0; e < 4; ++e) y[e] = gelu_tanh(y[e]);
        }
        if (EPI == kEpiBiasGateRes || EPI == kEpiBiasRes) {
          float res[4];
          load4(static_cast<const ResT*>(ep.res) + static_cast<size_t>(m) * ep.ldr + n0, res);
          if (EPI == kEpiBiasGateRes) {
            const float4 gm4 = *reinterpret_cast<const float4*>(
                ep.mod + (static_cast<size_t>(sidx) * 6 + ep.gate_row) * ep.dim + n0);
            const float4 gt4 = *reinterpret_cast<const float4*>(
                ep.mod_table + static_cast<size_t>(ep.gate_row) * ep.dim + n0);
            const float gate[4] = {gm4.x + gt4.x, gm4.y + gt4.y, gm4.z + gt4.z, gm4.w + gt4.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) y[e] = res[e] + gate[e] * y[e];
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) y[e] = res[e] + y[e];
          }
        }
        store4(C + static_cast<size_t>(m) * ldc + n0, y);
      }
    }
  }
}

}  // namespace

template <int EPI, typename ResT, typename OutT>
static void launch_t(hipStream_t st, const bf16_t* A, int lda, const bf16_t* W, int ldw, void* C,
                     int ldc, int M, int N, int K, const GemmEpiArgs& ep, int tiles_m,
                     int tiles_n, int per_xcd) {
  hipLaunchKernelGGL((gemm_kernel<EPI, ResT, OutT>), dim3(per_xcd * kNumXcd), dim3(256), 0, st,
                     A, lda, W, ldw, static_cast<OutT*>(C), ldc, M, N, K, ep, tiles_m, tiles_n,
                     per_xcd);
}

hipError_t launch_gemm(hipStream_t st, int epi, const bf16_t* A, int lda, const bf16_t* W,
                       int ldw, void* C, int ldc, int M, int N, int K, const GemmEpiArgs& ep) {
  if (M == 0) return hipSuccess;
  const int tiles_m = (M + BM - 1) / BM, tiles_n = N / BN;
  const int total = tiles_m * tiles_n;
  const int per_xcd = (total + kNumXcd - 1) / kNumXcd;
  const bool rf = ep.res_f32, of = ep.out_f32;
#define ARDIT_GEMM(E, R, O) launch_t<E, R, O>(st, A, lda, W, ldw, C, ldc, M, N, K, ep, tiles_m, tiles_n, per_xcd)
  switch (epi) {
    case kEpiBias:
      if (of) ARDIT_GEMM(kEpiBias, bf16_t, float); else ARDIT_GEMM(kEpiBias, bf16_t, bf16_t);
      break;
    case kEpiBiasGelu:
      ARDIT_GEMM(kEpiBiasGelu, bf16_t, bf16_t);
      break;
    case kEpiBiasGateRes:
      if (rf && of) ARDIT_GEMM(kEpiBiasGateRes, float, float);
      else if (rf) ARDIT_GEMM(kEpiBiasGateRes, float, bf16_t);
      else if (of) ARDIT_GEMM(kEpiBiasGateRes, bf16_t, float);
      else ARDIT_GEMM(kEpiBiasGateRes, bf16_t, bf16_t);
      break;
    case kEpiBiasRes:
      if (rf && of) ARDIT_GEMM(kEpiBiasRes, float, float);
      else if (rf) ARDIT_GEMM(kEpiBiasRes, float, bf16_t);
      else if (of) ARDIT_GEMM(kEpiBiasRes, bf16_t, float);
      else ARDIT_GEMM(kEpiBiasRes, bf16_t, bf16_t);
      break;
    default:
      return hipErrorInvalidValue;
  }
#undef ARDIT_GEMM
  return hipGetLastError();
}

}  // namespace ardit
