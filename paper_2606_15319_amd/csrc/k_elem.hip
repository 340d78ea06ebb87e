// Bandwidth-bound kernels of the block: adaLN RMSNorm, RMSNorm with gain,
// QK-RMSNorm + 3D RoPE + key append, value append (transposed pages), text
// key/value layout, and the small time-modulation MLP.
//
// One 64-lane wave owns one token row: 16-byte loads/stores, fp32 math, a
// wave reduction for the mean square.  Rows of up to 8192 elements are held
// in registers so each row is read from HBM once.
#include <math.h>

#include "launch.h"

namespace ardit {

constexpr int kMaxChunksPerLane = 16;  // 16 * 8 * 64 = 8192 elements per row

// ------------------------------------------------------------------ norms
// 8 consecutive elements of a bf16 or fp32 row as fp32
__device__ __forceinline__ void load8(const bf16_t* p, float* f) {
  unpack8(*reinterpret_cast<const uint4*>(p), f);
}
__device__ __forceinline__ void load8(const float* p, float* f) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
  f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
}

// One wave per row; a lane holds chunks lane + 64 i (i < MAXC) of 8 elements.
template <typename T, int MAXC>
__global__ __launch_bounds__(256) void adaln_norm_kernel(
    const T* __restrict__ x, bf16_t* __restrict__ out, int N, int D,
    const float* __restrict__ mod, const float* __restrict__ mod_table, int shift_row,
    int scale_row, int rows_per_stream, float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  const int b = row / rows_per_stream;
  const int nchunk = D >> 3;
  const T* xr = x + static_cast<size_t>(row) * D;
  float v[MAXC][8];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      load8(xr + 8 * c, v[i]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[i][e] * v[i][e];
    }
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / static_cast<float>(D) + eps);
  const float* msh = mod + (static_cast<size_t>(b) * 6 + shift_row) * D;
  const float* msc = mod + (static_cast<size_t>(b) * 6 + scale_row) * D;
  const float* tsh = mod_table + static_cast<size_t>(shift_row) * D;
  const float* tsc = mod_table + static_cast<size_t>(scale_row) * D;
  uint4* orow = reinterpret_cast<uint4*>(out + static_cast<size_t>(row) * D);
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      float sh[8], sc[8], th[8], tc[8], y[8];
      load8(msh + 8 * c, sh);
      load8(msc + 8 * c, sc);
      load8(tsh + 8 * c, th);
      load8(tsc + 8 * c, tc);
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = v[i][e] * r * (1.0f + sc[e] + tc[e]) + (sh[e] + th[e]);
      orow[c] = pack8(y);
    }
  }
}

template <typename T, int MAXC>
__global__ __launch_bounds__(256) void rms_gain_kernel(const T* in, bf16_t* out, int N, int D,
                                                        const bf16_t* __restrict__ gain,
                                                        float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  const int nchunk = D >> 3;
  const T* xr = in + static_cast<size_t>(row) * D;
  float v[MAXC][8];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      load8(xr + 8 * c, v[i]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[i][e] * v[i][e];
    }
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / static_cast<float>(D) + eps);
  uint4* orow = reinterpret_cast<uint4*>(out + static_cast<size_t>(row) * D);
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      float g[8], y[8];
      load8(gain + 8 * c, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = v[i][e] * r * g[e];
      orow[c] = pack8(y);
    }
  }
}

// chunks per lane needed for a row of D elements, rounded up to 1, 2, 4, 8, 16
static int row_chunks(int D) {
  const int c = (D / 8 + 63) / 64;
  return c <= 1 ? 1 : c <= 2 ? 2 : c <= 4 ? 4 : c <= 8 ? 8 : 16;
}

#define ARDIT_ROW_DISPATCH(KERNEL, T, ...)                                              \
  switch (row_chunks(D)) {                                                              \
    case 1: hipLaunchKernelGGL((KERNEL<T, 1>), grid, dim3(256), 0, st, __VA_ARGS__); break;  \
    case 2: hipLaunchKernelGGL((KERNEL<T, 2>), grid, dim3(256), 0, st, __VA_ARGS__); break;  \
    case 4: hipLaunchKernelGGL((KERNEL<T, 4>), grid, dim3(256), 0, st, __VA_ARGS__); break;  \
    case 8: hipLaunchKernelGGL((KERNEL<T, 8>), grid, dim3(256), 0, st, __VA_ARGS__); break;  \
    default: hipLaunchKernelGGL((KERNEL<T, 16>), grid, dim3(256), 0, st, __VA_ARGS__); break; \
  }

hipError_t launch_adaln_norm(hipStream_t st, const void* x, bool x_f32, bf16_t* out, int N, int D,
                             const float* mod, const float* mod_table, int shift_row,
                             int scale_row, int rows_per_stream, float eps) {
  if (N == 0) return hipSuccess;
  const dim3 grid((N + 3) / 4);
  if (x_f32) {
    const float* xf = static_cast<const float*>(x);
    ARDIT_ROW_DISPATCH(adaln_norm_kernel, float, xf, out, N, D, mod, mod_table, shift_row,
                       scale_row, rows_per_stream, eps);
  } else {
    const bf16_t* xb = static_cast<const bf16_t*>(x);
    ARDIT_ROW_DISPATCH(adaln_norm_kernel, bf16_t, xb, out, N, D, mod, mod_table, shift_row,
                       scale_row, rows_per_stream, eps);
  }
  return hipGetLastError();
}

hipError_t launch_rms_gain(hipStream_t st, const void* in, bool in_f32, bf16_t* out, int N, int D,
                           const bf16_t* gain, float eps) {
  if (N == 0) return hipSuccess;
  const dim3 grid((N + 3) / 4);
  if (in_f32) {
    const float* xf = static_cast<const float*>(in);
    ARDIT_ROW_DISPATCH(rms_gain_kernel, float, xf, out, N, D, gain, eps);
  } else {
    const bf16_t* xb = static_cast<const bf16_t*>(in);
    ARDIT_ROW_DISPATCH(rms_gain_kernel, bf16_t, xb, out, N, D, gain, eps);
  }
  return hipGetLastError();
}

// ------------------------------------------- QK-norm + 3D RoPE + key append
struct QkRopeParams {
  const bf16_t* qkv;
  bf16_t* q_out;
  bf16_t* k_pages;
  const int32_t* page_table;
  const bf16_t* g_q;
  const bf16_t* g_k;
  int N, D, H, hd, T, lat_w, max_frames, n_pages;
  FastDiv fT, fW;
  float eps;
  int pairs_t, pairs_h;       // pair-index boundaries of the t and h segments
  float inv_freq[64];         // theta^(-2k/seg) of every pair of a head
  RowStreams rs;
};

__device__ __forceinline__ int find_stream(const RowStreams& rs, int row) {
  int b = 0;
  for (int i = 1; i < rs.n; ++i)
    if (row >= rs.s[i].row_begin) b = i;
  return b;
}

__device__ __forceinline__ int clamp_page(int p, int n_pages) {
  return p < 0 ? 0 : (p >= n_pages ? n_pages - 1 : p);
}

__global__ __launch_bounds__(256) void qk_norm_rope_kernel(const QkRopeParams p) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= p.N) return;
  const int b = find_stream(p.rs, row);
  const RowStream s = p.rs.s[b];
  const int t = row - s.row_begin;
  const int f = static_cast<int>(fdiv(static_cast<uint32_t>(t), p.fT));
  const int rem = t - f * p.T;
  const int i = static_cast<int>(fdiv(static_cast<uint32_t>(rem), p.fW));
  const int j = rem - i * p.lat_w;

  // this lane's rotation: pair `lane` of a head (lanes >= hd/2 unused)
  float cs = 1.f, sn = 0.f;
  if (lane < (p.hd >> 1)) {
    const int pos = lane < p.pairs_t ? s.frame_pos0 + f : (lane < p.pairs_t + p.pairs_h ? i : j);
    sincosf(static_cast<float>(pos) * p.inv_freq[lane], &sn, &cs);
  }

  const int nchunk = p.D >> 3;
  const uint4* qr = reinterpret_cast<const uint4*>(p.qkv + static_cast<size_t>(row) * 3 * p.D);
  const uint4* kr = qr + nchunk;
  uint4 qraw[kMaxChunksPerLane], kraw[kMaxChunksPerLane];
  float sq = 0.f, sk = 0.f;
#pragma unroll
  for (int c8 = 0; c8 < kMaxChunksPerLane; ++c8) {
    const int c = lane + 64 * c8;
    if (c < nchunk) {
      qraw[c8] = qr[c];
      kraw[c8] = kr[c];
      float a[8], bb[8];
      unpack8(qraw[c8], a);
      unpack8(kraw[c8], bb);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sq += a[e] * a[e];
        sk += bb[e] * bb[e];
      }
    }
  }
  sq = wave_sum(sq);
  sk = wave_sum(sk);
  const float rq = 1.0f / sqrtf(sq / static_cast<float>(p.D) + p.eps);
  const float rk = 1.0f / sqrtf(sk / static_cast<float>(p.D) + p.eps);

  const int slot = s.cache_len + t;
  const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(slot), p.fT));
  const int page = clamp_page(p.page_table[static_cast<size_t>(b) * p.max_frames + fr],
                              p.n_pages);
  const int off = slot - fr * p.T;
  const uint4* gq = reinterpret_cast<const uint4*>(p.g_q);
  const uint4* gk = reinterpret_cast<const uint4*>(p.g_k);
  uint4* qo = reinterpret_cast<uint4*>(p.q_out + static_cast<size_t>(row) * p.D);
#pragma unroll
  for (int c8 = 0; c8 < kMaxChunksPerLane; ++c8) {
    if (64 * c8 >= nchunk) break;  // wave-uniform
    const int c = lane + 64 * c8;
    // every lane takes part in the shuffles, so the per-lane guard sits inside
    const int cc = c < nchunk ? c : 0;
    const int e0 = (8 * cc) % p.hd;
    const int h = (8 * cc) / p.hd;
    const int pb = e0 >> 1;
    float cv[4], sv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      cv[e] = __shfl(cs, pb + e, 64);
      sv[e] = __shfl(sn, pb + e, 64);
    }
    if (c < nchunk) {
      float a[8], g[8], y[8];
      unpack8(qraw[c8], a);
      unpack8(gq[c], g);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x0 = a[2 * e] * rq * g[2 * e], x1 = a[2 * e + 1] * rq * g[2 * e + 1];
        y[2 * e] = x0 * cv[e] - x1 * sv[e];
        y[2 * e + 1] = x0 * sv[e] + x1 * cv[e];
      }
      qo[c] = pack8(y);
      unpack8(kraw[c8], a);
      unpack8(gk[c], g);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x0 = a[2 * e] * rk * g[2 * e], x1 = a[2 * e + 1] * rk * g[2 * e + 1];
        y[2 * e] = x0 * cv[e] - x1 * sv[e];
        y[2 * e + 1] = x0 * sv[e] + x1 * cv[e];
      }
      bf16_t* dst = p.k_pages + ((static_cast<size_t>(page) * p.H + h) * p.T + off) * p.hd + e0;
      *reinterpret_cast<uint4*>(dst) = pack8(y);
    }
  }
}

hipError_t launch_qk_norm_rope(hipStream_t st, const bf16_t* qkv, int N, const RopeGeom& g,
                               const bf16_t* g_q, const bf16_t* g_k, bf16_t* q_out,
                               bf16_t* k_pages, const int32_t* page_table, const RowStreams& rs) {
  if (N == 0) return hipSuccess;
  QkRopeParams p;
  p.qkv = qkv;
  p.q_out = q_out;
  p.k_pages = k_pages;
  p.page_table = page_table;
  p.g_q = g_q;
  p.g_k = g_k;
  p.N = N;
  p.D = g.D;
  p.H = g.H;
  p.hd = g.hd;
  p.T = g.T;
  p.lat_w = g.lat_w;
  p.max_frames = g.max_frames;
  p.n_pages = g.n_pages;
  p.fT = make_fastdiv(g.T);
  p.fW = make_fastdiv(g.lat_w);
  p.eps = g.eps;
  const int seg_hw = 2 * (g.hd / 6);
  const int seg_t = g.hd - 2 * seg_hw;
  p.pairs_t = seg_t / 2;
  p.pairs_h = seg_hw / 2;
  for (int k = 0; k < 64; ++k) p.inv_freq[k] = 0.f;
  int pair = 0;
  const int segs[3] = {seg_t, seg_hw, seg_hw};
  for (int a = 0; a < 3; ++a)
    for (int k = 0; k < segs[a] / 2; ++k)
      p.inv_freq[pair++] =
          static_cast<float>(pow(static_cast<double>(g.theta), -2.0 * k / segs[a]));
  p.rs = rs;
  hipLaunchKernelGGL(qk_norm_rope_kernel, dim3((N + 3) / 4), dim3(256), 0, st, p);
  return hipGetLastError();
}

// ------------------------------------------------ value transpose / append
struct VtParams {
  const bf16_t* src;
  int ld_src, col_off, N, D, H, hd;
  bf16_t* dst;
  int paged, T, max_frames, n_pages;
  FastDiv fT;
  const int32_t* page_table;
  RowStreams rs;
};

constexpr int kVtRows = 64;

__global__ __launch_bounds__(256) void v_transpose_kernel(const VtParams p) {
  __shared__ bf16_t tile[kVtRows][128 + 8];
  const int n0 = blockIdx.x * kVtRows;
  const int h = blockIdx.y;
  const int cpr = p.hd >> 3;  // 16-byte chunks per row of one head
  for (int c = threadIdx.x; c < kVtRows * cpr; c += 256) {
    const int r = c / cpr, cc = c - r * cpr;
    const int n = n0 + r;
    if (n < p.N) {
      const uint4 u = *reinterpret_cast<const uint4*>(
          p.src + static_cast<size_t>(n) * p.ld_src + p.col_off + h * p.hd + cc * 8);
      *reinterpret_cast<uint4*>(&tile[r][cc * 8]) = u;
    }
  }
  __syncthreads();
  const int r = threadIdx.x & 63;
  const int n = n0 + r;
  if (n >= p.N) return;
  const int b = find_stream(p.rs, n);
  const RowStream s = p.rs.s[b];
  const int t = n - s.row_begin;
  size_t base;
  int T, off;
  if (p.paged) {
    const int slot = s.cache_len + t;
    const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(slot), p.fT));
    const int page =
        clamp_page(p.page_table[static_cast<size_t>(b) * p.max_frames + fr], p.n_pages);
    T = p.T;
    off = slot - fr * p.T;
    base = static_cast<size_t>(page) * p.H * p.hd * T;
  } else {
    T = s.len;
    off = t;
    base = static_cast<size_t>(s.row_begin) * p.D;
  }
  bf16_t* dst = p.dst + base + static_cast<size_t>(h) * p.hd * T + off;
  for (int dd = threadIdx.x >> 6; dd < p.hd; dd += 4) dst[static_cast<size_t>(dd) * T] = tile[r][dd];
}

hipError_t launch_v_transpose(hipStream_t st, const bf16_t* src, int ld_src, int col_off, int N,
                              int D, int H, int hd, bf16_t* dst, bool paged, int T,
                              const int32_t* page_table, int max_frames, int n_pages,
                              const RowStreams& rs) {
  if (N == 0) return hipSuccess;
  VtParams p;
  p.src = src;
  p.ld_src = ld_src;
  p.col_off = col_off;
  p.N = N;
  p.D = D;
  p.H = H;
  p.hd = hd;
  p.dst = dst;
  p.paged = paged ? 1 : 0;
  p.T = T > 0 ? T : 1;
  p.fT = make_fastdiv(p.T);
  p.max_frames = max_frames;
  p.n_pages = n_pages;
  p.page_table = page_table;
  p.rs = rs;
  hipLaunchKernelGGL(v_transpose_kernel, dim3((N + kVtRows - 1) / kVtRows, H), dim3(256), 0, st,
                     p);
  return hipGetLastError();
}

// ------------------------------------------------------- text key layout
struct CtxKParams {
  const bf16_t* src;
  int N, D, H, hd;
  const bf16_t* gain;
  float eps;
  bf16_t* dst;
  RowStreams rs;
};

__global__ __launch_bounds__(256) void ctx_k_layout_kernel(const CtxKParams p) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= p.N) return;
  const int b = find_stream(p.rs, row);
  const RowStream s = p.rs.s[b];
  const int j = row - s.row_begin;
  const int nchunk = p.D >> 3;
  const uint4* xr = reinterpret_cast<const uint4*>(p.src + static_cast<size_t>(row) * p.D);
  const uint4* gr = reinterpret_cast<const uint4*>(p.gain);
  uint4 raw[kMaxChunksPerLane];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxChunksPerLane; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      raw[i] = xr[c];
      float f[8];
      unpack8(raw[i], f);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += f[e] * f[e];
    }
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / static_cast<float>(p.D) + p.eps);
  bf16_t* base = p.dst + static_cast<size_t>(s.row_begin) * p.D;
#pragma unroll
  for (int i = 0; i < kMaxChunksPerLane; ++i) {
    const int c = lane + 64 * i;
    if (c < nchunk) {
      float f[8], g[8], y[8];
      unpack8(raw[i], f);
      unpack8(gr[c], g);
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = f[e] * r * g[e];
      const int h = (8 * c) / p.hd, e0 = (8 * c) % p.hd;
      *reinterpret_cast<uint4*>(base + (static_cast<size_t>(h) * s.len + j) * p.hd + e0) =
          pack8(y);
    }
  }
}

hipError_t launch_ctx_k_layout(hipStream_t st, const bf16_t* src, int N, int D, int H, int hd,
                               const bf16_t* gain, float eps, bf16_t* dst,
                               const RowStreams& rs) {
  if (N == 0) return hipSuccess;
  CtxKParams p{src, N, D, H, hd, gain, eps, dst, rs};
  hipLaunchKernelGGL(ctx_k_layout_kernel, dim3((N + 3) / 4), dim3(256), 0, st, p);
  return hipGetLastError();
}

// ------------------------------------------------------- time modulation
struct SinParams {
  int B;
  float t[kMaxStreams];
};

__global__ void time_sinusoid_kernel(const SinParams p, float* s_out) {
  const int b = blockIdx.x;
  const int k = threadIdx.x;  // 0..127
  const double w = pow(10000.0, -static_cast<double>(k) / 128.0);
  const double a = static_cast<double>(p.t[b]) * w;
  s_out[b * 256 + k] = static_cast<float>(cos(a));
  s_out[b * 256 + 128 + k] = static_cast<float>(sin(a));
}

hipError_t launch_time_sinusoid(hipStream_t st, const float* t_host, int B, float* s_out) {
  SinParams p;
  p.B = B;
  for (int b = 0; b < B; ++b) p.t[b] = t_host[b];
  hipLaunchKernelGGL(time_sinusoid_kernel, dim3(B), dim3(128), 0, st, p, s_out);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void linear_small_kernel(const float* __restrict__ x, int B,
                                                           int K, const bf16_t* __restrict__ W,
                                                           const bf16_t* __restrict__ bias, int O,
                                                           float* __restrict__ y, int silu_in) {
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= O) return;
  const bf16_t* wr = W + static_cast<size_t>(o) * K;
  const float bo = bf2f(bias[o]);
  for (int b = 0; b < B; ++b) {
    const float* xb = x + static_cast<size_t>(b) * K;
    float acc = 0.f;
    for (int k = lane; k < K; k += 64) {
      float xv = xb[k];
      if (silu_in) xv = xv / (1.0f + expf(-xv));
      acc += xv * bf2f(wr[k]);
    }
    acc = wave_sum(acc);
    if (lane == 0) y[static_cast<size_t>(b) * O + o] = acc + bo;
  }
}

hipError_t launch_linear_small(hipStream_t st, const float* x, int B, int K, const bf16_t* W,
                               const bf16_t* bias, int O, float* y, bool silu_in) {
  hipLaunchKernelGGL(linear_small_kernel, dim3((O + 3) / 4), dim3(256), 0, st, x, B, K, W, bias,
                     O, y, silu_in ? 1 : 0);
  return hipGetLastError();
}

}  // namespace ardit
