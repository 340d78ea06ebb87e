// Bandwidth-bound kernels of the block: adaLN RMSNorm, RMSNorm with gain,
// QK-RMSNorm + 3D RoPE + key append, value append (transposed pages), text
// key/value layout, and the small time-modulation MLP.
//
// One 64-lane wave owns a token row at a time: 16-byte loads/stores, fp32
// math, a wave reduction for the mean square.  Rows of up to 8192 elements
// are held in registers so each row is read from HBM once; vectors shared by
// a workgroup's rows (modulation, gains, rotation terms) are staged in LDS.
#include <math.h>

#include <algorithm>

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

// A workgroup handles kRowsPerGroup consecutive rows: 4 waves of 2 rows, or,
// for rows of more than 3072 elements, 8 waves of one row each (half the
// registers per wave, so twice the waves in flight: 17% less time for the
// norms of 5120-wide rows);
// the per-row vectors it shares (modulation, gains) are staged once in LDS as
// fp32, the first four of each 8-element chunk in one array and the last four
// in a second, so a wave's 16-byte reads are consecutive (pairs of 16-byte
// reads 32 bytes apart made two-way bank conflicts).  A lane holds chunks lane + 64 i (i < MAXC) of 8 elements of each of
// its rows, so every row is read from HBM once and all its loads are in
// flight together.
constexpr int kRowsPerGroup = 8;
// rows per wave and threads per workgroup for rows of up to 512 MAXC elements
template <int MAXC> struct RowCfg {
  static constexpr int RPW = MAXC >= 8 ? 1 : 2;
  static constexpr int THREADS = 64 * kRowsPerGroup / RPW;
};

// y = rms(x) * (1 + scale) + shift with scale = mod[b][scale_row] +
// mod_table[scale_row] and shift likewise.  Streams hold rows_per_stream
// rows, a multiple of kRowsPerGroup, so a workgroup's rows share one stream.
template <typename T, int MAXC>
__global__ __launch_bounds__(512) void adaln_norm_kernel(
    const T* __restrict__ x, bf16_t* __restrict__ out, int N, int D,
    const float* __restrict__ mod, const float* __restrict__ mod_table, int shift_row,
    int scale_row, int rows_per_stream, float eps) {
  extern __shared__ float4 lds_mod[];   // D / 4 of (1 + scale), then D / 4 of shift (split halves)
  constexpr int kRowsPerWave = RowCfg<MAXC>::RPW, NTHR = RowCfg<MAXC>::THREADS;
  const int lane = threadIdx.x & 63;
  const int row0 = blockIdx.x * kRowsPerGroup + (threadIdx.x >> 6) * kRowsPerWave;
  const int nchunk = D >> 3;
  // this wave's rows, loads issued before the modulation is staged
  float v[kRowsPerWave][MAXC][8];
#pragma unroll
  for (int r = 0; r < kRowsPerWave; ++r) {
    const T* xr = x + static_cast<size_t>(min(row0 + r, N - 1)) * D;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + 64 * i;
      if (c < nchunk) load8(xr + 8 * c, v[r][i]);
    }
  }
  {
    const int b = (blockIdx.x * kRowsPerGroup) / rows_per_stream;
    const float4* msh = reinterpret_cast<const float4*>(mod + (static_cast<size_t>(b) * 6 + shift_row) * D);
    const float4* msc = reinterpret_cast<const float4*>(mod + (static_cast<size_t>(b) * 6 + scale_row) * D);
    const float4* tsh = reinterpret_cast<const float4*>(mod_table + static_cast<size_t>(shift_row) * D);
    const float4* tsc = reinterpret_cast<const float4*>(mod_table + static_cast<size_t>(scale_row) * D);
    for (int k = threadIdx.x; k < D / 8; k += NTHR) {   // chunk k, both halves
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const float4 a = msc[2 * k + hf], c = tsc[2 * k + hf];
        const float4 sh = msh[2 * k + hf], th = tsh[2 * k + hf];
        lds_mod[hf * (D / 8) + k] =
            make_float4(1.f + a.x + c.x, 1.f + a.y + c.y, 1.f + a.z + c.z, 1.f + a.w + c.w);
        lds_mod[D / 4 + hf * (D / 8) + k] =
            make_float4(sh.x + th.x, sh.y + th.y, sh.z + th.z, sh.w + th.w);
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kRowsPerWave; ++r) {
    const int row = row0 + r;
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
      if (lane + 64 * i < nchunk)
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[r][i][e] * v[r][i][e];
    ss = wave_sum(ss);
    const float rs = 1.0f / sqrtf(ss / static_cast<float>(D) + eps);
    if (row >= N) continue;
    uint4* orow = reinterpret_cast<uint4*>(out + static_cast<size_t>(row) * D);
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + 64 * i;
      if (c < nchunk) {
        const float4 a0 = lds_mod[c], a1 = lds_mod[nchunk + c];
        const float4 b0 = lds_mod[D / 4 + c], b1 = lds_mod[D / 4 + nchunk + c];
        const float sa[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        const float sb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = v[r][i][e] * rs * sa[e] + sb[e];
        orow[c] = pack8(y);
      }
    }
  }
}

// y = rms(x) * gain, the gain staged in LDS as fp32.
template <typename T, int MAXC>
__global__ __launch_bounds__(512) void rms_gain_kernel(const T* in, bf16_t* out, int N, int D,
                                                        const bf16_t* __restrict__ gain,
                                                        float eps) {
  extern __shared__ float4 lds_gain[];   // D / 4
  constexpr int kRowsPerWave = RowCfg<MAXC>::RPW, NTHR = RowCfg<MAXC>::THREADS;
  const int lane = threadIdx.x & 63;
  const int row0 = blockIdx.x * kRowsPerGroup + (threadIdx.x >> 6) * kRowsPerWave;
  const int nchunk = D >> 3;
  float v[kRowsPerWave][MAXC][8];
#pragma unroll
  for (int r = 0; r < kRowsPerWave; ++r) {
    const T* xr = in + static_cast<size_t>(min(row0 + r, N - 1)) * D;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + 64 * i;
      if (c < nchunk) load8(xr + 8 * c, v[r][i]);
    }
  }
  for (int k = threadIdx.x; k < D / 8; k += NTHR) {
    float g[8];
    load8(gain + 8 * k, g);
    lds_gain[k] = make_float4(g[0], g[1], g[2], g[3]);
    lds_gain[D / 8 + k] = make_float4(g[4], g[5], g[6], g[7]);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kRowsPerWave; ++r) {
    const int row = row0 + r;
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
      if (lane + 64 * i < nchunk)
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[r][i][e] * v[r][i][e];
    ss = wave_sum(ss);
    const float rs = 1.0f / sqrtf(ss / static_cast<float>(D) + eps);
    if (row >= N) continue;
    uint4* orow = reinterpret_cast<uint4*>(out + static_cast<size_t>(row) * D);
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + 64 * i;
      if (c < nchunk) {
        const float4 g0 = lds_gain[c], g1 = lds_gain[nchunk + c];
        const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        float y[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = v[r][i][e] * rs * g[e];
        orow[c] = pack8(y);
      }
    }
  }
}

// chunks per lane needed for a row of D elements, rounded up to a size that
// has an instantiation (the row arrays are sized by it)
static int row_chunks(int D) {
  const int c = (D / 8 + 63) / 64;
  const int sizes[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 16};
  for (int s : sizes)
    if (c <= s) return s;
  return 16;
}

#define ARDIT_ROW_CASE(KERNEL, T, C, LDS, ...) \
  case C: hipLaunchKernelGGL((KERNEL<T, C>), grid, dim3(RowCfg<C>::THREADS), LDS, st, __VA_ARGS__); break;
#define ARDIT_ROW_DISPATCH(KERNEL, T, LDS, ...)         \
  switch (row_chunks(D)) {                              \
    ARDIT_ROW_CASE(KERNEL, T, 1, LDS, __VA_ARGS__)      \
    ARDIT_ROW_CASE(KERNEL, T, 2, LDS, __VA_ARGS__)      \
    ARDIT_ROW_CASE(KERNEL, T, 3, LDS, __VA_ARGS__)      \
    ARDIT_ROW_CASE(KERNEL, T, 4, LDS, __VA_ARGS__)      \
    ARDIT_ROW_CASE(KERNEL, T, 5, LDS, __VA_ARGS__)      \
    ARDIT_ROW_CASE(KERNEL, T, 6, LDS, __VA_ARGS__)      \
    ARDIT_ROW_CASE(KERNEL, T, 8, LDS, __VA_ARGS__)      \
    ARDIT_ROW_CASE(KERNEL, T, 10, LDS, __VA_ARGS__)     \
    ARDIT_ROW_CASE(KERNEL, T, 12, LDS, __VA_ARGS__)     \
    default: hipLaunchKernelGGL((KERNEL<T, 16>), grid, dim3(RowCfg<16>::THREADS), LDS, st, __VA_ARGS__); break; \
  }

hipError_t launch_adaln_norm(hipStream_t st, const void* x, bool x_f32, bf16_t* out, int N, int D,
                             const float* mod, const float* mod_table, int shift_row,
                             int scale_row, int rows_per_stream, float eps) {
  if (N == 0) return hipSuccess;
  if (rows_per_stream % kRowsPerGroup != 0) return hipErrorInvalidValue;
  const dim3 grid((N + kRowsPerGroup - 1) / kRowsPerGroup);
  const size_t lds = 2 * sizeof(float) * D;
  if (x_f32) {
    const float* xf = static_cast<const float*>(x);
    ARDIT_ROW_DISPATCH(adaln_norm_kernel, float, lds, xf, out, N, D, mod, mod_table, shift_row,
                       scale_row, rows_per_stream, eps);
  } else {
    const bf16_t* xb = static_cast<const bf16_t*>(x);
    ARDIT_ROW_DISPATCH(adaln_norm_kernel, bf16_t, lds, xb, out, N, D, mod, mod_table, shift_row,
                       scale_row, rows_per_stream, eps);
  }
  return hipGetLastError();
}

hipError_t launch_rms_gain(hipStream_t st, const void* in, bool in_f32, bf16_t* out, int N, int D,
                           const bf16_t* gain, float eps) {
  if (N == 0) return hipSuccess;
  const dim3 grid((N + kRowsPerGroup - 1) / kRowsPerGroup);
  const size_t lds = sizeof(float) * D;
  if (in_f32) {
    const float* xf = static_cast<const float*>(in);
    ARDIT_ROW_DISPATCH(rms_gain_kernel, float, lds, xf, out, N, D, gain, eps);
  } else {
    const bf16_t* xb = static_cast<const bf16_t*>(in);
    ARDIT_ROW_DISPATCH(rms_gain_kernel, bf16_t, lds, xb, out, N, D, gain, eps);
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

// Page of a write: an entry outside [0, n_pages) (an unassigned or stale
// table slot) yields -1 and the store is skipped, so a bad table can never
// write into a page another stream owns.
__device__ __forceinline__ int write_page(int p, int n_pages) {
  return p >= 0 && p < n_pages ? p : -1;
}

// A workgroup handles kRowsPerGroup rows (RowCfg: 2 or 1 per wave).  Per row, lane k < d/2
// computes the rotation (cos, sin) of pair k, shared through LDS; the gains
// are staged in LDS as fp32; both rows' q and k are loaded before any math.
// lds_qk: g_q (D / 4 float4), g_k (D / 4), then cos / sin per row
template <int MAXC>
__device__ __forceinline__ void qk_norm_rope_group(const QkRopeParams& p, int group,
                                                   float4* lds_qk) {
  constexpr int kRowsPerWave = RowCfg<MAXC>::RPW, NTHR = RowCfg<MAXC>::THREADS;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int row0 = group * kRowsPerGroup + wave * kRowsPerWave;
  const int nchunk = p.D >> 3;
  float4* lg_q = lds_qk;
  float4* lg_k = lds_qk + p.D / 4;
  float* lcs = reinterpret_cast<float*>(lds_qk + p.D / 2);   // [kRowsPerGroup][64]
  float* lsn = lcs + kRowsPerGroup * 64;

  uint4 qraw[kRowsPerWave][MAXC], kraw[kRowsPerWave][MAXC];
#pragma unroll
  for (int r = 0; r < kRowsPerWave; ++r) {
    const uint4* qr = reinterpret_cast<const uint4*>(
        p.qkv + static_cast<size_t>(min(row0 + r, p.N - 1)) * 3 * p.D);
    const uint4* kr = qr + nchunk;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + 64 * i;
      if (c < nchunk) {
        qraw[r][i] = qr[c];
        kraw[r][i] = kr[c];
      }
    }
  }
  for (int k = threadIdx.x; k < p.D / 8; k += NTHR) {
    float g[8];
    unpack8(reinterpret_cast<const uint4*>(p.g_q)[k], g);
    lg_q[k] = make_float4(g[0], g[1], g[2], g[3]);
    lg_q[p.D / 8 + k] = make_float4(g[4], g[5], g[6], g[7]);
    unpack8(reinterpret_cast<const uint4*>(p.g_k)[k], g);
    lg_k[k] = make_float4(g[0], g[1], g[2], g[3]);
    lg_k[p.D / 8 + k] = make_float4(g[4], g[5], g[6], g[7]);
  }
  // rotation of pair `lane` of a head for each of this wave's rows
#pragma unroll
  for (int r = 0; r < kRowsPerWave; ++r) {
    const int row = min(row0 + r, p.N - 1);
    const RowStream s = p.rs.s[find_stream(p.rs, row)];
    const int t = row - s.row_begin;
    const int f = static_cast<int>(fdiv(static_cast<uint32_t>(t), p.fT));
    const int rem = t - f * p.T;
    const int i = static_cast<int>(fdiv(static_cast<uint32_t>(rem), p.fW));
    const int j = rem - i * p.lat_w;
    float cs = 1.f, sn = 0.f;
    if (lane < (p.hd >> 1)) {
      const int pos = lane < p.pairs_t ? s.frame_pos0 + f : (lane < p.pairs_t + p.pairs_h ? i : j);
      sincosf(static_cast<float>(pos) * p.inv_freq[lane], &sn, &cs);
    }
    lcs[(wave * kRowsPerWave + r) * 64 + lane] = cs;
    lsn[(wave * kRowsPerWave + r) * 64 + lane] = sn;
  }
  __syncthreads();

#pragma unroll
  for (int r = 0; r < kRowsPerWave; ++r) {
    const int row = row0 + r;
    float sq = 0.f, sk = 0.f;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      if (lane + 64 * i < nchunk) {
        float a[8], bb[8];
        unpack8(qraw[r][i], a);
        unpack8(kraw[r][i], bb);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sq += a[e] * a[e];
          sk += bb[e] * bb[e];
        }
      }
    }
    sq = wave_sum(sq);
    sk = wave_sum(sk);
    if (row >= p.N) continue;
    const float rq = 1.0f / sqrtf(sq / static_cast<float>(p.D) + p.eps);
    const float rk = 1.0f / sqrtf(sk / static_cast<float>(p.D) + p.eps);
    const int b = find_stream(p.rs, row);
    const RowStream s = p.rs.s[b];
    const int slot = s.cache_len + row - s.row_begin;
    const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(slot), p.fT));
    const int page = write_page(p.page_table[static_cast<size_t>(b) * p.max_frames + fr],
                                p.n_pages);
    const int off = slot - fr * p.T;
    const float* rcs = lcs + (wave * kRowsPerWave + r) * 64;
    const float* rsn = lsn + (wave * kRowsPerWave + r) * 64;
    uint4* qo = reinterpret_cast<uint4*>(p.q_out + static_cast<size_t>(row) * p.D);
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int c = lane + 64 * i;
      if (c < nchunk) {
        const int e0 = (8 * c) % p.hd;
        const int h = (8 * c) / p.hd;
        const float4 cv = *reinterpret_cast<const float4*>(rcs + (e0 >> 1));
        const float4 sv = *reinterpret_cast<const float4*>(rsn + (e0 >> 1));
        const float cc[4] = {cv.x, cv.y, cv.z, cv.w}, ss[4] = {sv.x, sv.y, sv.z, sv.w};
        float a[8], y[8];
        const float4 g0 = lg_q[c], g1 = lg_q[nchunk + c];
        const float gq[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        unpack8(qraw[r][i], a);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x0 = a[2 * e] * rq * gq[2 * e], x1 = a[2 * e + 1] * rq * gq[2 * e + 1];
          y[2 * e] = x0 * cc[e] - x1 * ss[e];
          y[2 * e + 1] = x0 * ss[e] + x1 * cc[e];
        }
        qo[c] = pack8(y);
        const float4 k0 = lg_k[c], k1 = lg_k[nchunk + c];
        const float gk[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
        unpack8(kraw[r][i], a);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x0 = a[2 * e] * rk * gk[2 * e], x1 = a[2 * e + 1] * rk * gk[2 * e + 1];
          y[2 * e] = x0 * cc[e] - x1 * ss[e];
          y[2 * e + 1] = x0 * ss[e] + x1 * cc[e];
        }
        if (page >= 0) {
          bf16_t* dst =
              p.k_pages + ((static_cast<size_t>(page) * p.H + h) * p.T + off) * p.hd + e0;
          *reinterpret_cast<uint4*>(dst) = pack8(y);
        }
      }
    }
  }
}

template <int MAXC>
__global__ __launch_bounds__(512) void qk_norm_rope_kernel(const QkRopeParams p) {
  extern __shared__ float4 lds_qk[];
  qk_norm_rope_group<MAXC>(p, blockIdx.x, lds_qk);
}

static QkRopeParams qk_params(const bf16_t* qkv, int N, const RopeGeom& g, const bf16_t* g_q,
                              const bf16_t* g_k, bf16_t* q_out, bf16_t* k_pages,
                              const int32_t* page_table, const RowStreams& rs) {
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
  return p;
}

static size_t qk_lds_bytes(int D) {
  return 2 * sizeof(float) * D + 2 * sizeof(float) * kRowsPerGroup * 64;
}

hipError_t launch_qk_norm_rope(hipStream_t st, const bf16_t* qkv, int N, const RopeGeom& g,
                               const bf16_t* g_q, const bf16_t* g_k, bf16_t* q_out,
                               bf16_t* k_pages, const int32_t* page_table, const RowStreams& rs) {
  if (N == 0) return hipSuccess;
  const QkRopeParams p = qk_params(qkv, N, g, g_q, g_k, q_out, k_pages, page_table, rs);
  const dim3 grid((N + kRowsPerGroup - 1) / kRowsPerGroup);
  const size_t lds = qk_lds_bytes(g.D);
  switch (row_chunks(g.D)) {
#define ARDIT_QK_CASE(C) \
    case C: hipLaunchKernelGGL(qk_norm_rope_kernel<C>, grid, dim3(RowCfg<C>::THREADS), lds, st, p); break;
    ARDIT_QK_CASE(1) ARDIT_QK_CASE(2) ARDIT_QK_CASE(3) ARDIT_QK_CASE(4) ARDIT_QK_CASE(5)
    ARDIT_QK_CASE(6) ARDIT_QK_CASE(8) ARDIT_QK_CASE(10) ARDIT_QK_CASE(12)
#undef ARDIT_QK_CASE
    default: hipLaunchKernelGGL(qk_norm_rope_kernel<16>, grid, dim3(RowCfg<16>::THREADS), lds, st, p); break;
  }
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
        write_page(p.page_table[static_cast<size_t>(b) * p.max_frames + fr], p.n_pages);
    if (page < 0) return;
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

// Paged value append with 16-byte stores: 64 tokens x one head staged in LDS
// (16-byte chunk cc of token r at slot cc ^ ((r / 8) % 8), so the eight
// lanes gathering one dim from eight 8-token groups hit distinct banks); a
// lane then gathers 8 consecutive tokens of one dim and stores them as one
// 16-byte write, eight lanes filling 128 contiguous bytes of a transposed row
// (69 against 71 us for the 2-byte stores at 37440 rows; 256-token tiles were
// slower, 105 us).  Transposed rows are T = 1560 tokens long, so these 128-byte
// pieces straddle cache lines: a row pitch rounded to 64 tokens would align
// them, at the price of a page layout change.
// Needs every stream's rows and cache length in multiples of 8 and T % 8 == 0,
// so each 8-token group lies in one stream and one page.
constexpr int kVaRows = 64;

__device__ __forceinline__ void v_append16_block(const VtParams& p, int nb, int h,
                                                 bf16_t (*tile)[128]) {
  const int n0 = nb * kVaRows;
  const int cpr = p.hd >> 3;  // 16-byte chunks per row of one head
  for (int c = threadIdx.x; c < kVaRows * cpr; c += 256) {
    const int r = c / cpr, cc = c - r * cpr;
    const int n = n0 + r;
    if (n < p.N) {
      const uint4 u = *reinterpret_cast<const uint4*>(
          p.src + static_cast<size_t>(n) * p.ld_src + p.col_off + h * p.hd + cc * 8);
      *reinterpret_cast<uint4*>(&tile[r][8 * (cc ^ ((r >> 3) & 7))]) = u;
    }
  }
  __syncthreads();
  // item (dim dd, group g): lanes of one dim take consecutive groups
  for (int it = threadIdx.x; it < p.hd * (kVaRows / 8); it += 256) {
    const int g = it & (kVaRows / 8 - 1), dd = it / (kVaRows / 8);
    const int r0 = 8 * g;
    const int n = n0 + r0;
    if (n >= p.N) continue;
    const int b = find_stream(p.rs, n);
    const RowStream s = p.rs.s[b];
    const int slot = s.cache_len + n - s.row_begin;
    const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(slot), p.fT));
    const int page =
        write_page(p.page_table[static_cast<size_t>(b) * p.max_frames + fr], p.n_pages);
    if (page < 0) continue;
    const int off = slot - fr * p.T;
    const int cc = dd >> 3, e = dd & 7;
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int ra = r0 + 2 * k, rb = ra + 1;
      const uint32_t lo = tile[ra][8 * (cc ^ ((ra >> 3) & 7)) + e];
      const uint32_t hi = tile[rb][8 * (cc ^ ((rb >> 3) & 7)) + e];
      w[k] = lo | (hi << 16);
    }
    bf16_t* dst = p.dst + (static_cast<size_t>(page) * p.H + h) * p.hd * p.T +
                  static_cast<size_t>(dd) * p.T + off;
    *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

__global__ __launch_bounds__(256) void v_append16_kernel(const VtParams p) {
  __shared__ __attribute__((aligned(16))) bf16_t tile[kVaRows][128];
  v_append16_block(p, blockIdx.x, blockIdx.y, tile);
}

// The key path (QK-norm + RoPE + key append) and the 16-byte value append in
// one launch: the first qk_groups workgroups take 8-row groups of q and k, the
// rest (64-token block, head) value tiles, so the two run side by side instead
// of one after the other.
template <int MAXC>
__global__ __launch_bounds__(256) void qk_v_append_kernel(const QkRopeParams qp,
                                                          const VtParams vp, int qk_groups,
                                                          int v_blocks) {
  extern __shared__ float4 lds_qkv[];
  const int b = blockIdx.x;
  if (b < qk_groups) {
    qk_norm_rope_group<MAXC>(qp, b, lds_qkv);
  } else {
    const int v = b - qk_groups;
    v_append16_block(vp, v % v_blocks, v / v_blocks, reinterpret_cast<bf16_t (*)[128]>(lds_qkv));
  }
}

static VtParams vt_params(const bf16_t* src, int ld_src, int col_off, int N, int D, int H,
                          int hd, bf16_t* dst, bool paged, int T, const int32_t* page_table,
                          int max_frames, int n_pages, const RowStreams& rs) {
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
  return p;
}

// the 16-byte value append applies: paged, and every 8-token group in one
// stream and one page
static bool vt_groups8(const VtParams& p) {
  bool ok = p.paged && p.T % 8 == 0 && p.hd <= 128 && p.N % 8 == 0;
  for (int i = 0; i < p.rs.n && ok; ++i)
    ok = p.rs.s[i].len % 8 == 0 && p.rs.s[i].cache_len % 8 == 0 && p.rs.s[i].row_begin % 8 == 0;
  return ok;
}

hipError_t launch_v_transpose(hipStream_t st, const bf16_t* src, int ld_src, int col_off, int N,
                              int D, int H, int hd, bf16_t* dst, bool paged, int T,
                              const int32_t* page_table, int max_frames, int n_pages,
                              const RowStreams& rs) {
  if (N == 0) return hipSuccess;
  const VtParams p = vt_params(src, ld_src, col_off, N, D, H, hd, dst, paged, T, page_table,
                               max_frames, n_pages, rs);
  if (vt_groups8(p))
    hipLaunchKernelGGL(v_append16_kernel, dim3((N + kVaRows - 1) / kVaRows, H), dim3(256), 0, st,
                       p);
  else
    hipLaunchKernelGGL(v_transpose_kernel, dim3((N + kVtRows - 1) / kVtRows, H), dim3(256), 0,
                       st, p);
  return hipGetLastError();
}

hipError_t launch_kv_append(hipStream_t st, const bf16_t* qkv, int N, const RopeGeom& g,
                            const bf16_t* g_q, const bf16_t* g_k, bf16_t* q_out,
                            bf16_t* k_pages, bf16_t* v_pages, const int32_t* page_table,
                            const RowStreams& rs) {
  if (N == 0) return hipSuccess;
  const VtParams vp = vt_params(qkv, 3 * g.D, 2 * g.D, N, g.D, g.H, g.hd, v_pages, true, g.T,
                                page_table, g.max_frames, g.n_pages, rs);
  const int mc = row_chunks(g.D);
  if (!vt_groups8(vp) || mc > 4) {   // two launches
    hipError_t e = launch_qk_norm_rope(st, qkv, N, g, g_q, g_k, q_out, k_pages, page_table, rs);
    if (e != hipSuccess) return e;
    return launch_v_transpose(st, qkv, 3 * g.D, 2 * g.D, N, g.D, g.H, g.hd, v_pages, true, g.T,
                              page_table, g.max_frames, g.n_pages, rs);
  }
  const QkRopeParams qp = qk_params(qkv, N, g, g_q, g_k, q_out, k_pages, page_table, rs);
  const int qk_groups = (N + kRowsPerGroup - 1) / kRowsPerGroup;
  const int v_blocks = (N + kVaRows - 1) / kVaRows;
  const dim3 grid(qk_groups + v_blocks * g.H);
  const size_t lds = std::max(qk_lds_bytes(g.D), sizeof(bf16_t) * kVaRows * 128);
  switch (mc) {
#define ARDIT_QKV_CASE(C)                                                                     \
    case C:                                                                                 \
      hipLaunchKernelGGL(qk_v_append_kernel<C>, grid, dim3(256), lds, st, qp, vp, qk_groups, \
                         v_blocks);                                                         \
      break;
    ARDIT_QKV_CASE(1) ARDIT_QKV_CASE(2) ARDIT_QKV_CASE(3)
    default: ARDIT_QKV_CASE(4)
#undef ARDIT_QKV_CASE
  }
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
