// Block selection of block-sparse self-attention on gfx950.
//
// The sparsity knob rho of a fidelity configuration skips the attention blocks
// that a sparse mask leaves out (paper, Section 2.1, fidelity knobs; rho in
// {0, 0.6, 0.7, 0.8, 0.9}, Appendix A).  The paper names Light Forcing as the
// method but gives no selection rule; the one computed here: for each item
// (stream, head, 256-query tile) the score of key tile j (64 logical keys of
// [cache | chunk]) is mean(q over the item's rows) . mean(k over the tile's
// keys), both means in fp32, and the item keeps the
// n_keep = ceil((1 - rho) n - 1e-3) highest-scoring of its n key tiles (at
// least one), ties to the lower tile index.  The attention kernel then runs
// the item over its kept tiles only.
//
// key_mean_kernel: one wave per (stream, head, key tile) reads the tile's keys
// through the page table, 16 bytes per lane, and writes their fp32 mean.  It
// reads every key of the sparse streams once, the selection's HBM cost.
//
// select_kernel: one 256-thread workgroup per item forms the query mean, the
// scores against its head's tile means, the n_keep-th largest score by a
// 32-step radix search over order-preserving integer keys, and writes the
// kept tiles in ascending order using two ballot scans (the second resolves
// ties at the threshold by index).
#include <math.h>

#include "launch.h"

namespace ardit {

namespace {

constexpr int SEL_THR = 256;

// Order-preserving unsigned key of a score: larger score, larger key.  NaN
// ranks as -inf and -0 as +0.
__device__ __forceinline__ uint32_t order_key(float s) {
  if (s != s) s = -INFINITY;
  if (s == 0.f) s = 0.f;
  const uint32_t b = __float_as_uint(s);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Sum of v over the workgroup (every thread gets it); sh holds 4 ints.
__device__ __forceinline__ int block_sum(int v, int* sh) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  const int t = sh[0] + sh[1] + sh[2] + sh[3];
  __syncthreads();
  return t;
}

// Exclusive prefix count of f over the workgroup in thread order; *total gets
// the count of the whole workgroup.
__device__ __forceinline__ int block_excl_scan(bool f, int* total, int* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(f);
  const int within = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) sh[wave] = __popcll(m);
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SEL_THR / 64; ++w) {
    const int c = sh[w];
    before += w < wave ? c : 0;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return before + within;
}

// Physical page of logical frame fr of a stream, clamped into the pool.
__device__ __forceinline__ int page_of(const AttnArgs& a, const AttnStream& S, int fr) {
  const int p = a.page_table[static_cast<size_t>(S.stream) * a.max_frames + fr];
  return p < 0 ? 0 : (p >= a.n_pages ? a.n_pages - 1 : p);
}

// Mean key of (stream, head, tile) number g of the sparse plan, rows of kbar
// ordered the same way (streams in plan order, then head, then tile).
template <int HD>
__global__ __launch_bounds__(SEL_THR) void key_mean_kernel(const AttnArgs a, int total) {
  constexpr int LPR = HD / 8;        // lanes per key row, 8 dims (16 bytes) each
  constexpr int RPS = 64 / LPR;      // key rows per wave step
  const int lane = threadIdx.x & 63;
  const int g = blockIdx.x * (SEL_THR / 64) + (threadIdx.x >> 6);
  if (g >= total) return;
  int si = 0, base = 0;
  for (; si < a.n_streams - 1; ++si) {
    const int cnt = a.H * a.s[si].n_tiles;
    if (g < base + cnt) break;
    base += cnt;
  }
  const AttnStream& S = a.s[si];
  if (S.n_keep >= S.n_tiles) return;   // nothing to select
  const int r = g - base;
  const int h = r / S.n_tiles, j = r - h * S.n_tiles;
  const int j0 = j * kAttnKTile;
  const int cnt = min(kAttnKTile, S.kv_len - j0);
  const int dc = lane % LPR, ro = lane / LPR;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int k = ro; k < cnt; k += RPS) {
    const int key = j0 + k;
    const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(key), a.fT));
    const int p = page_of(a, S, fr);
    const bf16_t* src =
        a.k + ((static_cast<size_t>(p) * a.H + h) * a.T + (key - fr * a.T)) * HD + 8 * dc;
    float f[8];
    unpack8(*reinterpret_cast<const uint4*>(src), f);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += f[e];
  }
#pragma unroll
  for (int m = LPR; m < 64; m <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], m, kWave);
  if (ro == 0) {
    const float n = static_cast<float>(cnt);
    float* out = a.kbar + static_cast<size_t>(g) * HD + 8 * dc;
    *reinterpret_cast<float4*>(out) =
        make_float4(acc[0] / n, acc[1] / n, acc[2] / n, acc[3] / n);
    *reinterpret_cast<float4*>(out + 4) =
        make_float4(acc[4] / n, acc[5] / n, acc[6] / n, acc[7] / n);
  }
}

template <int HD>
__global__ __launch_bounds__(SEL_THR) void select_kernel(const AttnArgs a) {
  constexpr int LPR = HD / 8;          // threads per query row, 8 dims each
  constexpr int RPS = SEL_THR / LPR;   // query rows per step
  __shared__ uint32_t key[kSparseMaxTiles];
  __shared__ float red[RPS][HD];
  __shared__ float qbar[HD];
  __shared__ int sh[SEL_THR / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  const int L = blockIdx.x;
  int si = 0;
  for (int i = 1; i < a.n_streams; ++i)
    if (L >= a.s[i].item_begin) si = i;
  const AttnStream& S = a.s[si];
  const int it = L - S.item_begin;
  const int h = it / S.n_qtiles;
  const int qt = it - h * S.n_qtiles;
  const int ld = a.blk_ld ? a.blk_ld : S.n_keep;
  int32_t* out = a.blocks + S.blk_off + static_cast<int64_t>(it) * ld;
  const int n = S.n_tiles, nk = S.n_keep;
  if (nk >= n) {   // dense stream: every tile, in order
    for (int t = tid; t < ld; t += SEL_THR) out[t] = t < n ? t : -1;
    return;
  }

  // ---- query mean over the item's rows
  const int r0 = qt * kAttnQTile;
  const int rows = min(kAttnQTile, S.q_len - r0);
  {
    const int dc = tid % LPR, ro = tid / LPR;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int r = ro; r < rows; r += RPS) {
      const bf16_t* src = a.q + static_cast<size_t>(S.q_off + r0 + r) * a.ldq + h * HD + 8 * dc;
      float f[8];
      unpack8(*reinterpret_cast<const uint4*>(src), f);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += f[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) red[ro][8 * dc + e] = acc[e];
  }
  __syncthreads();
  if (tid < HD) {
    float s = 0.f;
#pragma unroll 8
    for (int r = 0; r < RPS; ++r) s += red[r][tid];
    qbar[tid] = s / static_cast<float>(rows);
  }
  __syncthreads();

  // ---- scores: a wave per tile, two dims per lane (HD = 64: two tiles per wave)
  {
    int kb = 0;   // first kbar row of this stream
    for (int i = 0; i < si; ++i) kb += a.H * a.s[i].n_tiles;
    const float* kbar = a.kbar + (static_cast<size_t>(kb) + static_cast<size_t>(h) * n) * HD;
    constexpr int LPT = HD / 2;          // lanes per tile
    constexpr int TPW = 64 / LPT;        // tiles per wave step
    const int dp = lane % LPT, sub = lane / LPT;
    const float2 qv = make_float2(qbar[2 * dp], qbar[2 * dp + 1]);
    for (int j0 = wave * TPW; j0 < n; j0 += (SEL_THR / 64) * TPW) {
      const int j = j0 + sub;
      float p = 0.f;
      if (j < n) {
        const float2 kv = *reinterpret_cast<const float2*>(kbar + static_cast<size_t>(j) * HD + 2 * dp);
        p = qv.x * kv.x + qv.y * kv.y;
      }
#pragma unroll
      for (int m = LPT / 2; m >= 1; m >>= 1) p += __shfl_xor(p, m, kWave);
      if (dp == 0 && j < n) key[j] = order_key(p);
    }
  }
  __syncthreads();

  // ---- threshold: the nk-th largest key, found bit by bit from the top
  uint32_t thr = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = thr | (1u << bit);
    int c = 0;
    for (int j = tid; j < n; j += SEL_THR) c += key[j] >= cand ? 1 : 0;
    if (block_sum(c, sh) >= nk) thr = cand;
  }
  int gt = 0;
  for (int j = tid; j < n; j += SEL_THR) gt += key[j] > thr ? 1 : 0;
  const int need = nk - block_sum(gt, sh);   // tiles taken at the threshold, lowest index first

  // ---- kept tiles in ascending order
  int carry_eq = 0, carry_keep = 0;
  for (int base = 0; base < n; base += SEL_THR) {
    const int j = base + tid;
    const uint32_t kj = j < n ? key[j] : 0u;
    const bool eq = j < n && kj == thr;
    int eq_tot, keep_tot;
    const int eq_before = carry_eq + block_excl_scan(eq, &eq_tot, sh);
    const bool keep = j < n && (kj > thr || (eq && eq_before < need));
    const int pos = carry_keep + block_excl_scan(keep, &keep_tot, sh);
    if (keep) out[pos] = j;
    carry_eq += eq_tot;
    carry_keep += keep_tot;
  }
  for (int t = nk + tid; t < ld; t += SEL_THR) out[t] = -1;
}

}  // namespace

int sparse_keep_count(int n_tiles, float rho) {
  if (n_tiles <= 0) return 0;
  const double keep = ceil((1.0 - static_cast<double>(rho)) * n_tiles - 1e-3);
  if (!(keep >= 1.0)) return 1;
  return keep >= n_tiles ? n_tiles : static_cast<int>(keep);
}

size_t sparse_kbar_floats(const AttnArgs& a, int head_dim) {
  size_t n = 0;
  for (int i = 0; i < a.n_streams; ++i)
    if (a.s[i].q_len > 0)
      n += static_cast<size_t>(a.H) * ((a.s[i].kv_len + kAttnKTile - 1) / kAttnKTile) * head_dim;
  return n;
}

void plan_sparse_attention(AttnArgs& a, const float* rho, int32_t* blocks, int32_t blk_ld,
                           float* kbar) {
  // per stream in batch order: tiles, kept tiles, offset of its lists
  AttnStream tmp[kMaxStreams];
  int n = 0;
  int64_t packed = 0, rows = 0;
  for (int i = 0; i < a.n_streams; ++i) {
    AttnStream s = a.s[i];
    s.n_qtiles = (s.q_len + kAttnQTile - 1) / kAttnQTile;
    s.n_tiles = (s.kv_len + kAttnKTile - 1) / kAttnKTile;
    s.n_keep = sparse_keep_count(s.n_tiles, rho ? rho[i] : 0.f);
    s.blk_off = static_cast<int32_t>(blk_ld ? rows * blk_ld : packed);
    s.main_tiles = s.n_tiles;
    s.tail_begin = 0;
    rows += static_cast<int64_t>(a.H) * s.n_qtiles;
    packed += static_cast<int64_t>(a.H) * s.n_qtiles * s.n_keep;
    if (s.q_len > 0) tmp[n++] = s;
  }
  // longest items first
  for (int i = 1; i < n; ++i) {
    AttnStream x = tmp[i];
    int j = i - 1;
    while (j >= 0 && tmp[j].n_keep < x.n_keep) {
      tmp[j + 1] = tmp[j];
      --j;
    }
    tmp[j + 1] = x;
  }
  int items = 0;
  for (int i = 0; i < n; ++i) {
    tmp[i].item_begin = items;
    items += tmp[i].n_qtiles * a.H;
    a.s[i] = tmp[i];
  }
  a.n_streams = n;
  a.total_items = items;
  a.per_xcd = (items + kNumXcd - 1) / kNumXcd;
  a.split_blocks = 0;
  a.total_tiles = 0;
  a.split_tiles = 0;
  a.part_o = nullptr;
  a.part_ml = nullptr;
  a.blocks = blocks;
  a.blk_ld = blk_ld;
  a.kbar = kbar;
}

hipError_t launch_sparse_select(hipStream_t st, const AttnArgs& a, int head_dim) {
  if (a.total_items == 0) return hipSuccess;
  int total = 0;
  for (int i = 0; i < a.n_streams; ++i) total += a.H * a.s[i].n_tiles;
  const dim3 g_mean((total + SEL_THR / 64 - 1) / (SEL_THR / 64));
  if (head_dim == 128) {
    hipLaunchKernelGGL((key_mean_kernel<128>), g_mean, dim3(SEL_THR), 0, st, a, total);
    hipLaunchKernelGGL((select_kernel<128>), dim3(a.total_items), dim3(SEL_THR), 0, st, a);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL((key_mean_kernel<64>), g_mean, dim3(SEL_THR), 0, st, a, total);
    hipLaunchKernelGGL((select_kernel<64>), dim3(a.total_items), dim3(SEL_THR), 0, st, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ardit
