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
// Three kernels, all on the sparse streams only:
//  - query_mean_kernel: per item, the fp32 mean of its (up to) 256 queries,
//    every row's load issued before the first add;
//  - key_score_kernel: one wave per (stream, head, key tile) reads the tile's
//    keys through the page table (16 bytes per lane, all rows in flight at
//    once), keeps their mean in registers and scores it against the mean query
//    of each query tile of that head.  It reads every key of the sparse
//    streams once, the selection's HBM cost;
//  - select_kernel: one wave per item, its order keys in registers (up to 1024
//    tiles) or LDS, finds the n_keep-th largest score by a 32-step radix search
//    over order-preserving integer keys, counting with ballots, then writes
//    the kept tiles in ascending order from two ballot scans (the second
//    resolves ties at the threshold by index).
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

// Physical page of logical frame fr of a stream, clamped into the pool.
__device__ __forceinline__ int page_of(const AttnArgs& a, const AttnStream& S, int fr) {
  const int p = a.page_table[static_cast<size_t>(S.stream) * a.max_frames + fr];
  return p < 0 ? 0 : (p >= a.n_pages ? a.n_pages - 1 : p);
}

// First score row of each stream: items in plan order, n_tiles scores each.
__device__ __forceinline__ size_t score_base(const AttnArgs& a, int si) {
  size_t off = 0;
  for (int i = 0; i < si; ++i)
    off += static_cast<size_t>(a.H) * a.s[i].n_qtiles * a.s[i].n_tiles;
  return off;
}

// Mean query of every item of the sparse streams: qbar[item][HD], fp32.
template <int HD>
__global__ __launch_bounds__(SEL_THR) void query_mean_kernel(const AttnArgs a) {
  constexpr int LPR = HD / 8;          // threads per query row, 8 dims each
  constexpr int RPS = SEL_THR / LPR;   // query rows per step
  __shared__ float red[RPS][HD];
  const int tid = threadIdx.x;
  const int L = blockIdx.x;
  int si = 0;
  for (int i = 1; i < a.n_streams; ++i)
    if (L >= a.s[i].item_begin) si = i;
  const AttnStream& S = a.s[si];
  if (S.n_keep >= S.n_tiles) return;   // dense stream
  const int it = L - S.item_begin;
  const int h = it / S.n_qtiles;
  const int qt = it - h * S.n_qtiles;
  const int r0 = qt * kAttnQTile;
  const int rows = min(kAttnQTile, S.q_len - r0);
  const int dc = tid % LPR, ro = tid / LPR;
  const bf16_t* src = a.q + static_cast<size_t>(S.q_off + r0) * a.ldq + h * HD + 8 * dc;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  // all rows of the thread issued together: one load latency per item
  uint4 v[kAttnQTile / RPS];
#pragma unroll
  for (int i = 0; i < kAttnQTile / RPS; ++i) {
    const int r = ro + i * RPS;
    v[i] = r < rows ? *reinterpret_cast<const uint4*>(src + static_cast<size_t>(r) * a.ldq)
                    : make_uint4(0u, 0u, 0u, 0u);
  }
#pragma unroll
  for (int i = 0; i < kAttnQTile / RPS; ++i) {
    float f[8];
    unpack8(v[i], f);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += f[e];
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[ro][8 * dc + e] = acc[e];
  __syncthreads();
  if (tid < HD) {
    float sum = 0.f;
#pragma unroll 8
    for (int r = 0; r < RPS; ++r) sum += red[r][tid];
    a.qbar[static_cast<size_t>(L) * HD + tid] = sum / static_cast<float>(rows);
  }
}

// One wave per (stream, head, key tile) of the sparse streams: the tile's mean
// key (fp32, kept in registers) and its score against the mean query of every
// query tile of the same stream and head.
template <int HD>
__global__ __launch_bounds__(SEL_THR) void key_score_kernel(const AttnArgs a, int total) {
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
  if (S.n_keep >= S.n_tiles) return;   // dense stream
  const int r = g - base;
  const int h = r / S.n_tiles, j = r - h * S.n_tiles;
  const int j0 = j * kAttnKTile;
  const int cnt = min(kAttnKTile, S.kv_len - j0);
  // the tile's keys start at offset off0 of frame fr and may continue on the
  // next frame's page (frames hold T >= 64 keys)
  const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(j0), a.fT));
  const int off0 = j0 - fr * a.T;
  const int p0 = page_of(a, S, fr);
  const int p1 = (off0 + kAttnKTile > a.T && (fr + 1) * a.T < S.kv_len) ? page_of(a, S, fr + 1) : p0;
  const size_t hs = static_cast<size_t>(a.T) * HD;
  const bf16_t* k0 = a.k + (static_cast<size_t>(p0) * a.H + h) * hs;
  const bf16_t* k1 = a.k + (static_cast<size_t>(p1) * a.H + h) * hs;
  const int dc = lane % LPR, ro = lane / LPR;
  uint4 v[kAttnKTile / RPS];
#pragma unroll
  for (int i = 0; i < kAttnKTile / RPS; ++i) {
    const int k = ro + i * RPS;
    const int o = off0 + k;
    const bf16_t* src = (o < a.T ? k0 + static_cast<size_t>(o) * HD
                                 : k1 + static_cast<size_t>(o - a.T) * HD) + 8 * dc;
    v[i] = k < cnt ? *reinterpret_cast<const uint4*>(src) : make_uint4(0u, 0u, 0u, 0u);
  }
  float kb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) kb[e] = 0.f;
#pragma unroll
  for (int i = 0; i < kAttnKTile / RPS; ++i) {
    float f[8];
    unpack8(v[i], f);
#pragma unroll
    for (int e = 0; e < 8; ++e) kb[e] += f[e];
  }
  // every lane ends with the sums of its 8 dims over all rows of the tile
#pragma unroll
  for (int m = LPR; m < 64; m <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) kb[e] += __shfl_xor(kb[e], m, kWave);
  const float n = static_cast<float>(cnt);
#pragma unroll
  for (int e = 0; e < 8; ++e) kb[e] = kb[e] / n;
  // row group ro scores query tiles ro, ro + RPS, ...
  const int nq = S.n_qtiles;
  const int it0 = S.item_begin + h * nq;
  float* sc = a.scores + score_base(a, si) + static_cast<size_t>(h) * nq * S.n_tiles + j;
  for (int i = ro; i < nq; i += RPS) {
    const float* qb = a.qbar + static_cast<size_t>(it0 + i) * HD + 8 * dc;
    const float4 x0 = *reinterpret_cast<const float4*>(qb);
    const float4 x1 = *reinterpret_cast<const float4*>(qb + 4);
    float p = x0.x * kb[0] + x0.y * kb[1] + x0.z * kb[2] + x0.w * kb[3] +
              x1.x * kb[4] + x1.y * kb[5] + x1.z * kb[6] + x1.w * kb[7];
#pragma unroll
    for (int m = LPR / 2; m >= 1; m >>= 1) p += __shfl_xor(p, m, kWave);
    if (dc == 0) sc[static_cast<size_t>(i) * S.n_tiles] = p;
  }
}

// Key source of the selection: order keys of up to 64 KPL tiles in registers
// (KPL per lane, lane-strided), or of any count in LDS.  Slots past n hold
// key 0, below every real key (order_key(-inf) > 0), so they are never counted.
template <int KPL>
struct RegKeys {
  uint32_t k[KPL];
  __device__ __forceinline__ void load(const float* sc, int n, int lane) {
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int j = 64 * i + lane;
      k[i] = j < n ? order_key(sc[j]) : 0u;
    }
  }
  __device__ __forceinline__ int count_ge(uint32_t c, int) const {
    int s = 0;
#pragma unroll
    for (int i = 0; i < KPL; ++i) s += __popcll(__ballot(k[i] >= c));
    return s;
  }
  __device__ __forceinline__ uint32_t at(int i) const {
    uint32_t v = 0u;
#pragma unroll
    for (int q = 0; q < KPL; ++q) v = q == i ? k[q] : v;
    return v;
  }
};

struct LdsKeys {
  uint32_t* k;
  int lane;
  __device__ __forceinline__ void load(const float* sc, int n, int ln) {
    lane = ln;
    const int slots = (n + 63) & ~63;   // the launch provides this many
#pragma unroll 8
    for (int j = lane; j < slots; j += 64) k[j] = j < n ? order_key(sc[j]) : 0u;
    __syncthreads();
  }
  __device__ __forceinline__ int count_ge(uint32_t c, int n) const {
    int s = 0;
#pragma unroll 8
    for (int b = 0; b < n; b += 64) s += __popcll(__ballot(k[b + lane] >= c));
    return s;
  }
  __device__ __forceinline__ uint32_t at(int i) const { return k[64 * i + lane]; }
};

// The n_keep best of n scores (one wave), written ascending to out.
template <class Keys>
__device__ __forceinline__ void select_top(Keys& K, int n, int nk, int lane, int32_t* out) {
  // threshold: the nk-th largest key, found bit by bit from the top; counts
  // are popcounts of ballots (scalar, no data moves between lanes)
  uint32_t thr = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = thr | (1u << bit);
    if (K.count_ge(cand, n) >= nk) thr = cand;
  }
  // taken at the threshold, lowest index first (thr + 1 cannot wrap: the
  // largest order key, that of +inf, is 0xff800000)
  const int need = nk - K.count_ge(thr + 1u, n);
  // kept tiles in ascending order, 64 candidates per step
  const uint64_t below = (1ull << lane) - 1ull;
  int carry_eq = 0, carry_keep = 0;
  for (int i = 0; 64 * i < n; ++i) {
    const uint32_t kj = K.at(i);
    const bool eq = kj == thr;
    const uint64_t me = __ballot(eq);
    const bool keep = kj > thr || (eq && carry_eq + __popcll(me & below) < need);
    const uint64_t mk = __ballot(keep);
    if (keep) out[carry_keep + __popcll(mk & below)] = 64 * i + lane;
    carry_eq += __popcll(me);
    carry_keep += __popcll(mk);
  }
}

// Per item, one wave: the n_keep best of its scores, written ascending, keys
// in registers when the stream has at most 64 KPL tiles (KPL > 0), else in
// LDS (KPL = 0).
template <int KPL>
__global__ __launch_bounds__(64) void select_kernel(const AttnArgs a) {
  extern __shared__ uint32_t lds_keys[];
  const int lane = threadIdx.x;
  const int L = blockIdx.x;
  int si = 0;
  for (int i = 1; i < a.n_streams; ++i)
    if (L >= a.s[i].item_begin) si = i;
  const AttnStream& S = a.s[si];
  const int it = L - S.item_begin;
  const int ld = a.blk_ld ? a.blk_ld : S.n_keep;
  int32_t* out = a.blocks + S.blk_off + static_cast<int64_t>(it) * ld;
  const int n = S.n_tiles, nk = S.n_keep;
  if (nk >= n) {   // dense stream: every tile, in order
    for (int t = lane; t < ld; t += 64) out[t] = t < n ? t : -1;
    return;
  }
  const float* sc = a.scores + score_base(a, si) + static_cast<size_t>(it) * n;
  if constexpr (KPL > 0) {
    RegKeys<KPL> K;
    K.load(sc, n, lane);
    select_top(K, n, nk, lane, out);
  } else {
    LdsKeys K;
    K.k = lds_keys;
    K.load(sc, n, lane);
    select_top(K, n, nk, lane, out);
  }
  for (int t = nk + lane; t < ld; t += 64) out[t] = -1;
}

}  // namespace

int sparse_keep_count(int n_tiles, float rho) {
  if (n_tiles <= 0) return 0;
  const double keep = ceil((1.0 - static_cast<double>(rho)) * n_tiles - 1e-3);
  if (!(keep >= 1.0)) return 1;
  return keep >= n_tiles ? n_tiles : static_cast<int>(keep);
}

void finish_plan(AttnArgs& a, bool sparse) {
  AttnStream tmp[kMaxStreams];
  int n = 0;
  for (int i = 0; i < a.n_streams; ++i)
    if (a.s[i].q_len > 0) tmp[n++] = a.s[i];
  // longest items first
  auto cost = [&](const AttnStream& x) { return sparse ? x.n_keep : x.n_tiles; };
  for (int i = 1; i < n; ++i) {
    AttnStream x = tmp[i];
    int j = i - 1;
    while (j >= 0 && cost(tmp[j]) < cost(x)) {
      tmp[j + 1] = tmp[j];
      --j;
    }
    tmp[j + 1] = x;
  }
  int items = 0;
  for (int i = 0; i < n; ++i) {
    tmp[i].item_begin = items;
    tmp[i].main_tiles = tmp[i].n_tiles;
    tmp[i].tail_begin = 0;
    items += tmp[i].n_qtiles * a.H;
    a.s[i] = tmp[i];
  }
  a.n_streams = n;
  a.total_items = items;
  a.split_blocks = 0;
  a.total_tiles = 0;
  a.split_tiles = 0;
  a.part_o = nullptr;
  a.part_ml = nullptr;
  balance_items_over_xcds(a, sparse);
}

void plan_sparse_attention(AttnArgs& a, const float* rho, int32_t* blocks, int32_t blk_ld,
                           float* qbar, float* scores) {
  // per stream in batch order: tiles, kept tiles, offset of its lists
  int64_t packed = 0, rows = 0;
  for (int i = 0; i < a.n_streams; ++i) {
    AttnStream& s = a.s[i];
    s.n_qtiles = (s.q_len + kAttnQTile - 1) / kAttnQTile;
    s.n_tiles = (s.kv_len + kAttnKTile - 1) / kAttnKTile;
    s.n_keep = sparse_keep_count(s.n_tiles, rho ? rho[i] : 0.f);
    s.blk_off = static_cast<int32_t>(blk_ld ? rows * blk_ld : packed);
    rows += static_cast<int64_t>(a.H) * s.n_qtiles;
    packed += static_cast<int64_t>(a.H) * s.n_qtiles * s.n_keep;
  }
  finish_plan(a, true);
  a.blocks = blocks;
  a.blk_ld = blk_ld;
  a.qbar = qbar;
  a.scores = scores;
}

hipError_t launch_sparse_select(hipStream_t st, const AttnArgs& a, int head_dim) {
  if (a.total_items == 0) return hipSuccess;
  int total = 0;
  for (int i = 0; i < a.n_streams; ++i) total += a.H * a.s[i].n_tiles;
  const dim3 g_key((total + SEL_THR / 64 - 1) / (SEL_THR / 64));
  const dim3 g_item(a.total_items);
  if (head_dim == 128) {
    hipLaunchKernelGGL((query_mean_kernel<128>), g_item, dim3(SEL_THR), 0, st, a);
    hipLaunchKernelGGL((key_score_kernel<128>), g_key, dim3(SEL_THR), 0, st, a, total);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL((query_mean_kernel<64>), g_item, dim3(SEL_THR), 0, st, a);
    hipLaunchKernelGGL((key_score_kernel<64>), g_key, dim3(SEL_THR), 0, st, a, total);
  } else {
    return hipErrorInvalidValue;
  }
  int max_tiles = 0;
  for (int i = 0; i < a.n_streams; ++i)
    if (a.s[i].n_keep < a.s[i].n_tiles) max_tiles = max(max_tiles, a.s[i].n_tiles);
  if (max_tiles <= 64 * 16) {
    hipLaunchKernelGGL(select_kernel<16>, g_item, dim3(64), 0, st, a);
  } else {
    const size_t lds = sizeof(uint32_t) * 64 * ((max_tiles + 63) / 64);
    hipLaunchKernelGGL(select_kernel<0>, g_item, dim3(64), lds, st, a);
  }
  return hipGetLastError();
}

}  // namespace ardit
