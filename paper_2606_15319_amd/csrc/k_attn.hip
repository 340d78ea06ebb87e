// Flash attention of a chunk's queries over a stream's keys on gfx950 MFMA.
//
// o = softmax(q K^T / sqrt(d)) V per (stream, head) over keys [0, kv_len),
// every key visible (the chunk attends to its whole cache and to itself; the
// block-causal structure across chunks is what the cache holds).  Keys come
// either from frame pages through the stream's page table (self-attention)
// or from one contiguous per-stream block (text cross-attention); both store
// keys [H][T][d] and values transposed [H][d][T].
//
// Work item = (stream, head, 128-query tile); 4 waves x 32 query rows.  Key
// tiles of 64 are staged in LDS (keys row-major, values d-major), double
// buffered with register prefetch.  Per wave and tile:
//   S^T = K Q^T   on v_mfma_f32_32x32x16_bf16 (K from LDS, Q held in VGPRs),
//   online softmax in fp32 with exp2 (log2(e)/sqrt(d) folded into one FMA),
//   O^T += V^T P^T on the same MFMA, P taken straight from the S registers.
// Computing the transposed products puts one query row in each lane, so the
// row max/sum need only one cross-lane exchange (lanes l and l^32).  The
// keys of each 32-key block are stored in LDS in the order
//   kappa(8j + 4g + i) = 16(j/2) + 8g + 4(j%2) + i
// (j = acc group, g = lane half, i = element), which makes the S values a
// lane holds for PV step s exactly keys 16s + 8g .. 16s + 8g + 7: the P
// operand needs no shuffle and the V^T operand is one 16-byte LDS read.
#include <math.h>

#include "launch.h"

namespace ardit {

namespace {

constexpr int BQ = 128;   // queries per work item
constexpr int BKV = 64;   // keys per tile

// LDS row (within a 32-key block) that holds physical key p
__device__ __forceinline__ int kappa_inv(int p) {
  const int a = p >> 4, g = (p >> 3) & 1, b = (p >> 2) & 1, i = p & 3;
  return 8 * (2 * a + b) + 4 * g + i;
}

// physical key (within a 32-key block) of MFMA row r
__device__ __forceinline__ int kappa(int r) {
  const int j = r >> 3, g = (r >> 2) & 1, i = r & 3;
  return 16 * (j >> 1) + 8 * g + 4 * (j & 1) + i;
}

// Keys of one 64-key tile: [j0, j0 + 64) starts at offset off0 of page p0 and,
// when it runs past the page end T, continues at offset 0 of page p1.  T >= 64
// for frame pages, so a tile touches at most two pages.  Contiguous (text)
// keys behave as one unbounded page.
struct TileMap {
  const bf16_t* k0;   // key row of offset 0 in page p0 (this head)
  const bf16_t* k1;
  const bf16_t* v0;   // value column of offset 0 in page p0 (this head, dim 0)
  const bf16_t* v1;
  int off0;
  int T;
};

template <int HD, bool PAGED>
__device__ __forceinline__ TileMap map_tile(const AttnArgs& a, const AttnStream& S, int h, int j0) {
  TileMap m;
  if (PAGED) {
    const int32_t* pt = a.page_table + static_cast<size_t>(S.stream) * a.max_frames;
    const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(j0), a.fT));
    m.off0 = j0 - fr * a.T;
    m.T = a.T;
    int p0 = pt[fr];
    p0 = p0 < 0 ? 0 : (p0 >= a.n_pages ? a.n_pages - 1 : p0);
    int p1 = p0;
    // the next page is read only when it holds keys of this stream
    if (m.off0 + BKV > a.T && (fr + 1) * a.T < S.kv_len) {
      p1 = pt[fr + 1];
      p1 = p1 < 0 ? 0 : (p1 >= a.n_pages ? a.n_pages - 1 : p1);
    }
    const size_t hs = static_cast<size_t>(a.T) * HD;
    m.k0 = a.k + (static_cast<size_t>(p0) * a.H + h) * hs;
    m.k1 = a.k + (static_cast<size_t>(p1) * a.H + h) * hs;
    m.v0 = a.v + (static_cast<size_t>(p0) * a.H + h) * hs;
    m.v1 = a.v + (static_cast<size_t>(p1) * a.H + h) * hs;
  } else {
    const size_t hs = static_cast<size_t>(S.T) * HD;
    m.k0 = m.k1 = a.k + static_cast<size_t>(S.base_off) + h * hs;
    m.v0 = m.v1 = a.v + static_cast<size_t>(S.base_off) + h * hs;
    m.off0 = j0;
    m.T = 0x7fffffff;   // never crossed
  }
  return m;
}

// VEC: values of 8 consecutive keys are one aligned 16-byte load (frame pages;
// text blocks whose length is a multiple of 8).  GUARD: the tile holds keys at
// or past kv_len (last tile only); those are loaded as zeros.
template <int HD, bool VEC, bool GUARD, int NK, int NV>
__device__ __forceinline__ void load_tile(const TileMap& m, int vstride, int j0, int kv_len,
                                          const int (&k_row)[NK], int k_cc, const int (&v_dd)[NV],
                                          int v_kc, u32x4 (&rk)[NK], u32x4 (&rv)[NV]) {
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < NK; ++i) {
    const int o = m.off0 + k_row[i];
    const bf16_t* p = (o < m.T ? m.k0 + static_cast<size_t>(o) * HD
                               : m.k1 + static_cast<size_t>(o - m.T) * HD) + k_cc * 8;
    if (!GUARD || j0 + k_row[i] < kv_len)
      rk[i] = *reinterpret_cast<const u32x4*>(p);
    else
      rk[i] = zero4;
  }
  const int o = m.off0 + 8 * v_kc;
  const bf16_t* vb = o < m.T ? m.v0 + o : m.v1 + (o - m.T);
  const int jv = j0 + 8 * v_kc;
  if (VEC && (!GUARD || jv + 8 <= kv_len)) {
#pragma unroll
    for (int i = 0; i < NV; ++i)
      rv[i] = *reinterpret_cast<const u32x4*>(vb + static_cast<size_t>(v_dd[i]) * vstride);
  } else {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (jv + e < kv_len) {
          const uint32_t x = vb[static_cast<size_t>(v_dd[i]) * vstride + e];
          w[e >> 1] |= x << (16 * (e & 1));
        }
      }
      rv[i] = u32x4{w[0], w[1], w[2], w[3]};
    }
  }
}

template <int HD, bool PAGED, bool VEC>
__global__ __launch_bounds__(256, 2) void attn_kernel(const AttnArgs a) {
  constexpr int KLD = HD + 8;          // padded LDS row of the key tile
  constexpr int VLD = BKV + 8;         // padded LDS row of the value tile
  constexpr int NK = BKV * HD / 8 / 256;   // 16-byte key chunks per thread per tile
  constexpr int NV = HD * BKV / 8 / 256;   // 16-byte value chunks per thread per tile
  constexpr int KS = HD / 16;          // MFMA k-steps over d
  constexpr int DB = HD / 32;          // 32-wide output blocks over d
  __shared__ __attribute__((aligned(16))) bf16_t sK[2][BKV * KLD];
  __shared__ __attribute__((aligned(16))) bf16_t sV[2][HD * VLD];

  // ---- work item (XCD-aware: consecutive items share an XCD and its L2)
  const int pid = blockIdx.x;
  const int L = (pid % kNumXcd) * a.per_xcd + pid / kNumXcd;
  if (L >= a.total_items) return;
  int si = 0;
  for (int i = 1; i < a.n_streams; ++i)
    if (L >= a.s[i].item_begin) si = i;
  const AttnStream S = a.s[si];
  const int it = L - S.item_begin;
  const int h = it / S.n_qtiles;
  const int qt = it - h * S.n_qtiles;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;

  // ---- Q fragments (B operand of S^T = K Q^T): lane holds row l32, dims 16ks + 8g..
  const int q_local = qt * BQ + wave * 32 + l32;
  const int q_row = min(q_local, S.q_len - 1);
  const bf16_t* qp = a.q + static_cast<size_t>(S.q_off + q_row) * a.ldq + h * HD;
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qp + 16 * ks + 8 * g);

  const int kv_len = S.kv_len;
  const int vstride = PAGED ? a.T : S.T;   // distance between value dims

  // K chunk i of this thread: key row k_row[i], 16-byte column k_cc
  constexpr int CPR = HD / 8;
  const int k_cc = tid % CPR;
  int k_row[NK], k_lds[NK];
#pragma unroll
  for (int i = 0; i < NK; ++i) {
    const int kr = (tid + 256 * i) / CPR;
    k_row[i] = kr;
    k_lds[i] = ((kr & 32) | kappa_inv(kr & 31)) * KLD + k_cc * 8;
  }
  // V chunk i: dim v_dd[i], keys 8 * v_kc .. + 8
  const int v_kc = tid & 7;
  int v_dd[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v_dd[i] = (tid + 256 * i) >> 3;

  u32x4 rk[NK], rv[NV];
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float m_run = -INFINITY;   // running max (scaled, log2 units) used for this lane's row
  float l_run = 0.f;         // this lane's half of the running denominator
  const float c = a.scale_log2;

  const int ntiles = (kv_len + BKV - 1) / BKV;
  const int nfull = kv_len / BKV;   // tiles whose 64 keys are all valid

#define ARDIT_LOAD(tile)                                                                   \
  {                                                                                        \
    const int j0_ = (tile) * BKV;                                                          \
    const TileMap tm_ = map_tile<HD, PAGED>(a, S, h, j0_);                                 \
    if ((tile) < nfull)                                                                    \
      load_tile<HD, VEC, false>(tm_, vstride, j0_, kv_len, k_row, k_cc, v_dd, v_kc, rk, rv); \
    else                                                                                   \
      load_tile<HD, VEC, true>(tm_, vstride, j0_, kv_len, k_row, k_cc, v_dd, v_kc, rk, rv);  \
  }
#define ARDIT_STORE(buf)                                                                   \
  {                                                                                        \
    _Pragma("unroll") for (int i = 0; i < NK; ++i)                                         \
        *reinterpret_cast<u32x4*>(&sK[buf][k_lds[i]]) = rk[i];                             \
    _Pragma("unroll") for (int i = 0; i < NV; ++i)                                         \
        *reinterpret_cast<u32x4*>(&sV[buf][v_dd[i] * VLD + 8 * v_kc]) = rv[i];             \
  }

  ARDIT_LOAD(0);
  ARDIT_STORE(0);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) ARDIT_LOAD(t + 1);

    // S^T = K Q^T for the tile's two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) s[kb][v] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(&sK[buf][(kb * 32 + l32) * KLD + 16 * ks + 8 * g]);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[kb], 0, 0, 0);
      }
    }
    if (t >= nfull) {   // keys past the end (last tile only)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = t * BKV + kb * 32 + kappa(8 * (v >> 2) + 4 * g + (v & 3));
          if (key >= kv_len) s[kb][v] = -INFINITY;
        }
    }
    // online softmax in scaled log2 units; the running max is raised only when
    // a row's tile max exceeds it by more than 8 (p <= 2^8 otherwise), so the
    // O / l rescale is skipped on almost every tile
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kb][v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c;
    if (__any(mx > m_run + 8.0f)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
    }
    bf16x8 pf[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float pv = __builtin_amdgcn_exp2f(fmaf(s[st >> 1][8 * (st & 1) + e], c, -m_run));
        l_run += pv;
        pf[st][e] = static_cast<__bf16>(pv);
      }
    }
    // O^T += V^T P^T
#pragma unroll
    for (int st = 0; st < 4; ++st) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 vf =
            *reinterpret_cast<const bf16x8*>(&sV[buf][(db * 32 + l32) * VLD + 16 * st + 8 * g]);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[st], o[db], 0, 0, 0);
      }
    }
    if (t + 1 < ntiles) ARDIT_STORE(buf ^ 1);
    __syncthreads();
  }
#undef ARDIT_LOAD
#undef ARDIT_STORE

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  if (q_local < S.q_len) {
    bf16_t* op = a.o + static_cast<size_t>(S.q_off + q_local) * a.ldo + h * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        uint2 w;
        w.x = pack_bf16x2(o[db][4 * jj] * inv, o[db][4 * jj + 1] * inv);
        w.y = pack_bf16x2(o[db][4 * jj + 2] * inv, o[db][4 * jj + 3] * inv);
        *reinterpret_cast<uint2*>(op + 32 * db + 8 * jj + 4 * g) = w;
      }
  }
}

}  // namespace

void plan_attention(AttnArgs& a, int /*head_dim*/) {
  // order streams by decreasing key count so the longest items start first
  AttnStream tmp[kMaxStreams];
  int n = 0;
  for (int i = 0; i < a.n_streams; ++i)
    if (a.s[i].q_len > 0) tmp[n++] = a.s[i];
  for (int i = 1; i < n; ++i) {
    AttnStream x = tmp[i];
    int j = i - 1;
    while (j >= 0 && tmp[j].kv_len < x.kv_len) {
      tmp[j + 1] = tmp[j];
      --j;
    }
    tmp[j + 1] = x;
  }
  int items = 0;
  for (int i = 0; i < n; ++i) {
    tmp[i].n_qtiles = (tmp[i].q_len + BQ - 1) / BQ;
    tmp[i].item_begin = items;
    items += tmp[i].n_qtiles * a.H;
    a.s[i] = tmp[i];
  }
  a.n_streams = n;
  a.total_items = items;
  a.per_xcd = (items + kNumXcd - 1) / kNumXcd;
}

hipError_t launch_attention(hipStream_t st, const AttnArgs& a, int head_dim, bool paged) {
  if (a.total_items == 0) return hipSuccess;
  const dim3 grid(a.per_xcd * kNumXcd), block(256);
  // contiguous keys take the 16-byte value path only when every block length is a multiple of 8
  bool vec = true;
  if (!paged)
    for (int i = 0; i < a.n_streams; ++i) vec = vec && (a.s[i].T % 8 == 0);
#define ARDIT_ATTN(HD, P, V) hipLaunchKernelGGL((attn_kernel<HD, P, V>), grid, block, 0, st, a)
  if (head_dim == 128) {
    if (paged) ARDIT_ATTN(128, true, true);
    else if (vec) ARDIT_ATTN(128, false, true);
    else ARDIT_ATTN(128, false, false);
  } else if (head_dim == 64) {
    if (paged) ARDIT_ATTN(64, true, true);
    else if (vec) ARDIT_ATTN(64, false, true);
    else ARDIT_ATTN(64, false, false);
  } else {
    return hipErrorInvalidValue;
  }
#undef ARDIT_ATTN
  return hipGetLastError();
}

}  // namespace ardit
