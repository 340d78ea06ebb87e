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

constexpr int BQ = 256;   // queries per work item
constexpr int BKV = 64;   // keys per tile

// Key order of a 64-key tile for 16x16x32 MFMAs: row r of 16-key block kb
// holds physical key kappa(kb, r) = 32 (kb/2) + 8 (r/4) + 4 (kb%2) + r%4, so
// the S^T values a lane holds for blocks 2s and 2s+1 are exactly keys
// 32 s + 8 g .. 32 s + 8 g + 7 (g = lane / 16): the P operand of PV step s.
__device__ __forceinline__ int kappa16(int kb, int r) {
  return 32 * (kb >> 1) + 8 * (r >> 2) + 4 * (kb & 1) + (r & 3);
}
// LDS row that holds physical key p of the tile
__device__ __forceinline__ int kappa16_inv(int p) {
  const int ps = p >> 5, g = (p >> 3) & 3, hh = (p >> 2) & 1, i = p & 3;
  return 16 * (2 * ps + hh) + 4 * g + i;
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

// Tile inside one page (the common case): uniform bases plus per-lane byte
// offsets fixed for the whole kernel, so each load is scalar base + 32-bit
// vector offset with no per-tile address arithmetic.
template <int NK, int NV>
__device__ __forceinline__ void load_tile_fast(const char* kb, const char* vb,
                                               const uint32_t (&k_off)[NK],
                                               const uint32_t (&v_off)[NV], u32x4 (&rk)[NK],
                                               u32x4 (&rv)[NV]) {
#pragma unroll
  for (int i = 0; i < NK; ++i) rk[i] = *reinterpret_cast<const u32x4*>(kb + k_off[i]);
#pragma unroll
  for (int i = 0; i < NV; ++i) rv[i] = *reinterpret_cast<const u32x4*>(vb + v_off[i]);
}

template <int HD, bool PAGED, bool VEC>
__global__ __launch_bounds__(512, 1) void attn_kernel(const AttnArgs a) {
  constexpr int KLD = HD + 8;          // padded LDS row of the key tile
  constexpr int VLD = BKV + 8;         // padded LDS row of the value tile
  constexpr int NK = BKV * HD / 8 / 512;   // 16-byte key chunks per thread per tile
  constexpr int NV = HD * BKV / 8 / 512;   // 16-byte value chunks per thread per tile
  constexpr int KS = HD / 32;          // 16x16x32 MFMA k-steps over d
  constexpr int DB = HD / 16;          // 16-wide output blocks over d
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
  const int l16 = lane & 15, g = lane >> 4;

  // ---- Q fragments (B operand of S^T = K Q^T): the wave's 32 rows are two
  // 16-row blocks; lane holds row l16 of block qb, dims 32 ks + 8 g ..
  int q_local[2];
  bf16x8 qf[2][KS];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    q_local[qb] = qt * BQ + wave * 32 + 16 * qb + l16;
    const int q_row = min(q_local[qb], S.q_len - 1);
    const bf16_t* qp = a.q + static_cast<size_t>(S.q_off + q_row) * a.ldq + h * HD;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[qb][ks] = *reinterpret_cast<const bf16x8*>(qp + 32 * ks + 8 * g);
  }

  const int kv_len = S.kv_len;
  const int vstride = PAGED ? a.T : S.T;   // distance between value dims

  // K chunk i of this thread: key row k_row[i], 16-byte column k_cc
  constexpr int CPR = HD / 8;
  const int k_cc = tid % CPR;
  int k_row[NK], k_lds[NK];
#pragma unroll
  for (int i = 0; i < NK; ++i) {
    const int kr = (tid + 512 * i) / CPR;
    k_row[i] = kr;
    k_lds[i] = kappa16_inv(kr) * KLD + k_cc * 8;
  }
  // V chunk i: dim v_dd[i], keys 8 * v_kc .. + 8
  const int v_kc = tid & 7;
  int v_dd[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v_dd[i] = (tid + 512 * i) >> 3;

  u32x4 rk[2][NK], rv[2][NV];
  // byte offsets of this thread's chunks relative to the tile's first key
  uint32_t k_off[NK], v_off[NV];
#pragma unroll
  for (int i = 0; i < NK; ++i) k_off[i] = static_cast<uint32_t>((k_row[i] * HD + k_cc * 8) * 2);
#pragma unroll
  for (int i = 0; i < NV; ++i) v_off[i] = static_cast<uint32_t>((v_dd[i] * vstride + 8 * v_kc) * 2);
  f32x4 o[2][DB];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int v = 0; v < 4; ++v) o[qb][db][v] = 0.f;
  float m_run[2] = {-INFINITY, -INFINITY};   // running max (scaled, log2) of the lane's rows
  float l_run[2] = {0.f, 0.f};               // this lane's quarter of each running denominator
  const float c = a.scale_log2;

  const int ntiles = (kv_len + BKV - 1) / BKV;
  const int nfull = kv_len / BKV;   // tiles whose 64 keys are all valid

#define ARDIT_LOAD(tile, set)                                                              \
  {                                                                                        \
    const int j0_ = (tile) * BKV;                                                          \
    const TileMap tm_ = map_tile<HD, PAGED>(a, S, h, j0_);                                 \
    if ((tile) < nfull && tm_.off0 + BKV <= tm_.T && VEC)                                  \
      load_tile_fast(reinterpret_cast<const char*>(tm_.k0 + static_cast<size_t>(tm_.off0) * HD), \
                     reinterpret_cast<const char*>(tm_.v0 + tm_.off0), k_off, v_off, rk[set], rv[set]); \
    else if ((tile) < nfull)                                                               \
      load_tile<HD, VEC, false>(tm_, vstride, j0_, kv_len, k_row, k_cc, v_dd, v_kc, rk[set], rv[set]); \
    else                                                                                   \
      load_tile<HD, VEC, true>(tm_, vstride, j0_, kv_len, k_row, k_cc, v_dd, v_kc, rk[set], rv[set]);  \
  }
#define ARDIT_STORE(buf, set)                                                              \
  {                                                                                        \
    _Pragma("unroll") for (int i = 0; i < NK; ++i)                                         \
        *reinterpret_cast<u32x4*>(&sK[buf][k_lds[i]]) = rk[set][i];                        \
    _Pragma("unroll") for (int i = 0; i < NV; ++i)                                         \
        *reinterpret_cast<u32x4*>(&sV[buf][v_dd[i] * VLD + 8 * v_kc]) = rv[set][i];        \
  }

  // two tiles of loads in flight: register set (t & 1) holds tile t until stored
  ARDIT_LOAD(0, 0);
  if (ntiles > 1) ARDIT_LOAD(1, 1);
  ARDIT_STORE(0, 0);
  __syncthreads();
  for (int t0 = 0; t0 < ntiles; t0 += 2) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
    const int t = t0 + half;
    if (t < ntiles) {
    const int buf = half;
    if (t + 2 < ntiles) ARDIT_LOAD(t + 2, half);
    // S^T = K Q^T: four 16-key blocks x two 16-query blocks, 8 accumulators
    f32x4 s[4][2];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int v = 0; v < 4; ++v) s[kb][qb][v] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(&sK[buf][(kb * 16 + l16) * KLD + 32 * ks + 8 * g]);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
          s[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qb][ks], s[kb][qb], 0, 0, 0);
      }
    }
    if (t >= nfull) {   // keys past the end (last tile only)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int key = t * BKV + kappa16(kb, 4 * g + v);
          if (key >= kv_len) {
            s[kb][0][v] = -INFINITY;
            s[kb][1][v] = -INFINITY;
          }
        }
    }
    // online softmax in scaled log2 units; the running max is raised only when
    // a row's tile max exceeds it by more than 8 (p <= 2^8 otherwise), so the
    // O / l rescale is skipped on almost every tile
    bf16x8 pf[2][2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int v = 0; v < 4; ++v) mx = fmaxf(mx, s[kb][qb][v]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c;
      if (__any(mx > m_run[qb] + 8.0f)) {
        const float m_new = fmaxf(m_run[qb], mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int v = 0; v < 4; ++v) o[qb][db][v] *= alpha;
      }
      const float mr = m_run[qb];
#pragma unroll
      for (int ps = 0; ps < 2; ++ps) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = __builtin_amdgcn_exp2f(fmaf(s[2 * ps + (e >> 2)][qb][e & 3], c, -mr));
          pf[qb][ps][e] = static_cast<__bf16>(pv);
        }
        const bf16x2 one2 = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const bf16x2 pp = {pf[qb][ps][e], pf[qb][ps][e + 1]};
          l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(pp, one2, l_run[qb], false);
        }
      }
    }
    // O^T += V^T P^T: 16-dim blocks x two query blocks, 16 accumulators
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 vf =
            *reinterpret_cast<const bf16x8*>(&sV[buf][(db * 16 + l16) * VLD + 32 * ps + 8 * g]);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
          o[qb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qb][ps], o[qb][db], 0, 0, 0);
      }
    }
    if (t + 1 < ntiles) ARDIT_STORE(buf ^ 1, half ^ 1);
    __syncthreads();
    }
    }
  }
#undef ARDIT_LOAD
#undef ARDIT_STORE

#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 16, 64);
    l_tot += __shfl_xor(l_tot, 32, 64);
    const float inv = 1.0f / l_tot;
    if (q_local[qb] < S.q_len) {
      bf16_t* op = a.o + static_cast<size_t>(S.q_off + q_local[qb]) * a.ldo + h * HD;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        uint2 w;
        w.x = pack_bf16x2(o[qb][db][0] * inv, o[qb][db][1] * inv);
        w.y = pack_bf16x2(o[qb][db][2] * inv, o[qb][db][3] * inv);
        *reinterpret_cast<uint2*>(op + 16 * db + 4 * g) = w;
      }
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
  const dim3 grid(a.per_xcd * kNumXcd), block(512);
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
