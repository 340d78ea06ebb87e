// Flash attention of a chunk's queries over a stream's keys on gfx950 MFMA.
//
// o = softmax(q K^T / sqrt(d)) V per (stream, head) over keys [0, kv_len),
// every key visible (the chunk attends to its whole cache and to itself; the
// block-causal structure across chunks is what the cache holds).  Keys come
// either from frame pages through the stream's page table (self-attention)
// or from one contiguous per-stream block (text cross-attention); both store
// keys [H][T][d] and values transposed [H][d][T].
//
// Work item = (stream, head, 256-query tile): a 512-thread workgroup, eight
// waves of 32 query rows.  Key tiles of 64 are staged in LDS (keys row-major,
// values d-major, 16-byte chunks XOR-swizzled across banks) in two buffers,
// with the global loads of the next two tiles in flight in registers.  Per
// wave and tile:
//   S^T = K Q^T   on v_mfma_f32_16x16x32_bf16 (K from LDS, Q held in VGPRs),
//   online softmax in fp32 with exp2 (log2(e)/sqrt(d) folded into one FMA),
//   O^T += V^T P^T on the same MFMA, P taken straight from the S registers.
// Computing the transposed products puts one query row in each lane column,
// so the row max needs two cross-lane exchanges and no LDS round trip.  The
// keys of a tile are stored in LDS in the order kappa16 below, which makes
// the S values a lane holds for PV step s exactly the 8 keys that lane
// supplies to the P operand: P needs no shuffle and each V^T operand is one
// 16-byte LDS read.  Fragment reads are issued four ahead of the MFMAs that
// consume them.
//
// When the items are so few that one workgroup per item would leave more than
// a quarter of the CUs idle, each item keeps the first part of its key range
// and the idle workgroups share the remaining parts; the pieces leave partial
// results (unnormalised O, running max and denominator in fp32) that a second
// kernel merges.
#include <math.h>
#include <string.h>

#include "launch.h"

namespace ardit {

namespace {

constexpr int BQ = 256;        // queries per work item
constexpr int BKV = 64;        // keys per tile
constexpr int NTHR = 512;      // threads per workgroup
constexpr int LDS_AHEAD = 4;   // fragment reads in flight ahead of the MFMAs

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
// 16-byte chunk c of LDS row r sits at chunk c ^ swz(r): 16 consecutive rows
// then cover every bank for a fixed c.  Rows of 256 bytes (keys, d = 128) use
// r % 16, rows of 128 bytes (keys d = 64, values) (r / 2) % 8.
template <int ROWB>
__device__ __forceinline__ int swz(int r) { return ROWB == 256 ? (r & 15) : ((r >> 1) & 7); }

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

// Normalised bf16 output of one item.
template <int HD>
__device__ __forceinline__ void store_output(const AttnArgs& a, const AttnStream& S, int h, int qt,
                                             const f32x4 (&o)[2][HD / 16], const float (&l_run)[2]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const float l_tot = rows4_sum(l_run[qb]);
    const float inv = 1.0f / l_tot;
    const int ql = qt * BQ + wave * 32 + 16 * qb + l16;
    if (ql < S.q_len) {
      bf16_t* op = a.o + static_cast<size_t>(S.q_off + ql) * a.ldo + h * HD;
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) {
        uint2 w;
        w.x = pack_bf16x2(o[qb][db][0] * inv, o[qb][db][1] * inv);
        w.y = pack_bf16x2(o[qb][db][2] * inv, o[qb][db][3] * inv);
        *reinterpret_cast<uint2*>(op + 16 * db + 4 * g) = w;
      }
    }
  }
}

// Partial results of a piece of a split item into slot `slot`: fp32 o, running
// max and denominator per query row of the item.
template <int HD>
__device__ __forceinline__ void store_partial(const AttnArgs& a, size_t slot,
                                              const f32x4 (&o)[2][HD / 16],
                                              const float (&m_run)[2], const float (&l_run)[2]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const float l_tot = rows4_sum(l_run[qb]);
    const int row = wave * 32 + 16 * qb + l16;
    float* po = a.part_o + (slot * BQ + row) * HD;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db)
      *reinterpret_cast<float4*>(po + 16 * db + 4 * g) =
          make_float4(o[qb][db][0], o[qb][db][1], o[qb][db][2], o[qb][db][3]);
    if (g == 0) {
      a.part_ml[slot * 2 * BQ + row] = m_run[qb];
      a.part_ml[slot * 2 * BQ + BQ + row] = l_tot;
    }
  }
}

// Runs key tiles [tb, te) of item (S, head h, query tile qt) over the
// workgroup's 256 queries, then writes the normalised output (slot < 0) or
// the partial results into slot `slot`.  LIST: positions [tb, te) index the
// tile list tl (block-sparse attention) instead of being the tiles themselves.
template <int HD, bool PAGED, bool VEC, bool LIST = false>
__device__ __forceinline__ void attn_range(const AttnArgs& a, const AttnStream& S, int h, int qt,
                                           int tb, int te, bf16_t (&sK)[2][BKV * HD],
                                           bf16_t (&sV)[2][HD * BKV], int64_t slot,
                                           const int32_t* tl = nullptr) {
  constexpr int KLD = HD;              // LDS row of the key tile
  constexpr int VLD = BKV;             // LDS row of the value tile
  constexpr int NK = BKV * HD / 8 / NTHR;   // 16-byte key chunks per thread per tile
  constexpr int NV = HD * BKV / 8 / NTHR;   // 16-byte value chunks per thread per tile
  constexpr int KS = HD / 32;          // 16x16x32 MFMA k-steps over d
  constexpr int DB = HD / 16;          // 16-wide output blocks over d
  static_assert(NK >= 1 && NV >= 1 && 4 * KS > LDS_AHEAD && 2 * DB > LDS_AHEAD, "tile shape");
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;

  // K chunk i of this thread: key row k_row[i], 16-byte column k_cc
  constexpr int CPR = HD / 8;
  const int k_cc = tid % CPR;
  int k_row[NK], k_lds[NK];
#pragma unroll
  for (int i = 0; i < NK; ++i) {
    const int kr = (tid + NTHR * i) / CPR;
    k_row[i] = kr;
    const int R = kappa16_inv(kr);
    k_lds[i] = R * KLD + 8 * (k_cc ^ swz<HD * 2>(R));
  }
  // V chunk i: dim v_dd[i], keys 8 * v_kc .. + 8
  const int v_kc = tid & 7;
  int v_dd[NV], v_lds[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v_dd[i] = (tid + NTHR * i) >> 3;
    v_lds[i] = v_dd[i] * VLD + 8 * (v_kc ^ swz<BKV * 2>(v_dd[i]));
  }
  // fragment read offsets: rows kb * 16 + l16 / db * 16 + l16 share the swizzle of l16
  int k_frag[KS], v_frag[2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) k_frag[ks] = l16 * KLD + 8 * ((4 * ks + g) ^ swz<HD * 2>(l16));
#pragma unroll
  for (int ps = 0; ps < 2; ++ps) v_frag[ps] = l16 * VLD + 8 * ((4 * ps + g) ^ swz<BKV * 2>(l16));
  const float c = a.scale_log2;

  // ---- Q fragments (B operand of S^T = K Q^T): the wave's 32 rows are two
  // 16-row blocks; lane holds row l16 of block qb, dims 32 ks + 8 g ..
  bf16x8 qf[2][KS];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int q_row = min(qt * BQ + wave * 32 + 16 * qb + l16, S.q_len - 1);
    const bf16_t* qp = a.q + static_cast<size_t>(S.q_off + q_row) * a.ldq + h * HD;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[qb][ks] = *reinterpret_cast<const bf16x8*>(qp + 32 * ks + 8 * g);
  }

  const int kv_len = S.kv_len;
  const int vstride = PAGED ? a.T : S.T;   // distance between value dims

  u32x4 rk[2][NK], rv[2][NV];
  // byte offsets of this thread's chunks relative to the tile's first key
  uint32_t k_off[NK], v_off[NV];
  f32x4 o[2][DB];
#pragma unroll
  for (int i = 0; i < NK; ++i) k_off[i] = static_cast<uint32_t>((k_row[i] * HD + k_cc * 8) * 2);
#pragma unroll
  for (int i = 0; i < NV; ++i)
    v_off[i] = static_cast<uint32_t>((v_dd[i] * vstride + 8 * v_kc) * 2);
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int v = 0; v < 4; ++v) o[qb][db][v] = 0.f;
  float m_run[2] = {-INFINITY, -INFINITY};   // running max (scaled, log2) of the lane's rows
  float l_run[2] = {0.f, 0.f};               // this lane's quarter of each running denominator

  const int nfull = kv_len / BKV;         // tiles whose 64 keys are all valid

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
      *reinterpret_cast<u32x4*>(&sV[buf][v_lds[i]]) = rv[set][i];                        \
}

  // list entries are clamped into the stream's tiles, so a corrupt list cannot
  // send the loads outside the pages
#define ARDIT_TIX(t) (LIST ? min(max(tl[(t)], 0), S.n_tiles - 1) : (t))
  // two tiles of loads in flight: register set (t - tb) & 1 holds tile t until stored
  ARDIT_LOAD(ARDIT_TIX(tb), 0);
  if (tb + 1 < te) ARDIT_LOAD(ARDIT_TIX(tb + 1), 1);
  ARDIT_STORE(0, 0);
  __syncthreads();
  for (int t0 = tb; t0 < te; t0 += 2) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int t = t0 + half;
      if (t < te) {
        const int buf = half;
        if (t + 2 < te) ARDIT_LOAD(ARDIT_TIX(t + 2), half);
        // S^T = K Q^T: four 16-key blocks x two 16-query blocks, 8 accumulators
        f32x4 s[4][2];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int v = 0; v < 4; ++v) s[kb][qb][v] = 0.f;
        {
          bf16x8 kf[KS][4];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
              kf[ks][kb] = *reinterpret_cast<const bf16x8*>(&sK[buf][kb * 16 * KLD + k_frag[ks]]);
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
              for (int qb = 0; qb < 2; ++qb)
                s[kb][qb] =
                    __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ks][kb], qf[qb][ks], s[kb][qb], 0, 0, 0);
          // schedule: LDS_AHEAD reads, then one read per pair of MFMAs
          __builtin_amdgcn_sched_group_barrier(0x100, LDS_AHEAD, 0);
#pragma unroll
          for (int i = 0; i < 4 * KS - LDS_AHEAD; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, 2 * LDS_AHEAD, 0);
        }
        const int tile = ARDIT_TIX(t);
        if (tile >= nfull) {   // keys past the end (last tile only)
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int key = tile * BKV + kappa16(kb, 4 * g + v);
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
          mx = rows4_max(mx) * c;
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
            uint32_t pw[4];
            const bf16x2 one2 = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
              const int e = 2 * e2;
              const float p0 =
                  __builtin_amdgcn_exp2f(fmaf(s[2 * ps + (e >> 2)][qb][e & 3], c, -mr));
              const float p1 = __builtin_amdgcn_exp2f(
                  fmaf(s[2 * ps + ((e + 1) >> 2)][qb][(e + 1) & 3], c, -mr));
              pw[e2] = pack_bf16x2(p0, p1);
              l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw[e2]),
                                                          one2, l_run[qb], false);
            }
            pf[qb][ps] = __builtin_bit_cast(bf16x8, u32x4{pw[0], pw[1], pw[2], pw[3]});
          }
        }
        // O^T += V^T P^T: 16-dim blocks x two query blocks, 16 accumulators
        {
          bf16x8 vf[2][DB];
#pragma unroll
          for (int ps = 0; ps < 2; ++ps)
#pragma unroll
            for (int db = 0; db < DB; ++db)
              vf[ps][db] = *reinterpret_cast<const bf16x8*>(&sV[buf][db * 16 * VLD + v_frag[ps]]);
#pragma unroll
          for (int ps = 0; ps < 2; ++ps)
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
              for (int qb = 0; qb < 2; ++qb)
                o[qb][db] =
                    __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[ps][db], pf[qb][ps], o[qb][db], 0, 0, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, LDS_AHEAD, 0);
#pragma unroll
          for (int i = 0; i < 2 * DB - LDS_AHEAD; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, 2 * LDS_AHEAD, 0);
        }
        if (t + 1 < te) ARDIT_STORE(buf ^ 1, half ^ 1);
        __syncthreads();
      }
    }
  }
#undef ARDIT_LOAD
#undef ARDIT_STORE
#undef ARDIT_TIX
  if (slot < 0)
    store_output<HD>(a, S, h, qt, o, l_run);
  else
    store_partial<HD>(a, static_cast<size_t>(slot), o, m_run, l_run);
}

// One workgroup per item.  The tile loop is the same as attn_range's; it is
// kept in the kernel itself because routing it through the inlined function
// changes the register allocation (copies of the output accumulators every
// tile) and costs about 2% on long key ranges.
template <int HD, bool PAGED, bool VEC>
__global__ __launch_bounds__(NTHR, 1) void attn_kernel(const AttnArgs a) {
  constexpr int KLD = HD;
  constexpr int VLD = BKV;
  constexpr int NK = BKV * HD / 8 / NTHR;   // 16-byte key chunks per thread per tile
  constexpr int NV = HD * BKV / 8 / NTHR;   // 16-byte value chunks per thread per tile
  constexpr int KS = HD / 32;          // 16x16x32 MFMA k-steps over d
  constexpr int DB = HD / 16;          // 16-wide output blocks over d
  __shared__ __attribute__((aligned(16))) bf16_t sK[2][BKV * KLD];
  __shared__ __attribute__((aligned(16))) bf16_t sV[2][HD * VLD];

  // ---- work item (XCD-aware: each XCD runs a contiguous range of items, so
  // the items of one head share its L2, the ranges balanced by tile count)
  const int pid = blockIdx.x;
  const int xcd = pid % kNumXcd;
  const int L = a.xcd_begin[xcd] + pid / kNumXcd;
  if (L >= a.xcd_begin[xcd + 1]) return;
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
    const int kr = (tid + NTHR * i) / CPR;
    k_row[i] = kr;
    const int R = kappa16_inv(kr);
    k_lds[i] = R * KLD + 8 * (k_cc ^ swz<HD * 2>(R));
  }
  // V chunk i: dim v_dd[i], keys 8 * v_kc .. + 8
  const int v_kc = tid & 7;
  int v_dd[NV], v_lds[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v_dd[i] = (tid + NTHR * i) >> 3;
    v_lds[i] = v_dd[i] * VLD + 8 * (v_kc ^ swz<BKV * 2>(v_dd[i]));
  }
  int k_frag[KS], v_frag[2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) k_frag[ks] = l16 * KLD + 8 * ((4 * ks + g) ^ swz<HD * 2>(l16));
#pragma unroll
  for (int ps = 0; ps < 2; ++ps) v_frag[ps] = l16 * VLD + 8 * ((4 * ps + g) ^ swz<BKV * 2>(l16));

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
        *reinterpret_cast<u32x4*>(&sV[buf][v_lds[i]]) = rv[set][i];                        \
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
    {
      bf16x8 kf[KS][4];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          kf[ks][kb] = *reinterpret_cast<const bf16x8*>(&sK[buf][kb * 16 * KLD + k_frag[ks]]);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            s[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ks][kb], qf[qb][ks], s[kb][qb], 0, 0, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, LDS_AHEAD, 0);
#pragma unroll
      for (int i = 0; i < 4 * KS - LDS_AHEAD; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * LDS_AHEAD, 0);
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
      mx = rows4_max(mx) * c;
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
        // keys 2 e2, 2 e2 + 1 of the step packed into one register, which both
        // feeds the P operand and is summed into the denominator (a plain
        // array: filling a 4-word vector element by element here compiled to
        // dot products that all read its first word)
        uint32_t pw[4];
        const bf16x2 one2 = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const int e = 2 * e2;
          const float p0 = __builtin_amdgcn_exp2f(fmaf(s[2 * ps + (e >> 2)][qb][e & 3], c, -mr));
          const float p1 =
              __builtin_amdgcn_exp2f(fmaf(s[2 * ps + ((e + 1) >> 2)][qb][(e + 1) & 3], c, -mr));
          pw[e2] = pack_bf16x2(p0, p1);
          l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw[e2]), one2,
                                                      l_run[qb], false);
        }
        pf[qb][ps] = __builtin_bit_cast(bf16x8, u32x4{pw[0], pw[1], pw[2], pw[3]});
      }
    }
    // O^T += V^T P^T: 16-dim blocks x two query blocks, 16 accumulators
    {
      bf16x8 vf[2][DB];
#pragma unroll
      for (int ps = 0; ps < 2; ++ps)
#pragma unroll
        for (int db = 0; db < DB; ++db)
          vf[ps][db] = *reinterpret_cast<const bf16x8*>(&sV[buf][db * 16 * VLD + v_frag[ps]]);
#pragma unroll
      for (int ps = 0; ps < 2; ++ps)
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            o[qb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[ps][db], pf[qb][ps], o[qb][db], 0, 0, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, LDS_AHEAD, 0);
#pragma unroll
      for (int i = 0; i < 2 * DB - LDS_AHEAD; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * LDS_AHEAD, 0);
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
    const float l_tot = rows4_sum(l_run[qb]);
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


// Split schedule: each item runs its first main_tiles tiles in its own
// workgroup; the remaining workgroups take equal ranges of the concatenated tails.
template <int HD, bool PAGED, bool VEC>
__global__ __launch_bounds__(NTHR, 1) void attn_split_kernel(const AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t sK[2][BKV * HD];
  __shared__ __attribute__((aligned(16))) bf16_t sV[2][HD * BKV];

  const int pid = blockIdx.x;
  const int xcd = pid % kNumXcd, j = pid / kNumXcd;

  // XCD x runs items [pre, pre + nx), then its share of the tail ranges
  const int ipx = a.total_items / kNumXcd, irem = a.total_items % kNumXcd;
  const int nx = ipx + (xcd < irem ? 1 : 0);
  const int pre = xcd * ipx + min(xcd, irem);
  if (j < nx) {
    const int gi = pre + j;
    int si = 0;
    for (int i = 1; i < a.n_streams; ++i)
      if (gi >= a.s[i].item_begin) si = i;
    const AttnStream S = a.s[si];
    const int item = gi - S.item_begin;
    const int h = item / S.n_qtiles, qt = item - h * S.n_qtiles;
    attn_range<HD, PAGED, VEC>(a, S, h, qt, 0, S.main_tiles, sK, sV,
                               S.main_tiles == S.n_tiles ? -1 : gi);
    return;
  }
  const int r = a.per_xcd * xcd + j - (pre + nx);   // tail range
  if (r >= a.split_blocks - a.total_items) return;
  int pos = r * a.split_tiles;
  const int end = min(pos + a.split_tiles, a.total_tiles);
  while (pos < end) {
    int si = 0;
    for (int i = 1; i < a.n_streams; ++i)
      if (pos >= a.s[i].tail_begin) si = i;
    const AttnStream S = a.s[si];
    const int tl = S.n_tiles - S.main_tiles;
    const int rel = pos - S.tail_begin;
    const int item = rel / tl;
    const int tb = S.main_tiles + (rel - item * tl);
    const int te = min(S.n_tiles, tb + (end - pos));
    pos += te - tb;
    const int h = item / S.n_qtiles, qt = item - h * S.n_qtiles;
    // piece (range r, item i) -> slot total_items + i + r: items increase within a
    // range and the next range starts at the last one's last item, so slots differ
    attn_range<HD, PAGED, VEC>(a, S, h, qt, tb, te, sK, sV,
                               static_cast<int64_t>(a.total_items) + S.item_begin + item + r);
  }
}

// Combines the partial results of the items that a split schedule cut:
// o = sum_j 2^(m_j - M) O_j / sum_j 2^(m_j - M) l_j, M = max_j m_j, over the
// item's main part (slot = item) and the pieces of its tail [w0, w1) of the
// concatenated tails, held by ranges w0 / W .. (w1 - 1) / W (slot
// total_items + item + range).
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(const AttnArgs a) {
  constexpr int TPR = HD / 4;          // threads per row, 4 dims each
  constexpr int RPB = 256 / TPR;       // rows per workgroup
  const int gi = blockIdx.x / (BQ / RPB);
  const int row = (blockIdx.x % (BQ / RPB)) * RPB + threadIdx.x / TPR;
  int si = 0;
  for (int i = 1; i < a.n_streams; ++i)
    if (gi >= a.s[i].item_begin) si = i;
  const AttnStream& S = a.s[si];
  const int item = gi - S.item_begin;
  const int tl = S.n_tiles - S.main_tiles;
  if (tl == 0) return;   // written whole by its main part
  const int w0 = S.tail_begin + item * tl, w1 = w0 + tl;
  const int W = a.split_tiles;
  const int b_lo = w0 / W, b_hi = (w1 - 1) / W;
  const int h = item / S.n_qtiles;
  const int qt = item - h * S.n_qtiles;
  const int d4 = threadIdx.x % TPR;
  const int ql = qt * BQ + row;
  if (ql >= S.q_len) return;
  {
    float M = a.part_ml[static_cast<size_t>(gi) * 2 * BQ + row];
    for (int b = b_lo; b <= b_hi; ++b) {
      const size_t slot = static_cast<size_t>(a.total_items) + gi + b;
      M = fmaxf(M, a.part_ml[slot * 2 * BQ + row]);
    }
    float l = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int b = b_lo - 1; b <= b_hi; ++b) {
      const size_t slot = b < b_lo ? static_cast<size_t>(gi) : static_cast<size_t>(a.total_items) + gi + b;
      const float wgt = __builtin_amdgcn_exp2f(a.part_ml[slot * 2 * BQ + row] - M);
      l += wgt * a.part_ml[slot * 2 * BQ + BQ + row];
      const float4 p = *reinterpret_cast<const float4*>(a.part_o + (slot * BQ + row) * HD + 4 * d4);
      acc.x += wgt * p.x;
      acc.y += wgt * p.y;
      acc.z += wgt * p.z;
      acc.w += wgt * p.w;
    }
    const float inv = 1.0f / l;
    uint2 w;
    w.x = pack_bf16x2(acc.x * inv, acc.y * inv);
    w.y = pack_bf16x2(acc.z * inv, acc.w * inv);
    *reinterpret_cast<uint2*>(a.o + static_cast<size_t>(S.q_off + ql) * a.ldo + h * HD + 4 * d4) = w;
  }
}

// Block-sparse attention: one workgroup per item over the item's kept tiles,
// read from its list (written by the block selection).
template <int HD>
__global__ __launch_bounds__(NTHR, 1) void attn_sparse_kernel(const AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t sK[2][BKV * HD];
  __shared__ __attribute__((aligned(16))) bf16_t sV[2][HD * BKV];
  const int pid = blockIdx.x;
  const int xcd = pid % kNumXcd;
  const int L = a.xcd_begin[xcd] + pid / kNumXcd;
  if (L >= a.xcd_begin[xcd + 1]) return;
  int si = 0;
  for (int i = 1; i < a.n_streams; ++i)
    if (L >= a.s[i].item_begin) si = i;
  const AttnStream S = a.s[si];
  const int it = L - S.item_begin;
  const int h = it / S.n_qtiles;
  const int qt = it - h * S.n_qtiles;
  const int ld = a.blk_ld ? a.blk_ld : S.n_keep;
  const int32_t* tl = a.blocks + S.blk_off + static_cast<int64_t>(it) * ld;
  attn_range<HD, true, true, true>(a, S, h, qt, 0, S.n_keep, sK, sV, -1, tl);
}

}  // namespace

hipError_t launch_sparse_attention(hipStream_t st, const AttnArgs& a, int head_dim) {
  if (a.total_items == 0) return hipSuccess;
  const dim3 grid(a.per_xcd * kNumXcd);
  if (head_dim == 128)
    hipLaunchKernelGGL((attn_sparse_kernel<128>), grid, dim3(NTHR), 0, st, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL((attn_sparse_kernel<64>), grid, dim3(NTHR), 0, st, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

namespace {

constexpr int kCusPerXcd = 32;   // MI355X: 8 XCDs of 32 CUs

// Item costs in plan order as runs: the items of one stream are contiguous
// and cost the same (its key tiles, or its kept tiles when sparse), so run r
// covers items [begin[r], begin[r + 1]) at cost[r].
struct CostRuns {
  int n;
  int32_t begin[kMaxStreams + 1];
  int32_t cost[kMaxStreams];
};

// List schedule of items [i, n) (plan order) onto one XCD's CUs, each CU
// taking the next item when it frees (how the dispatcher hands out an XCD's
// workgroups in order, one 512-thread workgroup per CU).  Returns the first
// item past those that finish by makespan M; with share > 0 it also stops once
// the XCD's cost reaches share.
int fill_xcd(const CostRuns& c, int i, int n, int64_t M, int64_t share) {
  int64_t fin[kCusPerXcd] = {};
  int64_t taken = 0;
  int r = 0;
  while (r + 1 < c.n && i >= c.begin[r + 1]) ++r;
  for (; i < n; ++i) {
    while (i >= c.begin[r + 1]) ++r;
    const int64_t cost = c.cost[r];
    if (share > 0 && taken >= share) break;
    int k = 0;
    for (int u = 1; u < kCusPerXcd; ++u) k = fin[u] < fin[k] ? u : k;
    if (fin[k] + cost > M) break;
    fin[k] += cost;
    taken += cost;
  }
  return i;
}

int64_t runs_cost(const CostRuns& c, int i0, int i1) {
  int64_t t = 0;
  for (int r = 0; r < c.n; ++r) {
    const int lo = c.begin[r] > i0 ? c.begin[r] : i0;
    const int hi = c.begin[r + 1] < i1 ? c.begin[r + 1] : i1;
    if (hi > lo) t += static_cast<int64_t>(hi - lo) * c.cost[r];
  }
  return t;
}

// Contiguous split of the items over the XCDs that minimises the makespan of
// the slowest XCD under list scheduling (binary search on the makespan), with
// the items spread evenly by cost where that makespan allows.
void split_by_makespan(const CostRuns& c, int n, int64_t total, int32_t* begin) {
  int64_t lo = 0, hi = total;
  for (int r = 0; r < c.n; ++r)
    if (c.begin[r + 1] > c.begin[r]) lo = c.cost[r] > lo ? c.cost[r] : lo;
  auto feasible = [&](int64_t M) {
    int i = 0;
    for (int x = 0; x < kNumXcd && i < n; ++x) i = fill_xcd(c, i, n, M, 0);
    return i == n;
  };
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (feasible(mid)) hi = mid;
    else lo = mid + 1;
  }
  // even spread first, bounded by the makespan; the greedy fill if that fails
  for (int pass = 0; pass < 2; ++pass) {
    int i = 0;
    int64_t done = 0;
    begin[0] = 0;
    for (int x = 0; x < kNumXcd; ++x) {
      int64_t share = 0;
      if (pass == 0 && x < kNumXcd - 1) {
        share = (total - done) / (kNumXcd - x);
        share = share > 0 ? share : 1;
      }
      const int e = fill_xcd(c, i, n, lo, share);
      done += runs_cost(c, i, e);
      i = e;
      begin[x + 1] = i;
    }
    if (i == n) return;
  }
}

// The last plan's XCD split, reused while the item costs repeat (every layer
// and denoising step of a chunk has the same geometry).  Fixed-size, so
// planning makes no host allocation.
struct XcdSplitCache {
  int32_t key[2 * kMaxStreams + 1];
  int key_len = -1;
  int32_t begin[kNumXcd + 1];
};

}  // namespace

void balance_items_over_xcds(AttnArgs& a, bool sparse) {
  // per-stream item runs in plan order, also the cache key
  thread_local XcdSplitCache cache;
  int32_t key[2 * kMaxStreams + 1];
  int key_len = 0;
  key[key_len++] = a.H;
  CostRuns runs;
  runs.n = a.n_streams;
  int64_t total = 0;
  for (int i = 0; i < a.n_streams; ++i) {
    const int32_t c = sparse ? a.s[i].n_keep : a.s[i].n_tiles;
    key[key_len++] = a.s[i].n_qtiles;
    key[key_len++] = c;
    runs.begin[i] = a.s[i].item_begin;
    runs.cost[i] = c;
    total += static_cast<int64_t>(a.s[i].n_qtiles) * a.H * c;
  }
  const int n = a.total_items;
  runs.begin[a.n_streams] = n;
  const bool same = key_len == cache.key_len &&
                    memcmp(key, cache.key, sizeof(int32_t) * static_cast<size_t>(key_len)) == 0;
  if (!same) {
    if (n <= 65536) {
      split_by_makespan(runs, n, total, cache.begin);
    } else {   // very large batches: equal item counts
      for (int x = 0; x <= kNumXcd; ++x)
        cache.begin[x] = static_cast<int32_t>(static_cast<int64_t>(n) * x / kNumXcd);
    }
    memcpy(cache.key, key, sizeof(int32_t) * static_cast<size_t>(key_len));
    cache.key_len = key_len;
  }
  int most = 0;
  for (int x = 0; x <= kNumXcd; ++x) a.xcd_begin[x] = cache.begin[x];
  for (int x = 0; x < kNumXcd; ++x)
    most = a.xcd_begin[x + 1] - a.xcd_begin[x] > most ? a.xcd_begin[x + 1] - a.xcd_begin[x] : most;
  a.per_xcd = most;
}

size_t attention_split_bytes(int head_dim) {
  return static_cast<size_t>(2) * kAttnSplitBlocks * BQ * (head_dim + 2) * sizeof(float);
}

void plan_attention(AttnArgs& a, int head_dim, float* split_ws) {
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
  int64_t work = 0;
  for (int i = 0; i < n; ++i) {
    tmp[i].n_qtiles = (tmp[i].q_len + BQ - 1) / BQ;
    tmp[i].n_tiles = (tmp[i].kv_len + BKV - 1) / BKV;
    tmp[i].main_tiles = tmp[i].n_tiles;
    tmp[i].tail_begin = 0;
    tmp[i].item_begin = items;
    items += tmp[i].n_qtiles * a.H;
    work += static_cast<int64_t>(tmp[i].n_qtiles) * a.H * tmp[i].n_tiles;
  }
  a.n_streams = n;
  a.total_items = items;
  a.total_tiles = 0;
  a.split_blocks = 0;
  a.split_tiles = 0;
  a.part_o = nullptr;
  a.part_ml = nullptr;
  // Split when the items fit one round of workgroups but leave more than a
  // quarter of them idle: every item keeps its first W tiles (W = the even
  // share of all tiles per workgroup) and the idle workgroups take equal ranges
  // of the remaining tails.  Items of one head still run their main parts in
  // step, sharing key tiles through L2.  The tail ranges cost more per tile
  // (short segments, partial writes, the merge), which outweighs the gain when
  // few workgroups are idle.
  const int spare = kAttnSplitBlocks - items;
  if (split_ws && items > 0 && spare * 4 > kAttnSplitBlocks &&
      work >= 8 * static_cast<int64_t>(kAttnSplitBlocks) && work < (static_cast<int64_t>(1) << 30)) {
    const int W = static_cast<int>((work + kAttnSplitBlocks - 1) / kAttnSplitBlocks);
    int64_t tails = 0;
    for (int i = 0; i < n; ++i) {
      tmp[i].main_tiles = min(tmp[i].n_tiles, W);
      tmp[i].tail_begin = static_cast<int32_t>(tails);
      tails += static_cast<int64_t>(tmp[i].n_qtiles) * a.H * (tmp[i].n_tiles - tmp[i].main_tiles);
    }
    if (tails > 0) {
      a.split_blocks = kAttnSplitBlocks;
      a.total_tiles = static_cast<int32_t>(tails);
      a.split_tiles = static_cast<int32_t>((tails + spare - 1) / spare);
      a.part_o = split_ws;
      a.part_ml = split_ws + static_cast<size_t>(2) * kAttnSplitBlocks * BQ * head_dim;
      a.per_xcd = kAttnSplitBlocks / kNumXcd;
    } else {
      for (int i = 0; i < n; ++i) tmp[i].main_tiles = tmp[i].n_tiles;
    }
  }
  for (int i = 0; i < n; ++i) a.s[i] = tmp[i];
  if (!a.split_blocks) balance_items_over_xcds(a, false);
}

template <int HD, bool P, bool V>
static void launch_attn_t(hipStream_t st, const AttnArgs& a, dim3 grid) {
  if (a.split_blocks) {
    hipLaunchKernelGGL((attn_split_kernel<HD, P, V>), grid, dim3(NTHR), 0, st, a);
    hipLaunchKernelGGL((attn_merge_kernel<HD>), dim3(a.total_items * (BQ / (256 / (HD / 4)))),
                       dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL((attn_kernel<HD, P, V>), grid, dim3(NTHR), 0, st, a);
  }
}

hipError_t launch_attention(hipStream_t st, const AttnArgs& a, int head_dim, bool paged) {
  if (a.total_items == 0) return hipSuccess;
  const dim3 grid(a.per_xcd * kNumXcd);
  // contiguous keys take the 16-byte value path only when every block length is a multiple of 8
  bool vec = true;
  if (!paged)
    for (int i = 0; i < a.n_streams; ++i) vec = vec && (a.s[i].T % 8 == 0);
  if (head_dim == 128) {
    if (paged) launch_attn_t<128, true, true>(st, a, grid);
    else if (vec) launch_attn_t<128, false, true>(st, a, grid);
    else launch_attn_t<128, false, false>(st, a, grid);
  } else if (head_dim == 64) {
    if (paged) launch_attn_t<64, true, true>(st, a, grid);
    else if (vec) launch_attn_t<64, false, true>(st, a, grid);
    else launch_attn_t<64, false, false>(st, a, grid);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ardit
