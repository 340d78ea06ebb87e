// FP8 attention on gfx950 (the quantisation knob Q of a fidelity configuration).
//
// Attention is computed on OCP E4M3 operands with power-of-two (E8M0) scales
// per 32 elements along each product's reduction axis (paper, Section 2.1
// fidelity knobs and Section 5: activations are quantised online inside
// attention, weights never):
//   q, k  per token and head, 32 consecutive dims;
//   v     per head and dim, 32 consecutive keys of the logical sequence;
//   p     per query row, 32 consecutive keys, after the exponential.
// A block's exponent is e = floor(log2 max|x|) - 7, so the block maximum lands
// in [128, 256) and every element converts without saturation; the codes are
// round-to-nearest-even E4M3 of x / 2^e.  Logits, the running maximum and the
// softmax denominator (a sum of the unquantised weights) stay fp32.
//
// A pre-pass quantises q (rows of the packed activations) and, per stream
// and head, the keys (row-major, [pad][d]) and values (dim-major, [d][pad])
// read through the page table, into the workspace; pad = 64 n_tiles and keys
// past kv_len are zero.  The attention kernel then works on 256-query items
// like the bf16 kernel (8 waves of 32 rows), with 64-key tiles of E4M3 in LDS,
// on v_mfma_scale_f32_32x32x64_f8f6f4, whose E8M0 scale operands apply the
// block scales in hardware:
//   S^T (64 keys x 32 queries) = K Q^T: 2 key blocks x 2 dim steps of 64;
//   O^T (128 dims x 32 queries) += V^T P^T: 4 dim blocks, k = the 64 keys.
// The MFMA's k layout (measured on the device): lane m + 32 h holds, for row
// (or column) m, k = 16 h + 0..15 in its bytes 0..15 and k = 32 + 16 h + 0..15
// in bytes 16..31, and lane m + 32 b supplies the scale of k-block b.  Keys
// are stored in LDS in the order that makes the 32 S values a lane holds
// exactly the 32 P bytes it supplies to the PV product, so the weights are
// quantised in registers: a block's maximum needs one exchange with lane
// n ^ 32, which holds the block's other 16 keys.  LDS rows have their 16-byte
// chunks XOR-swizzled by row so that the 16 lanes served together read 16
// different slots of the 64 banks: key rows of 128 bytes by (row / 2) % 8,
// value rows of 64 bytes by (row / 4) % 4 (swizzling by row % 8 and
// (row / 2) % 4 left two-way conflicts: 7% slower).
#include <math.h>

#include "launch.h"

namespace ardit {

namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int F8_BQ = 256;     // queries per item
constexpr int F8_BKV = 64;     // keys per tile
constexpr int F8_NTHR = 512;   // threads per workgroup
constexpr int F8_HD = 128;     // head dim of the FP8 kernel

// e = floor(log2(amax)) - 7, clamped to [-127, 127]; -127 for amax == 0.
__device__ __forceinline__ int mx_exponent(float amax) {
  const uint32_t b = __float_as_uint(amax);
  int fl;
  if (b & 0x7f800000u) {
    fl = static_cast<int>((b >> 23) & 0xff) - 127;
  } else {
    if ((b & 0x7fffffu) == 0u) return -127;
    fl = -118 - static_cast<int>(__clz(b & 0x7fffffu));   // subnormal: 31 - clz(m) - 149
  }
  const int e = fl - 7;
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// 2^-e as a float (e <= 120 for any finite fp32 block maximum, so 127 - e >= 7)
__device__ __forceinline__ float mx_inv_scale(int e) {
  return __uint_as_float(static_cast<uint32_t>(127 - e) << 23);
}

// floor(log2 amax) - 7 clamped to [-127, 127], -127 for 0, without branches
// (the exponent instruction handles subnormal inputs); amax >= 0 and finite
__device__ __forceinline__ int mx_exponent_nb(float amax) {
  const int e = __builtin_amdgcn_frexp_expf(amax) - 8;
  return amax > 0.f ? min(max(e, -127), 127) : -127;
}

// max of x over lanes l and l ^ 32 (one swap of the wave's halves, no LDS)
__device__ __forceinline__ float half_pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// four floats (|x| < 256) -> four E4M3 bytes, first value in the low byte (the
// first conversion's untouched half is overwritten by the second, so it starts
// from a's bits instead of a zeroed register)
__device__ __forceinline__ uint32_t pack4_e4m3(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, __float_as_int(a), false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return static_cast<uint32_t>(w);
}

// 8 bf16 values, block-quantised with the other lanes of their 4-lane group
// (32 consecutive elements): codes of this lane's 8 and the block's exponent.
__device__ __forceinline__ uint2 quantize8(const float (&f)[8], int& e_out) {
  float m = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = fmaxf(m, fabsf(f[i]));
  m = fmaxf(m, __shfl_xor(m, 1, 64));
  m = fmaxf(m, __shfl_xor(m, 2, 64));
  const int e = mx_exponent(m);
  const float s = mx_inv_scale(e);
  e_out = e;
  return make_uint2(pack4_e4m3(f[0] * s, f[1] * s, f[2] * s, f[3] * s),
                    pack4_e4m3(f[4] * s, f[5] * s, f[6] * s, f[7] * s));
}

// ------------------------------------------------------------- pre-pass
// Rows of bf16: one lane per 8 columns, one wave per 512 columns of a row.
__global__ __launch_bounds__(256) void mx_quant_rows_kernel(const bf16_t* x, int64_t rows, int cols,
                                                            int ld, uint8_t* codes,
                                                            uint8_t* scales) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int segs = (cols + 511) / 512;
  const int64_t row = wave / segs;
  if (row >= rows) return;
  const int c0 = static_cast<int>(wave - row * segs) * 512 + 8 * lane;
  const bool in = c0 < cols;
  float f[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (in) unpack8(*reinterpret_cast<const uint4*>(x + row * ld + c0), f);
  int e;
  const uint2 q = quantize8(f, e);
  if (in) {
    *reinterpret_cast<uint2*>(codes + row * cols + c0) = q;
    if ((lane & 3) == 0) scales[row * (cols / 32) + c0 / 32] = static_cast<uint8_t>(e + 127);
  }
}

__device__ __forceinline__ int page_at(const AttnArgs& a, const AttnStream& S, int fr) {
  const int p = a.page_table[static_cast<size_t>(S.stream) * a.max_frames + fr];
  return p < 0 ? 0 : (p >= a.n_pages ? a.n_pages - 1 : p);
}

// Keys and values of one (stream, head, 64-key tile) per 256-thread
// workgroup: each thread quantises 4 chunks of 8 key dims and 4 chunks of 8
// keys of one value dim, every load issued before the first conversion.  A
// 32-element block is 4 consecutive chunks, held by 4 consecutive lanes.
__global__ __launch_bounds__(256) void fp8_kv_prep_kernel(const AttnArgs a, int total_tiles) {
  const int tid = threadIdx.x;
  int g = blockIdx.x;
  if (g >= total_tiles) return;
  int si = 0, before = 0;
  for (int i = 0; i < a.n_streams; ++i) {
    const int n = a.H * a.s[i].n_tiles;
    if (g < before + n) {
      si = i;
      break;
    }
    before += n;
  }
  const AttnStream& S = a.s[si];
  g -= before;
  const int h = g / S.n_tiles, t = g - h * S.n_tiles;
  const int pad = F8_BKV * S.n_tiles;
  const int j0 = F8_BKV * t;
  // the tile starts at offset off0 of frame fr and may continue on the next page
  const int fr = static_cast<int>(fdiv(static_cast<uint32_t>(j0), a.fT));
  const int off0 = j0 - fr * a.T;
  const int p0 = page_at(a, S, fr);
  const int p1 = (off0 + F8_BKV > a.T && (fr + 1) * a.T < S.kv_len) ? page_at(a, S, fr + 1) : p0;
  const size_t head0 = static_cast<size_t>(a.H) * S.base_off + static_cast<size_t>(h) * pad;
  uint4 kraw[4], vraw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = tid + 256 * i;
    // key chunk: key kk of the tile, dims 8 kc .. + 8
    const int kk = ch >> 4, kc = ch & 15;
    const int ok = off0 + kk;
    const bf16_t* ksrc = a.k + ((static_cast<size_t>(ok < a.T ? p0 : p1) * a.H + h) * a.T +
                                (ok < a.T ? ok : ok - a.T)) * F8_HD + 8 * kc;
    kraw[i] = j0 + kk < S.kv_len ? *reinterpret_cast<const uint4*>(ksrc) : make_uint4(0u, 0u, 0u, 0u);
    // value chunk: dim vdm, keys 8 vc .. + 8 of the tile
    const int vdm = ch >> 3, vc = ch & 7;
    const int ov = off0 + 8 * vc;
    const bf16_t* vsrc = a.v + ((static_cast<size_t>(ov < a.T ? p0 : p1) * a.H + h) * F8_HD + vdm) * a.T +
                         (ov < a.T ? ov : ov - a.T);
    const int jv = j0 + 8 * vc;
    if (jv + 8 <= S.kv_len) {
      vraw[i] = *reinterpret_cast<const uint4*>(vsrc);
    } else {
      uint32_t w[4] = {0u, 0u, 0u, 0u};
      for (int e = 0; e < 8 && jv + e < S.kv_len; ++e)
        w[e >> 1] |= static_cast<uint32_t>(vsrc[e]) << (16 * (e & 1));
      vraw[i] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = tid + 256 * i;
    float f[8];
    int e;
    unpack8(kraw[i], f);
    const uint2 kq = quantize8(f, e);
    const int kk = ch >> 4, kc = ch & 15;
    *reinterpret_cast<uint2*>(a.k8 + (head0 + j0 + kk) * F8_HD + 8 * kc) = kq;
    if ((kc & 3) == 0) a.k8s[(head0 + j0 + kk) * (F8_HD / 32) + kc / 4] = static_cast<uint8_t>(e + 127);
    unpack8(vraw[i], f);
    const uint2 vq = quantize8(f, e);
    const int vdm = ch >> 3, vc = ch & 7;
    *reinterpret_cast<uint2*>(a.v8 + head0 * F8_HD + static_cast<size_t>(vdm) * pad + j0 + 8 * vc) = vq;
    if ((vc & 3) == 0)
      a.v8s[(head0 / 32 + j0 / 32 + vc / 4) * F8_HD + vdm] = static_cast<uint8_t>(e + 127);
  }
}

// ------------------------------------------------------------ attention
// LDS row of physical key p of a tile: key block b = p / 32 holds in MFMA row
// r = 8 (i / 4) + 4 h + i % 4 the key 32 b + 16 h + i.
__device__ __forceinline__ int f8_lds_row(int p) {
  const int b = p >> 5, h = (p >> 4) & 1, i = p & 15;
  return 32 * b + 8 * (i >> 2) + 4 * h + (i & 3);
}

template <bool LIST>
__global__ __launch_bounds__(F8_NTHR, 1) void attn_fp8_kernel(const AttnArgs a) {
  constexpr int KROW = F8_HD;    // bytes per key row
  constexpr int VROW = F8_BKV;   // bytes per value (dim) row
  __shared__ __attribute__((aligned(16))) uint8_t sK[2][F8_BKV * KROW];
  __shared__ __attribute__((aligned(16))) uint8_t sV[2][F8_HD * VROW];
  __shared__ __attribute__((aligned(16))) uint32_t sKs[2][F8_BKV];     // 4 scale bytes per LDS key row
  __shared__ __attribute__((aligned(16))) uint8_t sVs[2][2 * F8_HD];    // [key block][dim]

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
  const int32_t* tl = nullptr;
  int te = S.n_tiles;
  if (LIST) {
    const int ld = a.blk_ld ? a.blk_ld : S.n_keep;
    tl = a.blocks + S.blk_off + static_cast<int64_t>(it) * ld;
    te = S.n_keep;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hh = lane >> 5;

  // ---- Q fragments (B operand of S^T = K Q^T) and their scales
  i32x8 qf[2];
  int qsc[2];
  {
    const int q_row = min(qt * F8_BQ + wave * 32 + n, S.q_len - 1);
    const size_t row = static_cast<size_t>(S.q_off + q_row);
    const uint8_t* qp = a.q8 + row * a.ldq + h * F8_HD;
    const uint8_t* qs = a.q8s + row * (a.ldq / 32) + h * (F8_HD / 32);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const uint4 c0 = *reinterpret_cast<const uint4*>(qp + 64 * ks + 16 * hh);
      const uint4 c1 = *reinterpret_cast<const uint4*>(qp + 64 * ks + 32 + 16 * hh);
      qf[ks] = i32x8{static_cast<int>(c0.x), static_cast<int>(c0.y), static_cast<int>(c0.z),
                     static_cast<int>(c0.w), static_cast<int>(c1.x), static_cast<int>(c1.y),
                     static_cast<int>(c1.z), static_cast<int>(c1.w)};
      qsc[ks] = qs[2 * ks + hh];
    }
  }

  // ---- staging: one 16-byte chunk of keys and one of values per thread
  const int pad = F8_BKV * S.n_tiles;
  const size_t head0 = static_cast<size_t>(a.H) * S.base_off + static_cast<size_t>(h) * pad;
  const uint8_t* kg = a.k8 + head0 * F8_HD;
  const uint8_t* ksg = a.k8s + head0 * (F8_HD / 32);
  const uint8_t* vg = a.v8 + head0 * F8_HD;
  const uint8_t* vsg = a.v8s + (head0 / 32) * F8_HD;
  const int kr = tid >> 3, kc = tid & 7;
  const int kR = f8_lds_row(kr);
  const int k_lds = kR * KROW + ((kc ^ ((kR >> 1) & 7)) << 4);
  const int vd = tid >> 2, vc = tid & 3;
  const int v_lds = vd * VROW + ((vc ^ ((vd >> 2) & 3)) << 4);
  const float c = a.scale_log2;
  const int kv_len = S.kv_len;

  uint4 rk0, rk1, rv0, rv1, rs0, rs1;
  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m_run = -INFINITY;
  float l_run = 0.f;

#define F8_TIX(t) (LIST ? min(max(tl[(t)], 0), S.n_tiles - 1) : (t))
#define F8_LOAD(tile, SET)                                                                     \
  {                                                                                            \
    const int t_ = (tile);                                                                     \
    rk##SET = *reinterpret_cast<const uint4*>(kg + static_cast<size_t>(F8_BKV * t_ + kr) * F8_HD + 16 * kc); \
    rv##SET = *reinterpret_cast<const uint4*>(vg + static_cast<size_t>(vd) * pad + F8_BKV * t_ + 16 * vc);  \
    if (tid < 16)                                                                              \
      rs##SET = *reinterpret_cast<const uint4*>(ksg + static_cast<size_t>(F8_BKV * t_) * 4 + 16 * tid);     \
    else if (tid < 32)                                                                         \
      rs##SET = *reinterpret_cast<const uint4*>(vsg + static_cast<size_t>(2 * t_) * F8_HD + 16 * (tid - 16)); \
  }
#define F8_STORE(BUF, SET)                                                                     \
  {                                                                                            \
    *reinterpret_cast<uint4*>(&sK[BUF][k_lds]) = rk##SET;                                      \
    *reinterpret_cast<uint4*>(&sV[BUF][v_lds]) = rv##SET;                                      \
    if (tid < 16) {                                                                            \
      sKs[BUF][f8_lds_row(4 * tid)] = rs##SET.x;                                               \
      sKs[BUF][f8_lds_row(4 * tid + 1)] = rs##SET.y;                                           \
      sKs[BUF][f8_lds_row(4 * tid + 2)] = rs##SET.z;                                           \
      sKs[BUF][f8_lds_row(4 * tid + 3)] = rs##SET.w;                                           \
    } else if (tid < 32) {                                                                     \
      *reinterpret_cast<uint4*>(&sVs[BUF][16 * (tid - 16)]) = rs##SET;                         \
    }                                                                                          \
  }

  // one 64-key tile from LDS buffer buf: scores, online softmax, P in E4M3, PV
  auto tile_step = [&](const int t, const int buf) {
    // ---- S^T = K Q^T: two 32-key blocks, two 64-dim steps
    // all K fragments read first (two 16-byte halves each), then the four MFMAs
    i32x8 kf[2][2];
    uint32_t ksc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int R = 32 * kb + n;
      ksc[kb] = sKs[buf][R];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int c0 = 4 * ks + hh, c1 = 4 * ks + 2 + hh;
        const i32x4 a0 = *reinterpret_cast<const i32x4*>(&sK[buf][R * KROW + ((c0 ^ ((R >> 1) & 7)) << 4)]);
        const i32x4 a1 = *reinterpret_cast<const i32x4*>(&sK[buf][R * KROW + ((c1 ^ ((R >> 1) & 7)) << 4)]);
        kf[kb][ks] = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int sa = static_cast<int>((ksc[kb] >> (8 * (2 * ks + hh))) & 0xffu);
        s[kb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf[kb][ks], qf[ks], s[kb], 0, 0, 0, sa,
                                                                0, qsc[ks]);
      }
    }
    // V fragments for the PV product, read now so the softmax hides their latency
    i32x8 vf[4];
    int vsc[4];
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      const int R = 32 * db + n;
      const int c0 = hh, c1 = 2 + hh;
      const i32x4 v0 = *reinterpret_cast<const i32x4*>(&sV[buf][R * VROW + ((c0 ^ ((R >> 2) & 3)) << 4)]);
      const i32x4 v1 = *reinterpret_cast<const i32x4*>(&sV[buf][R * VROW + ((c1 ^ ((R >> 2) & 3)) << 4)]);
      vf[db] = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
      vsc[db] = sVs[buf][hh * F8_HD + R];
    }
    __builtin_amdgcn_sched_barrier(0);
    const int tile = F8_TIX(t);
    if (F8_BKV * tile + F8_BKV > kv_len) {   // keys past the end (last tile only)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (F8_BKV * tile + 32 * kb + 16 * hh + i >= kv_len) s[kb][i] = -INFINITY;
    }
    // ---- online softmax (scaled log2 units, lazy rescale by more than 2^8).
    // Each 32-key block's largest score gives its largest weight (exp2 is
    // monotonic), hence the block's E4M3 exponent before any weight exists;
    // the exponent is folded into the exp2 argument, so the weights come out
    // already divided by their block scale.
    float sb0 = -INFINITY, sb1 = -INFINITY;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      sb0 = fmaxf(sb0, s[0][i]);
      sb1 = fmaxf(sb1, s[1][i]);
    }
    sb0 = half_pair_max(sb0);
    sb1 = half_pair_max(sb1);
    const float mx = fmaxf(sb0, sb1) * c;
    if (__any(mx > m_run + 8.0f)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
    }
    const int e0 = mx_exponent_nb(__builtin_amdgcn_exp2f(fmaf(sb0, c, -m_run)));
    const int e1 = mx_exponent_nb(__builtin_amdgcn_exp2f(fmaf(sb1, c, -m_run)));
    const float m0 = m_run + static_cast<float>(e0), m1 = m_run + static_cast<float>(e1);
    float ps0 = 0.f, ps1 = 0.f;   // block sums of the scaled weights
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float p0 = __builtin_amdgcn_exp2f(fmaf(s[0][i], c, -m0));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(s[1][i], c, -m1));
      s[0][i] = p0;
      s[1][i] = p1;
      ps0 += p0;
      ps1 += p1;
    }
    l_run = fmaf(ps0, __uint_as_float(static_cast<uint32_t>(127 + e0) << 23),
                 fmaf(ps1, __uint_as_float(static_cast<uint32_t>(127 + e1) << 23), l_run));
    // ---- P in E4M3, one scale per 32-key block (this lane supplies block hh's)
    i32x8 pf;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      pf[w] = static_cast<int>(pack4_e4m3(s[0][4 * w], s[0][4 * w + 1], s[0][4 * w + 2], s[0][4 * w + 3]));
      pf[4 + w] = static_cast<int>(pack4_e4m3(s[1][4 * w], s[1][4 * w + 1], s[1][4 * w + 2], s[1][4 * w + 3]));
    }
    const int psc = (hh ? e1 : e0) + 127;
    // ---- O^T += V^T P^T: four 32-dim blocks
#pragma unroll
    for (int db = 0; db < 4; ++db)
      o[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vf[db], pf, o[db], 0, 0, 0, vsc[db], 0,
                                                              psc);
  };

  // two tiles of loads in flight: register set t & 1 holds tile t until stored
  F8_LOAD(F8_TIX(0), 0);
  if (1 < te) F8_LOAD(F8_TIX(1), 1);
  F8_STORE(0, 0);
  __syncthreads();
  for (int t0 = 0; t0 < te; t0 += 2) {
    {
      const int t = t0;
      if (t + 2 < te) F8_LOAD(F8_TIX(t + 2), 0);
      tile_step(t, 0);
      if (t + 1 < te) F8_STORE(1, 1);
      __syncthreads();
    }
    if (t0 + 1 < te) {
      const int t = t0 + 1;
      if (t + 2 < te) F8_LOAD(F8_TIX(t + 2), 1);
      tile_step(t, 1);
      if (t + 1 < te) F8_STORE(0, 0);
      __syncthreads();
    }
  }
#undef F8_LOAD
#undef F8_STORE
#undef F8_TIX
  // ---- normalised bf16 output: lane holds dims 32 db + 8 g + 4 hh + 0..3 of its query
  const auto lp = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run), __float_as_uint(l_run),
                                                    false, false);
  const float l_tot = __uint_as_float(lp[0]) + __uint_as_float(lp[1]);
  const float inv = 1.0f / l_tot;
  const int ql = qt * F8_BQ + wave * 32 + n;
  if (ql < S.q_len) {
    bf16_t* op = a.o + static_cast<size_t>(S.q_off + ql) * a.ldo + h * F8_HD;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 w;
        w.x = pack_bf16x2(o[db][4 * g] * inv, o[db][4 * g + 1] * inv);
        w.y = pack_bf16x2(o[db][4 * g + 2] * inv, o[db][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(op + 32 * db + 8 * g + 4 * hh) = w;
      }
  }
}

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

hipError_t launch_mx_quantize_rows(hipStream_t st, const bf16_t* x, int64_t rows, int cols, int ld,
                                   uint8_t* codes, uint8_t* scales) {
  if (rows == 0) return hipSuccess;
  if (cols % 32 != 0 || ld % 8 != 0 || cols <= 0) return hipErrorInvalidValue;
  const int64_t waves = rows * ((cols + 511) / 512);
  hipLaunchKernelGGL(mx_quant_rows_kernel, dim3(static_cast<unsigned>((waves + 3) / 4)), dim3(256),
                     0, st, x, rows, cols, ld, codes, scales);
  return hipGetLastError();
}

size_t plan_fp8_buffers(AttnArgs& a, int head_dim, uint8_t* base) {
  int64_t keys = 0;
  for (int i = 0; i < a.n_streams; ++i) {
    a.s[i].base_off = static_cast<int32_t>(keys);
    keys += static_cast<int64_t>(F8_BKV) * a.s[i].n_tiles;
  }
  const size_t kb = static_cast<size_t>(a.H) * keys * head_dim;
  const size_t sb = kb / 32;
  if (base) {
    a.k8 = base;
    a.k8s = base + up256(kb);
    a.v8 = a.k8s + up256(sb);
    a.v8s = a.v8 + up256(kb);
  }
  return 2 * (up256(kb) + up256(sb));
}

hipError_t launch_fp8_kv_prep(hipStream_t st, const AttnArgs& a, int head_dim) {
  if (a.total_items == 0) return hipSuccess;
  if (head_dim != F8_HD) return hipErrorInvalidValue;
  int tiles = 0;
  for (int i = 0; i < a.n_streams; ++i) tiles += a.H * a.s[i].n_tiles;
  hipLaunchKernelGGL(fp8_kv_prep_kernel, dim3(tiles), dim3(256), 0, st, a, tiles);
  return hipGetLastError();
}

hipError_t launch_attention_fp8(hipStream_t st, const AttnArgs& a, int head_dim, bool lists) {
  if (a.total_items == 0) return hipSuccess;
  if (head_dim != F8_HD) return hipErrorInvalidValue;
  const dim3 grid(a.per_xcd * kNumXcd);
  if (lists)
    hipLaunchKernelGGL(attn_fp8_kernel<true>, grid, dim3(F8_NTHR), 0, st, a);
  else
    hipLaunchKernelGGL(attn_fp8_kernel<false>, grid, dim3(F8_NTHR), 0, st, a);
  return hipGetLastError();
}

}  // namespace ardit
