// bf16 GEMM with fp32 accumulation on gfx950 MFMA, C = epilogue(A W^T).
//
// A [M][K] and W [N][K] are both K-contiguous (every projection of the block
// stores its weight [out][in]).  A 512-thread workgroup computes a 128 x 256
// or a 192 x 256 tile (the height picked per shape, see choose_bm); its eight
// waves own 64 x 64 or 96 x 64 pieces (2 x 4) as 4 x 4 or 6 x 4 blocks of
// v_mfma_f32_16x16x32_bf16.  K advances in steps of 64 through LDS stages
// (three for the 128-row tile, two for the 192-row one) filled by direct
// global->LDS loads (global_load_lds_dwordx4): the loads of a later step are
// in flight while step k is multiplied, and the loaded bytes never pass
// through registers.  The loads are issued from inline asm:
// the compiler's own form makes every later LDS read wait for all of them,
// which would leave no load in flight; the kernel waits on the vector-memory
// counter itself before the barrier that publishes a stage.  Each LDS row
// is 128 bytes with its eight 16-byte chunks XOR-swizzled by (row / 2) % 8,
// so the fragment reads of 16 consecutive rows spread over all banks.  The
// fragment reads run half a step ahead of the MFMAs: the second 32-wide half
// of step k is read under the first half's MFMAs and the first half of step
// k+1 under the second half's, so the LDS reads never stand alone between
// barriers (8% faster than reading a step's fragments up front).
//
// The MFMA computes C^T = W A^T: W rows feed the A operand and A rows the B
// operand, so each lane ends up owning one output row m and four
// consecutive columns n per block.  The epilogue applies bias / GELU /
// gate * y + residual in fp32, staging the tile through LDS so that the
// residual is read and C written one contiguous row at a time.
// Rows past M read a clamped row and store nothing; an N ending on a
// half tile (N % 256 == 128) clamps W rows the same way.
#include <type_traits>

#include "launch.h"

namespace ardit {

namespace {

// 16 bytes per lane from base + off to LDS byte address m0 + 16 * lane.  base
// and m0 are the same for every lane of the wave and live in scalar
// registers, so issuing a load costs no vector instruction.
__device__ __forceinline__ void lds_dma16(const char* base, uint32_t off, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %2"
               :: "v"(off), "s"(m0), "s"(base) : "m0");
}

// A pointer the compiler may hold in vector registers, made scalar (it is the
// same in every lane).  readfirstlane returns int, so each half goes through
// uint32_t before it is widened: a low half with bit 31 set must not be
// sign-extended into the high half.
__device__ __forceinline__ const char* uniform_ptr(const void* p) {
  const uint64_t b = reinterpret_cast<uint64_t>(p);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b)));
  return reinterpret_cast<const char*>((static_cast<uint64_t>(hi) << 32) | lo);
}

constexpr int BN = 256, BK = 64, NT = 512;
constexpr int NWAVES = NT / 64;
constexpr int WN = 64, NB = WN / 16;
constexpr int NWN = BN / WN;
constexpr int ROW_BYTES = BK * 2;
constexpr int W_BYTES = BN * ROW_BYTES;
constexpr int W_INS = W_BYTES / 1024 / NWAVES;
constexpr int GROUP_M = 8;   // m-tiles per raster group (L2 reuse of W columns)
constexpr int CROW = BN * 4 + 16;   // epilogue: fp32 tile row in LDS, padded by 16 bytes

// Tile height BM: 128 rows with three LDS stages, or 192 rows with two (the
// waves then own 96 x 64 pieces, 6 x 4 blocks; fragment reads per MFMA fall
// by a sixth and the tile count suits other shapes).  The epilogue stages
// the fp32 tile in passes of PASS_ROWS rows that fit the stages' LDS.
template <int BM_>
struct Cfg {
  static constexpr int BM = BM_;
  static constexpr int STAGES = BM_ == 128 ? 3 : 2;
  static constexpr int WM = BM / 2, MB = WM / 16;
  static constexpr int A_BYTES = BM * ROW_BYTES;
  static constexpr int STAGE_BYTES = A_BYTES + W_BYTES;
  static constexpr int A_INS = A_BYTES / 1024 / NWAVES;   // 1 KB load instructions per wave per K step
  static constexpr int PASS_ROWS = BM * CROW <= STAGES * STAGE_BYTES ? BM : BM / 2;
  static constexpr int NPASS = BM / PASS_ROWS;
  static constexpr int RB = PASS_ROWS / (NWAVES * 2);     // rows per batch and wave, two batches a pass
  static_assert(A_INS * NWAVES * 1024 == A_BYTES && W_INS * NWAVES * 1024 == W_BYTES, "");
  static_assert(STAGES * STAGE_BYTES <= 160 * 1024, "LDS");
  static_assert(PASS_ROWS * CROW <= STAGES * STAGE_BYTES && PASS_ROWS % 16 == 0, "C tile in LDS");
  static_assert(RB * NWAVES * 2 == PASS_ROWS, "row batches");
};

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

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
template <int BM_, int EPI, typename ResT, typename OutT>
__global__ __launch_bounds__(NT, 1) void gemm_kernel(const bf16_t* __restrict__ A, int lda,
                                                     const bf16_t* __restrict__ W, int ldw,
                                                     OutT* __restrict__ C, int ldc, int M,
                                                     int N, int K, const GemmEpiArgs ep,
                                                     int tiles_m, int tiles_n, int per_xcd) {
  using G = Cfg<BM_>;
  constexpr int BM = G::BM, STAGES = G::STAGES, WM = G::WM, MB = G::MB;
  constexpr int A_BYTES = G::A_BYTES, STAGE_BYTES = G::STAGE_BYTES, A_INS = G::A_INS;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[STAGES * STAGE_BYTES];

  // XCD-aware tile order: consecutive logical tiles land on one XCD (shared L2)
  const int p = blockIdx.x;
  const int L = (p % kNumXcd) * per_xcd + p / kNumXcd;
  if (L >= tiles_m * tiles_n) return;
  const int group = GROUP_M * tiles_n;
  const int g0 = (L / group) * GROUP_M;
  const int gm = min(tiles_m - g0, GROUP_M);
  const int tm = g0 + (L % group) % gm;
  const int tn = (L % group) / gm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int wm = wave / NWN, wn = wave % NWN;

  // Load instruction j of this wave fills the 8 LDS rows 8 (wave * INS + j) .. + 7: lane i
  // writes slot i % 8 of row 8 (...) + i / 8, which holds chunk (i % 8) ^ swz(row).  The
  // tile's first row (scalar) plus a per-lane byte offset fixed for the whole K loop.
  const char* a_base = uniform_ptr(A + static_cast<size_t>(tm) * BM * lda);
  const char* w_base = uniform_ptr(W + static_cast<size_t>(tn) * BN * ldw);
  uint32_t a_off[A_INS], w_off[W_INS];
#pragma unroll
  for (int j = 0; j < A_INS; ++j) {
    const int r = 8 * (wave * A_INS + j) + (lane >> 3);
    const int c = (lane & 7) ^ swz(r);
    a_off[j] = static_cast<uint32_t>((min(tm * BM + r, M - 1) - tm * BM) * lda * 2 + c * 16);
  }
#pragma unroll
  for (int j = 0; j < W_INS; ++j) {
    const int r = 8 * (wave * W_INS + j) + (lane >> 3);
    const int c = (lane & 7) ^ swz(r);
    w_off[j] = static_cast<uint32_t>((min(tn * BN + r, N - 1) - tn * BN) * ldw * 2 + c * 16);
  }
  // LDS byte addresses of this wave's first 1 KB blocks of the A and W parts
  // of stage 0 (the wave index made scalar: it is the same in every lane)
  const uint32_t wave_s = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(wave));
  const uint32_t smem_s = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const char*)smem))));
  const uint32_t lds_a = smem_s + wave_s * (A_INS * 1024u);
  const uint32_t lds_w = smem_s + A_BYTES + wave_s * (W_INS * 1024u);
  auto issue = [&](int kt) {
    const uint32_t so = static_cast<uint32_t>((kt % STAGES) * STAGE_BYTES);
    const int koff = kt * ROW_BYTES;
#pragma unroll
    for (int j = 0; j < A_INS; ++j) lds_dma16(a_base + koff, a_off[j], lds_a + so + 1024u * j);
#pragma unroll
    for (int j = 0; j < W_INS; ++j) lds_dma16(w_base + koff, w_off[j], lds_w + so + 1024u * j);
  };

  f32x4 acc[MB][NB];
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[a][b][v] = 0.f;

  const int nk = K / BK;
  // fragments of one 32-wide half of a K step from a stage
  auto read_half = [&](const unsigned char* st, int kk, bf16x8 (&fa)[MB], bf16x8 (&fw)[NB])
      __attribute__((always_inline)) {
    const bf16_t* cA = reinterpret_cast<const bf16_t*>(st);
    const bf16_t* cW = reinterpret_cast<const bf16_t*>(st + A_BYTES);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int r = WN * wn + 16 * nb + l16;
      fw[nb] = *reinterpret_cast<const bf16x8*>(&cW[r * BK + 8 * ((4 * kk + g) ^ swz(r))]);
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int r = WM * wm + 16 * mb + l16;
      fa[mb] = *reinterpret_cast<const bf16x8*>(&cA[r * BK + 8 * ((4 * kk + g) ^ swz(r))]);
    }
  };
  auto mma = [&](const bf16x8 (&fa)[MB], const bf16x8 (&fw)[NB]) __attribute__((always_inline)) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[nb], fa[mb], acc[mb][nb], 0, 0, 0);
  };
  // the MB * NB MFMAs of one half issued in MB + NB groups, each followed by
  // one fragment read of the next half (groups of 3 first, then of 2)
  constexpr int NREAD = MB + NB, EXTRA = MB * NB - 2 * NREAD;
  static_assert(EXTRA >= 0 && EXTRA <= NREAD, "MFMA groups");
  auto interleave = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < EXTRA; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#pragma unroll
    for (int i = EXTRA; i < NREAD; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
  };

  // The fragment reads run one half step ahead of the MFMAs: the second half
  // of step kt is read under the first half's MFMAs, and the first half of
  // step kt+1 under the second half's, after the barrier that publishes stage
  // kt+1.  That barrier also closes every read of stage kt.  With three
  // stages, step kt+2 is requested at the top of step kt (into the slot of
  // step kt-1); with two, right after that barrier (into the slot of step kt).
  // Either way a request has one and a half or one full step to land.
  issue(0);
  if (STAGES == 3 && nk > 1) {
    issue(1);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(A_INS + W_INS));
  } else {
    asm volatile("s_waitcnt vmcnt(0)");
  }
  __syncthreads();
  if (STAGES == 2 && nk > 1) issue(1);
  bf16x8 fa0[MB], fw0[NB], fa1[MB], fw1[NB];
  read_half(smem, 0, fa0, fw0);
  // one K step on stage S (a constant: the loop runs the stages in turn, so
  // every LDS address is a register plus an immediate)
  auto step = [&](int kt, auto s_c) __attribute__((always_inline)) {
    constexpr int S = decltype(s_c)::value;
    if (STAGES == 3 && kt + 2 < nk) issue(kt + 2);
    read_half(smem + S * STAGE_BYTES, 1, fa1, fw1);
    mma(fa0, fw0);
    interleave();
    if (kt + 1 < nk) {
      if (STAGES == 3 && kt + 2 < nk) {
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(A_INS + W_INS));
      } else {
        asm volatile("s_waitcnt vmcnt(0)");
      }
      __syncthreads();
      if (STAGES == 2 && kt + 2 < nk) issue(kt + 2);
      read_half(smem + ((S + 1) % STAGES) * STAGE_BYTES, 0, fa0, fw0);
    }
    mma(fa1, fw1);
    interleave();
  };
  static_assert(STAGES == 2 || STAGES == 3, "the K loop is unrolled over the stages");
  for (int kt = 0; kt < nk; kt += STAGES) {
    step(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < nk) step(kt + 1, std::integral_constant<int, 1>{});
    if constexpr (STAGES == 3) {
      if (kt + 2 < nk) step(kt + 2, std::integral_constant<int, 2>{});
    }
  }

  // epilogue through LDS (free once every wave has read its last fragments),
  // in passes of PASS_ROWS tile rows: the waves holding a pass's rows write
  // y = acc + bias (GELU applied) for their row and four columns of every
  // block into a row-major fp32 tile, and the workgroup then walks the pass
  // one row per wave, each lane taking four consecutive columns, so the
  // residual is read and C written as whole contiguous rows.  The residual
  // and gate loads of a wave's rows go out in two batches, the first before
  // the pass is staged and the second before the first is used, so their
  // latency hides behind the staging and the stores.  Rows are padded by 16
  // bytes: the 16 lanes of one write then cover all 64 banks.
  constexpr int PASS_ROWS = G::PASS_ROWS, NPASS = G::NPASS, RB = G::RB;
  constexpr bool HAS_RES = EPI == kEpiBiasGateRes || EPI == kEpiBiasRes;
  const bool cols_in = tn * BN + WN * wn < N;   // (a tile may end on a half tile)
  const int cl = 4 * lane;
  const bool lane_in = tn * BN + cl < N;
  const int n0 = min(tn * BN + cl, N - 4);      // lanes past N load a valid column, store nothing
  float res[2][RB][4], gmod[2][RB][4];
  auto load_batch = [&](int pass, int b) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int m = min(tm * BM + PASS_ROWS * pass + wave + NWAVES * (RB * b + i), M - 1);
      if (HAS_RES)
        load4(static_cast<const ResT*>(ep.res) + static_cast<size_t>(m) * ep.ldr + n0, res[b][i]);
      if (EPI == kEpiBiasGateRes)
        load4(ep.mod + (static_cast<size_t>(m / ep.rows_per_stream) * 6 + ep.gate_row) * ep.dim + n0,
              gmod[b][i]);
    }
  };
  float gt4[4] = {0.f, 0.f, 0.f, 0.f};
  if (EPI == kEpiBiasGateRes) load4(ep.mod_table + static_cast<size_t>(ep.gate_row) * ep.dim + n0, gt4);
  float bias[NB][4];
  if (cols_in) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) load4(ep.bias + tn * BN + WN * wn + 16 * nb + 4 * g, bias[nb]);
  }
#pragma unroll
  for (int pass = 0; pass < NPASS; ++pass) {
    load_batch(pass, 0);
    __syncthreads();
    if (cols_in) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int r = WM * wm + 16 * mb + l16 - PASS_ROWS * pass;
        if (NPASS > 1 && (WM * wm + 16 * mb) / PASS_ROWS != pass) continue;   // (wave-uniform)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int c = WN * wn + 16 * nb + 4 * g;
          float y[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) y[e] = acc[mb][nb][e] + bias[nb][e];
          if (EPI == kEpiBiasGelu) {
#pragma unroll
            for (int e = 0; e < 4; ++e) y[e] = gelu_tanh(y[e]);
          }
          *reinterpret_cast<float4*>(smem + r * CROW + c * 4) = make_float4(y[0], y[1], y[2], y[3]);
        }
      }
    }
    __syncthreads();
    load_batch(pass, 1);
    if (lane_in) {
#pragma unroll
      for (int b = 0; b < 2; ++b) {
#pragma unroll
        for (int i = 0; i < RB; ++i) {
          const int rr = wave + NWAVES * (RB * b + i);
          const int m = tm * BM + PASS_ROWS * pass + rr;
          if (m < M) {
            const float4 t = *reinterpret_cast<const float4*>(smem + rr * CROW + cl * 4);
            float y[4] = {t.x, t.y, t.z, t.w};
            if (EPI == kEpiBiasGateRes) {
#pragma unroll
              for (int e = 0; e < 4; ++e) y[e] = res[b][i][e] + (gmod[b][i][e] + gt4[e]) * y[e];
            } else if (EPI == kEpiBiasRes) {
#pragma unroll
              for (int e = 0; e < 4; ++e) y[e] = res[b][i][e] + y[e];
            }
            store4(C + static_cast<size_t>(m) * ldc + n0, y);
          }
        }
      }
    }
  }
}

}  // namespace

// Tile height for an M x N product.  Both heights give bit-identical C (the
// same MFMA sequence per output element), so the choice is speed only: the
// 192-row tile is taken when it needs clearly fewer rounds of 256
// workgroups, counting one of its rounds as 1.38 rounds of 128-row tiles
// (1.5 times the work at 92% of the time per unit of work).
static int choose_bm(int M, int N) {
  const long tn = (N + BN - 1) / BN;
  const long r128 = ((M + 127) / 128 * tn + 255) / 256;
  const long r192 = ((M + 191) / 192 * tn + 255) / 256;
  return 1.38 * static_cast<double>(r192) < static_cast<double>(r128) ? 192 : 128;
}

template <int BM_, int EPI, typename ResT, typename OutT>
static void launch_t(hipStream_t st, const bf16_t* A, int lda, const bf16_t* W, int ldw, void* C,
                     int ldc, int M, int N, int K, const GemmEpiArgs& ep) {
  const int tiles_m = (M + BM_ - 1) / BM_, tiles_n = (N + BN - 1) / BN;
  const int total = tiles_m * tiles_n;
  const int per_xcd = (total + kNumXcd - 1) / kNumXcd;
  hipLaunchKernelGGL((gemm_kernel<BM_, EPI, ResT, OutT>), dim3(per_xcd * kNumXcd), dim3(NT), 0, st,
                     A, lda, W, ldw, static_cast<OutT*>(C), ldc, M, N, K, ep, tiles_m, tiles_n,
                     per_xcd);
}

template <int EPI, typename ResT, typename OutT>
static void launch_bm(hipStream_t st, const bf16_t* A, int lda, const bf16_t* W, int ldw, void* C,
                      int ldc, int M, int N, int K, const GemmEpiArgs& ep) {
  if (choose_bm(M, N) == 192)
    launch_t<192, EPI, ResT, OutT>(st, A, lda, W, ldw, C, ldc, M, N, K, ep);
  else
    launch_t<128, EPI, ResT, OutT>(st, A, lda, W, ldw, C, ldc, M, N, K, ep);
}

hipError_t launch_gemm(hipStream_t st, int epi, const bf16_t* A, int lda, const bf16_t* W,
                       int ldw, void* C, int ldc, int M, int N, int K, const GemmEpiArgs& ep) {
  if (M == 0) return hipSuccess;
  if (N % 128 != 0 || K % BK != 0 || K == 0) return hipErrorInvalidValue;
  const bool rf = ep.res_f32, of = ep.out_f32;
#define ARDIT_GEMM(E, R, O) launch_bm<E, R, O>(st, A, lda, W, ldw, C, ldc, M, N, K, ep)
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
