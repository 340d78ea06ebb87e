// Host-side launchers of the gfx950 kernels (internal to libardit).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace ardit {

constexpr int kMaxStreams = 64;
// workgroups of a split attention schedule (one per CU of an MI355X)
constexpr int kAttnSplitBlocks = 256;
// attention work-item shape: 256 queries by 64-key tiles; block-sparse
// attention selects whole tiles per (stream, head, query tile)
constexpr int kAttnQTile = 256;
constexpr int kAttnKTile = 64;
// key tiles of one stream that the block selection can rank (64 KB of LDS)
constexpr int kSparseMaxTiles = 16384;

// ---------------------------------------------------------------- GEMM
enum GemmEpi : int {
  kEpiBias = 0,         // C = A W^T + b
  kEpiBiasGelu = 1,     // C = GELU_tanh(A W^T + b)
  kEpiBiasGateRes = 2,  // C = R + gate[stream(row)] * (A W^T + b)
  kEpiBiasRes = 3,      // C = R + (A W^T + b)
};

struct GemmEpiArgs {
  const bf16_t* bias = nullptr;      // [N]
  const void* res = nullptr;         // [M][ldr], bf16 or fp32 (res_f32)
  int ldr = 0;
  bool res_f32 = false;              // residual stored fp32
  bool out_f32 = false;              // C stored fp32
  const float* mod = nullptr;        // [streams][6][dim]
  const float* mod_table = nullptr;  // [6][dim]
  int gate_row = 0;
  int dim = 0;
  int rows_per_stream = 1;
};

// C[M][N] (row stride ldc, bf16 or fp32 per ep.out_f32) = epilogue(A[M][K] (lda) * W[N][K]^T
// (ldw)).  Requires N % 128 == 0, K % 64 == 0, 16-byte aligned rows.
hipError_t launch_gemm(hipStream_t st, int epi, const bf16_t* A, int lda, const bf16_t* W,
                       int ldw, void* C, int ldc, int M, int N, int K, const GemmEpiArgs& ep);

// ----------------------------------------------------------- attention
struct AttnStream {
  int32_t q_off;       // first row of the stream in q / o
  int32_t q_len;
  int32_t kv_len;      // keys [0, kv_len)
  int32_t item_begin;  // first work item of the stream
  int32_t n_qtiles;
  int32_t stream;      // row of the page table (paged) ...
  int32_t base_off;    // ... or element offset of the stream's keys (contiguous)
  int32_t T;           // tokens per page (contiguous: kv_len)
  int32_t n_tiles;     // 64-key tiles of kv_len
  int32_t main_tiles;  // split schedule: tiles [0, main_tiles) run in the item's own workgroup
  int32_t tail_begin;  // split schedule: first tail tile of the stream's items, concatenated
  int32_t n_keep;      // block-sparse: key tiles kept per item (n_tiles when dense)
  int32_t blk_off;     // block-sparse: element offset of the stream's kept-tile lists
};

struct AttnArgs {
  const bf16_t* q;
  int32_t ldq;
  bf16_t* o;
  int32_t ldo;
  const bf16_t* k;
  const bf16_t* v;
  const int32_t* page_table;
  int32_t max_frames;
  int32_t n_pages;
  int32_t T;           // page tokens (paged)
  FastDiv fT;
  int32_t H;
  float scale_log2;    // log2(e) / sqrt(d)
  int32_t n_streams;
  int32_t total_items;
  int32_t per_xcd;       // workgroups per XCD (grid = per_xcd * kNumXcd)
  int32_t xcd_begin[kNumXcd + 1];  // one workgroup per item: XCD x runs items
                                   // [xcd_begin[x], xcd_begin[x + 1]), in order
  int32_t split_blocks;  // 0: one workgroup per item; else the workgroups of a split schedule
  int32_t total_tiles;   // split: tail tiles of all items, concatenated
  int32_t split_tiles;   // split: tail tiles per spare workgroup
  float* part_o;         // [2 split_blocks][256][d] partial unnormalised outputs
  float* part_ml;        // [2 split_blocks][2][256] partial running max, denominator
  int32_t* blocks;       // block-sparse: kept tiles of item (h, qt) of stream S at
                         // blocks + S.blk_off + (h n_qtiles + qt) * ld, ascending
  int32_t blk_ld;        // row stride of those lists; 0: the stream's n_keep
  uint8_t* q8;           // FP8: E4M3 queries [rows][D] and their E8M0 scales [rows][D / 32]
  uint8_t* q8s;
  uint8_t* k8;           // FP8: per stream (base_off = first key) and head, keys [pad][d]
  uint8_t* k8s;          //      with scales [pad][d / 32], values [d][pad] with scales
  uint8_t* v8;           //      [pad / 32][d]; pad = 64 n_tiles, keys past kv_len zero
  uint8_t* v8s;
  float* qbar;           // block-sparse: fp32 mean query of every item
  float* scores;         // block-sparse: fp32 scores, n_tiles per item, streams in plan order
  AttnStream s[kMaxStreams];
};
static_assert(sizeof(AttnArgs) <= 4096, "attention arguments must fit the kernel-argument buffer");

// Splits the planned items (streams in order, n_qtiles * H items each, costing
// n_keep tiles each when sparse, else n_tiles) into kNumXcd contiguous ranges
// of equal total cost: xcd_begin and per_xcd.  Contiguous ranges keep the
// items of one head on one XCD, sharing its L2.
void balance_items_over_xcds(AttnArgs& a, bool sparse);
// Device bytes of the partial results of a split schedule.
size_t attention_split_bytes(int head_dim);
// Fills the schedule fields from the streams' lengths, ordering streams by
// decreasing key count.  split_ws (attention_split_bytes, or null to never
// split) receives the partial results when the items are cut between workgroups.
void plan_attention(AttnArgs& a, int head_dim, float* split_ws);
hipError_t launch_attention(hipStream_t st, const AttnArgs& a, int head_dim, bool paged);

// ---------------------------------------------------------- FP8 attention
// E4M3 codes and E8M0 scales of rows of bf16: each 32 consecutive columns
// share 2^e, e = floor(log2 max|x|) - 7; codes[r][c] = E4M3(x / 2^e), scales
// [r][c / 32] = e + 127.  cols % 32 == 0, ld % 8 == 0.
hipError_t launch_mx_quantize_rows(hipStream_t st, const bf16_t* x, int64_t rows, int cols, int ld,
                                   uint8_t* codes, uint8_t* scales);
// Sets base_off of the planned streams to their first key in the FP8 key and
// value buffers (64 n_tiles keys each, in the plan's order) and returns the
// bytes of k8, k8s, v8, v8s together (each part 256-byte aligned).
size_t plan_fp8_buffers(AttnArgs& a, int head_dim, uint8_t* base);
// Quantises the keys and values of the planned streams from the pages.
hipError_t launch_fp8_kv_prep(hipStream_t st, const AttnArgs& a, int head_dim);
// FP8 attention of the planned items (lists: the block-sparse lists apply).
hipError_t launch_attention_fp8(hipStream_t st, const AttnArgs& a, int head_dim, bool lists);

// ------------------------------------------------- block-sparse attention
// Key tiles kept per query tile at sparsity rho: ceil((1 - rho) n - 1e-3) in [1, n].
int sparse_keep_count(int n_tiles, float rho);
// Plans a block-sparse self-attention over paged keys: n_keep per stream from
// rho (batch order, before planning), one workgroup per item, streams ordered
// by decreasing n_keep.  blocks / blk_ld: where the selection writes its lists
// (blk_ld 0: packed per stream); qbar: [items][head_dim] and scores:
// [items][n_tiles of the item's stream] fp32 scratch.
void plan_sparse_attention(AttnArgs& a, const float* rho, int32_t* blocks, int32_t blk_ld,
                           float* qbar, float* scores);
// Numbers the items of the streams in a.s (n_qtiles, n_tiles and, when
// sparse, n_keep set): drops empty streams, orders them by decreasing cost
// (n_keep when sparse, else n_tiles), one workgroup per item, XCDs balanced.
void finish_plan(AttnArgs& a, bool sparse);
// Selection: per item the scores mean(q) . mean(k) of its key tiles and its
// n_keep best tiles, written ascending (padded with -1 up to blk_ld).
hipError_t launch_sparse_select(hipStream_t st, const AttnArgs& a, int head_dim);
// Attention of every item over its kept tiles only.
hipError_t launch_sparse_attention(hipStream_t st, const AttnArgs& a, int head_dim);

// --------------------------------------------------------- elementwise
struct RowStream {
  int32_t row_begin;
  int32_t len;
  int32_t cache_len;   // paged: logical slot of the first row
  int32_t frame_pos0;
};

struct RowStreams {
  int32_t n;
  RowStream s[kMaxStreams];
};

// x: bf16 or fp32 rows (x_f32); out: bf16 rows
hipError_t launch_adaln_norm(hipStream_t st, const void* x, bool x_f32, bf16_t* out, int N, int D,
                             const float* mod, const float* mod_table, int shift_row,
                             int scale_row, int rows_per_stream, float eps);
hipError_t launch_rms_gain(hipStream_t st, const void* in, bool in_f32, bf16_t* out, int N, int D,
                           const bf16_t* gain, float eps);

struct RopeGeom {
  int D, H, hd, T, lat_w, max_frames, n_pages;
  float eps, theta;
};
hipError_t launch_qk_norm_rope(hipStream_t st, const bf16_t* qkv, int N, const RopeGeom& g,
                               const bf16_t* g_q, const bf16_t* g_k, bf16_t* q_out,
                               bf16_t* k_pages, const int32_t* page_table, const RowStreams& rs);

// Writes rows of src (columns [col_off + h*hd, +hd) per head) into transposed
// value storage [H][hd][T].  paged: slot = cache_len + row - row_begin through
// the page table; otherwise stream b's block starts at element row_begin * D
// of dst with T = len.
hipError_t launch_v_transpose(hipStream_t st, const bf16_t* src, int ld_src, int col_off,
                              int N, int D, int H, int hd, bf16_t* dst, bool paged, int T,
                              const int32_t* page_table, int max_frames, int n_pages,
                              const RowStreams& rs);

// QK-norm + RoPE + key append and the value append of the QKV rows (q, k, v
// at columns 0, D, 2D of rows 3D wide) into paged storage: one launch when the
// 16-byte value append applies and rows are at most 2048 wide, else
// launch_qk_norm_rope then launch_v_transpose.
hipError_t launch_kv_append(hipStream_t st, const bf16_t* qkv, int N, const RopeGeom& g,
                            const bf16_t* g_q, const bf16_t* g_k, bf16_t* q_out,
                            bf16_t* k_pages, bf16_t* v_pages, const int32_t* page_table,
                            const RowStreams& rs);

// rms(src row) * gain written as [H][len][hd] per stream (block at row_begin * D).
hipError_t launch_ctx_k_layout(hipStream_t st, const bf16_t* src, int N, int D, int H, int hd,
                               const bf16_t* gain, float eps, bf16_t* dst,
                               const RowStreams& rs);

// y[b][o] = act_out(sum_k act_in(x[b][k]) W[o][k] + bias[o]); x, y fp32; W, bias bf16.
hipError_t launch_linear_small(hipStream_t st, const float* x, int B, int K, const bf16_t* W,
                               const bf16_t* bias, int O, float* y, bool silu_in);
hipError_t launch_time_sinusoid(hipStream_t st, const float* t_host, int B, float* s_out);

// ------------------------------------------------------- chunk sampler
// Rows [0, rows) of x, v, eps, out ([rows][vec_per_row * 8] bf16, stream
// b = row / rows_per_stream): out = x0_hat = x - tau_b v when tau_next_b < 0,
// else (1 - tau_next_b) x0_hat + tau_next_b eps (eps may then be null only if
// no stream of the rows has tau_next >= 0).  out may alias x.
struct SamplerArgs {
  float tau[kMaxStreams];
  float tau_next[kMaxStreams];
  int32_t rows;
  int32_t rows_per_stream;
  int32_t vec_per_row;
};
hipError_t launch_sampler(hipStream_t st, const bf16_t* x, const bf16_t* v, const bf16_t* eps,
                          bf16_t* out, const SamplerArgs& a);

// ------------------------------------------------------ measurement
// flops one wave performs per iteration of the MFMA peak kernel
double micro_mfma_flops_per_wave_iter(int dtype);
// dtype 0: bf16 (v_mfma_f32_16x16x32_bf16), 1: fp8 e4m3 (v_mfma_scale_f32_32x32x64_f8f6f4);
// workgroups of 256 threads (4 waves); sink: workgroups * 256 floats
hipError_t launch_micro_mfma(hipStream_t st, int dtype, int workgroups, int iters, float* sink);
// dst = src, bytes / 16 chunks of 16 bytes (16-byte aligned)
hipError_t launch_micro_copy(hipStream_t st, const void* src, void* dst, size_t bytes);
// reads bytes / 16 chunks of 16 bytes of src, one word per workgroup into sink
// (micro_read_workgroups(bytes) words)
int micro_read_workgroups(size_t bytes);
hipError_t launch_micro_read(hipStream_t st, const void* src, size_t bytes, uint32_t* sink);
// dst filled with a 32-bit value, bytes / 16 chunks of 16 bytes
hipError_t launch_fill(hipStream_t st, void* dst, size_t bytes, uint32_t value);

}  // namespace ardit
