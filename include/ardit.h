/*
 * ardit.h -- C ABI of the AR-DiT chunk-denoise block library (libardit.so).
 *
 * What is computed.  An autoregressive diffusion transformer generates video
 * one chunk of latent frames at a time; every denoising step of a chunk runs
 * the transformer stack on the chunk's tokens, each block attending over the
 * stream's KV cache of earlier chunks plus the chunk itself, and the chunk is
 * appended to that cache once generated (paper, Section 2.1, "AR-DiT").  The
 * cache is paged at latent-frame granularity behind a logical page table, and
 * different streams hold different cache lengths (Section 3.2, the State
 * Plane paragraph and its footnote; Section 4.4, "Unified KV management").
 * The block's internals are not given by the paper; this library computes,
 * per block and per stream b:
 *
 *   M      = mod[b] + mod_table                       rows: shift1 scale1 gate1 shift2 scale2 gate2
 *   h1     = rms(x) * (1 + scale1) + shift1
 *   q,k,v  = split(h1 W_qkv^T + b_qkv)
 *   q~,k~  = rope3d(rms(q) * g_q), rope3d(rms(k) * g_k)   (rms over the full width D)
 *   K,V    = [cache | k~], [cache | v]                (k~, v written into the stream's pages)
 *   o      = softmax(q~ K^T / sqrt(d)) V per head, every key visible
 *   x1     = x + gate1 * (o W_o^T + b_o)
 *   q_c    = rms(rms(x1) * g_n3 W_cq^T + b_cq) * g_cq
 *   x2     = x1 + (softmax(q_c K_c^T / sqrt(d)) V_c) W_co^T + b_co
 *   out    = x2 + gate2 * (GELU_tanh((rms(x2) * (1 + scale2) + shift2) W_1^T + b_1) W_2^T + b_2)
 *
 * with rms(z) = z / sqrt(mean(z^2) + eps), linears y = x W^T + b (W stored
 * [out][in]), 3D RoPE over (latent frame, row, column) with head-dim
 * segments (d - 4 floor(d/6), 2 floor(d/6), 2 floor(d/6)) and adjacent
 * pairs, and K_c, V_c the per-stream text keys/values (ardit_ctx_kv).
 *
 * Conventions for every call below.
 *  - Precision: activations, weights, pages and outputs are bf16; biases and
 *    gains bf16; modulation tensors fp32.  All accumulation and all norm,
 *    softmax, RoPE and GELU arithmetic is fp32; fp32 -> bf16 rounds to
 *    nearest even.
 *  - Ownership: the caller allocates and owns every buffer; the library
 *    never allocates device memory in these calls and keeps no pointer after
 *    the call returns.  "device" pointers are HIP device memory, "host"
 *    pointers are read during the call only.
 *  - Asynchrony: each call enqueues its kernels on `stream` and returns
 *    without synchronising.  Host-side checks run before anything is
 *    enqueued; when one fails the call returns a negative status, enqueues
 *    nothing and leaves every output untouched.  A device-side failure shows
 *    up as ARDIT_EHIP from a later call (ardit_last_error has the detail).
 *  - Threading: calls may be made from several host threads; the last error
 *    message is kept per thread.
 *  - Layout of one frame page (T = lat_h * lat_w tokens of one latent frame,
 *    H heads of d dims): keys [H][T][d], values transposed [H][d][T].  A
 *    head's slice of a page is contiguous in both.  Logical token j of stream
 *    b lives in page page_table[b * max_frames + j / T] at offset j % T.
 *  - Text keys/values of stream b start at element offset ctx_off_b * D of
 *    ctx_k / ctx_v, where ctx_off_b is the sum of the earlier streams'
 *    ctx_lens; within a stream keys are [H][L_x][d] and values [H][d][L_x].
 *  - Supported shapes: head_dim in {64, 128}; dim = n_heads * head_dim and
 *    dim, ffn_dim multiples of 128; T = lat_h * lat_w a multiple of 8 with
 *    T + gcd(T, 64) >= 64 (a 64-key attention tile spans at most two frame
 *    pages: T in {8, 16, 24, 40} is rejected); at most ARDIT_MAX_STREAMS
 *    streams per call.
 */
#ifndef ARDIT_H
#define ARDIT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ARDIT_MAX_STREAMS 64
#define ARDIT_TIME_FREQ_DIM 256
#define ARDIT_MAX_STEPS 16     /* denoising steps of one chunk in ardit_chunk_generate */

typedef enum {
  ARDIT_OK = 0,
  ARDIT_EINVAL = -1,      /* null pointer or meaningless argument */
  ARDIT_ESHAPE = -2,      /* dims inconsistent with each other or with a length */
  ARDIT_ECAPACITY = -3,   /* a stream's keys exceed its page table or a length is out of range */
  ARDIT_EWORKSPACE = -4,  /* workspace smaller than ardit_workspace_size reports */
  ARDIT_EUNSUPPORTED = -5,/* shape outside what the kernels support (see above) */
  ARDIT_EHIP = -6,        /* the HIP runtime reported an error */
  ARDIT_EHOST = -7        /* host memory ran out inside the call */
} ardit_status;

/* Model and chunk geometry (host struct). */
typedef struct {
  int32_t dim;               /* D, hidden width */
  int32_t n_heads;           /* H */
  int32_t head_dim;          /* d; D == H * d */
  int32_t ffn_dim;           /* F */
  int32_t frames_per_chunk;  /* latent frames per chunk (n_f) */
  int32_t lat_h, lat_w;      /* latent grid of one frame; T = lat_h * lat_w tokens per frame page */
  float eps;                 /* RMSNorm epsilon (1e-6) */
  float rope_theta;          /* RoPE base (10000) */
} ardit_dims;

/* One batch of streams (host struct, host arrays of n_streams entries).
 * Tokens of stream b occupy rows [sum_{b'<b} q_lens[b'], ... + q_lens[b]) of
 * the packed activations. */
typedef struct {
  int32_t n_streams;          /* 1 .. ARDIT_MAX_STREAMS */
  const int32_t* q_lens;      /* chunk tokens per stream (<= 2^22 in all); block calls:
                                 frames_per_chunk * T each */
  const int32_t* cache_lens;  /* tokens already in the stream's cache; a multiple of T, <= 2^30 */
  const int32_t* frame_pos0;  /* absolute latent-frame index of the chunk's first frame (RoPE t) */
  const int32_t* ctx_lens;    /* text tokens per stream (>= 1) */
  const float* sparsity;      /* attention sparsity rho per stream in [0, 1], or NULL for all 0
                                 (block-sparse self-attention, see ardit_sparse_select) */
  const int32_t* quant;       /* self-attention precision per stream (ardit_quant), or NULL for
                                 all ARDIT_QUANT_BF16 */
} ardit_batch;

/* Precision of a stream's self-attention (the paper's quantisation knob Q,
 * Section 2.1; Section 5: activations quantised online, weights never).
 * ARDIT_QUANT_FP8 (head_dim 128 only): q, k, v and the softmax weights are
 * OCP E4M3 with a power-of-two scale per 32 elements along each product's
 * reduction axis (q, k: 32 dims; v, weights: 32 keys), the scale exponent
 * floor(log2 max|x|) - 7 of the block (ardit_mx_quantize); logits, running
 * max and denominator stay fp32.  Everything else in the block stays bf16. */
typedef enum { ARDIT_QUANT_BF16 = 0, ARDIT_QUANT_FP8 = 1 } ardit_quant;

/* Frame-paged KV cache of one layer (device memory). */
typedef struct {
  void* k_pages;               /* [n_pages][H][T][d] bf16 */
  void* v_pages;               /* [n_pages][H][d][T] bf16 */
  const int32_t* page_table;   /* [n_streams][max_frames] int32, physical page of each logical frame */
  int32_t n_pages;             /* pages in the pool.  A table entry outside [0, n_pages) is a caller
                                  error: reads clamp it into the pool, writes skip it (the chunk's
                                  keys/values for that frame are dropped, no other page changes);
                                  ardit_debug_checks(1) rejects such a table before any launch */
  int32_t max_frames;          /* row length of page_table */
} ardit_kv_paged;

/* Weights of one block (device pointers, bf16 unless noted, matrices [out][in]). */
typedef struct {
  const void *w_qkv, *b_qkv;   /* [3D][D], [3D]  rows: q, k, v */
  const void *g_q, *g_k;       /* [D] QK-RMSNorm gains */
  const void *w_o, *b_o;       /* [D][D], [D] */
  const void *g_n3;            /* [D] cross-attention pre-norm gain */
  const void *w_cq, *b_cq;     /* [D][D], [D] */
  const void *g_cq;            /* [D] */
  const void *w_ck, *b_ck;     /* [D][D], [D]   used by ardit_ctx_kv only */
  const void *g_ck;            /* [D]           used by ardit_ctx_kv only */
  const void *w_cv, *b_cv;     /* [D][D], [D]   used by ardit_ctx_kv only */
  const void *w_co, *b_co;     /* [D][D], [D] */
  const void *w_1, *b_1;       /* [F][D], [F] */
  const void *w_2, *b_2;       /* [D][F], [D] */
  const float* mod_table;      /* [6][D] fp32, added to the stream's time modulation */
} ardit_block_weights;

/* Shared time MLP (device pointers, bf16): 256 -> D -> D -> 6D. */
typedef struct {
  const void *w_t1, *b_t1;     /* [D][256], [D] */
  const void *w_t2, *b_t2;     /* [D][D], [D] */
  const void *w_m, *b_m;       /* [6D][D], [6D] */
} ardit_time_weights;

/* Name of a status code; never NULL. */
const char* ardit_status_str(int status);
/* Detail of the calling thread's last failed call ("" if none). */
const char* ardit_last_error(void);
/* ABI version (major * 100 + minor): 502. */
int ardit_version(void);

/* Workspace bytes needed by any call below for this geometry and batch
 * (block, stack, context and time-modulation calls share one workspace). */
int ardit_workspace_size(const ardit_dims* dims, const ardit_batch* batch, size_t* bytes);

/* Time modulation, once per stream per denoising step (the timestep that
 * conditions each of the S denoising steps of a chunk, Section 2.1; the
 * paper gives no embedding, this is the DiT-family form): sinusoid of t (256
 * features: cos then sin of t * 10000^(-k/128)), then
 * m = W_m SiLU(W_t2 SiLU(W_t1 s + b_t1) + b_t2) + b_m.
 * t_host: host [n_streams] timesteps.  mod_out: device fp32 [n_streams][6][D]. */
int ardit_time_mod(hipStream_t stream, const ardit_dims* dims, int32_t n_streams,
                   const float* t_host, const ardit_time_weights* tw, float* mod_out,
                   void* ws, size_t ws_bytes);

/* Text keys/values of each stream for one block (the conditioning embeddings
 * the DiT attends to, Section 2.1, "Video Generation"): K_c = rms(ctx W_ck^T + b_ck) * g_ck,
 * V_c = ctx W_cv^T + b_cv, written in the layout described above.
 * ctx: device bf16 [sum ctx_lens][D], streams packed in order.  Only
 * batch->n_streams and batch->ctx_lens are read. */
int ardit_ctx_kv(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                 const void* ctx, const ardit_block_weights* w, void* ctx_k, void* ctx_v,
                 void* ws, size_t ws_bytes);

/* The QK-norm / RoPE / append step alone (a chunk's keys and values enter the
 * stream's rolling cache, Section 2.1, "AR-DiT"; frame pages behind the
 * logical page table, Section 4.4): from packed projections qkv
 * (device bf16 [sum q_lens][3D], columns q | k | v), writes q~ (device bf16
 * [sum q_lens][D]) and the chunk's k~ and v into logical slots
 * [cache_len, cache_len + q_len) of each stream's pages.  g_q, g_k: device
 * bf16 [D].  Nothing else of the pool is written. */
int ardit_kv_append(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                    const void* qkv, const void* g_q, const void* g_k,
                    const ardit_kv_paged* kv, void* q_out);

/* Paged attention alone (a chunk attends to the KV cache of the stream's
 * earlier chunks and to itself, Section 2.1, "AR-DiT"; pages per latent frame,
 * Section 4.4; per-stream cache lengths, Section 3.2 footnote):
 * o = softmax(q K^T / sqrt(d)) V per stream and head
 * over logical keys [0, cache_len + q_len) of the stream's pages (the chunk's
 * own keys must already be in the pages).  q, o: device bf16 [sum q_lens][H][d].
 * ws / ws_bytes as for the block calls (ardit_workspace_size of this batch):
 * when the (stream, head, query tile) items are too few to fill the GPU, their
 * key ranges are split between workgroups and the partial results combined
 * through the workspace.  When batch->sparsity gives some stream rho > 0 the
 * attention is block-sparse: each query tile attends only to the keys of the
 * tiles ardit_sparse_select would list for it (selection and attention both
 * run in this call, the lists live in the workspace). */
int ardit_attn_fwd(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                   const void* q, const ardit_kv_paged* kv, void* o, void* ws, size_t ws_bytes);

/* Paged attention without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops and harnesses
 * that forbid hipMalloc).  Computes exactly what ardit_attn_fwd computes, with
 * the same kernels and schedule, for batches whose streams all run bf16
 * attention (dense or block-sparse); the scratch those kernels need (the
 * split schedule's partial results, or the block selection's means, scores
 * and lists) lives in a static device array of the library instead of the
 * caller's workspace.  Limits: at most 72 MiB of scratch (the dense split
 * schedule takes (2 * 256 * 256 * (head_dim + 2)) * 4 bytes: 65 MiB at
 * head_dim 128; a sparse batch its ardit_sparse_select regions), else
 * ARDIT_EWORKSPACE; a stream in FP8: ARDIT_EUNSUPPORTED; `stream` (NULL: the
 * null stream of the current device) must belong to the current device, else
 * ARDIT_EINVAL.  Each GPU holds one copy of the array, taken when the library
 * is loaded and kept until the process ends, and every call on that GPU
 * shares it: calls that overlap on one GPU (two streams, two threads) race on
 * it and must be ordered by the caller.  Nothing needs clearing between calls
 * (every scratch entry is written before it is read).  The call makes no
 * device or host allocation, no memset and no copy; it records no timing
 * events and skips ardit_debug_checks. */
int ardit_attn_fwd_noalloc(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                           const void* q, const ardit_kv_paged* kv, void* o);

/* The FP8 block quantisation the FP8 attention applies to its operands:
 * rows of bf16 x (device, row stride ld elements, ld % 8 == 0) to E4M3 codes
 * (device uint8 [rows][cols]) and E8M0 scales (device uint8 [rows][cols / 32]):
 * each 32 consecutive columns take e = floor(log2 max|x|) - 7 (-127 for an
 * all-zero block), scale byte e + 127, codes = round-to-nearest-even E4M3 of
 * x / 2^e (|x / 2^e| < 256, no saturation).  cols % 32 == 0. */
int ardit_mx_quantize(hipStream_t stream, const void* x, int64_t rows, int32_t cols, int32_t ld,
                      void* codes, void* scales);

/* Block selection of block-sparse self-attention (paper, Section 2.1: the
 * sparsity knob rho skips attention blocks a sparse mask leaves out; Section 5
 * names Light Forcing as the method, whose rule the paper does not give).
 * The rule computed: an item is (stream b, head h, query tile i of 256 rows of
 * the chunk); key tile j is 64 logical keys [64 j, 64 j + 64) of the stream's
 * [cache | chunk] (the last tile may hold fewer).  Its score is
 * mean(q~ over the tile's rows) . mean(k~ over the key tile), fp32, and the item
 * keeps the n_keep = min(n, max(1, ceil((1 - rho_b) n - 1e-3))) tiles of
 * highest score among its n = ceil((cache_len + q_len) / 64), ties to the
 * lower index; rho_b = 0 keeps every tile.  NaN scores rank as -inf.
 * q: device bf16 [sum q_lens][H][d] (rotated queries); the stream's keys must be
 * in the pages.  blocks: device int32, one row of row_stride entries per item,
 * rows of stream b starting at row H * sum_{b' < b} ceil(q_lens[b'] / 256),
 * then head-major, then query tile; a row holds its kept tiles ascending,
 * then -1 up to row_stride.  row_stride must be at least every stream's
 * n_keep.  Streams with q_len 0 have no rows.  ws / ws_bytes:
 * ardit_workspace_size of this batch.  Deterministic: the same inputs give the
 * same lists as the selection inside ardit_attn_fwd and the block calls. */
int ardit_sparse_select(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                        const void* q, const ardit_kv_paged* kv, int32_t* blocks,
                        int32_t row_stride, void* ws, size_t ws_bytes);

/* One block, one stream (dense self-attention): one denoising step of one DiT
 * block on a chunk over the stream's KV cache (Section 2.1, "AR-DiT"; the
 * block internals are the contract at the top of this file).
 * x, out: device bf16 [L_q][D] (L_q = frames_per_chunk * T);
 * kv.page_table has one row.  mod: device fp32 [6][D] (from ardit_time_mod).
 * ctx_k / ctx_v from ardit_ctx_kv with ctx_len text tokens.  Writes the
 * chunk's keys/values into slots [cache_len, cache_len + L_q); the caller
 * commits the chunk by advancing cache_len (or rotating its page table). */
int ardit_block_fwd(hipStream_t stream, const ardit_dims* dims, const void* x,
                    ardit_kv_paged kv, int32_t cache_len, int32_t frame_pos0,
                    const float* mod, const void* ctx_k, const void* ctx_v, int32_t ctx_len,
                    const ardit_block_weights* w, void* out, void* ws, size_t ws_bytes);

/* One block over a ragged batch of streams sharing the weights (one GPU's share
 * of the streams; streams hold different KV lengths, Section 3.2 footnote, and
 * a worker serves several streams, Section 3.1).  x, out: device bf16 [sum q_lens][D]; mod: device fp32
 * [n_streams][6][D]; page_table rows follow the batch order.  Streams with
 * batch->sparsity > 0 run block-sparse self-attention (ardit_sparse_select). */
int ardit_block_fwd_varlen(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                           const void* x, const ardit_kv_paged* kv, const float* mod,
                           const void* ctx_k, const void* ctx_v, const ardit_block_weights* w,
                           void* out, void* ws, size_t ws_bytes);

/* n_layers blocks applied in sequence (one denoising step of the DiT, Section
 * 2.1: the model denoises the chunk's latent over S such steps).
 * kv, w, ctx_k, ctx_v: host arrays of n_layers entries.  x is not modified. */
int ardit_stack_fwd(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                    int32_t n_layers, const void* x, const ardit_kv_paged* kv, const float* mod,
                    const void* const* ctx_k, const void* const* ctx_v,
                    const ardit_block_weights* w, void* out, void* ws, size_t ws_bytes);

/* Page table of one stream under a sink + sliding-window cache (paper,
 * Section 2.1: the cache keeps a few sink chunks plus the most recent W
 * chunks; Sections 3.2 and 4.4: frame pages behind a logical table).  While
 * chunk `chunk` (0-based) is generated, the stream's cache holds chunks
 * 0 .. min(sink, chunk) - 1 and max(sink, chunk - window) .. chunk - 1, in that
 * order.  Chunk k lives in slot k when k < sink, else in slot
 * sink + (k - sink) mod (window + 1), so the slot of the chunk being generated
 * never holds a chunk still in the window; slot s owns pages
 * page_base + s * frames_per_chunk + f, f < frames_per_chunk.  A stream thus
 * needs (sink + window + 1) * frames_per_chunk pages.  Writes the held
 * chunks' pages followed by chunk `chunk`'s into table[0 ..
 * (held + 1) * frames_per_chunk) (host int32, max_frames entries; the rest is
 * untouched) and the held frame count to *cache_frames: the stream's
 * cache_len is *cache_frames * lat_h * lat_w.  Keys keep the RoPE positions
 * of their absolute frames, so frame_pos0 stays chunk * frames_per_chunk.
 * Host only: makes no HIP call.  ARDIT_ECAPACITY when max_frames is too short
 * or the pages overflow int32. */
int ardit_window_pages(int32_t chunk, int32_t sink, int32_t window, int32_t frames_per_chunk,
                       int32_t page_base, int32_t* table, int32_t max_frames,
                       int32_t* cache_frames);

/* One chunk of every stream of the batch, end to end (paper, Section 2.1,
 * "AR-DiT": a chunk is denoised in S steps by the stack attending to the
 * stream's cache, then appended to it; Appendix A: S is a fidelity knob).
 * The paper does not give the sampler or the commit; computed here:
 *  - step i of stream b (timestep t = t_host[b * t_ld + i] in [0, 1000], tau = t / 1000):
 *    M = ardit_time_mod(t); v = ardit_stack_fwd(x_tau) (the velocity);
 *    x0_hat = x_tau - tau v; the next step starts from
 *    (1 - tau') x0_hat + tau' eps_{i+1}, tau' its timestep / 1000; the last step
 *    keeps x0_hat (the clean chunk, written to x0_out).  The update runs in
 *    fp32 on bf16 operands and stores bf16.
 *  - the commit: one more pass of the stack on x0_hat at t = 0, whose keys and
 *    values are what slots [cache_len, cache_len + L_q) of every layer's pages
 *    hold when the call's work completes (the caller then commits the chunk
 *    through its page table, e.g. ardit_window_pages for the next chunk).
 * Streams run in lockstep: pass i covers the streams with n_steps[b] >= i, as
 * step i of those with n_steps[b] > i and the commit of those with
 * n_steps[b] == i; n_steps must be non-increasing along the batch so each pass
 * is a prefix of it.  A pass that only commits skips the work after the last
 * layer's key/value append (its output is not used).
 *   n_steps: host [n_streams], each in [1, ARDIT_MAX_STEPS].
 *   t_host:  host, row b of t_ld >= n_steps[0] entries: the stream's timesteps.
 *   x_init:  device bf16 [sum q_lens][D], the starting noise x_{tau_0} (read only).
 *   noise:   device bf16 [n_steps[0] - 1][sum q_lens][D]; slab i is eps_{i+1}
 *            (rows of streams without a step i + 1 are not read); may be NULL
 *            when n_steps[0] == 1.
 *   kv, ctx_k, ctx_v, w: per-layer host arrays of n_layers entries, as for
 *            ardit_stack_fwd; tw: the shared time MLP.
 *   x0_out:  device bf16 [sum q_lens][D], the clean chunk; must not overlap
 *            x_init, noise or the workspace.
 *   ws:      ardit_workspace_size of this batch (it includes the modulation
 *            and velocity buffers this call needs).
 * batch->sparsity and batch->quant apply to every pass. */
int ardit_chunk_generate(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                         int32_t n_layers, const int32_t* n_steps, const float* t_host,
                         int32_t t_ld, const void* x_init, const void* noise,
                         const ardit_kv_paged* kv, const ardit_time_weights* tw,
                         const void* const* ctx_k, const void* const* ctx_v,
                         const ardit_block_weights* w, void* x0_out, void* ws, size_t ws_bytes);

/* Kernel timing.  ardit_timing_enable(mask) turns on HIP events recorded on
 * the launch stream around each launch of the kinds in mask: bit 0 (1) the
 * self-attention kernel (for sparse streams the attention over the kept
 * tiles, after the block selection; for FP8 streams the FP8 attention after
 * its quantisation pre-pass), bit 1 (2) the block's six GEMMs, bit 2 (4) its
 * elementwise kernels (both adaLN norms, both RMS-gain norms, QK-norm / RoPE /
 * key append, value append); 0 turns timing off.  The events of the GEMM and
 * elementwise kinds sit between kernels that otherwise follow each other on
 * the stream, so timing them can add small gaps.  ardit_timing_collect_kind
 * waits for the recorded events of one kind (0, 1 or 2), returns the number of
 * launches and their summed duration in ms, and clears that kind's record;
 * ardit_timing_collect is the same for kind 0.  ARDIT_EINVAL for a mask or
 * kind out of range. */
int ardit_timing_enable(int enable);
int ardit_timing_collect(int32_t* launches, double* total_ms);
int ardit_timing_collect_kind(int32_t kind, int32_t* launches, double* total_ms);

/* Cold timing and per-launch records.  ardit_timing_flush(buf, bytes) makes
 * every timed launch (the kinds enabled by ardit_timing_enable) first read
 * device buffer buf (16-byte aligned, bytes % 16 == 0, at least 128 KiB; its
 * last 64 KiB receive the read's checksum words) with a kernel outside its
 * events, so a buffer larger than L2 and the last-level cache leaves the
 * launch's operands cold and the caches holding clean lines (a write would
 * leave dirty lines to be written back during the timed launch); (NULL, 0)
 * turns it off.
 * ardit_timing_records waits for the recorded launches of one kind and
 * returns, in launch order, each launch's name (a static string of the
 * library) and duration in ms, clearing them; ARDIT_ECAPACITY (nothing
 * cleared, *n_records set to the count) when more than max_records are held. */
int ardit_timing_flush(void* buf, size_t bytes);
int ardit_timing_records(int32_t kind, int32_t max_records, const char** names, double* ms,
                         int32_t* n_records);

/* Debug validation of page tables (off by default; for callers that want a
 * bad table reported rather than silently dropped or clamped).  With
 * ardit_debug_checks(1) every call that reads a page table first copies it to
 * the host on the call's stream and synchronises that stream, then returns
 * ARDIT_ECAPACITY when an entry that a stream reads or writes lies outside
 * [0, n_pages), and ARDIT_EINVAL when a page that the call writes (a chunk's
 * frames) is written by two streams, twice by one, or read as cache by another
 * stream; nothing is enqueued then.  The synchronisation makes it unsuitable
 * for timed or captured runs.  0 turns it off; other values: ARDIT_EINVAL. */
int ardit_debug_checks(int enable);

#ifdef __cplusplus
}
#endif

#endif /* ARDIT_H */
