// C ABI of libardit: argument validation, workspace layout and the launch
// chains of the block.  Every check runs before the first launch, so a
// failing call enqueues nothing and leaves its outputs untouched.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "ardit.h"
#include "ardit_micro.h"
#include "launch.h"

using namespace ardit;

namespace {

// a fixed buffer: recording an error never allocates, so it also works when
// host memory has run out
thread_local char g_last_error[512];

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(ARDIT_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define ARDIT_TRY(expr)                        \
  do {                                         \
    int _s = (expr);                           \
    if (_s != ARDIT_OK) return _s;             \
  } while (0)

#define ARDIT_HIP(expr, what)                  \
  do {                                         \
    hipError_t _e = (expr);                    \
    if (_e != hipSuccess) return hip_fail(_e, what); \
  } while (0)

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

int check_dims(const ardit_dims* d) {
  if (!d) return fail(ARDIT_EINVAL, "dims is NULL");
  if (d->dim <= 0 || d->n_heads <= 0 || d->head_dim <= 0 || d->ffn_dim <= 0 ||
      d->frames_per_chunk <= 0 || d->lat_h <= 0 || d->lat_w <= 0)
    return fail(ARDIT_ESHAPE, "dims must be positive");
  if (static_cast<int64_t>(d->n_heads) * d->head_dim != d->dim)
    return fail(ARDIT_ESHAPE, "dim %d != n_heads %d * head_dim %d", d->dim, d->n_heads,
                d->head_dim);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(ARDIT_EUNSUPPORTED, "head_dim %d not in {64, 128}", d->head_dim);
  if (d->dim % 128 != 0 || d->ffn_dim % 128 != 0)
    return fail(ARDIT_EUNSUPPORTED, "dim %d and ffn_dim %d must be multiples of 128", d->dim,
                d->ffn_dim);
  if (d->dim > 8192) return fail(ARDIT_EUNSUPPORTED, "dim %d above 8192", d->dim);
  if (d->ffn_dim > 65536) return fail(ARDIT_EUNSUPPORTED, "ffn_dim %d above 65536", d->ffn_dim);
  const int64_t T = static_cast<int64_t>(d->lat_h) * d->lat_w;
  if (T % 8 != 0) return fail(ARDIT_EUNSUPPORTED, "lat_h * lat_w = %lld not a multiple of 8",
                              static_cast<long long>(T));
  // a 64-key attention tile may span at most two frame pages: tiles start at
  // multiples of 64, so the furthest one reaches T - gcd(T, 64) + 63 < 2 T
  {
    int64_t gcd = 64;
    while (T % gcd != 0) gcd >>= 1;
    if (T > 0 && T + gcd < 64)
      return fail(ARDIT_EUNSUPPORTED,
                  "lat_h * lat_w = %lld: a 64-key tile would span more than two frames",
                  static_cast<long long>(T));
  }
  if (T * d->frames_per_chunk > (1 << 20)) return fail(ARDIT_ESHAPE, "chunk too large");
  if (!(d->eps > 0.f) || !(d->rope_theta > 0.f))
    return fail(ARDIT_EINVAL, "eps and rope_theta must be positive");
  return ARDIT_OK;
}

int tokens_per_frame(const ardit_dims* d) { return d->lat_h * d->lat_w; }
int chunk_tokens(const ardit_dims* d) { return d->frames_per_chunk * tokens_per_frame(d); }

enum BatchUse : unsigned {
  kUseQ = 1, kUseCache = 2, kUsePos = 4, kUseCtx = 8, kChunkQ = 16,
};

int check_batch(const ardit_dims* d, const ardit_batch* b, unsigned use) {
  if (!b) return fail(ARDIT_EINVAL, "batch is NULL");
  if (b->n_streams < 1 || b->n_streams > ARDIT_MAX_STREAMS)
    return fail(ARDIT_EINVAL, "n_streams %d not in [1, %d]", b->n_streams, ARDIT_MAX_STREAMS);
  if ((use & kUseQ) && !b->q_lens) return fail(ARDIT_EINVAL, "batch q_lens is NULL");
  if ((use & kUseCache) && !b->cache_lens) return fail(ARDIT_EINVAL, "batch cache_lens is NULL");
  if ((use & kUsePos) && !b->frame_pos0) return fail(ARDIT_EINVAL, "batch frame_pos0 is NULL");
  if ((use & kUseCtx) && !b->ctx_lens) return fail(ARDIT_EINVAL, "batch ctx_lens is NULL");
  const int T = tokens_per_frame(d);
  int64_t nq = 0, nc = 0;
  for (int i = 0; i < b->n_streams; ++i) {
    if (use & kUseQ) {
      const int q = b->q_lens[i];
      if (q < 0) return fail(ARDIT_ESHAPE, "q_lens[%d] = %d is negative", i, q);
      if ((use & kChunkQ) && q != chunk_tokens(d))
        return fail(ARDIT_ESHAPE, "q_lens[%d] = %d != frames_per_chunk * lat_h * lat_w = %d", i, q,
                    chunk_tokens(d));
      nq += q;
    }
    if (use & kUseCache) {
      const int c = b->cache_lens[i];
      if (c < 0 || c % T != 0)
        return fail(ARDIT_ESHAPE, "cache_lens[%d] = %d is not a non-negative multiple of %d", i,
                    c, T);
      // with at most 2^22 queries, cache + chunk stays below 2^31 keys
      if (c > (1 << 30)) return fail(ARDIT_ECAPACITY, "cache_lens[%d] = %d above 2^30", i, c);
    }
    if ((use & kUsePos) && b->frame_pos0[i] < 0)
      return fail(ARDIT_EINVAL, "frame_pos0[%d] = %d is negative", i, b->frame_pos0[i]);
    if (use & kUseCtx) {
      const int c = b->ctx_lens[i];
      if (c < 1) return fail(ARDIT_ESHAPE, "ctx_lens[%d] = %d must be >= 1", i, c);
      nc += c;
    }
  }
  if (nq > (1 << 22) || nc > (1 << 22))
    return fail(ARDIT_ECAPACITY, "more than 2^22 tokens in one batch");
  // the text keys / values of a stream are addressed by a 32-bit element offset
  if (nc * d->dim >= (int64_t(1) << 31))
    return fail(ARDIT_ECAPACITY, "%lld text tokens of width %d exceed 2^31 elements",
                static_cast<long long>(nc), d->dim);
  if (b->sparsity)
    for (int i = 0; i < b->n_streams; ++i) {
      const float r = b->sparsity[i];
      if (!(r >= 0.f && r <= 1.f))
        return fail(ARDIT_EINVAL, "sparsity[%d] = %g not in [0, 1]", i, static_cast<double>(r));
    }
  if (b->quant)
    for (int i = 0; i < b->n_streams; ++i) {
      if (b->quant[i] != ARDIT_QUANT_BF16 && b->quant[i] != ARDIT_QUANT_FP8)
        return fail(ARDIT_EINVAL, "quant[%d] = %d is not a quantisation mode", i, b->quant[i]);
      if (b->quant[i] == ARDIT_QUANT_FP8 && d->head_dim != 128)
        return fail(ARDIT_EUNSUPPORTED, "FP8 attention needs head_dim 128 (got %d)", d->head_dim);
    }
  return ARDIT_OK;
}

// true when some stream of the batch runs FP8 attention
bool batch_fp8(const ardit_batch* b) {
  if (!b->quant) return false;
  for (int i = 0; i < b->n_streams; ++i)
    if (b->quant[i] == ARDIT_QUANT_FP8) return true;
  return false;
}

constexpr size_t kAlign = 256;
size_t up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// true when some stream of the batch runs block-sparse self-attention
bool batch_sparse(const ardit_batch* b) {
  if (!b->sparsity) return false;
  for (int i = 0; i < b->n_streams; ++i)
    if (b->sparsity[i] > 0.f) return true;
  return false;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Bytes of the block selection's scratch for this batch: the fp32 mean query
// of every item, its fp32 score per key tile, and the kept-tile lists packed
// per stream.
struct SparseBytes {
  size_t qbar = 0, scores = 0, lists = 0;
  size_t f8q = 0, f8kv = 0;   // FP8: query codes + scales; key / value codes + scales
  int64_t f8_keys = 0;        // FP8: keys of all FP8 streams, padded to whole tiles
};
SparseBytes sparse_ws_bytes(const ardit_dims* d, const ardit_batch* b) {
  SparseBytes z;
  if (batch_fp8(b) && b->q_lens && b->cache_lens) {
    int64_t N = 0, keys = 0;
    for (int i = 0; i < b->n_streams; ++i) {
      N += b->q_lens[i];
      if (b->quant[i] == ARDIT_QUANT_FP8 && b->q_lens[i] > 0)
        keys += kAttnKTile * ceil_div(static_cast<int64_t>(b->cache_lens[i]) + b->q_lens[i], kAttnKTile);
    }
    z.f8_keys = keys;
    const size_t qb = static_cast<size_t>(N) * d->dim;
    z.f8q = up(qb) + up(qb / 32);
    const size_t kb = static_cast<size_t>(d->n_heads) * keys * d->head_dim;
    z.f8kv = 2 * (up(kb) + up(kb / 32));
  }
  if (!batch_sparse(b) || !b->q_lens || !b->cache_lens) return z;
  for (int i = 0; i < b->n_streams; ++i) {
    const int64_t q = b->q_lens[i];
    if (q <= 0) continue;
    const int64_t nt = ceil_div(b->cache_lens[i] + q, kAttnKTile);
    const int64_t nk = sparse_keep_count(static_cast<int>(nt), b->sparsity[i]);
    const int64_t items = d->n_heads * ceil_div(q, kAttnQTile);
    z.qbar += sizeof(float) * static_cast<size_t>(items * d->head_dim);
    z.scores += sizeof(float) * static_cast<size_t>(items * nt);
    z.lists += sizeof(int32_t) * static_cast<size_t>(items * nk);
  }
  return z;
}

// Limits of the block selection, on a batch whose q_lens and cache_lens passed check_batch.
int check_sparse(const ardit_dims* d, const ardit_batch* b) {
  if (sparse_ws_bytes(d, b).f8_keys >= (int64_t(1) << 31))
    return fail(ARDIT_ECAPACITY, "FP8 streams hold more than 2^31 keys in all");
  if (!b->sparsity) return ARDIT_OK;
  int64_t lists = 0, scores = 0;
  for (int i = 0; i < b->n_streams; ++i) {
    const int64_t q = b->q_lens[i];
    if (q <= 0) continue;
    const int64_t nt = ceil_div(b->cache_lens[i] + q, kAttnKTile);
    if (b->sparsity[i] > 0.f && nt > kSparseMaxTiles)
      return fail(ARDIT_EUNSUPPORTED, "stream %d: %lld key tiles above the %d the selection ranks",
                  i, static_cast<long long>(nt), kSparseMaxTiles);
    lists += d->n_heads * ceil_div(q, kAttnQTile) *
             sparse_keep_count(static_cast<int>(nt), b->sparsity[i]);
    scores += d->n_heads * ceil_div(q, kAttnQTile) * nt;
  }
  if (lists >= (int64_t(1) << 31)) return fail(ARDIT_ECAPACITY, "kept-tile lists above 2^31 entries");
  if (scores >= (int64_t(1) << 31)) return fail(ARDIT_ECAPACITY, "block scores above 2^31 entries");
  return ARDIT_OK;
}

int check_kv(const ardit_dims* d, const ardit_batch* b, const ardit_kv_paged* kv) {
  if (!kv) return fail(ARDIT_EINVAL, "kv is NULL");
  if (!kv->k_pages || !kv->v_pages || !kv->page_table)
    return fail(ARDIT_EINVAL, "kv pointers must be non-NULL");
  if (misaligned(kv->k_pages) || misaligned(kv->v_pages))
    return fail(ARDIT_EINVAL, "kv pages must be 16-byte aligned");
  if (kv->n_pages < 1 || kv->max_frames < 1)
    return fail(ARDIT_EINVAL, "n_pages and max_frames must be >= 1");
  const int64_t T = tokens_per_frame(d);
  if (static_cast<int64_t>(kv->n_pages) * d->dim * T > (int64_t(1) << 40))
    return fail(ARDIT_ECAPACITY, "page pool too large");
  for (int i = 0; i < b->n_streams; ++i) {
    const int64_t keys = static_cast<int64_t>(b->cache_lens[i]) + b->q_lens[i];
    const int64_t frames = (keys + T - 1) / T;
    if (frames > kv->max_frames)
      return fail(ARDIT_ECAPACITY, "stream %d needs %lld frames > max_frames %d", i,
                  static_cast<long long>(frames), kv->max_frames);
  }
  return ARDIT_OK;
}

// Opt-in validation of the page tables against the pool (ardit_debug_checks).
std::atomic<int> g_debug_checks{0};

// With the debug checks on: copies the page table to the host (synchronising
// `st`) and checks every entry a stream reads or writes against the pool, and
// that no page the batch writes is used by another stream or twice.
int check_pages(hipStream_t st, const ardit_dims* d, const ardit_batch* b,
                const ardit_kv_paged* kv, bool writes) {
  if (!g_debug_checks.load(std::memory_order_relaxed)) return ARDIT_OK;
  const int64_t T = tokens_per_frame(d);
  const size_t n = static_cast<size_t>(b->n_streams) * kv->max_frames;
  std::vector<int32_t> table(n);
  ARDIT_HIP(hipMemcpyAsync(table.data(), kv->page_table, n * sizeof(int32_t),
                           hipMemcpyDeviceToHost, st), "page table copy");
  ARDIT_HIP(hipStreamSynchronize(st), "page table copy");
  std::vector<int32_t> owner(static_cast<size_t>(kv->n_pages), -1);   // stream writing the page
  for (int i = 0; i < b->n_streams; ++i) {
    if (b->q_lens[i] == 0) continue;
    const int64_t keys = static_cast<int64_t>(b->cache_lens[i]) + b->q_lens[i];
    const int64_t frames = (keys + T - 1) / T;
    for (int64_t f = 0; f < frames; ++f) {
      const int32_t p = table[static_cast<size_t>(i) * kv->max_frames + f];
      if (p < 0 || p >= kv->n_pages)
        return fail(ARDIT_ECAPACITY, "stream %d frame %lld: page %d outside the pool of %d", i,
                    static_cast<long long>(f), p, kv->n_pages);
      if (writes && f >= b->cache_lens[i] / T) {
        if (owner[p] >= 0)
          return fail(ARDIT_EINVAL, "page %d is written by streams %d and %d", p, owner[p], i);
        owner[p] = i;
      }
    }
  }
  if (writes)
    for (int i = 0; i < b->n_streams; ++i) {
      if (b->q_lens[i] == 0) continue;
      const int64_t cached = b->cache_lens[i] / T;
      for (int64_t f = 0; f < cached; ++f) {
        const int32_t p = table[static_cast<size_t>(i) * kv->max_frames + f];
        if (owner[p] >= 0)
          return fail(ARDIT_EINVAL, "stream %d reads page %d that stream %d writes", i, p,
                      owner[p]);
      }
    }
  return ARDIT_OK;
}

int check_ptr(const void* p, const char* name) {
  if (!p) return fail(ARDIT_EINVAL, "%s is NULL", name);
  if (misaligned(p)) return fail(ARDIT_EINVAL, "%s must be 16-byte aligned", name);
  return ARDIT_OK;
}

int check_block_weights(const ardit_block_weights* w, bool ctx) {
  if (!w) return fail(ARDIT_EINVAL, "weights is NULL");
  if (ctx) {
    ARDIT_TRY(check_ptr(w->w_ck, "w_ck"));
    ARDIT_TRY(check_ptr(w->b_ck, "b_ck"));
    ARDIT_TRY(check_ptr(w->g_ck, "g_ck"));
    ARDIT_TRY(check_ptr(w->w_cv, "w_cv"));
    ARDIT_TRY(check_ptr(w->b_cv, "b_cv"));
    return ARDIT_OK;
  }
  const void* p[] = {w->w_qkv, w->b_qkv, w->g_q, w->g_k, w->w_o, w->b_o, w->g_n3, w->w_cq,
                     w->b_cq, w->g_cq, w->w_co, w->b_co, w->w_1, w->b_1, w->w_2, w->b_2,
                     w->mod_table};
  const char* n[] = {"w_qkv", "b_qkv", "g_q", "g_k", "w_o", "b_o", "g_n3", "w_cq", "b_cq",
                     "g_cq", "w_co", "b_co", "w_1", "b_1", "w_2", "b_2", "mod_table"};
  for (size_t i = 0; i < sizeof(p) / sizeof(p[0]); ++i) ARDIT_TRY(check_ptr(p[i], n[i]));
  return ARDIT_OK;
}

// ------------------------------------------------------------ workspace

struct Ws {
  size_t tsin, te1, te2;             // fp32 time-MLP scratch
  size_t h, qkv, q, o, x1, x2, u;    // bf16 block activations
  size_t ck, cv;                     // bf16 text projections
  size_t attn;                       // fp32 partial results of split attention
  size_t sp_qbar, sp_scores, sp_lists;   // block-sparse selection (last, sized by the batch)
  size_t f8q, f8kv;                      // FP8 attention operands
  size_t gmod, gv;                       // chunk generation: fp32 modulation, bf16 velocity
  size_t total;
};

Ws ws_layout(const ardit_dims* d, int B, int64_t N, int64_t Nc,
             const SparseBytes& sp = SparseBytes()) {
  Ws w;
  size_t off = 0;
  const size_t D = d->dim, F = d->ffn_dim;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += up(bytes);
    return o;
  };
  w.tsin = take(sizeof(float) * B * ARDIT_TIME_FREQ_DIM);
  w.te1 = take(sizeof(float) * B * D);
  w.te2 = take(sizeof(float) * B * D);
  w.h = take(2 * N * D);
  w.qkv = take(2 * N * 3 * D);
  w.q = take(2 * N * D);
  w.o = take(2 * N * D);
  w.x1 = take(4 * N * D);   // fp32: the residual stream inside a block stays fp32
  w.x2 = take(4 * N * D);
  w.u = take(2 * N * F);
  w.ck = take(2 * Nc * D);
  w.cv = take(2 * Nc * D);
  w.attn = take(attention_split_bytes(d->head_dim));
  w.sp_qbar = take(sp.qbar);
  w.sp_scores = take(sp.scores);
  w.sp_lists = take(sp.lists);
  w.f8q = take(sp.f8q);
  w.f8kv = take(sp.f8kv);
  w.gmod = take(sizeof(float) * B * 6 * D);
  w.gv = take(2 * N * D);
  w.total = off;
  return w;
}

int64_t sum_q(const ardit_batch* b) {
  int64_t n = 0;
  if (b->q_lens)
    for (int i = 0; i < b->n_streams; ++i) n += b->q_lens[i];
  return n;
}
int64_t sum_ctx(const ardit_batch* b) {
  int64_t n = 0;
  if (b->ctx_lens)
    for (int i = 0; i < b->n_streams; ++i) n += b->ctx_lens[i];
  return n;
}

int check_ws(const ardit_dims* d, const ardit_batch* b, const void* ws, size_t ws_bytes,
             Ws* out) {
  *out = ws_layout(d, b->n_streams, sum_q(b), sum_ctx(b), sparse_ws_bytes(d, b));
  if (!ws) return fail(ARDIT_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
    return fail(ARDIT_EINVAL, "workspace must be %zu-byte aligned", kAlign);
  if (ws_bytes < out->total)
    return fail(ARDIT_EWORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, out->total);
  return ARDIT_OK;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

RowStreams q_streams(const ardit_batch* b) {
  RowStreams rs;
  rs.n = b->n_streams;
  int row = 0;
  for (int i = 0; i < b->n_streams; ++i) {
    rs.s[i].row_begin = row;
    rs.s[i].len = b->q_lens[i];
    rs.s[i].cache_len = b->cache_lens ? b->cache_lens[i] : 0;
    rs.s[i].frame_pos0 = b->frame_pos0 ? b->frame_pos0[i] : 0;
    row += b->q_lens[i];
  }
  return rs;
}

RowStreams ctx_streams(const ardit_batch* b) {
  RowStreams rs;
  rs.n = b->n_streams;
  int row = 0;
  for (int i = 0; i < b->n_streams; ++i) {
    rs.s[i].row_begin = row;
    rs.s[i].len = b->ctx_lens[i];
    rs.s[i].cache_len = 0;
    rs.s[i].frame_pos0 = 0;
    row += b->ctx_lens[i];
  }
  return rs;
}

// ---------------------------------------------------------------- timing
// kinds of timed launches (bits of the enable mask)
enum TimedKind : int { kTimeAttn = 0, kTimeGemm = 1, kTimeElem = 2, kTimeKinds = 3 };

struct TimedRec {
  int kind;
  const char* what;   // static string naming the launch
  hipEvent_t e0, e1;
};

struct Timing {
  std::mutex mu;
  unsigned mask = 0;
  void* flush = nullptr;     // read before every timed launch when set (cold caches)
  size_t flush_bytes = 0;
  uint32_t* flush_sink = nullptr;   // one word per workgroup of the flush read
  std::vector<hipEvent_t> pool;
  std::vector<TimedRec> rec;
};
Timing& timing() {
  static Timing t;
  return t;
}

hipEvent_t take_event(Timing& t) {
  if (!t.pool.empty()) {
    hipEvent_t e = t.pool.back();
    t.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Events around one launch while timing of its kind is on: begin() before
// the launch, end() after it.
struct TimedLaunch {
  hipStream_t st;
  int kind;
  const char* what;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  void* flush = nullptr;
  size_t flush_bytes = 0;
  uint32_t* flush_sink = nullptr;
  TimedLaunch(hipStream_t s, int k, const char* w) : st(s), kind(k), what(w) {
    Timing& tm = timing();
    std::lock_guard<std::mutex> g(tm.mu);
    if (tm.mask & (1u << k)) {
      e0 = take_event(tm);
      e1 = take_event(tm);
      flush = tm.flush;
      flush_bytes = tm.flush_bytes;
      flush_sink = tm.flush_sink;
    }
  }
  hipError_t begin() {
    if (!(e0 && e1)) return hipSuccess;
    if (flush) {
      const hipError_t f = launch_micro_read(st, flush, flush_bytes, flush_sink);
      if (f != hipSuccess) return f;
    }
    return hipEventRecord(e0, st);
  }
  hipError_t end() {
    if (!(e0 && e1)) return hipSuccess;
    const hipError_t e = hipEventRecord(e1, st);
    Timing& tm = timing();
    std::lock_guard<std::mutex> g(tm.mu);
    tm.rec.push_back(TimedRec{kind, what, e0, e1});
    e0 = e1 = nullptr;
    return e;
  }
  // events not handed to the record (a failed launch, or only one event
  // created) go back to the pool
  ~TimedLaunch() {
    if (!e0 && !e1) return;
    Timing& tm = timing();
    std::lock_guard<std::mutex> g(tm.mu);
    for (hipEvent_t e : {e0, e1}) {
      if (!e) continue;
      try {
        tm.pool.push_back(e);
      } catch (...) {
        (void)hipEventDestroy(e);
      }
    }
  }
};

#define ARDIT_TIMED(kind, expr, what)                              \
  do {                                                             \
    TimedLaunch tl_(st, kind, what);                               \
    ARDIT_HIP(tl_.begin(), "hipEventRecord");                      \
    ARDIT_HIP(expr, what);                                         \
    ARDIT_HIP(tl_.end(), "hipEventRecord");                        \
  } while (0)

// launches the self-attention kernels (block selection first when sparse);
// while timing is on, events bracket the attention kernel itself
int run_self_attention(hipStream_t st, const AttnArgs& a, int hd) {
  if (a.blocks) ARDIT_HIP(launch_sparse_select(st, a, hd), "block selection launch");
  if (a.blocks)
    ARDIT_TIMED(kTimeAttn, launch_sparse_attention(st, a, hd), "block-sparse attention launch");
  else
    ARDIT_TIMED(kTimeAttn, launch_attention(st, a, hd, true), "self-attention launch");
  return ARDIT_OK;
}

// Self-attention over the pages, streams in batch order, not yet planned.
AttnArgs self_attn_base(const ardit_dims* d, const ardit_batch* b, const void* q,
                        const ardit_kv_paged* kv, void* o) {
  AttnArgs a;
  memset(&a, 0, sizeof(a));
  a.q = static_cast<const bf16_t*>(q);
  a.ldq = d->dim;
  a.o = static_cast<bf16_t*>(o);
  a.ldo = d->dim;
  a.k = static_cast<const bf16_t*>(kv->k_pages);
  a.v = static_cast<const bf16_t*>(kv->v_pages);
  a.page_table = kv->page_table;
  a.max_frames = kv->max_frames;
  a.n_pages = kv->n_pages;
  a.T = tokens_per_frame(d);
  a.fT = make_fastdiv(a.T);
  a.H = d->n_heads;
  a.scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(d->head_dim)));
  a.n_streams = b->n_streams;
  int row = 0;
  for (int i = 0; i < b->n_streams; ++i) {
    AttnStream& s = a.s[i];
    s.q_off = row;
    s.q_len = b->q_lens[i];
    s.kv_len = b->cache_lens[i] + b->q_lens[i];
    s.stream = i;
    s.base_off = 0;
    s.T = a.T;
    row += b->q_lens[i];
  }
  return a;
}

// Planned self-attention.  Sparse batches run the block-sparse kernels with
// their lists and key means in the workspace regions of L.
AttnArgs self_attn_args(const ardit_dims* d, const ardit_batch* b, const void* q,
                        const ardit_kv_paged* kv, void* o, void* ws, const Ws& L) {
  AttnArgs a = self_attn_base(d, b, q, kv, o);
  if (batch_sparse(b))
    plan_sparse_attention(a, b->sparsity, at<int32_t>(ws, L.sp_lists), 0, at<float>(ws, L.sp_qbar),
                          at<float>(ws, L.sp_scores));
  else
    plan_attention(a, d->head_dim, at<float>(ws, L.attn));
  return a;
}

// The streams of a planned batch whose quantisation mode is `mode`, renumbered.
AttnArgs stream_subset(const AttnArgs& all, const ardit_batch* b, int mode, bool sparse) {
  AttnArgs a = all;
  int n = 0;
  for (int i = 0; i < all.n_streams; ++i) {
    const int m = b->quant ? b->quant[all.s[i].stream] : ARDIT_QUANT_BF16;
    if (m == mode) a.s[n++] = all.s[i];
  }
  a.n_streams = n;
  finish_plan(a, sparse);
  return a;
}

// Self-attention of a batch: block selection first when a stream is sparse,
// then the 16-bit streams on the bf16 kernels and the FP8 streams through the
// quantisation pre-pass and the FP8 kernel.
int self_attention(hipStream_t st, const ardit_dims* d, const ardit_batch* b, const void* q,
                   const ardit_kv_paged* kv, void* o, void* ws, const Ws& L) {
  const int hd = d->head_dim;
  if (!batch_fp8(b)) return run_self_attention(st, self_attn_args(d, b, q, kv, o, ws, L), hd);
  const bool sparse = batch_sparse(b);
  AttnArgs all = self_attn_base(d, b, q, kv, o);
  if (sparse) {
    plan_sparse_attention(all, b->sparsity, at<int32_t>(ws, L.sp_lists), 0,
                          at<float>(ws, L.sp_qbar), at<float>(ws, L.sp_scores));
    ARDIT_HIP(launch_sparse_select(st, all, hd), "block selection launch");
  } else {
    for (int i = 0; i < all.n_streams; ++i) {
      AttnStream& s = all.s[i];
      s.n_qtiles = static_cast<int32_t>(ceil_div(s.q_len, kAttnQTile));
      s.n_tiles = static_cast<int32_t>(ceil_div(s.kv_len, kAttnKTile));
      s.n_keep = s.n_tiles;
    }
  }
  AttnArgs a16 = stream_subset(all, b, ARDIT_QUANT_BF16, sparse);
  if (a16.total_items > 0) {
    if (sparse) {
      ARDIT_HIP(launch_sparse_attention(st, a16, hd), "block-sparse attention launch");
    } else {
      plan_attention(a16, hd, at<float>(ws, L.attn));
      ARDIT_HIP(launch_attention(st, a16, hd, true), "self-attention launch");
    }
  }
  AttnArgs a8 = stream_subset(all, b, ARDIT_QUANT_FP8, sparse);
  if (a8.total_items > 0) {
    uint8_t* f8q = at<uint8_t>(ws, L.f8q);
    const size_t qb = static_cast<size_t>(sum_q(b)) * d->dim;
    a8.q8 = f8q;
    a8.q8s = f8q + up(qb);
    plan_fp8_buffers(a8, hd, at<uint8_t>(ws, L.f8kv));
    ARDIT_HIP(launch_mx_quantize_rows(st, static_cast<const bf16_t*>(q), sum_q(b), d->dim, d->dim,
                                      a8.q8, a8.q8s), "FP8 query quantisation");
    ARDIT_HIP(launch_fp8_kv_prep(st, a8, hd), "FP8 key / value quantisation");
    ARDIT_TIMED(kTimeAttn, launch_attention_fp8(st, a8, hd, sparse), "FP8 attention launch");
  }
  return ARDIT_OK;
}

AttnArgs cross_attn_args(const ardit_dims* d, const ardit_batch* b, const void* q,
                         const void* ctx_k, const void* ctx_v, void* o, float* split_ws) {
  AttnArgs a;
  memset(&a, 0, sizeof(a));
  a.q = static_cast<const bf16_t*>(q);
  a.ldq = d->dim;
  a.o = static_cast<bf16_t*>(o);
  a.ldo = d->dim;
  a.k = static_cast<const bf16_t*>(ctx_k);
  a.v = static_cast<const bf16_t*>(ctx_v);
  a.T = 1;
  a.fT = make_fastdiv(1);
  a.H = d->n_heads;
  a.scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(d->head_dim)));
  a.n_streams = b->n_streams;
  int row = 0, crow = 0;
  for (int i = 0; i < b->n_streams; ++i) {
    AttnStream& s = a.s[i];
    s.q_off = row;
    s.q_len = b->q_lens[i];
    s.kv_len = b->ctx_lens[i];
    s.stream = i;
    s.base_off = crow * d->dim;
    s.T = b->ctx_lens[i];
    row += b->q_lens[i];
    crow += b->ctx_lens[i];
  }
  plan_attention(a, d->head_dim, split_ws);
  return a;
}

// the block chain on validated arguments
// (kv_only: stop once the chunk's keys and values are in the pages; out is
// not written)
int block_chain(hipStream_t st, const ardit_dims* d, const ardit_batch* b, const void* xin,
                const ardit_kv_paged* kv, const float* mod, const void* ctx_k, const void* ctx_v,
                const ardit_block_weights* w, void* out, void* ws, const Ws& L,
                bool kv_only = false) {
  const int N = static_cast<int>(sum_q(b));
  const int D = d->dim, F = d->ffn_dim, H = d->n_heads, hd = d->head_dim;
  const int Lq = chunk_tokens(d);
  const bf16_t* x = static_cast<const bf16_t*>(xin);
  bf16_t* h = at<bf16_t>(ws, L.h);
  bf16_t* qkv = at<bf16_t>(ws, L.qkv);
  bf16_t* q = at<bf16_t>(ws, L.q);
  bf16_t* o = at<bf16_t>(ws, L.o);
  float* x1 = at<float>(ws, L.x1);
  float* x2 = at<float>(ws, L.x2);
  bf16_t* u = at<bf16_t>(ws, L.u);
  bf16_t* y = static_cast<bf16_t*>(out);
  const float* mt = w->mod_table;
  const RowStreams rs = q_streams(b);
  auto B16 = [](const void* p) { return static_cast<const bf16_t*>(p); };

  // adaLN RMSNorm #1 and the QKV projection
  ARDIT_TIMED(kTimeElem, launch_adaln_norm(st, x, false, h, N, D, mod, mt, 0, 1, Lq, d->eps),
              "adaln_norm");
  GemmEpiArgs e;
  e.bias = B16(w->b_qkv);
  ARDIT_TIMED(kTimeGemm, launch_gemm(st, kEpiBias, h, D, B16(w->w_qkv), D, qkv, 3 * D, N, 3 * D, D, e),
              "qkv gemm");
  // QK-norm, 3D RoPE, append k~ and v to the pages
  RopeGeom rg{D, H, hd, tokens_per_frame(d), d->lat_w, kv->max_frames, kv->n_pages, d->eps,
              d->rope_theta};
  ARDIT_TIMED(kTimeElem,
              launch_kv_append(st, qkv, N, rg, B16(w->g_q), B16(w->g_k), q,
                               static_cast<bf16_t*>(kv->k_pages),
                               static_cast<bf16_t*>(kv->v_pages), kv->page_table, rs),
              "qk_norm_rope / kv append");
  if (kv_only) return ARDIT_OK;
  // self-attention over [cache | chunk]
  ARDIT_TRY(self_attention(st, d, b, q, kv, o, ws, L));
  // x1 = x + gate1 * (o W_o^T + b_o)
  e = GemmEpiArgs();
  e.bias = B16(w->b_o);
  e.res = x;
  e.ldr = D;
  e.mod = mod;
  e.mod_table = mt;
  e.gate_row = 2;
  e.dim = D;
  e.rows_per_stream = Lq;
  e.out_f32 = true;
  ARDIT_TIMED(kTimeGemm, launch_gemm(st, kEpiBiasGateRes, o, D, B16(w->w_o), D, x1, D, N, D, D, e),
              "o gemm");
  // cross-attention query: rms(rms(x1) g_n3 W_cq^T + b_cq) g_cq
  ARDIT_TIMED(kTimeElem, launch_rms_gain(st, x1, true, h, N, D, B16(w->g_n3), d->eps),
              "cross pre-norm");
  e = GemmEpiArgs();
  e.bias = B16(w->b_cq);
  ARDIT_TIMED(kTimeGemm, launch_gemm(st, kEpiBias, h, D, B16(w->w_cq), D, q, D, N, D, D, e),
              "cq gemm");
  ARDIT_TIMED(kTimeElem, launch_rms_gain(st, q, false, q, N, D, B16(w->g_cq), d->eps),
              "cross q-norm");
  const AttnArgs ca = cross_attn_args(d, b, q, ctx_k, ctx_v, o, at<float>(ws, L.attn));
  ARDIT_HIP(launch_attention(st, ca, hd, false), "cross-attention");
  // x2 = x1 + o_c W_co^T + b_co
  e = GemmEpiArgs();
  e.bias = B16(w->b_co);
  e.res = x1;
  e.ldr = D;
  e.res_f32 = true;
  e.out_f32 = true;
  ARDIT_TIMED(kTimeGemm, launch_gemm(st, kEpiBiasRes, o, D, B16(w->w_co), D, x2, D, N, D, D, e),
              "co gemm");
  // FFN: out = x2 + gate2 * (GELU(adaLN2(x2) W_1^T + b_1) W_2^T + b_2)
  ARDIT_TIMED(kTimeElem, launch_adaln_norm(st, x2, true, h, N, D, mod, mt, 3, 4, Lq, d->eps),
              "adaln_norm 2");
  e = GemmEpiArgs();
  e.bias = B16(w->b_1);
  ARDIT_TIMED(kTimeGemm, launch_gemm(st, kEpiBiasGelu, h, D, B16(w->w_1), D, u, F, N, F, D, e),
              "ffn up");
  e = GemmEpiArgs();
  e.bias = B16(w->b_2);
  e.res = x2;
  e.ldr = D;
  e.res_f32 = true;
  e.mod = mod;
  e.mod_table = mt;
  e.gate_row = 5;
  e.dim = D;
  e.rows_per_stream = Lq;
  ARDIT_TIMED(kTimeGemm, launch_gemm(st, kEpiBiasGateRes, u, F, B16(w->w_2), F, y, D, N, D, F, e),
              "ffn down");
  return ARDIT_OK;
}

int check_time_weights(const ardit_time_weights* tw) {
  if (!tw) return fail(ARDIT_EINVAL, "time weights NULL");
  const void* p[] = {tw->w_t1, tw->b_t1, tw->w_t2, tw->b_t2, tw->w_m, tw->b_m};
  const char* n[] = {"w_t1", "b_t1", "w_t2", "b_t2", "w_m", "b_m"};
  for (int i = 0; i < 6; ++i) ARDIT_TRY(check_ptr(p[i], n[i]));
  return ARDIT_OK;
}

// sinusoid of t, then the time MLP, into mod_out [B][6][D]
int time_mod_chain(hipStream_t st, const ardit_dims* d, int B, const float* t_host,
                   const ardit_time_weights* tw, float* mod_out, void* ws, const Ws& L) {
  const int D = d->dim;
  float* s = at<float>(ws, L.tsin);
  float* e1 = at<float>(ws, L.te1);
  float* e2 = at<float>(ws, L.te2);
  auto B16 = [](const void* q) { return static_cast<const bf16_t*>(q); };
  ARDIT_HIP(launch_time_sinusoid(st, t_host, B, s), "time sinusoid");
  ARDIT_HIP(launch_linear_small(st, s, B, ARDIT_TIME_FREQ_DIM, B16(tw->w_t1), B16(tw->b_t1), D,
                                e1, false), "time mlp 1");
  ARDIT_HIP(launch_linear_small(st, e1, B, D, B16(tw->w_t2), B16(tw->b_t2), D, e2, true),
            "time mlp 2");
  ARDIT_HIP(launch_linear_small(st, e2, B, D, B16(tw->w_m), B16(tw->b_m), 6 * D, mod_out, true),
            "time modulation");
  return ARDIT_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return na && nb && x < y + nb && y < x + na;
}

int check_block_args(hipStream_t st, const ardit_dims* d, const ardit_batch* b, const void* x,
                     const ardit_kv_paged* kv, const float* mod, const void* ctx_k,
                     const void* ctx_v, const ardit_block_weights* w, const void* out) {
  ARDIT_TRY(check_dims(d));
  ARDIT_TRY(check_batch(d, b, kUseQ | kUseCache | kUsePos | kUseCtx | kChunkQ));
  ARDIT_TRY(check_kv(d, b, kv));
  ARDIT_TRY(check_sparse(d, b));
  ARDIT_TRY(check_ptr(x, "x"));
  ARDIT_TRY(check_ptr(out, "out"));
  ARDIT_TRY(check_ptr(mod, "mod"));
  ARDIT_TRY(check_ptr(ctx_k, "ctx_k"));
  ARDIT_TRY(check_ptr(ctx_v, "ctx_v"));
  ARDIT_TRY(check_block_weights(w, false));
  return check_pages(st, d, b, kv, true);
}

// ------------------------------------------------ allocation-free attention
// Scratch of ardit_attn_fwd_noalloc: the split schedule's partial results
// (dense batches) or the block selection's means, scores and lists (sparse
// batches).  One copy per GPU the library runs on, held until the process
// ends.  Host code never uses the array's name as an address: the device
// address comes from hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = static_cast<size_t>(72) << 20;
constexpr int kScratchDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on device dev, which must be current.
int scratch_address(int dev, void** out) {
  static std::mutex mu;
  static void* addr[kScratchDevices] = {};
  if (dev < 0 || dev >= kScratchDevices)
    return fail(ARDIT_EUNSUPPORTED, "device %d beyond the %d the scratch table covers", dev,
                kScratchDevices);
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    ARDIT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!p) return fail(ARDIT_EHIP, "hipGetSymbolAddress(scratch) gave a null address");
    addr[dev] = p;
  }
  *out = addr[dev];
  return ARDIT_OK;
}

// Scratch bytes a batch's self-attention needs: the sparse selection's
// regions, else the split schedule's partial results.
size_t noalloc_scratch_bytes(const ardit_dims* d, const ardit_batch* b) {
  if (batch_sparse(b)) {
    const SparseBytes sp = sparse_ws_bytes(d, b);
    return up(sp.qbar) + up(sp.scores) + up(sp.lists);
  }
  return up(attention_split_bytes(d->head_dim));
}

}  // namespace

namespace ardit {
// the calling thread's error detail, for the controller's translation unit
int set_error(int status, const char* msg) { return fail(status, "%s", msg); }
// every entry point ends here when a host-side exception (an allocation that
// failed) would otherwise leave the library through its C interface
int host_failure() { return fail(ARDIT_EHOST, "host memory exhausted"); }
}  // namespace ardit

// ======================================================================== ABI
extern "C" {

const char* ardit_status_str(int s) {
  switch (s) {
    case ARDIT_OK: return "ARDIT_OK";
    case ARDIT_EINVAL: return "ARDIT_EINVAL";
    case ARDIT_ESHAPE: return "ARDIT_ESHAPE";
    case ARDIT_ECAPACITY: return "ARDIT_ECAPACITY";
    case ARDIT_EWORKSPACE: return "ARDIT_EWORKSPACE";
    case ARDIT_EUNSUPPORTED: return "ARDIT_EUNSUPPORTED";
    case ARDIT_EHIP: return "ARDIT_EHIP";
    case ARDIT_EHOST: return "ARDIT_EHOST";
    default: return "ARDIT_UNKNOWN";
  }
}

const char* ardit_last_error(void) { return g_last_error; }

int ardit_version(void) { return 502; }

int ardit_workspace_size(const ardit_dims* dims, const ardit_batch* batch, size_t* bytes) try {
  ARDIT_TRY(check_dims(dims));
  if (!bytes) return fail(ARDIT_EINVAL, "bytes is NULL");
  ARDIT_TRY(check_batch(dims, batch, 0));
  if (batch->q_lens) ARDIT_TRY(check_batch(dims, batch, kUseQ));
  if (batch->cache_lens) ARDIT_TRY(check_batch(dims, batch, kUseCache));
  if (batch->ctx_lens) ARDIT_TRY(check_batch(dims, batch, kUseCtx));
  if (batch_sparse(batch)) {
    if (!batch->q_lens || !batch->cache_lens)
      return fail(ARDIT_EINVAL, "a sparse batch needs q_lens and cache_lens");
    ARDIT_TRY(check_batch(dims, batch, kUseQ | kUseCache));
    ARDIT_TRY(check_sparse(dims, batch));
  }
  *bytes = ws_layout(dims, batch->n_streams, sum_q(batch), sum_ctx(batch),
                     sparse_ws_bytes(dims, batch)).total;
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_time_mod(hipStream_t stream, const ardit_dims* dims, int32_t n_streams,
                   const float* t_host, const ardit_time_weights* tw, float* mod_out, void* ws,
                   size_t ws_bytes) try {
  ARDIT_TRY(check_dims(dims));
  if (n_streams < 1 || n_streams > ARDIT_MAX_STREAMS)
    return fail(ARDIT_EINVAL, "n_streams %d not in [1, %d]", n_streams, ARDIT_MAX_STREAMS);
  if (!t_host) return fail(ARDIT_EINVAL, "t_host is NULL");
  ARDIT_TRY(check_time_weights(tw));
  ARDIT_TRY(check_ptr(mod_out, "mod_out"));
  ARDIT_TRY(check_ptr(ws, "ws"));
  const Ws L = ws_layout(dims, n_streams, 0, 0);
  if (ws_bytes < L.h) return fail(ARDIT_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.h);
  return time_mod_chain(stream, dims, n_streams, t_host, tw, mod_out, ws, L);
} catch (...) {
  return host_failure();
}

int ardit_ctx_kv(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                 const void* ctx, const ardit_block_weights* w, void* ctx_k, void* ctx_v,
                 void* ws, size_t ws_bytes) try {
  ARDIT_TRY(check_dims(dims));
  ARDIT_TRY(check_batch(dims, batch, kUseCtx));
  ARDIT_TRY(check_ptr(ctx, "ctx"));
  ARDIT_TRY(check_ptr(ctx_k, "ctx_k"));
  ARDIT_TRY(check_ptr(ctx_v, "ctx_v"));
  ARDIT_TRY(check_block_weights(w, true));
  ardit_batch cb = *batch;
  cb.q_lens = nullptr;
  Ws L;
  ARDIT_TRY(check_ws(dims, &cb, ws, ws_bytes, &L));
  const int Nc = static_cast<int>(sum_ctx(batch));
  const int D = dims->dim;
  bf16_t* ck = at<bf16_t>(ws, L.ck);
  bf16_t* cv = at<bf16_t>(ws, L.cv);
  const RowStreams rs = ctx_streams(batch);
  auto B16 = [](const void* q) { return static_cast<const bf16_t*>(q); };
  GemmEpiArgs e;
  e.bias = B16(w->b_ck);
  ARDIT_HIP(launch_gemm(stream, kEpiBias, B16(ctx), D, B16(w->w_ck), D, ck, D, Nc, D, D, e),
            "ctx k gemm");
  ARDIT_HIP(launch_ctx_k_layout(stream, ck, Nc, D, dims->n_heads, dims->head_dim, B16(w->g_ck),
                                dims->eps, static_cast<bf16_t*>(ctx_k), rs),
            "ctx k layout");
  e.bias = B16(w->b_cv);
  ARDIT_HIP(launch_gemm(stream, kEpiBias, B16(ctx), D, B16(w->w_cv), D, cv, D, Nc, D, D, e),
            "ctx v gemm");
  ARDIT_HIP(launch_v_transpose(stream, cv, D, 0, Nc, D, dims->n_heads, dims->head_dim,
                               static_cast<bf16_t*>(ctx_v), false, 0, nullptr, 0, 0, rs),
            "ctx v layout");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_kv_append(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                    const void* qkv, const void* g_q, const void* g_k, const ardit_kv_paged* kv,
                    void* q_out) try {
  ARDIT_TRY(check_dims(dims));
  ARDIT_TRY(check_batch(dims, batch, kUseQ | kUseCache | kUsePos | kChunkQ));
  ARDIT_TRY(check_kv(dims, batch, kv));
  ARDIT_TRY(check_ptr(qkv, "qkv"));
  ARDIT_TRY(check_ptr(g_q, "g_q"));
  ARDIT_TRY(check_ptr(g_k, "g_k"));
  ARDIT_TRY(check_ptr(q_out, "q_out"));
  ARDIT_TRY(check_pages(stream, dims, batch, kv, true));
  const int N = static_cast<int>(sum_q(batch));
  const RowStreams rs = q_streams(batch);
  const int D = dims->dim;
  RopeGeom rg{D, dims->n_heads, dims->head_dim, tokens_per_frame(dims), dims->lat_w,
              kv->max_frames, kv->n_pages, dims->eps, dims->rope_theta};
  ARDIT_HIP(launch_kv_append(stream, static_cast<const bf16_t*>(qkv), N, rg,
                             static_cast<const bf16_t*>(g_q), static_cast<const bf16_t*>(g_k),
                             static_cast<bf16_t*>(q_out), static_cast<bf16_t*>(kv->k_pages),
                             static_cast<bf16_t*>(kv->v_pages), kv->page_table, rs),
            "qk_norm_rope / kv append");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_attn_fwd(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                   const void* q, const ardit_kv_paged* kv, void* o, void* ws, size_t ws_bytes) try {
  ARDIT_TRY(check_dims(dims));
  ARDIT_TRY(check_batch(dims, batch, kUseQ | kUseCache));
  ARDIT_TRY(check_kv(dims, batch, kv));
  ARDIT_TRY(check_sparse(dims, batch));
  ARDIT_TRY(check_ptr(q, "q"));
  ARDIT_TRY(check_ptr(o, "o"));
  Ws L;
  ARDIT_TRY(check_ws(dims, batch, ws, ws_bytes, &L));
  ARDIT_TRY(check_pages(stream, dims, batch, kv, false));
  return self_attention(stream, dims, batch, q, kv, o, ws, L);
} catch (...) {
  return host_failure();
}

int ardit_attn_fwd_noalloc(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                           const void* q, const ardit_kv_paged* kv, void* o) try {
  ARDIT_TRY(check_dims(dims));
  ARDIT_TRY(check_batch(dims, batch, kUseQ | kUseCache));
  ARDIT_TRY(check_kv(dims, batch, kv));
  ARDIT_TRY(check_sparse(dims, batch));
  ARDIT_TRY(check_ptr(q, "q"));
  ARDIT_TRY(check_ptr(o, "o"));
  if (batch_fp8(batch))
    return fail(ARDIT_EUNSUPPORTED, "the allocation-free attention runs bf16 streams only");
  const size_t need = noalloc_scratch_bytes(dims, batch);
  if (need > kScratchBytes)
    return fail(ARDIT_EWORKSPACE, "batch needs %zu bytes of scratch, above the %zu the "
                "allocation-free attention holds", need, kScratchBytes);
  int dev = -1;
  ARDIT_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (stream) {
    hipDevice_t sdev = -1;
    ARDIT_HIP(hipStreamGetDevice(stream, &sdev), "hipStreamGetDevice");
    if (sdev != dev)
      return fail(ARDIT_EINVAL, "the stream belongs to device %d, device %d is current", sdev,
                  dev);
  }
  void* base = nullptr;
  ARDIT_TRY(scratch_address(dev, &base));
  AttnArgs a = self_attn_base(dims, batch, q, kv, o);
  const int hd = dims->head_dim;
  if (batch_sparse(batch)) {
    const SparseBytes sp = sparse_ws_bytes(dims, batch);
    char* c = static_cast<char*>(base);
    plan_sparse_attention(a, batch->sparsity, reinterpret_cast<int32_t*>(c + up(sp.qbar) +
                                                                           up(sp.scores)),
                          0, reinterpret_cast<float*>(c), reinterpret_cast<float*>(c + up(sp.qbar)));
    ARDIT_HIP(launch_sparse_select(stream, a, hd), "block selection launch");
    ARDIT_HIP(launch_sparse_attention(stream, a, hd), "block-sparse attention launch");
  } else {
    plan_attention(a, hd, static_cast<float*>(base));
    ARDIT_HIP(launch_attention(stream, a, hd, true), "self-attention launch");
  }
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_mx_quantize(hipStream_t stream, const void* x, int64_t rows, int32_t cols, int32_t ld,
                      void* codes, void* scales) try {
  if (!x || !codes || !scales) return fail(ARDIT_EINVAL, "pointers must be non-NULL");
  if (rows < 0 || cols <= 0 || cols % 32 != 0)
    return fail(ARDIT_ESHAPE, "cols %d must be a positive multiple of 32", cols);
  if (ld < cols || ld % 8 != 0) return fail(ARDIT_ESHAPE, "ld %d must be >= cols and a multiple of 8", ld);
  if (misaligned(x) || reinterpret_cast<uintptr_t>(codes) % 8 != 0)
    return fail(ARDIT_EINVAL, "x must be 16-byte and codes 8-byte aligned");
  ARDIT_HIP(launch_mx_quantize_rows(stream, static_cast<const bf16_t*>(x), rows, cols, ld,
                                    static_cast<uint8_t*>(codes), static_cast<uint8_t*>(scales)),
            "mx quantisation launch");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_sparse_select(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                        const void* q, const ardit_kv_paged* kv, int32_t* blocks,
                        int32_t row_stride, void* ws, size_t ws_bytes) try {
  ARDIT_TRY(check_dims(dims));
  ARDIT_TRY(check_batch(dims, batch, kUseQ | kUseCache));
  ARDIT_TRY(check_kv(dims, batch, kv));
  ARDIT_TRY(check_sparse(dims, batch));
  ARDIT_TRY(check_ptr(q, "q"));
  if (!blocks) return fail(ARDIT_EINVAL, "blocks is NULL");
  if (reinterpret_cast<uintptr_t>(blocks) % sizeof(int32_t) != 0)
    return fail(ARDIT_EINVAL, "blocks must be 4-byte aligned");
  int64_t rows = 0;
  int max_keep = 0;
  for (int i = 0; i < batch->n_streams; ++i) {
    const int64_t qn = batch->q_lens[i];
    if (qn <= 0) continue;
    const int nt = static_cast<int>(ceil_div(batch->cache_lens[i] + qn, kAttnKTile));
    const int nk = sparse_keep_count(nt, batch->sparsity ? batch->sparsity[i] : 0.f);
    max_keep = nk > max_keep ? nk : max_keep;
    rows += dims->n_heads * ceil_div(qn, kAttnQTile);
  }
  if (row_stride < max_keep)
    return fail(ARDIT_EINVAL, "row_stride %d below the %d tiles a row keeps", row_stride,
                max_keep);
  if (rows * row_stride >= (int64_t(1) << 31))
    return fail(ARDIT_ECAPACITY, "block lists above 2^31 entries");
  Ws L;
  ARDIT_TRY(check_ws(dims, batch, ws, ws_bytes, &L));
  ARDIT_TRY(check_pages(stream, dims, batch, kv, false));
  AttnArgs a = self_attn_base(dims, batch, q, kv, nullptr);
  plan_sparse_attention(a, batch->sparsity, blocks, row_stride, at<float>(ws, L.sp_qbar),
                        at<float>(ws, L.sp_scores));
  ARDIT_HIP(launch_sparse_select(stream, a, dims->head_dim), "block selection launch");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_block_fwd_varlen(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                           const void* x, const ardit_kv_paged* kv, const float* mod,
                           const void* ctx_k, const void* ctx_v, const ardit_block_weights* w,
                           void* out, void* ws, size_t ws_bytes) try {
  ARDIT_TRY(check_block_args(stream, dims, batch, x, kv, mod, ctx_k, ctx_v, w, out));
  Ws L;
  ARDIT_TRY(check_ws(dims, batch, ws, ws_bytes, &L));
  return block_chain(stream, dims, batch, x, kv, mod, ctx_k, ctx_v, w, out, ws, L);
} catch (...) {
  return host_failure();
}

int ardit_block_fwd(hipStream_t stream, const ardit_dims* dims, const void* x, ardit_kv_paged kv,
                    int32_t cache_len, int32_t frame_pos0, const float* mod, const void* ctx_k,
                    const void* ctx_v, int32_t ctx_len, const ardit_block_weights* w, void* out,
                    void* ws, size_t ws_bytes) try {
  ARDIT_TRY(check_dims(dims));
  const int32_t q_len = chunk_tokens(dims);
  ardit_batch b;
  b.n_streams = 1;
  b.q_lens = &q_len;
  b.cache_lens = &cache_len;
  b.frame_pos0 = &frame_pos0;
  b.ctx_lens = &ctx_len;
  b.sparsity = nullptr;
  b.quant = nullptr;
  return ardit_block_fwd_varlen(stream, dims, &b, x, &kv, mod, ctx_k, ctx_v, w, out, ws,
                                ws_bytes);
} catch (...) {
  return host_failure();
}

int ardit_stack_fwd(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                    int32_t n_layers, const void* x, const ardit_kv_paged* kv, const float* mod,
                    const void* const* ctx_k, const void* const* ctx_v,
                    const ardit_block_weights* w, void* out, void* ws, size_t ws_bytes) try {
  if (n_layers < 1) return fail(ARDIT_EINVAL, "n_layers %d must be >= 1", n_layers);
  if (!kv || !ctx_k || !ctx_v || !w) return fail(ARDIT_EINVAL, "per-layer arrays must be non-NULL");
  for (int l = 0; l < n_layers; ++l)
    ARDIT_TRY(check_block_args(stream, dims, batch, x, &kv[l], mod, ctx_k[l], ctx_v[l], &w[l], out));
  if (x == out) return fail(ARDIT_EINVAL, "stack input and output must differ");
  Ws L;
  ARDIT_TRY(check_ws(dims, batch, ws, ws_bytes, &L));
  // layer 0 reads x and writes out; later layers update out in place (a
  // layer reads its input only before it writes its output)
  for (int l = 0; l < n_layers; ++l)
    ARDIT_TRY(block_chain(stream, dims, batch, l == 0 ? x : out, &kv[l], mod, ctx_k[l], ctx_v[l],
                          &w[l], out, ws, L));
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_window_pages(int32_t chunk, int32_t sink, int32_t window, int32_t frames_per_chunk,
                       int32_t page_base, int32_t* table, int32_t max_frames,
                       int32_t* cache_frames) try {
  if (chunk < 0 || sink < 0 || window < 0 || frames_per_chunk < 1 || page_base < 0)
    return fail(ARDIT_EINVAL, "chunk %d, sink %d, window %d, page_base %d must be >= 0 and "
                "frames_per_chunk %d >= 1", chunk, sink, window, page_base, frames_per_chunk);
  if (!table || !cache_frames) return fail(ARDIT_EINVAL, "table and cache_frames must be non-NULL");
  const int64_t slots = static_cast<int64_t>(sink) + window + 1;
  if (page_base + slots * frames_per_chunk > INT32_MAX)
    return fail(ARDIT_ECAPACITY, "pages of the stream's slots exceed int32");
  // held chunks in logical order: the sink, then the last `window` before chunk
  const int64_t n_sink = chunk < sink ? chunk : sink;
  const int64_t w_begin = chunk - static_cast<int64_t>(window) > sink ? chunk - window : sink;
  const int64_t held = n_sink + (chunk > w_begin ? chunk - w_begin : 0);
  if ((held + 1) * frames_per_chunk > max_frames)
    return fail(ARDIT_ECAPACITY, "table of %d frames holds fewer than the %lld the window needs",
                max_frames, static_cast<long long>((held + 1) * frames_per_chunk));
  auto slot_of = [&](int64_t k) -> int64_t {
    return k < sink ? k : sink + (k - sink) % (static_cast<int64_t>(window) + 1);
  };
  int64_t f = 0;
  auto put = [&](int64_t k) {
    const int64_t first = page_base + slot_of(k) * frames_per_chunk;
    for (int j = 0; j < frames_per_chunk; ++j) table[f++] = static_cast<int32_t>(first + j);
  };
  for (int64_t k = 0; k < n_sink; ++k) put(k);
  for (int64_t k = w_begin; k < chunk; ++k) put(k);
  put(chunk);
  *cache_frames = static_cast<int32_t>(held * frames_per_chunk);
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_chunk_generate(hipStream_t stream, const ardit_dims* dims, const ardit_batch* batch,
                         int32_t n_layers, const int32_t* n_steps, const float* t_host,
                         int32_t t_ld, const void* x_init, const void* noise,
                         const ardit_kv_paged* kv, const ardit_time_weights* tw,
                         const void* const* ctx_k, const void* const* ctx_v,
                         const ardit_block_weights* w, void* x0_out, void* ws, size_t ws_bytes) try {
  ARDIT_TRY(check_dims(dims));
  ARDIT_TRY(check_batch(dims, batch, kUseQ | kUseCache | kUsePos | kUseCtx | kChunkQ));
  if (n_layers < 1) return fail(ARDIT_EINVAL, "n_layers %d must be >= 1", n_layers);
  if (!kv || !ctx_k || !ctx_v || !w) return fail(ARDIT_EINVAL, "per-layer arrays must be non-NULL");
  if (!n_steps || !t_host) return fail(ARDIT_EINVAL, "n_steps and t_host must be non-NULL");
  const int B = batch->n_streams;
  const int S0 = n_steps[0];
  for (int b = 0; b < B; ++b) {
    if (n_steps[b] < 1 || n_steps[b] > ARDIT_MAX_STEPS)
      return fail(ARDIT_EINVAL, "n_steps[%d] = %d not in [1, %d]", b, n_steps[b],
                  ARDIT_MAX_STEPS);
    if (b > 0 && n_steps[b] > n_steps[b - 1])
      return fail(ARDIT_EINVAL, "n_steps must be non-increasing along the batch (stream %d)", b);
  }
  if (t_ld < S0) return fail(ARDIT_EINVAL, "t_ld %d below n_steps[0] = %d", t_ld, S0);
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < n_steps[b]; ++i) {
      const float t = t_host[static_cast<size_t>(b) * t_ld + i];
      if (!(t >= 0.f && t <= 1000.f))
        return fail(ARDIT_EINVAL, "timestep %g of stream %d step %d not in [0, 1000]",
                    static_cast<double>(t), b, i);
    }
  ARDIT_TRY(check_time_weights(tw));
  ARDIT_TRY(check_ptr(x_init, "x_init"));
  ARDIT_TRY(check_ptr(x0_out, "x0_out"));
  if (S0 > 1) ARDIT_TRY(check_ptr(noise, "noise"));
  Ws L;
  ARDIT_TRY(check_ws(dims, batch, ws, ws_bytes, &L));
  float* mod = at<float>(ws, L.gmod);
  bf16_t* vel = at<bf16_t>(ws, L.gv);
  for (int l = 0; l < n_layers; ++l)
    ARDIT_TRY(check_block_args(stream, dims, batch, x_init, &kv[l], mod, ctx_k[l], ctx_v[l], &w[l],
                               vel));
  const int64_t N = sum_q(batch);
  const int D = dims->dim;
  const size_t xbytes = 2 * static_cast<size_t>(N) * D;
  if (overlaps(x0_out, xbytes, x_init, xbytes) ||
      (S0 > 1 && overlaps(x0_out, xbytes, noise, xbytes * (S0 - 1))) ||
      overlaps(x0_out, xbytes, ws, L.total))
    return fail(ARDIT_EINVAL, "x0_out overlaps x_init, noise or the workspace");

  const int Lq = chunk_tokens(dims);
  // pass i runs the streams with n_steps >= i (a prefix): denoising step i of
  // those with n_steps > i, the commit pass (t = 0) of those with n_steps == i
  for (int i = 0; i <= S0; ++i) {
    int active = 0, denoise = 0;
    float t[ARDIT_MAX_STREAMS];
    SamplerArgs sa;
    for (int b = 0; b < B; ++b) {
      if (n_steps[b] >= i) active = b + 1;
      if (n_steps[b] > i) denoise = b + 1;
      const bool step = i < n_steps[b];
      t[b] = step ? t_host[static_cast<size_t>(b) * t_ld + i] : 0.f;
      sa.tau[b] = static_cast<float>(static_cast<double>(t[b]) / 1000.0);
      sa.tau_next[b] = step && i + 1 < n_steps[b]
          ? static_cast<float>(static_cast<double>(t_host[static_cast<size_t>(b) * t_ld + i + 1]) /
                               1000.0)
          : -1.f;
    }
    ardit_batch sb = *batch;
    sb.n_streams = active;
    ARDIT_TRY(time_mod_chain(stream, dims, active, t, tw, mod, ws, L));
    const void* xin = i == 0 ? x_init : x0_out;
    // a pass that only commits needs no output of its last layer
    const bool commit_only = denoise == 0;
    for (int l = 0; l < n_layers; ++l)
      ARDIT_TRY(block_chain(stream, dims, &sb, l == 0 ? xin : vel, &kv[l], mod, ctx_k[l],
                            ctx_v[l], &w[l], vel, ws, L, commit_only && l == n_layers - 1));
    if (denoise > 0) {
      sa.rows = denoise * Lq;
      sa.rows_per_stream = Lq;
      sa.vec_per_row = D / 8;
      const bf16_t* eps = i + 1 < S0 ? static_cast<const bf16_t*>(noise) + i * N * D : nullptr;
      ARDIT_HIP(launch_sampler(stream, static_cast<const bf16_t*>(xin), vel, eps,
                               static_cast<bf16_t*>(x0_out), sa),
                "sampler");
    }
  }
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_debug_checks(int enable) try {
  if (enable != 0 && enable != 1) return fail(ARDIT_EINVAL, "debug checks %d not 0 or 1", enable);
  g_debug_checks.store(enable, std::memory_order_relaxed);
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_timing_enable(int enable) try {
  if (enable < 0 || enable >= (1 << kTimeKinds))
    return fail(ARDIT_EINVAL, "timing mask %d outside [0, %d]", enable, (1 << kTimeKinds) - 1);
  Timing& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  t.mask = static_cast<unsigned>(enable);
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_timing_collect_kind(int32_t kind, int32_t* launches, double* total_ms) try {
  if (!launches || !total_ms) return fail(ARDIT_EINVAL, "outputs must be non-NULL");
  if (kind < 0 || kind >= kTimeKinds) return fail(ARDIT_EINVAL, "timing kind %d", kind);
  Timing& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  double sum = 0.0;
  int n = 0;
  int status = ARDIT_OK;
  std::vector<TimedRec> keep;
  for (auto& r : t.rec) {
    if (r.kind != kind) {
      keep.push_back(r);
      continue;
    }
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.e1);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.e0, r.e1);
    if (e != hipSuccess && status == ARDIT_OK) status = hip_fail(e, "timing events");
    sum += ms;
    ++n;
    t.pool.push_back(r.e0);
    t.pool.push_back(r.e1);
  }
  t.rec.swap(keep);
  *launches = n;
  *total_ms = sum;
  return status;
} catch (...) {
  return host_failure();
}

int ardit_timing_collect(int32_t* launches, double* total_ms) try {
  return ardit_timing_collect_kind(kTimeAttn, launches, total_ms);
} catch (...) {
  return host_failure();
}

int ardit_timing_flush(void* buf, size_t bytes) try {
  if ((buf == nullptr) != (bytes == 0))
    return fail(ARDIT_EINVAL, "timing flush: buffer and size must be both set or both empty");
  if (buf && (misaligned(buf) || bytes % 16 != 0 || bytes < 128 * 1024))
    return fail(ARDIT_EINVAL, "timing flush buffer must be 16-byte aligned, its size a multiple "
                "of 16 of at least 128 KiB");
  Timing& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  // the read covers all but the last 64 KiB, which take the read's
  // per-workgroup words (at most 32 KiB of them)
  t.flush = buf;
  t.flush_bytes = buf ? bytes - 64 * 1024 : 0;
  t.flush_sink = buf ? reinterpret_cast<uint32_t*>(static_cast<char*>(buf) + t.flush_bytes)
                     : nullptr;
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_timing_records(int32_t kind, int32_t max_records, const char** names, double* ms,
                         int32_t* n_records) try {
  if (!n_records || (max_records > 0 && (!names || !ms)) || max_records < 0)
    return fail(ARDIT_EINVAL, "timing records: NULL output or negative room");
  if (kind < 0 || kind >= kTimeKinds) return fail(ARDIT_EINVAL, "timing kind %d", kind);
  Timing& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  int32_t n = 0;
  for (const auto& r : t.rec) n += r.kind == kind;
  *n_records = n;
  if (n > max_records)
    return fail(ARDIT_ECAPACITY, "%d timed launches of kind %d, room for %d", n, kind,
                max_records);
  int status = ARDIT_OK;
  std::vector<TimedRec> keep;
  int32_t i = 0;
  for (auto& r : t.rec) {
    if (r.kind != kind) {
      keep.push_back(r);
      continue;
    }
    float m = 0.f;
    hipError_t e = hipEventSynchronize(r.e1);
    if (e == hipSuccess) e = hipEventElapsedTime(&m, r.e0, r.e1);
    if (e != hipSuccess && status == ARDIT_OK) status = hip_fail(e, "timing events");
    names[i] = r.what;
    ms[i] = m;
    ++i;
    t.pool.push_back(r.e0);
    t.pool.push_back(r.e1);
  }
  t.rec.swap(keep);
  return status;
} catch (...) {
  return host_failure();
}

int ardit_micro_mfma(hipStream_t stream, int32_t dtype, int32_t workgroups, int32_t iters,
                     float* sink, double* flops) try {
  if (dtype != 0 && dtype != 1) return fail(ARDIT_EINVAL, "micro mfma dtype %d not 0 or 1", dtype);
  if (workgroups < 1 || workgroups > (1 << 20) || iters < 1)
    return fail(ARDIT_EINVAL, "micro mfma: workgroups %d, iters %d", workgroups, iters);
  if (!sink || !flops) return fail(ARDIT_EINVAL, "micro mfma: NULL sink or flops");
  *flops = static_cast<double>(workgroups) * 4 * iters * micro_mfma_flops_per_wave_iter(dtype);
  ARDIT_HIP(launch_micro_mfma(stream, dtype, workgroups, iters, sink), "micro mfma launch");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_micro_copy(hipStream_t stream, const void* src, void* dst, size_t bytes) try {
  if (!src || !dst || misaligned(src) || misaligned(dst) || bytes % 16 != 0)
    return fail(ARDIT_EINVAL, "micro copy: 16-byte aligned buffers and a multiple of 16 bytes");
  if (overlaps(src, bytes, dst, bytes)) return fail(ARDIT_EINVAL, "micro copy: buffers overlap");
  ARDIT_HIP(launch_micro_copy(stream, src, dst, bytes), "micro copy launch");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_micro_read(hipStream_t stream, const void* src, size_t bytes, void* sink,
                     size_t sink_bytes) try {
  if (!src || misaligned(src) || bytes % 16 != 0)
    return fail(ARDIT_EINVAL, "micro read: a 16-byte aligned buffer and a multiple of 16 bytes");
  const size_t need = sizeof(uint32_t) * static_cast<size_t>(micro_read_workgroups(bytes));
  if (!sink || reinterpret_cast<uintptr_t>(sink) % 4 != 0 || sink_bytes < need)
    return fail(ARDIT_EINVAL, "micro read: a 4-byte aligned sink of at least %zu bytes", need);
  ARDIT_HIP(launch_micro_read(stream, src, bytes, static_cast<uint32_t*>(sink)),
            "micro read launch");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

int ardit_micro_fill(hipStream_t stream, void* dst, size_t bytes, uint32_t value) try {
  if (!dst || misaligned(dst) || bytes % 16 != 0)
    return fail(ARDIT_EINVAL, "micro fill: a 16-byte aligned buffer and a multiple of 16 bytes");
  ARDIT_HIP(launch_fill(stream, dst, bytes, value), "micro fill launch");
  return ARDIT_OK;
} catch (...) {
  return host_failure();
}

}  // extern "C"
