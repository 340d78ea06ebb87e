"""ctypes binding of libardit (include/ardit.h).

Argument marshalling only: every function forwards to the C entry point of
the same name.  Tensor arguments may be torch tensors (their data_ptr() is
passed) or raw integer device addresses; `stream` is a HIP stream handle
(int) or None for torch's current stream.  The library must have been built
(``python -m paper_2606_15319_amd.build``); importing this module without it
raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libardit.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_15319_amd.build`")
# The library must run on the same HIP runtime instance as the framework that
# owns the streams and memory handed to it.  torch bundles its own
# libamdhip64.so.7; loading torch first makes the library's dependency on that
# soname resolve to torch's copy instead of pulling in a second runtime.
try:
    import torch  # noqa: F401
except ImportError:  # plain C-ABI use without torch
    pass
_lib = C.CDLL(LIB_PATH)

ARDIT_MAX_STREAMS = 64
ARDIT_MAX_STEPS = 16
STATUS = {0: "ARDIT_OK", -1: "ARDIT_EINVAL", -2: "ARDIT_ESHAPE", -3: "ARDIT_ECAPACITY",
          -4: "ARDIT_EWORKSPACE", -5: "ARDIT_EUNSUPPORTED", -6: "ARDIT_EHIP",
          -7: "ARDIT_EHOST"}


class ArditError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        super().__init__(f"{func}: {STATUS.get(status, status)}: {detail}")
        self.status = status
        self.func = func
        self.detail = detail


# ------------------------------------------------------------------ structs
class ardit_dims(C.Structure):
    _fields_ = [("dim", C.c_int32), ("n_heads", C.c_int32), ("head_dim", C.c_int32),
                ("ffn_dim", C.c_int32), ("frames_per_chunk", C.c_int32),
                ("lat_h", C.c_int32), ("lat_w", C.c_int32),
                ("eps", C.c_float), ("rope_theta", C.c_float)]


class ardit_batch(C.Structure):
    _fields_ = [("n_streams", C.c_int32), ("q_lens", C.POINTER(C.c_int32)),
                ("cache_lens", C.POINTER(C.c_int32)), ("frame_pos0", C.POINTER(C.c_int32)),
                ("ctx_lens", C.POINTER(C.c_int32)), ("sparsity", C.POINTER(C.c_float)),
                ("quant", C.POINTER(C.c_int32))]


class ardit_kv_paged(C.Structure):
    _fields_ = [("k_pages", C.c_void_p), ("v_pages", C.c_void_p), ("page_table", C.c_void_p),
                ("n_pages", C.c_int32), ("max_frames", C.c_int32)]


_BLOCK_FIELDS = ("w_qkv", "b_qkv", "g_q", "g_k", "w_o", "b_o", "g_n3", "w_cq", "b_cq", "g_cq",
                 "w_ck", "b_ck", "g_ck", "w_cv", "b_cv", "w_co", "b_co", "w_1", "b_1", "w_2",
                 "b_2", "mod_table")
_TIME_FIELDS = ("w_t1", "b_t1", "w_t2", "b_t2", "w_m", "b_m")


class ardit_block_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _BLOCK_FIELDS]


class ardit_time_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _TIME_FIELDS]


class ardit_fidelity(C.Structure):
    _fields_ = [("steps", C.c_int32), ("sparsity", C.c_float), ("window", C.c_int32),
                ("quant", C.c_int32), ("latency_ms", C.c_double), ("quality", C.c_double)]


class ardit_stream_state(C.Structure):
    _fields_ = [("worker", C.c_int32), ("slack_ms", C.c_double), ("remaining_ms", C.c_double)]


class ardit_stream_decision(C.Structure):
    _fields_ = [("cfg", C.c_int32), ("mode", C.c_int32), ("tier", C.c_int32),
                ("queue_pos", C.c_int32), ("credit_ms", C.c_double)]


_vp, _i32, _sz = C.c_void_p, C.c_int32, C.c_size_t
_P = C.POINTER
_SIGS = {
    "ardit_status_str": (C.c_char_p, [C.c_int]),
    "ardit_last_error": (C.c_char_p, []),
    "ardit_version": (C.c_int, []),
    "ardit_workspace_size": (C.c_int, [_P(ardit_dims), _P(ardit_batch), _P(_sz)]),
    "ardit_time_mod": (C.c_int, [_vp, _P(ardit_dims), _i32, _P(C.c_float),
                                 _P(ardit_time_weights), _vp, _vp, _sz]),
    "ardit_ctx_kv": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _vp,
                               _P(ardit_block_weights), _vp, _vp, _vp, _sz]),
    "ardit_kv_append": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _vp, _vp, _vp,
                                  _P(ardit_kv_paged), _vp]),
    "ardit_attn_fwd": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _vp,
                                 _P(ardit_kv_paged), _vp, _vp, _sz]),
    "ardit_attn_fwd_noalloc": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _vp,
                                         _P(ardit_kv_paged), _vp]),
    "ardit_mx_quantize": (C.c_int, [_vp, _vp, C.c_int64, _i32, _i32, _vp, _vp]),
    "ardit_sparse_select": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _vp,
                                      _P(ardit_kv_paged), _vp, _i32, _vp, _sz]),
    "ardit_block_fwd": (C.c_int, [_vp, _P(ardit_dims), _vp, ardit_kv_paged, _i32, _i32, _vp,
                                  _vp, _vp, _i32, _P(ardit_block_weights), _vp, _vp, _sz]),
    "ardit_block_fwd_varlen": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _vp,
                                         _P(ardit_kv_paged), _vp, _vp, _vp,
                                         _P(ardit_block_weights), _vp, _vp, _sz]),
    "ardit_stack_fwd": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _i32, _vp,
                                  _P(ardit_kv_paged), _vp, _P(_vp), _P(_vp),
                                  _P(ardit_block_weights), _vp, _vp, _sz]),
    "ardit_window_pages": (C.c_int, [_i32, _i32, _i32, _i32, _i32, _P(_i32), _i32, _P(_i32)]),
    "ardit_chunk_generate": (C.c_int, [_vp, _P(ardit_dims), _P(ardit_batch), _i32, _P(_i32),
                                       _P(C.c_float), _i32, _vp, _vp, _P(ardit_kv_paged),
                                       _P(ardit_time_weights), _P(_vp), _P(_vp),
                                       _P(ardit_block_weights), _vp, _vp, _sz]),
    "ardit_pareto_frontier": (C.c_int, [_i32, _P(ardit_fidelity), _P(_i32), _P(_i32),
                                        _P(C.c_double)]),
    "ardit_bmpr_select": (C.c_int, [_i32, _P(ardit_fidelity), _i32, _P(_i32), C.c_double,
                                    C.c_double, _P(_i32), _P(_i32)]),
    "ardit_control_tick": (C.c_int, [_i32, _i32, _P(ardit_fidelity), _i32, _P(_i32),
                                     C.c_double, _i32, _P(ardit_stream_state),
                                     _P(ardit_stream_decision)]),
    "ardit_timing_enable": (C.c_int, [C.c_int]),
    "ardit_timing_collect": (C.c_int, [_P(_i32), _P(C.c_double)]),
    "ardit_timing_collect_kind": (C.c_int, [_i32, _P(_i32), _P(C.c_double)]),
    "ardit_debug_checks": (C.c_int, [C.c_int]),
    "ardit_timing_flush": (C.c_int, [_vp, _sz]),
    "ardit_timing_records": (C.c_int, [_i32, _i32, _P(C.c_char_p), _P(C.c_double), _P(_i32)]),
    "ardit_micro_mfma": (C.c_int, [_vp, _i32, _i32, _i32, _vp, _P(C.c_double)]),
    "ardit_micro_copy": (C.c_int, [_vp, _vp, _vp, _sz]),
    "ardit_micro_read": (C.c_int, [_vp, _vp, _sz, _vp, _sz]),
    "ardit_micro_fill": (C.c_int, [_vp, _vp, _sz, C.c_uint32]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def exported_symbols():
    return tuple(_SIGS)


def has_symbol(name: str) -> bool:
    try:
        getattr(_lib, name)
        return True
    except AttributeError:
        return False


# ---------------------------------------------------------------- helpers
def _ptr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return int(s) if not hasattr(s, "cuda_stream") else s.cuda_stream


def _check(status: int, func: str):
    if status != 0:
        raise ArditError(status, func, ardit_last_error())


def ardit_status_str(status: int) -> str:
    return _lib.ardit_status_str(status).decode()


def ardit_last_error() -> str:
    return _lib.ardit_last_error().decode()


def ardit_version() -> int:
    return _lib.ardit_version()


def make_dims(dim, n_heads, head_dim, ffn_dim, frames_per_chunk, lat_h, lat_w, eps=1e-6,
              rope_theta=10000.0) -> ardit_dims:
    return ardit_dims(dim, n_heads, head_dim, ffn_dim, frames_per_chunk, lat_h, lat_w, eps,
                      rope_theta)


def dims_from_shape(shape) -> ardit_dims:
    """From any object with dim, n_heads, head_dim, ffn_dim, frames, lat_h, lat_w, eps, theta."""
    return make_dims(shape.dim, shape.n_heads, shape.head_dim, shape.ffn_dim, shape.frames,
                     shape.lat_h, shape.lat_w, shape.eps, shape.theta)


class Batch:
    """Host-side batch descriptor; keeps its int32 arrays alive."""

    def __init__(self, q_lens=None, cache_lens=None, frame_pos0=None, ctx_lens=None,
                 sparsity=None, quant=None):
        lens = [a for a in (q_lens, cache_lens, frame_pos0, ctx_lens) if a is not None]
        n = len(lens[0]) if lens else 0
        self._arrs = []

        def arr(a):
            if a is None:
                return None
            assert len(a) == n, "all per-stream arrays must have the same length"
            c = (C.c_int32 * n)(*[int(v) for v in a])
            self._arrs.append(c)
            return C.cast(c, C.POINTER(C.c_int32))

        sp = None
        if sparsity is not None:
            assert len(sparsity) == n, "all per-stream arrays must have the same length"
            c = (C.c_float * n)(*[float(v) for v in sparsity])
            self._arrs.append(c)
            sp = C.cast(c, C.POINTER(C.c_float))
        self.struct = ardit_batch(n, arr(q_lens), arr(cache_lens), arr(frame_pos0), arr(ctx_lens),
                                  sp, arr(quant))
        self.n = n
        self.q_lens = None if q_lens is None else [int(v) for v in q_lens]


def kv_paged(k_pages, v_pages, page_table, n_pages: int, max_frames: int) -> ardit_kv_paged:
    return ardit_kv_paged(_ptr(k_pages), _ptr(v_pages), _ptr(page_table), int(n_pages),
                          int(max_frames))


def block_weights(w: dict) -> ardit_block_weights:
    return ardit_block_weights(*[_ptr(w.get(n)) for n in _BLOCK_FIELDS])


def time_weights(w: dict) -> ardit_time_weights:
    return ardit_time_weights(*[_ptr(w[n]) for n in _TIME_FIELDS])


# ------------------------------------------------------------ entry points
def ardit_workspace_size(dims: ardit_dims, batch: Batch) -> int:
    n = C.c_size_t(0)
    _check(_lib.ardit_workspace_size(C.byref(dims), C.byref(batch.struct), C.byref(n)),
           "ardit_workspace_size")
    return n.value


def ardit_time_mod(stream, dims, t_values, tw: ardit_time_weights, mod_out, ws, ws_bytes):
    t = (C.c_float * len(t_values))(*[float(v) for v in t_values])
    _check(_lib.ardit_time_mod(_stream(stream), C.byref(dims), len(t_values), t, C.byref(tw),
                               _ptr(mod_out), _ptr(ws), int(ws_bytes)), "ardit_time_mod")


def ardit_ctx_kv(stream, dims, batch: Batch, ctx, w: ardit_block_weights, ctx_k, ctx_v, ws,
                 ws_bytes):
    _check(_lib.ardit_ctx_kv(_stream(stream), C.byref(dims), C.byref(batch.struct), _ptr(ctx),
                             C.byref(w), _ptr(ctx_k), _ptr(ctx_v), _ptr(ws), int(ws_bytes)),
           "ardit_ctx_kv")


def ardit_kv_append(stream, dims, batch: Batch, qkv, g_q, g_k, kv: ardit_kv_paged, q_out):
    _check(_lib.ardit_kv_append(_stream(stream), C.byref(dims), C.byref(batch.struct), _ptr(qkv),
                                _ptr(g_q), _ptr(g_k), C.byref(kv), _ptr(q_out)),
           "ardit_kv_append")


def ardit_attn_fwd(stream, dims, batch: Batch, q, kv: ardit_kv_paged, o, ws, ws_bytes):
    _check(_lib.ardit_attn_fwd(_stream(stream), C.byref(dims), C.byref(batch.struct), _ptr(q),
                               C.byref(kv), _ptr(o), _ptr(ws), int(ws_bytes)), "ardit_attn_fwd")


def ardit_attn_fwd_noalloc(stream, dims, batch: Batch, q, kv: ardit_kv_paged, o):
    _check(_lib.ardit_attn_fwd_noalloc(_stream(stream), C.byref(dims), C.byref(batch.struct),
                                       _ptr(q), C.byref(kv), _ptr(o)), "ardit_attn_fwd_noalloc")


QUANT_BF16, QUANT_FP8 = 0, 1


def ardit_mx_quantize(stream, x, rows, cols, ld, codes, scales):
    _check(_lib.ardit_mx_quantize(_stream(stream), _ptr(x), int(rows), int(cols), int(ld),
                                  _ptr(codes), _ptr(scales)), "ardit_mx_quantize")


def ardit_sparse_select(stream, dims, batch: Batch, q, kv: ardit_kv_paged, blocks, row_stride,
                        ws, ws_bytes):
    _check(_lib.ardit_sparse_select(_stream(stream), C.byref(dims), C.byref(batch.struct),
                                    _ptr(q), C.byref(kv), _ptr(blocks), int(row_stride), _ptr(ws),
                                    int(ws_bytes)), "ardit_sparse_select")


def ardit_block_fwd(stream, dims, x, kv: ardit_kv_paged, cache_len, frame_pos0, mod, ctx_k,
                    ctx_v, ctx_len, w: ardit_block_weights, out, ws, ws_bytes):
    _check(_lib.ardit_block_fwd(_stream(stream), C.byref(dims), _ptr(x), kv, int(cache_len),
                                int(frame_pos0), _ptr(mod), _ptr(ctx_k), _ptr(ctx_v),
                                int(ctx_len), C.byref(w), _ptr(out), _ptr(ws), int(ws_bytes)),
           "ardit_block_fwd")


def ardit_block_fwd_varlen(stream, dims, batch: Batch, x, kv: ardit_kv_paged, mod, ctx_k, ctx_v,
                           w: ardit_block_weights, out, ws, ws_bytes):
    _check(_lib.ardit_block_fwd_varlen(_stream(stream), C.byref(dims), C.byref(batch.struct),
                                       _ptr(x), C.byref(kv), _ptr(mod), _ptr(ctx_k), _ptr(ctx_v),
                                       C.byref(w), _ptr(out), _ptr(ws), int(ws_bytes)),
           "ardit_block_fwd_varlen")


def ardit_stack_fwd(stream, dims, batch: Batch, x, kvs, mod, ctx_ks, ctx_vs, ws_list, out, ws,
                    ws_bytes):
    L = len(kvs)
    kv_arr = (ardit_kv_paged * L)(*kvs)
    w_arr = (ardit_block_weights * L)(*ws_list)
    ck = (C.c_void_p * L)(*[_ptr(t) for t in ctx_ks])
    cv = (C.c_void_p * L)(*[_ptr(t) for t in ctx_vs])
    _check(_lib.ardit_stack_fwd(_stream(stream), C.byref(dims), C.byref(batch.struct), L, _ptr(x),
                                kv_arr, _ptr(mod), ck, cv, w_arr, _ptr(out), _ptr(ws),
                                int(ws_bytes)), "ardit_stack_fwd")


def ardit_window_pages(chunk, sink, window, frames_per_chunk, page_base=0, max_frames=None):
    """Returns (table entries of the held chunks then the chunk, cached frames)."""
    if max_frames is None:
        max_frames = (int(sink) + int(window) + 1) * int(frames_per_chunk)
    table = (C.c_int32 * max(int(max_frames), 1))()
    cached = C.c_int32(0)
    _check(_lib.ardit_window_pages(int(chunk), int(sink), int(window), int(frames_per_chunk),
                                   int(page_base), table, int(max_frames), C.byref(cached)),
           "ardit_window_pages")
    n = cached.value + int(frames_per_chunk)
    return [table[i] for i in range(n)], cached.value


def ardit_chunk_generate(stream, dims, batch: Batch, n_steps, timesteps, x_init, noise, kvs,
                         tw: ardit_time_weights, ctx_ks, ctx_vs, ws_list, x0_out, ws, ws_bytes):
    """timesteps: per stream, the list of its n_steps[b] timesteps."""
    L = len(kvs)
    B = len(n_steps)
    t_ld = max(1, max(int(s) for s in n_steps))
    t = (C.c_float * (B * t_ld))()
    for b, ts in enumerate(timesteps):
        for i, v in enumerate(ts):
            t[b * t_ld + i] = float(v)
    ns = (C.c_int32 * B)(*[int(v) for v in n_steps])
    kv_arr = (ardit_kv_paged * L)(*kvs)
    w_arr = (ardit_block_weights * L)(*ws_list)
    ck = (C.c_void_p * L)(*[_ptr(x) for x in ctx_ks])
    cv = (C.c_void_p * L)(*[_ptr(x) for x in ctx_vs])
    _check(_lib.ardit_chunk_generate(_stream(stream), C.byref(dims), C.byref(batch.struct), L, ns,
                                     t, t_ld, _ptr(x_init), _ptr(noise), kv_arr, C.byref(tw), ck,
                                     cv, w_arr, _ptr(x0_out), _ptr(ws), int(ws_bytes)),
           "ardit_chunk_generate")


TIME_ATTENTION, TIME_GEMM, TIME_ELEMENTWISE = 0, 1, 2


def ardit_timing_enable(enable):
    """enable: a bool (attention launches only) or a mask of 1 << TIME_* bits."""
    mask = int(enable) if not isinstance(enable, bool) else (1 if enable else 0)
    _check(_lib.ardit_timing_enable(mask), "ardit_timing_enable")


def ardit_timing_collect_kind(kind):
    n = C.c_int32(0)
    ms = C.c_double(0.0)
    _check(_lib.ardit_timing_collect_kind(int(kind), C.byref(n), C.byref(ms)),
           "ardit_timing_collect_kind")
    return n.value, ms.value


def ardit_timing_flush(buf, nbytes):
    """buf: device buffer written before every timed launch (None, 0: off)."""
    _check(_lib.ardit_timing_flush(_ptr(buf), int(nbytes)), "ardit_timing_flush")


def ardit_timing_records(kind, max_records=4096):
    """[(launch name, ms)] of the timed launches of one kind, in launch order."""
    names = (C.c_char_p * max(max_records, 1))()
    ms = (C.c_double * max(max_records, 1))()
    n = C.c_int32(0)
    _check(_lib.ardit_timing_records(int(kind), int(max_records), names, ms, C.byref(n)),
           "ardit_timing_records")
    return [(names[i].decode(), ms[i]) for i in range(n.value)]


def ardit_micro_mfma(stream, dtype, workgroups, iters, sink):
    """Launches the MFMA throughput kernel; returns the flops it performs."""
    f = C.c_double(0.0)
    _check(_lib.ardit_micro_mfma(_stream(stream), int(dtype), int(workgroups), int(iters),
                                 _ptr(sink), C.byref(f)), "ardit_micro_mfma")
    return f.value


def ardit_micro_copy(stream, src, dst, nbytes):
    _check(_lib.ardit_micro_copy(_stream(stream), _ptr(src), _ptr(dst), int(nbytes)),
           "ardit_micro_copy")


def ardit_micro_read(stream, src, nbytes, sink, sink_bytes):
    _check(_lib.ardit_micro_read(_stream(stream), _ptr(src), int(nbytes), _ptr(sink),
                                 int(sink_bytes)), "ardit_micro_read")


def ardit_micro_fill(stream, dst, nbytes, value=0):
    _check(_lib.ardit_micro_fill(_stream(stream), _ptr(dst), int(nbytes), int(value)),
           "ardit_micro_fill")


def ardit_debug_checks(enable):
    _check(_lib.ardit_debug_checks(int(enable)), "ardit_debug_checks")


def ardit_timing_collect():
    n = C.c_int32(0)
    ms = C.c_double(0.0)
    _check(_lib.ardit_timing_collect(C.byref(n), C.byref(ms)), "ardit_timing_collect")
    return n.value, ms.value


# ------------------------------------------------------------- controller
URGENT, NORMAL, RELAXED = 0, 1, 2
BMPR_QUALITY, BMPR_SPEED_RECOVERY = 0, 1


def fidelity_array(cfgs):
    """cfgs: sequence of (steps, sparsity, window, quant, latency_ms, quality)."""
    arr = (ardit_fidelity * len(cfgs))()
    for i, c in enumerate(cfgs):
        arr[i] = ardit_fidelity(int(c[0]), float(c[1]), int(c[2]), int(c[3]), float(c[4]),
                                float(c[5]))
    return arr


def ardit_pareto_frontier(cfgs):
    """Returns (frontier indices, quality floor)."""
    arr = cfgs if isinstance(cfgs, C.Array) else fidelity_array(cfgs)
    n = len(arr)
    f = (C.c_int32 * n)()
    m = C.c_int32(0)
    fl = C.c_double(0.0)
    _check(_lib.ardit_pareto_frontier(n, arr, f, C.byref(m), C.byref(fl)), "ardit_pareto_frontier")
    return [f[i] for i in range(m.value)], fl.value


def ardit_bmpr_select(cfgs, frontier, q_floor, budget_ms):
    arr = cfgs if isinstance(cfgs, C.Array) else fidelity_array(cfgs)
    f = (C.c_int32 * len(frontier))(*frontier)
    c, m = C.c_int32(0), C.c_int32(0)
    _check(_lib.ardit_bmpr_select(len(arr), arr, len(frontier), f, float(q_floor),
                                  float(budget_ms), C.byref(c), C.byref(m)), "ardit_bmpr_select")
    return c.value, m.value


def ardit_control_tick(n_workers, cfgs, frontier, q_floor, streams):
    """streams: sequence of (worker, slack_ms, remaining_ms).  Returns a list of
    ardit_stream_decision."""
    arr = cfgs if isinstance(cfgs, C.Array) else fidelity_array(cfgs)
    f = (C.c_int32 * len(frontier))(*frontier)
    n = len(streams)
    st = (ardit_stream_state * max(n, 1))()
    for i, s in enumerate(streams):
        st[i] = ardit_stream_state(int(s[0]), float(s[1]), float(s[2]))
    out = (ardit_stream_decision * max(n, 1))()
    _check(_lib.ardit_control_tick(int(n_workers), len(arr), arr, len(frontier), f,
                                   float(q_floor), n, st, out), "ardit_control_tick")
    return [out[i] for i in range(n)]
