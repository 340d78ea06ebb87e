"""Float64 reference of one AR-DiT block on one chunk -- TEST INFRASTRUCTURE ONLY.

What the paper fixes (Section 2.1, "AR-DiT" paragraph): video is generated
one chunk at a time; each chunk's generation uses the KV cache of the earlier
chunks, and a chunk is appended to a rolling KV cache once generated; the
cache keeps a sink plus the most recent W chunks.  Denoising runs S steps per
chunk (Section 2.1, fidelity knobs).  The paper says nothing about the
block's internals; this module computes the block as a fixed model contract
(adaLN-modulated RMSNorm, QKV projection, QK-RMSNorm over the full hidden
width, 3D RoPE, self-attention of the chunk over [cache | chunk], text
cross-attention, GELU-tanh FFN), each silent point taken as stated at the
function that computes it.

Conventions: every linear is y = x W^T + b with W stored [out][in];
rms(z) = z / sqrt(mean(z^2) + eps) over the last axis; float64 throughout.
Inputs are the bf16-exact fp32 arrays the workload generator draws.

Parity pins (tests/test_oracle_pins.py): brute-force scalar loops on tiny
shapes, softmax rows summing to 1, chunk-with-cache equal to the matching
slice of full-sequence block-causal attention, bit-identical earlier rows
when later chunks change, RoPE as a complex rotation and its relative-position
property, RMSNorm scale invariance, GELU-tanh odd part and its distance to
the erf GELU, closed-form attention special cases, zero gates.  The numerics
of a trained model are parity unpinned (no weights and no printed values).
"""
from __future__ import annotations

import math

import numpy as np

DTYPE = np.float64


def _f(a):
    return np.asarray(a, dtype=DTYPE)


def _bf16_round(a):
    """Round to the nearest bfloat16 (ties to even), returned as float32."""
    b = np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.uint32)
    b = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return b.view(np.float32)


# --------------------------------------------------------------------------
# elementary pieces
# --------------------------------------------------------------------------
def timestep_sinusoid(t: float, n: int = 256, max_period: float = 10000.0):
    """[cos(t w_k) for k<n/2] ++ [sin(t w_k) for k<n/2], w_k = max_period^(-k/(n/2)).

    Reading of the timestep embedding (the paper names no embedding)."""
    half = n // 2
    k = np.arange(half, dtype=DTYPE)
    w = max_period ** (-k / half)
    a = DTYPE(t) * w
    return np.concatenate([np.cos(a), np.sin(a)])


def silu(z):
    z = _f(z)
    return z / (1.0 + np.exp(-z))


def linear(x, w, b=None):
    """y = x W^T + b, W stored [out][in]."""
    y = _f(x) @ _f(w).T
    if b is not None:
        y = y + _f(b)
    return y


def rms_norm(z, eps: float, gain=None):
    """z / sqrt(mean(z^2) + eps) over the last axis, times an optional gain."""
    z = _f(z)
    ms = np.mean(z * z, axis=-1, keepdims=True)
    y = z / np.sqrt(ms + DTYPE(eps))
    if gain is not None:
        y = y * _f(gain)
    return y


def gelu_tanh(y):
    """GELU with the tanh form: y/2 * (1 + tanh(sqrt(2/pi) (y + 0.044715 y^3)))."""
    y = _f(y)
    c = math.sqrt(2.0 / math.pi)
    return 0.5 * y * (1.0 + np.tanh(c * (y + 0.044715 * y * y * y)))


# --------------------------------------------------------------------------
# 3D rotary position embedding
# --------------------------------------------------------------------------
def rope_split(head_dim: int):
    """Head-dim segments (d_t, d_h, d_w): d_h = d_w = 2 floor(d/6), d_t the rest."""
    dh = 2 * (head_dim // 6)
    return (head_dim - 2 * dh, dh, dh)


def rope_inv_freq(seg: int, theta: float):
    """theta^(-2k/seg) for the seg/2 pairs of one segment."""
    k = np.arange(seg // 2, dtype=DTYPE)
    return DTYPE(theta) ** (-2.0 * k / seg)


def chunk_positions(frames: int, lat_h: int, lat_w: int, frame_pos0: int):
    """(t, h, w) position of every token of a chunk, tokens frame-major then h then w."""
    f, i, j = np.meshgrid(np.arange(frames), np.arange(lat_h), np.arange(lat_w),
                          indexing="ij")
    pos = np.stack([f.ravel() + frame_pos0, i.ravel(), j.ravel()], axis=1)
    return pos.astype(np.int64)


def rope3d(z, positions, theta: float):
    """Rotate adjacent pairs (2k, 2k+1) of each head segment by angle p * theta_k.

    z: [L, H, d]; positions: [L, 3] integer (t, h, w).  Segment s of size d_s
    uses the s-th position component and theta_k = theta^(-2k/d_s)."""
    z = _f(z)
    L, H, d = z.shape
    out = z.copy()
    start = 0
    for axis, seg in enumerate(rope_split(d)):
        if seg == 0:
            continue
        inv = rope_inv_freq(seg, theta)                       # [seg/2]
        ang = positions[:, axis].astype(DTYPE)[:, None] * inv[None, :]   # [L, seg/2]
        c = np.cos(ang)[:, None, :]
        s = np.sin(ang)[:, None, :]
        a = z[:, :, start:start + seg:2]
        b = z[:, :, start + 1:start + seg:2]
        out[:, :, start:start + seg:2] = a * c - b * s
        out[:, :, start + 1:start + seg:2] = a * s + b * c
        start += seg
    return out


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------
def attention(q, k, v, mask=None, return_probs=False, q_block: int = 1024):
    """Per-head softmax(q k^T / sqrt(d)) v.

    q: [Lq, H, d], k and v: [Lk, H, d]; mask: optional [Lq, Lk] bool (True =
    visible).  Without a mask every key is visible.  Rows are processed in
    blocks of q_block queries only to bound memory."""
    q, k, v = _f(q), _f(k), _f(v)
    Lq, H, d = q.shape
    scale = 1.0 / math.sqrt(d)
    o = np.empty((Lq, H, d), dtype=DTYPE)
    probs = np.empty((H, Lq, k.shape[0]), dtype=DTYPE) if return_probs else None
    for h in range(H):
        kh = k[:, h, :]
        vh = v[:, h, :]
        for r0 in range(0, Lq, q_block):
            r1 = min(Lq, r0 + q_block)
            s = (q[r0:r1, h, :] @ kh.T) * scale
            if mask is not None:
                s = np.where(mask[r0:r1], s, -np.inf)
            s = s - np.max(s, axis=1, keepdims=True)
            p = np.exp(s)
            p = p / np.sum(p, axis=1, keepdims=True)
            o[r0:r1, h, :] = p @ vh
            if return_probs:
                probs[h, r0:r1] = p
    return (o, probs) if return_probs else o


# --------------------------------------------------------------------------
# time modulation and text context
# --------------------------------------------------------------------------
def time_modulation(t: float, tw: dict, dim: int):
    """Shared time MLP: s(t) -> e = W_t2 SiLU(W_t1 s + b_t1) + b_t2 ->
    m = W_m SiLU(e) + b_m, returned as rows (shift1, scale1, gate1, shift2,
    scale2, gate2) of width dim.  Evaluated once per stream per denoising step."""
    s = timestep_sinusoid(t, tw["w_t1"].shape[1])
    e = linear(silu(linear(s, tw["w_t1"], tw["b_t1"])), tw["w_t2"], tw["b_t2"])
    m = linear(silu(e), tw["w_m"], tw["b_m"])
    return m.reshape(6, dim)


def context_kv(ctx, w: dict, eps: float):
    """Cross-attention keys and values of one stream's text tokens:
    K_c = rms(ctx W_ck^T + b_ck) * g_ck,  V_c = ctx W_cv^T + b_cv.  [Lx, D] each."""
    kc = rms_norm(linear(ctx, w["w_ck"], w["b_ck"]), eps, w["g_ck"])
    vc = linear(ctx, w["w_cv"], w["b_cv"])
    return kc, vc


# --------------------------------------------------------------------------
# the block
# --------------------------------------------------------------------------
def _modulation(m_t, w):
    M = _f(m_t) + _f(w["mod_table"])
    return {"shift1": M[0], "scale1": M[1], "gate1": M[2],
            "shift2": M[3], "scale2": M[4], "gate2": M[5]}


def _qkv_rope(x, M, w, shape, positions):
    D, H, d = shape.dim, shape.n_heads, shape.head_dim
    h1 = rms_norm(x, shape.eps) * (1.0 + M["scale1"]) + M["shift1"]
    qkv = linear(h1, w["w_qkv"], w["b_qkv"])
    q, k, v = qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:]
    qn = rms_norm(q, shape.eps, w["g_q"]).reshape(-1, H, d)
    kn = rms_norm(k, shape.eps, w["g_k"]).reshape(-1, H, d)
    qr = rope3d(qn, positions, shape.theta)
    kr = rope3d(kn, positions, shape.theta)
    return qr, kr, v.reshape(-1, H, d)


def _after_self_attention(x, o, M, w, shape, ctx_k, ctx_v):
    D, H, d = shape.dim, shape.n_heads, shape.head_dim
    x1 = x + M["gate1"] * linear(o.reshape(-1, D), w["w_o"], w["b_o"])
    h3 = rms_norm(x1, shape.eps, w["g_n3"])
    qc = rms_norm(linear(h3, w["w_cq"], w["b_cq"]), shape.eps, w["g_cq"])
    oc = attention(qc.reshape(-1, H, d), _f(ctx_k).reshape(-1, H, d),
                   _f(ctx_v).reshape(-1, H, d)).reshape(-1, D)
    x2 = x1 + linear(oc, w["w_co"], w["b_co"])
    h2 = rms_norm(x2, shape.eps) * (1.0 + M["scale2"]) + M["shift2"]
    u = gelu_tanh(linear(h2, w["w_1"], w["b_1"]))
    out = x2 + M["gate2"] * linear(u, w["w_2"], w["b_2"])
    return {"x1": x1, "qc": qc, "oc": oc, "x2": x2, "u": u, "out": out}


def block_forward(x, cache_k, cache_v, frame_pos0: int, m_t, ctx_k, ctx_v,
                  w: dict, shape, rows=None, rho: float = 0.0, blocks=None, fp8: bool = False):
    """One block on one chunk of one stream.

    x: [L_q, D] chunk activations; cache_k / cache_v: [c, H, d] the stream's
    cached keys (already normalised and rotated) and values of earlier chunks,
    in logical order; frame_pos0: absolute latent-frame index of the chunk's
    first frame; m_t: [6, D] time modulation of this stream and step (the
    block adds its own mod_table); ctx_k / ctx_v: [L_x, D] from context_kv.

    The chunk's keys are appended after the cache and every query sees all
    c + L_q keys.  rows: optional query-row subset; keys and values are always
    computed for the whole chunk, the rest only for these rows.

    rho > 0 (or an explicit blocks [H, n_qblocks, n_keep] list) makes the
    self-attention block-sparse as sparse_ref defines it; the selection scores
    the bf16-rounded rotated q and k, the values the kernels store.  fp8 makes
    it the FP8 attention of fp8_ref, on the bf16-rounded q, k and v.

    Returns a dict with q (rotated, [L_q, H, d]), k_new, v_new ([L_q, H, d]),
    o (self-attention output, [R, D]), x1, qc, oc, x2, u, out ([R, ...])."""
    x = _f(x)
    M = _modulation(m_t, w)
    pos = chunk_positions(shape.frames, shape.lat_h, shape.lat_w, frame_pos0)
    q, k, v = _qkv_rope(x, M, w, shape, pos)
    K = np.concatenate([_f(cache_k), k], axis=0)
    V = np.concatenate([_f(cache_v), v], axis=0)
    sel = np.arange(x.shape[0]) if rows is None else np.asarray(rows)
    if fp8:
        from . import fp8_ref
        o = fp8_ref.fp8_attention(_bf16_round(q[sel]) if rows is not None else _bf16_round(q),
                                  _bf16_round(K), _bf16_round(V))[0].reshape(len(sel), shape.dim)
    elif rho > 0.0 or blocks is not None:
        from . import sparse_ref
        if blocks is None:
            n_k = (K.shape[0] + sparse_ref.K_BLOCK - 1) // sparse_ref.K_BLOCK
            scores = sparse_ref.block_scores(_bf16_round(q), _bf16_round(K))
            blocks = sparse_ref.select_blocks(scores, sparse_ref.keep_count(n_k, rho))
        o = sparse_ref.sparse_attention(q, K, V, blocks, rows=sel).reshape(len(sel), shape.dim)
    else:
        o = attention(q[sel], K, V).reshape(len(sel), shape.dim)
    res = _after_self_attention(x[sel], o, M, w, shape, ctx_k, ctx_v)
    res.update({"q": q, "k_new": k, "v_new": v, "o": o, "rows": sel, "blocks": blocks})
    return res


def full_sequence_forward(xs, m_ts, frame_pos0: int, ctx_k, ctx_v, w: dict,
                          shape, window=None, sink: int = 0):
    """Block-causal full-sequence version over chunks 0..C-1 of one stream.

    xs: list of [L_q, D] chunks; m_ts: per-chunk [6, D] time modulation.
    Chunk c's frames start at frame_pos0 + c * frames.  Token i sees token j
    iff chunk(j) <= chunk(i) (and, when a window of earlier chunks is given,
    chunk(i) - chunk(j) <= window or chunk(j) < sink: the sink chunks stay
    visible).  Used only to pin the chunk-with-cache form."""
    C = len(xs)
    Lq = shape.chunk_tokens
    x = np.concatenate([_f(a) for a in xs], axis=0)
    chunk_of = np.repeat(np.arange(C), Lq)
    Ms = [_modulation(m, w) for m in m_ts]
    Mtok = {key: np.concatenate([np.broadcast_to(M[key], (Lq, shape.dim)) for M in Ms])
            for key in Ms[0]}
    pos = np.concatenate([chunk_positions(shape.frames, shape.lat_h, shape.lat_w,
                                          frame_pos0 + c * shape.frames) for c in range(C)])
    q, k, v = _qkv_rope(x, Mtok, w, shape, pos)
    mask = chunk_of[None, :] <= chunk_of[:, None]
    if window is not None:
        mask &= ((chunk_of[:, None] - chunk_of[None, :]) <= window) | (chunk_of[None, :] < sink)
    o = attention(q, k, v, mask=mask).reshape(-1, shape.dim)
    res = _after_self_attention(x, o, Mtok, w, shape, ctx_k, ctx_v)
    res.update({"q": q, "k": k, "v": v, "o": o})
    return res
