"""Reference of FP8 attention (the quantisation knob Q) -- TEST INFRASTRUCTURE ONLY.

The quantisation knob of a fidelity configuration switches attention to FP8
(Section 2.1, fidelity knobs; Q in {FP16, FP8}, Appendix A).  The
implementation quantises activations online inside attention, following
SageAttention2, and never quantises weights (Section 5).  The paper gives no
format or granularity; this module takes these readings:

  - format: OCP FP8 E4M3 (finite values up to 448, subnormal step 2^-9),
    round to nearest, ties to even;
  - microscaled blocks of 32 consecutive elements along each product's
    reduction axis, each with a power-of-two scale 2^e:
      q, k: per token and head, 32 consecutive dims of the head;
      v:    per head and dim, 32 consecutive keys of the stream's logical key
            sequence (blocks start at key 0);
      p:    per query row, 32 consecutive keys (the unnormalised softmax
            weights, quantised after the exponential);
  - e = floor(log2(max |x| over the block)) - 7, so the block's largest
    magnitude lands in [128, 256) and no element reaches E4M3's top binade
    (no saturation path is needed); an all-zero block takes e = -127;
  - logits, the running max and the softmax denominator stay in full
    precision; the denominator sums the unquantised weights.

`fp8_attention` returns the attention of the dequantised q8, k8, v8 with
exact (unquantised) weights, together with an element-wise bound on what
quantising the weights, and the kernels' fp32 arithmetic, may add (see
`weight_quant_bound`), and the standard deviation that rounding the weights
gives each output element (`weight_quant_sigma`): the worst case grows with
the sum of |v| under the weights, the spread only with their root sum of
squares, which is what an output element itself scales with.  Pins
(tests/test_oracle_pins.py): every E4M3 code rounds to itself, midpoints round to even, the block exponent and the
[128, 256) landing of the block maximum, power-of-two scale invariance,
error within half a quantum, exactly representable inputs pass unchanged,
weight quantisation stays within the bound on random inputs, and the
statistical criterion built on sigma (tests/harness.py, fp8_parity) accepts
quantised weights at 14040 and 32760 keys while rejecting an all-zero
output, half the output and a 2% scale error.
"""
from __future__ import annotations

import math

import numpy as np

from .ardit_ref import attention

BLOCK = 32
E4M3_MAX = 448.0


def e4m3_values() -> np.ndarray:
    """The 254 finite values of OCP E4M3 (codes 0..255 without the two NaNs),
    from the format's definition: sign, 4-bit exponent (bias 7), 3-bit mantissa."""
    vals = []
    for code in range(256):
        if code & 0x7F == 0x7F:
            continue
        s = -1.0 if code & 0x80 else 1.0
        ex, m = (code >> 3) & 0xF, code & 7
        vals.append(s * (m / 8.0 * 2.0 ** -6 if ex == 0 else (1 + m / 8.0) * 2.0 ** (ex - 7)))
    return np.array(vals)


def e4m3_round(y):
    """Round to the nearest E4M3 value, ties to even mantissa.  |y| must stay
    below 464 (the midpoint between 448 and the first out-of-range value)."""
    y = np.asarray(y, dtype=np.float64)
    a = np.abs(y)
    if np.any(a >= 464.0) or np.any(~np.isfinite(y)):
        raise ValueError("value outside the E4M3 range handled here")
    # quantum: 2^(E - 3) in the normal range (E = floor(log2 |y|)), 2^-9 below 2^-6
    _, ex = np.frexp(np.where(a > 0, a, 1.0))     # a = f 2^ex, f in [0.5, 1)
    E = np.maximum(ex - 1, -6)
    quantum = np.ldexp(1.0, E - 3)
    return np.sign(y) * np.round(a / quantum) * quantum   # np.round: half to even


def block_exponent(amax):
    """floor(log2(amax)) - 7, clamped to [-127, 127]; -127 where amax == 0."""
    amax = np.asarray(amax, dtype=np.float64)
    _, ex = np.frexp(np.where(amax > 0, amax, 1.0))
    e = np.clip(ex - 1 - 7, -127, 127)
    return np.where(amax > 0, e, -127).astype(np.int64)


def mx_quantize(x, axis: int = -1, block: int = BLOCK):
    """Quantise x in blocks of `block` along `axis` (the last block may be
    shorter).  Returns (codes, e): codes are the E4M3 values x / 2^e of each
    element (exactly representable), e the block exponents broadcast to x's
    shape; the dequantised tensor is codes * 2^e."""
    x = np.moveaxis(np.asarray(x, dtype=np.float64), axis, -1)
    n = x.shape[-1]
    nb = (n + block - 1) // block
    pad = nb * block - n
    xp = np.concatenate([x, np.zeros(x.shape[:-1] + (pad,))], axis=-1) if pad else x
    xb = xp.reshape(x.shape[:-1] + (nb, block))
    e = block_exponent(np.max(np.abs(xb), axis=-1))[..., None]
    codes = e4m3_round(xb / np.ldexp(1.0, e))
    e_full = np.broadcast_to(e, xb.shape).reshape(xp.shape)[..., :n]
    codes = codes.reshape(xp.shape)[..., :n]
    return np.moveaxis(codes, -1, axis), np.moveaxis(e_full, -1, axis)


def mx_dequantize(codes, e):
    return np.asarray(codes, np.float64) * np.ldexp(1.0, np.asarray(e))


def quantize_qkv(q, k, v):
    """q: [Lq, H, d], k and v: [Lk, H, d] -> dequantised q8, k8, v8 (blocks of
    32 dims for q and k, of 32 keys for v)."""
    q8 = mx_dequantize(*mx_quantize(q, axis=-1))
    k8 = mx_dequantize(*mx_quantize(k, axis=-1))
    v8 = mx_dequantize(*mx_quantize(v, axis=0))
    return q8, k8, v8


def weight_quant_bound(p, v8, l):
    """Bound on |sum_j (p8_j - p_j) v_jd| / l for one head.

    p: [R, Lk] unnormalised weights (any common positive factor per row), v8:
    [Lk, d], l: [R] their row sums.  Quantising a weight in its block moves it
    by at most 2^-4 of itself (half an E4M3 step in the normal range) or by
    2^-10 2^e <= 2^-17 max(block) in the subnormal range.  2^-10 more of the
    weights covers the fp32 logits (products of 8-bit significands summed in
    fp32) and the hardware exp."""
    R, Lk = p.shape
    nb = (Lk + BLOCK - 1) // BLOCK
    pad = nb * BLOCK - Lk
    pb = np.concatenate([p, np.zeros((R, pad))], axis=1).reshape(R, nb, BLOCK)
    amax = np.repeat(pb.max(axis=2), BLOCK, axis=1)[:, :Lk]
    per = (2.0 ** -4 + 2.0 ** -10) * p + 2.0 ** -17 * amax
    return (per @ np.abs(v8)) / l[:, None]


def weight_quant_sigma(p, v8, l):
    """Standard deviation of sum_j (p8_j - p_j) v_jd / l for one head when each
    weight's rounding error is uniform within half its E4M3 quantum and
    independent of the others (round to nearest of values spread over many
    quanta).  p, v8, l as for weight_quant_bound; the quantum of weight j is
    that of p_j / 2^e in E4M3 times 2^e, e the exponent of its block of 32
    keys (block_exponent of the block's largest weight): 2^(E - 3) for
    E = floor(log2(p_j / 2^e)) >= -6, else 2^-9.  Variance quantum^2 / 12."""
    R, Lk = p.shape
    nb = (Lk + BLOCK - 1) // BLOCK
    pad = nb * BLOCK - Lk
    pb = np.concatenate([p, np.zeros((R, pad))], axis=1).reshape(R, nb, BLOCK)
    e = np.repeat(block_exponent(pb.max(axis=2)), BLOCK, axis=1)[:, :Lk]
    y = p / np.ldexp(1.0, e)
    _, ex = np.frexp(np.where(y > 0, y, 1.0))        # y = f 2^ex, f in [0.5, 1)
    E = np.where(y > 0, np.maximum(ex - 1, -6), -6)
    quantum = np.ldexp(1.0, E - 3 + e)
    var = quantum * quantum / 12.0
    return np.sqrt(var @ (v8 * v8)) / l[:, None]


def fp8_attention(q, k, v, mask=None, sigma=False):
    """FP8 attention of one stream: returns (o [Lq, H, d], bound [Lq, H, d]),
    and with sigma=True also sigma [Lq, H, d].

    o is softmax(q8 k8^T / sqrt(d)) v8 in float64 with the dequantised
    operands and unquantised weights; bound is weight_quant_bound per head (a
    worst case: every weight rounded by its largest error in one direction);
    sigma is weight_quant_sigma per head (the spread that rounding the weights
    to E4M3 gives an output element).  mask: optional [H, Lq, Lk] or [Lq, Lk]
    visibility (block-sparse use)."""
    q8, k8, v8 = quantize_qkv(q, k, v)
    Lq, H, d = q8.shape
    o = np.empty((Lq, H, d))
    bound = np.empty((Lq, H, d))
    sig = np.empty((Lq, H, d)) if sigma else None
    scale = 1.0 / math.sqrt(d)
    for h in range(H):
        s = (q8[:, h] @ k8[:, h].T) * scale
        if mask is not None:
            mh = mask[h] if np.ndim(mask) == 3 else mask
            s = np.where(mh, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        l = p.sum(axis=1)
        o[:, h] = (p @ v8[:, h]) / l[:, None]
        bound[:, h] = weight_quant_bound(p, v8[:, h], l)
        if sigma:
            sig[:, h] = weight_quant_sigma(p, v8[:, h], l)
    return (o, bound, sig) if sigma else (o, bound)


def fp8_attention_quantized_weights(q, k, v):
    """The same attention with the weights quantised too (per query row, blocks
    of 32 keys, relative to the row's final maximum).  Used only to pin the
    bound: |this - fp8_attention| <= bound."""
    q8, k8, v8 = quantize_qkv(q, k, v)
    Lq, H, d = q8.shape
    o = np.empty((Lq, H, d))
    for h in range(H):
        s = (q8[:, h] @ k8[:, h].T) / math.sqrt(d)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p8 = mx_dequantize(*mx_quantize(p, axis=1))
        o[:, h] = (p8 @ v8[:, h]) / p.sum(axis=1)[:, None]
    return o


def fp8_attention_dense_check(q, k, v):
    """Plain float64 attention of the dequantised operands (for pins)."""
    q8, k8, v8 = quantize_qkv(q, k, v)
    return attention(q8, k8, v8)
