"""Reference of block-sparse self-attention -- TEST INFRASTRUCTURE ONLY.

The sparsity knob rho of a fidelity configuration skips attention blocks that
a sparse mask does not select (Section 2.1, fidelity knobs); the candidate
values are rho in {0, 0.6, 0.7, 0.8, 0.9} (Appendix A, configuration space)
and the implementation follows Light Forcing (Section 5).  The paper gives
neither the block shape nor the selection rule.  This module takes these
readings, for one stream and one head at a time:

  - a query block is 256 consecutive rows of the chunk, a key block 64
    consecutive logical keys of the stream's [cache | chunk] sequence; the last
    block of either kind may hold fewer;
  - the score of (query block i, key block j) is mean(q over block i) .
    mean(k over block j), each mean over the rows the block holds (this is the
    mean of the block's logits q k^T, up to the 1/sqrt(d) that does not change
    the ranking);
  - a query block keeps the n_keep key blocks of highest score, ties going to
    the lower key-block index, with n_keep = ceil((1 - rho) n - 1e-3) clamped
    to [1, n] for n key blocks (the 1e-3 keeps a rho given in single precision,
    0.9f = 0.89999998, from adding a block to (1 - rho) n = 10.0000024);
  - each query of the block attends to the keys of its kept blocks only:
    softmax over those keys, the others get weight zero.

The scores decide which blocks run, an integer decision, so they are formed in
float32 (means as float32 sums divided by the count, then a float32 dot
product), the kernel's precision; the attention itself is float64.  A NaN
score counts as -inf.  rho = 0 keeps every block and is plain attention.

Pins (tests/test_oracle_pins.py): the float64 score equals the mean of the
brute-force logit block; the keep counts for the paper's rho values at
printed sizes; a planted key block whose mean aligns with the query mean is
always kept; selection invariant to permutations inside a block and to a
positive scale of q; sparse attention equals scalar-loop attention over the
kept keys only; rho = 0 equals dense attention; a ragged last key block is
averaged over its valid keys only.
"""
from __future__ import annotations

import math

import numpy as np

from .ardit_ref import attention

Q_BLOCK = 256
K_BLOCK = 64


def keep_count(n_blocks: int, rho: float) -> int:
    """Key blocks kept per query block: ceil((1 - rho) n - 1e-3) in [1, n]."""
    if n_blocks <= 0:
        return 0
    keep = math.ceil((1.0 - float(rho)) * n_blocks - 1e-3)
    return max(1, min(n_blocks, keep))


def block_means(x, block: int, dtype=np.float32):
    """[L, H, d] -> [ceil(L / block), H, d]: mean over the rows of each block
    (the last over the rows it holds), summed in `dtype`."""
    x = np.asarray(x)
    L = x.shape[0]
    nb = (L + block - 1) // block
    out = np.empty((nb,) + x.shape[1:], dtype=dtype)
    for b in range(nb):
        rows = x[b * block:min(L, (b + 1) * block)].astype(dtype)
        out[b] = rows.sum(axis=0, dtype=dtype) / dtype(rows.shape[0])
    return out


def block_scores(q, k, q_block: int = Q_BLOCK, k_block: int = K_BLOCK, dtype=np.float32):
    """Scores [H, n_qblocks, n_kblocks] = mean(q block) . mean(k block).

    q: [L_q, H, d] queries (after QK-norm and RoPE); k: [L_k, H, d] keys of the
    whole [cache | chunk] sequence."""
    qm = block_means(q, q_block, dtype)       # [nq, H, d]
    km = block_means(k, k_block, dtype)       # [nk, H, d]
    return np.einsum("ihd,jhd->hij", qm, km).astype(dtype)


def select_blocks(scores, n_keep: int):
    """Kept key blocks [H, n_qblocks, n_keep], ascending within a row: the
    n_keep highest scores of each row, ties to the lower index, NaN as -inf."""
    s = np.asarray(scores, dtype=np.float64)
    s = np.where(np.isnan(s), -np.inf, s)
    H, nq, nk = s.shape
    out = np.empty((H, nq, n_keep), dtype=np.int64)
    idx = np.arange(nk)
    for h in range(H):
        for i in range(nq):
            order = np.lexsort((idx, -s[h, i]))   # score descending, then index ascending
            out[h, i] = np.sort(order[:n_keep])
    return out


def block_mask(blocks_h, L_q: int, L_k: int, q_block: int = Q_BLOCK, k_block: int = K_BLOCK):
    """[L_q, L_k] visibility of one head: key j visible to query i iff key block
    j // k_block is among the kept blocks of query block i // q_block."""
    nq = (L_q + q_block - 1) // q_block
    nk = (L_k + k_block - 1) // k_block
    kept = np.zeros((nq, nk), dtype=bool)
    for i in range(nq):
        kept[i, np.asarray(blocks_h[i])] = True
    return kept[np.arange(L_q) // q_block][:, np.arange(L_k) // k_block]


def sparse_attention(q, k, v, blocks, q_block: int = Q_BLOCK, k_block: int = K_BLOCK, rows=None):
    """Per-head softmax(q K^T / sqrt(d)) V over the keys of the kept blocks.

    q: [L_q, H, d]; k, v: [L_k, H, d]; blocks: [H, n_qblocks, n_keep] key-block
    indices.  rows: optional subset of query rows (the blocks still refer to
    the full chunk's query blocks).  Returns [R, H, d] float64."""
    q = np.asarray(q)
    L_q, H, d = q.shape
    L_k = k.shape[0]
    sel = np.arange(L_q) if rows is None else np.asarray(rows)
    o = np.empty((len(sel), H, d), dtype=np.float64)
    for h in range(H):
        mask = block_mask(blocks[h], L_q, L_k, q_block, k_block)[sel]
        o[:, h:h + 1] = attention(q[sel, h:h + 1], k[:, h:h + 1], v[:, h:h + 1], mask=mask)
    return o


def sparse_self_attention(q, k, v, rho: float, q_block: int = Q_BLOCK, k_block: int = K_BLOCK,
                          rows=None, score_inputs=None):
    """Selection then sparse attention of one stream.  score_inputs: optional
    (q, k) to score with (for instance the bf16-stored values the kernel sees);
    defaults to q, k.  Returns (o [R, H, d], blocks [H, n_qblocks, n_keep])."""
    qs, ks = (q, k) if score_inputs is None else score_inputs
    n_k = (np.asarray(k).shape[0] + k_block - 1) // k_block
    blocks = select_blocks(block_scores(qs, ks, q_block, k_block), keep_count(n_k, rho))
    return sparse_attention(q, k, v, blocks, q_block, k_block, rows), blocks
