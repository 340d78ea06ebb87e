"""Reference of whole-chunk generation around the block -- TEST INFRASTRUCTURE ONLY.

An AR-DiT generates a stream chunk by chunk: each chunk is denoised in S
steps (S in {2, 3, 4}, Appendix A) by the transformer stack attending to the
stream's KV cache, then appended to the cache, which keeps a sink of the
first chunks plus the most recent W chunks (Section 2.1, "AR-DiT" and
fidelity knobs).  The paper does not spell out the sampler or the commit; this
module takes these readings:

  - the stack (L blocks on the chunk's latent tokens, with the time
    modulation of the step's timestep t in [0, 1000]) predicts the
    rectified-flow velocity v at x_tau, tau = t / 1000; a step forms
    x0_hat = x_tau - tau v and re-noises it for the next timestep tau' with
    fresh Gaussian noise eps': x_tau' = (1 - tau') x0_hat + tau' eps' (the
    few-step re-noising of distilled AR-DiT generators); the last step's
    x0_hat is the clean chunk;
  - the commit is one more pass of the stack on the clean chunk at t = 0,
    whose keys and values are what the cache keeps for the chunk;
  - the window: after chunk c is committed the stream's logical cache is the
    first `sink` chunks followed by the most recent W chunks, in order; keys
    keep the rotary positions of their absolute frames.  Physically, sink
    chunk k lives in slot k and a later chunk c in slot
    sink + (c - sink) mod (W + 1), so the current chunk never overwrites a
    chunk still in the window.

Pins (tests/test_oracle_pins.py): a step with the true velocity recovers x0
exactly, tau' = 0 returns x0_hat, the page map against a direct listing of
the window, and generating chunks with eviction equals the block-causal
full-sequence computation with a sink + window mask.
"""
from __future__ import annotations

import numpy as np

from .ardit_ref import block_forward, time_modulation


def sampler_step(x, v, t: float, t_next, eps_next):
    """x0_hat = x - tau v, then (1 - tau') x0_hat + tau' eps' (or x0_hat when
    there is no next timestep).  Timesteps in [0, 1000]."""
    tau = t / 1000.0
    x0 = np.asarray(x, np.float64) - tau * np.asarray(v, np.float64)
    if t_next is None:
        return x0
    tn = t_next / 1000.0
    return (1.0 - tn) * x0 + tn * np.asarray(eps_next, np.float64)


def window_chunks(c: int, sink: int, window: int):
    """Chunks held in the cache while chunk c is generated, in logical order."""
    held = [k for k in range(min(sink, c))]
    held += [k for k in range(max(sink, c - window), c)]
    return held


def chunk_slot(c: int, sink: int, window: int) -> int:
    """Physical chunk slot of chunk c (slots 0..sink-1 fixed, then a ring of W + 1)."""
    return c if c < sink else sink + (c - sink) % (window + 1)


def window_page_table(c: int, sink: int, window: int, frames: int):
    """Logical frame -> physical page (slot * frames + f) of a stream generating
    chunk c: its cached chunks then the chunk itself.  Returns (table, cached
    frames)."""
    held = window_chunks(c, sink, window)
    table = []
    for k in held + [c]:
        table += [chunk_slot(k, sink, window) * frames + f for f in range(frames)]
    return np.array(table, dtype=np.int64), len(held) * frames


def generate_chunk(x_init, noise, ts, caches, frame_pos0: int, tw: dict, ctx_kv, ws: list, shape,
                   store=None, rho: float = 0.0, fp8: bool = False):
    """One chunk of one stream through an L-layer stack.

    x_init: [L_q, D] starting noise; noise: fresh noise of the steps after the
    first ([S - 1][L_q, D]); ts: the S timesteps; caches: per layer (k, v) of
    the held chunks ([c, H, d] each, logical order); ctx_kv: per layer (K_c,
    V_c); ws: per-layer weights.  store: optional rounding applied where an
    implementation stores a tensor between operations (each layer's output,
    the sampler's result, the committed keys and values); None keeps float64
    throughout.  Returns (x0, committed per-layer (k, v) of the chunk, the
    per-step inputs x_tau).  rho and fp8 are the stream's attention knobs,
    applied in every pass as block_forward applies them."""
    keep = (lambda a: a) if store is None else (lambda a: np.asarray(store(a), np.float64))
    x = np.asarray(x_init, np.float64)
    xs = []
    for s, t in enumerate(ts):
        xs.append(x)
        m_t = time_modulation(t, tw, shape.dim)
        h = x
        for layer, w in enumerate(ws):
            ck, cv = caches[layer]
            h = keep(block_forward(h, ck, cv, frame_pos0, m_t, ctx_kv[layer][0], ctx_kv[layer][1],
                                   w, shape, rho=rho, fp8=fp8)["out"])
        nxt = ts[s + 1] if s + 1 < len(ts) else None
        x = keep(sampler_step(x, h, t, nxt, noise[s] if nxt is not None else None))
    x0 = x
    m0 = time_modulation(0.0, tw, shape.dim)
    committed = []
    h = x0
    for layer, w in enumerate(ws):
        ck, cv = caches[layer]
        r = block_forward(h, ck, cv, frame_pos0, m0, ctx_kv[layer][0], ctx_kv[layer][1], w, shape,
                          rho=rho, fp8=fp8)
        committed.append((keep(r["k_new"]), keep(r["v_new"])))
        h = keep(r["out"])
    return x0, committed, xs
