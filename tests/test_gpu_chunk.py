"""GPU checks of whole-chunk generation (ardit_chunk_generate) through the C ABI.

1. The call equals the same passes composed by hand from ardit_time_mod and
   ardit_stack_fwd, with the sampler update emulated on the host in the
   kernel's own arithmetic, bit for bit: x0 and every page of every layer
   (untouched pages keep their NaN sentinel).  Streams with different step
   counts exercise the lockstep passes (denoising and commit in one pass,
   then a commit-only pass).
2. A chain of chunks of two streams under sink + window caches, whose page
   tables come from ardit_window_pages, tracks the float64 oracle chunk by
   chunk: the clean chunk and the committed keys/values of every layer.  The
   oracle keeps its own committed keys/values (no GPU value feeds it) and
   rounds to bf16 where the library stores bf16 (layer outputs, the sampler
   result, the pages).  Evicted chunks' slots are reused by later chunks; a
   read of a page outside the window would mix in another chunk's keys and a
   read of a never-written page NaN.

Tolerance of (2): the parity bar (max |d| <= 2e-2 RMS(ref) + k half-ulps of
a quantum, cosine >= 0.9995) with k = 2 sqrt(n), n the bf16 stores on the
longest path to the compared tensor (layers times passes, over the chunks
whose keys it attends to): single-ulp rounding flips between the two sides
persist and add up as a random walk, as for the stack.  The quantum of a
stored key or value is its reference.  The clean chunk x0 = x - tau v is a
difference of two stored tensors that nearly cancel (with random weights the
stack is close to the identity, so v ~ x): a flip in x or v carries their
ulp, not x0's, so its quantum is |x| + tau |v| of the last step.
"""
import math

import numpy as np
import pytest

import oracle as O
from harness import PagedCache, dev_bf16, dev_i32, host_bits, host_f32, parity, upload_block_weights
from workloads import WORKLOADS, bf16_bits, bf16_round, bits_to_f32, make_rng, normal_bf16
from workloads.gen import draw_block_weights, draw_time_weights

pytestmark = pytest.mark.gpu

SH = WORKLOADS["tiny"].shape          # D 256, 4 x 64 heads, FFN 1024, 3 frames of 8 x 8
LQ = SH.chunk_tokens


@pytest.fixture(scope="module")
def A(gpu):
    from paper_2606_15319_amd import ardit
    return ardit


def _sync():
    import torch
    torch.cuda.synchronize()


def _sampler_bits(x, v, tau, tau_next, eps):
    """The sampler kernel's arithmetic on the host: r = fma(-tau, v, x) in
    fp32, then fma(1 - tau', r, fp32(tau' eps)) when there is a next step,
    stored bf16 (round to nearest even).  Operands hold bf16 values, so the
    products are exact in float64 and each fma is one rounding of the exact
    value (float64 holds the sums exactly unless the operands' exponents are
    more than 20 apart, where the first rounding cannot create an fp32 tie)."""
    tau32 = np.float64(np.float32(tau))
    r = (x.astype(np.float64) - tau32 * v.astype(np.float64)).astype(np.float32)
    if tau_next is not None:
        tn = np.float32(tau_next)
        keep = np.float32(np.float32(1.0) - tn)
        p = (np.float64(tn) * eps.astype(np.float64)).astype(np.float32)
        r = (np.float64(keep) * r.astype(np.float64) + p.astype(np.float64)).astype(np.float32)
    return bf16_bits(r)


class Model:
    """Tiny-shape stack of n_layers with per-stream text K/V, on the device."""

    def __init__(self, A, seed, n_layers, ctx_lens, shape=SH):
        import torch
        self.A = A
        self.shape = shape
        rng = make_rng(seed)
        self.rng = rng
        self.n_layers = n_layers
        self.time_w = draw_time_weights(rng, shape.dim, shape.time_freq_dim)
        self.block_w = [draw_block_weights(rng, shape) for _ in range(n_layers)]
        self.ctx = [normal_bf16(rng, (n, shape.dim)) for n in ctx_lens]
        self.ctx_lens = list(ctx_lens)
        self.dims = A.dims_from_shape(shape)
        self.tw_dev = {k: dev_bf16(v) for k, v in self.time_w.items()}
        self.tw = A.time_weights(self.tw_dev)
        self.w_dev = [upload_block_weights(w) for w in self.block_w]
        self.w = [A.block_weights(w) for w in self.w_dev]
        cb = A.Batch(ctx_lens=ctx_lens)
        ws_bytes = A.ardit_workspace_size(self.dims, cb)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        ctx_dev = dev_bf16(np.concatenate(self.ctx))
        n = sum(ctx_lens) * shape.dim
        self.ctx_k = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(n_layers)]
        self.ctx_v = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(n_layers)]
        for l in range(n_layers):
            A.ardit_ctx_kv(None, self.dims, cb, ctx_dev, self.w[l], self.ctx_k[l], self.ctx_v[l],
                           ws, ws_bytes)
        # oracle text K/V per stream and layer
        self.ctx_ref = [[O.context_kv(c, self.block_w[l], shape.eps) for l in range(n_layers)]
                        for c in self.ctx]

    def workspace(self, batch):
        import torch
        n = self.A.ardit_workspace_size(self.dims, batch)
        return torch.empty(n, dtype=torch.uint8, device="cuda"), n


def test_chunk_generate_equals_composed_passes(A):
    """Streams with 3, 2 and 1 steps (one block-sparse): the call equals the
    lockstep passes composed by hand, bit for bit."""
    import torch
    n_layers = 2
    n_steps = [3, 2, 1]
    ts = [[1000.0, 700.0, 350.0], [900.0, 400.0], [600.0]]
    cache_chunks = [2, 0, 1]
    B = len(n_steps)
    m = Model(A, 90, n_layers, [32, 17, 8])
    rng = m.rng
    page_ids, nxt = [], 0
    for c in cache_chunks:
        nf = (c + 1) * SH.frames
        page_ids.append(list(range(nxt, nxt + nf)))
        nxt += nf
    pools = [PagedCache(SH, page_ids, nxt + 2) for _ in range(n_layers)]   # 2 pages never used
    for p in pools:
        for b, c in enumerate(cache_chunks):
            if c:
                n = c * LQ
                p.fill_stream(b, normal_bf16(rng, (n, SH.n_heads, SH.head_dim)),
                              normal_bf16(rng, (n, SH.n_heads, SH.head_dim)))
    x_init = normal_bf16(rng, (B * LQ, SH.dim))
    noise = normal_bf16(rng, (max(n_steps) - 1, B * LQ, SH.dim))
    sparsity = [0.0, 0.5, 0.0]
    lens = dict(q=[LQ] * B, c=[c * LQ for c in cache_chunks], p=[3 * c for c in cache_chunks])
    batch = A.Batch(lens["q"], lens["c"], lens["p"], m.ctx_lens, sparsity=sparsity)
    ws, ws_bytes = m.workspace(batch)
    xi_dev, noise_dev = dev_bf16(x_init), dev_bf16(noise)

    # (a) one call
    for p in pools:
        p.upload()
    x0 = torch.empty_like(xi_dev)
    A.ardit_chunk_generate(None, m.dims, batch, n_steps, ts, xi_dev, noise_dev,
                           [p.kv(A) for p in pools], m.tw, m.ctx_k, m.ctx_v, m.w, x0, ws, ws_bytes)
    _sync()
    got_x0 = host_bits(x0)
    got_pages = [p.device_bits() for p in pools]

    # (b) the same passes by hand
    for p in pools:
        p.upload()
    mod = torch.empty((B, 6, SH.dim), dtype=torch.float32, device="cuda")
    vel = torch.empty_like(xi_dev)
    x_cur = bits_to_f32(bf16_bits(x_init))
    for i in range(max(n_steps) + 1):
        active = sum(1 for s in n_steps if s >= i)
        denoise = sum(1 for s in n_steps if s > i)
        sub = A.Batch(lens["q"][:active], lens["c"][:active], lens["p"][:active],
                      m.ctx_lens[:active], sparsity=sparsity[:active])
        t_pass = [ts[b][i] if i < n_steps[b] else 0.0 for b in range(active)]
        A.ardit_time_mod(None, m.dims, t_pass, m.tw, mod, ws, ws_bytes)
        A.ardit_stack_fwd(None, m.dims, sub, dev_bf16(x_cur[:active * LQ]),
                          [p.kv(A) for p in pools], mod, m.ctx_k, m.ctx_v, m.w, vel, ws, ws_bytes)
        _sync()
        v = host_f32(vel)
        nxt = x_cur.copy()
        for b in range(denoise):
            rows = slice(b * LQ, (b + 1) * LQ)
            tn = ts[b][i + 1] / 1000.0 if i + 1 < n_steps[b] else None
            bits = _sampler_bits(x_cur[rows], v[rows], ts[b][i] / 1000.0, tn,
                                 noise[i][rows] if tn is not None else None)
            nxt[rows] = bits_to_f32(bits)
        x_cur = nxt
    assert np.array_equal(got_x0, bf16_bits(x_cur))
    for l, p in enumerate(pools):
        kb, vb = p.device_bits()
        assert np.array_equal(got_pages[l][0], kb), f"layer {l} keys"
        assert np.array_equal(got_pages[l][1], vb), f"layer {l} values"
        # the two spare pages were never written
        assert (kb[-2:] == 0x7FC0).all() and (vb[-2:] == 0x7FC0).all()


def test_chunk_chain_sink_window_tracks_oracle(A):
    """Chunks 0..4 of two streams: stream 0 with 3 steps, sink 1 and window 2
    (chunk 4 evicts chunk 1 and reuses its slot), stream 1 with 2 steps, no
    sink and window 1 (a ring of two slots)."""
    import torch
    n_layers = 2
    cfg = [dict(steps=[1000.0, 750.0, 500.0], sink=1, window=2),
           dict(steps=[1000.0, 500.0], sink=0, window=1)]
    B = len(cfg)
    m = Model(A, 91, n_layers, [32, 24])
    rng = m.rng
    F = SH.frames
    slots = [c["sink"] + c["window"] + 1 for c in cfg]
    base = [0, slots[0] * F]
    n_pages = sum(slots) * F
    max_frames = max(slots) * F
    pools = [PagedCache(SH, [list(range(max_frames))] * B, n_pages) for _ in range(n_layers)]
    for p in pools:
        p.upload()                        # every page NaN until written
    committed = [[] for _ in range(B)]    # oracle: per stream, per chunk, per layer (k, v)
    n_chunks = 5
    for c in range(n_chunks):
        table = np.zeros((B, max_frames), dtype=np.int32)
        cache_lens, held = [], []
        for b, cf in enumerate(cfg):
            ids, cached = A.ardit_window_pages(c, cf["sink"], cf["window"], F, base[b], max_frames)
            table[b, :len(ids)] = ids
            cache_lens.append(cached * SH.tokens_per_frame)
            held.append(O.chunk_ref.window_chunks(c, cf["sink"], cf["window"]))
            assert cached == len(held[b]) * F
        table_dev = dev_i32(table)
        kvs = [A.kv_paged(p.k, p.v, table_dev, n_pages, max_frames) for p in pools]
        n_steps = [len(cf["steps"]) for cf in cfg]
        batch = A.Batch([LQ] * B, cache_lens, [F * c] * B, m.ctx_lens)
        ws, ws_bytes = m.workspace(batch)
        x_init = [normal_bf16(rng, (LQ, SH.dim)) for _ in range(B)]
        noise = [[normal_bf16(rng, (LQ, SH.dim)) for _ in range(s - 1)] for s in n_steps]
        noise_dev = np.zeros((max(n_steps) - 1, B * LQ, SH.dim), dtype=np.float32)
        for b in range(B):
            for i, e in enumerate(noise[b]):
                noise_dev[i, b * LQ:(b + 1) * LQ] = e
        x0 = torch.empty((B * LQ, SH.dim), dtype=torch.bfloat16, device="cuda")
        A.ardit_chunk_generate(None, m.dims, batch, n_steps, [cf["steps"] for cf in cfg],
                               dev_bf16(np.concatenate(x_init)), dev_bf16(noise_dev), kvs, m.tw,
                               m.ctx_k, m.ctx_v, m.w, x0, ws, ws_bytes)
        _sync()
        got = host_f32(x0)
        for b, cf in enumerate(cfg):
            caches = []
            for l in range(n_layers):
                ks = [committed[b][k][l][0] for k in held[b]]
                vs = [committed[b][k][l][1] for k in held[b]]
                empty = np.zeros((0, SH.n_heads, SH.head_dim))
                caches.append((np.concatenate(ks) if ks else empty,
                               np.concatenate(vs) if vs else empty))
            x0_ref, kv_ref, xs_ref = O.chunk_ref.generate_chunk(
                x_init[b], noise[b], cf["steps"], caches, F * c, m.time_w, m.ctx_ref[b],
                m.block_w, SH, store=bf16_round)
            committed[b].append(kv_ref)
            n_store = n_layers * (len(cf["steps"]) + 1) * (len(held[b]) + 1)
            k_ulps = 2.0 * np.sqrt(n_store)
            x_last = xs_ref[-1]
            tau = cf["steps"][-1] / 1000.0
            v_last = (x_last - x0_ref) / tau
            print(parity(got[b * LQ:(b + 1) * LQ], x0_ref, f"chunk {c} stream {b} x0",
                         quantum=np.abs(x_last) + tau * np.abs(v_last), half_ulps=k_ulps))
            ids = table[b][cache_lens[b] // SH.tokens_per_frame:][:F]
            for l, p in enumerate(pools):
                kb, vb = p.device_bits()
                k_pg = bits_to_f32(kb[ids])                       # [F][H][T][d]
                v_pg = bits_to_f32(vb[ids])                       # [F][H][d][T]
                k_got = np.transpose(k_pg, (0, 2, 1, 3)).reshape(LQ, SH.n_heads, SH.head_dim)
                v_got = np.transpose(v_pg, (0, 3, 1, 2)).reshape(LQ, SH.n_heads, SH.head_dim)
                print(parity(k_got, kv_ref[l][0], f"chunk {c} stream {b} layer {l} committed k",
                             quantum=kv_ref[l][0], half_ulps=k_ulps))
                print(parity(v_got, kv_ref[l][1], f"chunk {c} stream {b} layer {l} committed v",
                             quantum=kv_ref[l][1], half_ulps=k_ulps))


def test_controller_drives_batched_generation(A):
    """The controller picks each stream's configuration (BMPR over a latency
    table) and the streams then generate their chunks in one batched call
    with those step counts and windows (streams ordered by steps, as the
    call requires); every stream tracks its own float64 oracle run."""
    import torch
    n_layers = 2
    F = SH.frames
    # (S, rho, W, Q, ms per chunk, quality): a synthetic table; the median
    # quality (the floor) is 75
    table = [(4, 0.0, 3, 0, 300.0, 90.0), (4, 0.0, 1, 0, 220.0, 85.0),
             (3, 0.0, 3, 0, 200.0, 84.0), (3, 0.0, 1, 0, 150.0, 80.0),
             (2, 0.0, 3, 0, 130.0, 70.0), (2, 0.0, 1, 0, 100.0, 60.0),
             (2, 0.0, 7, 0, 400.0, 50.0), (3, 0.0, 7, 0, 500.0, 55.0)]
    frontier, floor = A.ardit_pareto_frontier(table)
    assert floor == 75.0
    # budget 210 ms: (3, 3) fits; 1000 ms: the best (4, 3); 40 ms: nothing fits,
    # speed recovery takes the fastest point above the floor, (3, 1)
    streams = [(0, 210.0, 0.0), (0, 1000.0, 0.0), (0, 50.0, 10.0)]
    dec = A.ardit_control_tick(1, table, frontier, floor, streams)
    cfg = [table[d.cfg] for d in dec]
    assert [d.cfg for d in dec] == [2, 0, 3]
    assert [d.mode for d in dec] == [A.BMPR_QUALITY, A.BMPR_QUALITY, A.BMPR_SPEED_RECOVERY]
    assert [d.tier for d in dec] == [A.URGENT, A.NORMAL, A.URGENT]
    assert [d.queue_pos for d in dec] == [1, 2, 0]
    order = sorted(range(3), key=lambda b: -cfg[b][0])        # non-increasing steps
    m = Model(A, 92, n_layers, [32, 32, 32])
    rng = m.rng
    chunk_idx = [5, 4, 6]
    slots = max(t[2] for t in table) + 1
    ids_all, cached_all, held_all = [], [], []
    for pos, b in enumerate(order):
        W = cfg[b][2]
        ids, cached = A.ardit_window_pages(chunk_idx[b], 0, W, F, pos * slots * F)
        ids_all.append(ids)
        cached_all.append(cached)
        held_all.append(O.chunk_ref.window_chunks(chunk_idx[b], 0, W))
    n_pages = 3 * slots * F
    pools = [PagedCache(SH, ids_all, n_pages) for _ in range(n_layers)]
    caches = [[None] * n_layers for _ in order]
    for l, p in enumerate(pools):
        for pos in range(3):
            n = cached_all[pos] * SH.tokens_per_frame
            k = normal_bf16(rng, (n, SH.n_heads, SH.head_dim))
            v = normal_bf16(rng, (n, SH.n_heads, SH.head_dim))
            if n:
                p.fill_stream(pos, k, v)
            caches[pos][l] = (k, v)
        p.upload()
    B = 3
    steps = [cfg[b][0] for b in order]
    ts = [[1000.0 * (1 - i / s) for i in range(s)] for s in steps]
    x_init = [normal_bf16(rng, (LQ, SH.dim)) for _ in range(B)]
    noise = [[normal_bf16(rng, (LQ, SH.dim)) for _ in range(s - 1)] for s in steps]
    noise_dev = np.zeros((max(steps) - 1, B * LQ, SH.dim), dtype=np.float32)
    for pos in range(B):
        for i, e in enumerate(noise[pos]):
            noise_dev[i, pos * LQ:(pos + 1) * LQ] = e
    batch = A.Batch([LQ] * B, [c * SH.tokens_per_frame for c in cached_all],
                    [F * chunk_idx[b] for b in order], m.ctx_lens)
    ws, ws_bytes = m.workspace(batch)
    x0 = torch.empty((B * LQ, SH.dim), dtype=torch.bfloat16, device="cuda")
    A.ardit_chunk_generate(None, m.dims, batch, steps, ts, dev_bf16(np.concatenate(x_init)),
                           dev_bf16(noise_dev), [p.kv(A) for p in pools], m.tw, m.ctx_k, m.ctx_v,
                           m.w, x0, ws, ws_bytes)
    _sync()
    got = host_f32(x0)
    for pos, b in enumerate(order):
        x0_ref, kv_ref, xs_ref = O.chunk_ref.generate_chunk(
            x_init[pos], noise[pos], ts[pos], caches[pos], F * chunk_idx[b], m.time_w,
            m.ctx_ref[pos], m.block_w, SH, store=bf16_round)
        tau = ts[pos][-1] / 1000.0
        v_last = (xs_ref[-1] - x0_ref) / tau
        k_ulps = 2.0 * np.sqrt(n_layers * (steps[pos] + 1) * (len(held_all[pos]) + 1))
        print(parity(got[pos * LQ:(pos + 1) * LQ], x0_ref,
                     f"stream {b} (S={steps[pos]}, W={cfg[b][2]}) x0",
                     quantum=np.abs(xs_ref[-1]) + tau * np.abs(v_last), half_ulps=k_ulps))
        own = ids_all[pos][cached_all[pos]:][:F]
        for l, p in enumerate(pools):
            kb, vb = p.device_bits()
            k_got = np.transpose(bits_to_f32(kb[own]), (0, 2, 1, 3)).reshape(LQ, SH.n_heads,
                                                                             SH.head_dim)
            print(parity(k_got, kv_ref[l][0], f"stream {b} layer {l} committed k",
                         quantum=kv_ref[l][0], half_ulps=k_ulps))


def test_chunk_generate_fp8_stream_tracks_oracle(A):
    """A stream with FP8 self-attention (the quantisation knob) and a bf16 one
    generate one chunk each in one call (head_dim 128, the FP8 kernel's);
    each tracks its float64 oracle run with the same knob.  The FP8 stream is
    held to 6e-2 of the RMS for the max error, as the FP8 block test: both
    sides quantise their own bf16 roundings of q, k and v, so an E4M3 code can
    differ by one step (2^-4 relative) where the two roundings straddle a
    rounding boundary; the cosine keeps 0.9995."""
    import torch
    from workloads import BlockShape
    sh = BlockShape(dim=256, n_heads=2, head_dim=128, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    lq = sh.chunk_tokens
    n_layers = 2
    m = Model(A, 93, n_layers, [24, 24], shape=sh)
    rng = m.rng
    B = 2
    steps = [[1000.0, 500.0], [1000.0, 500.0]]
    quant = [A.QUANT_FP8, A.QUANT_BF16]
    cache = lq                                            # one earlier chunk each
    ids = [list(range(0, 2 * sh.frames)), list(range(2 * sh.frames, 4 * sh.frames))]
    pools = [PagedCache(sh, ids, 4 * sh.frames) for _ in range(n_layers)]
    caches = [[None] * n_layers for _ in range(B)]
    for l, p in enumerate(pools):
        for b in range(B):
            k = normal_bf16(rng, (cache, sh.n_heads, sh.head_dim))
            v = normal_bf16(rng, (cache, sh.n_heads, sh.head_dim))
            p.fill_stream(b, k, v)
            caches[b][l] = (k, v)
        p.upload()
    batch = A.Batch([lq] * B, [cache] * B, [sh.frames] * B, m.ctx_lens, quant=quant)
    ws, ws_bytes = m.workspace(batch)
    x_init = [normal_bf16(rng, (lq, sh.dim)) for _ in range(B)]
    noise = [[normal_bf16(rng, (lq, sh.dim))] for _ in range(B)]
    x0 = torch.empty((B * lq, sh.dim), dtype=torch.bfloat16, device="cuda")
    A.ardit_chunk_generate(None, m.dims, batch, [2, 2], steps, dev_bf16(np.concatenate(x_init)),
                           dev_bf16(np.concatenate([n[0] for n in noise])[None]),
                           [p.kv(A) for p in pools], m.tw, m.ctx_k, m.ctx_v, m.w, x0, ws,
                           ws_bytes)
    _sync()
    got = host_f32(x0)
    for b in range(B):
        fp8 = quant[b] == A.QUANT_FP8
        x0_ref, kv_ref, xs_ref = O.chunk_ref.generate_chunk(
            x_init[b], noise[b], steps[b], caches[b], sh.frames, m.time_w, m.ctx_ref[b],
            m.block_w, sh, store=bf16_round, fp8=fp8)
        tau = steps[b][-1] / 1000.0
        v_last = (xs_ref[-1] - x0_ref) / tau
        k_ulps = 2.0 * np.sqrt(n_layers * 3 * 2)
        print(parity(got[b * lq:(b + 1) * lq], x0_ref, f"{'FP8' if fp8 else 'bf16'} stream x0",
                     tol=6e-2 if fp8 else 2e-2,
                     quantum=np.abs(xs_ref[-1]) + tau * np.abs(v_last), half_ulps=k_ulps))
        own = ids[b][cache // sh.tokens_per_frame:]
        for l, p in enumerate(pools):
            kb, vb = p.device_bits()
            k_got = np.transpose(bits_to_f32(kb[own]), (0, 2, 1, 3)).reshape(lq, sh.n_heads,
                                                                             sh.head_dim)
            print(parity(k_got, kv_ref[l][0], f"{'FP8' if fp8 else 'bf16'} layer {l} committed k",
                         tol=6e-2 if fp8 else 2e-2, quantum=kv_ref[l][0], half_ulps=k_ulps))
