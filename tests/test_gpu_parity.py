"""GPU parity of every entry point against the float64 oracle, plus the
bit-exact index/visibility checks (pages, sentinels, permutations, ragged
batches).  All calls go through the C ABI."""
import copy

import numpy as np
import pytest

import oracle as O
from harness import (BlockRun, PagedCache, NAN_BITS, dev_bf16, fp8_parity, host_bits, host_f32,
                     parity, ring_page_ids, sample_rows, upload_block_weights)
from workloads import BlockShape, WORKLOADS, bf16_round, make_rng, normal_bf16
from workloads.gen import draw_block_case, draw_time_weights, draw_block_weights

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def A(gpu):
    from paper_2606_15319_amd import ardit
    return ardit


def _sync():
    import torch
    torch.cuda.synchronize()


TINY = WORKLOADS["tiny"].shape


# ------------------------------------------------------------ time, context
@pytest.mark.parametrize("dim", [256, 1536])
def test_time_mod(A, dim):
    import torch
    sh = BlockShape(dim=dim, n_heads=dim // 64, head_dim=64, ffn_dim=1024, frames=3, lat_h=8,
                    lat_w=8)
    tw = draw_time_weights(make_rng(40), dim)
    ts = [1000.0, 750.0, 500.0, 250.0, 0.0]
    dims = A.dims_from_shape(sh)
    mod = torch.empty((len(ts), 6, dim), dtype=torch.float32, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    A.ardit_time_mod(None, dims, ts, A.time_weights({k: dev_bf16(v) for k, v in tw.items()}),
                     mod, ws, ws.numel())
    _sync()
    got = host_f32(mod)
    for i, t in enumerate(ts):
        parity(got[i], O.time_modulation(t, tw, dim), f"time_mod t={t}")


def test_ctx_kv(A):
    import torch
    from paper_2606_15319_amd.layout import ctx_from_device_layout
    sh = TINY
    w = draw_block_weights(make_rng(41), sh)
    rng = make_rng(42)
    lens = [32, 20, 64, 1]
    ctx = [normal_bf16(rng, (n, sh.dim)) for n in lens]
    dims = A.dims_from_shape(sh)
    batch = A.Batch(ctx_lens=lens)
    wd = upload_block_weights(w)
    nct = sum(lens)
    ck = torch.empty(nct * sh.dim, dtype=torch.bfloat16, device="cuda")
    cv = torch.empty_like(ck)
    ws_bytes = A.ardit_workspace_size(dims, batch)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    A.ardit_ctx_kv(None, dims, batch, dev_bf16(np.concatenate(ctx)), A.block_weights(wd), ck, cv,
                   ws, ws_bytes)
    _sync()
    kf, vf = host_f32(ck), host_f32(cv)
    off = 0
    for b, n in enumerate(lens):
        k, v = ctx_from_device_layout(kf[off * sh.dim:(off + n) * sh.dim],
                                      vf[off * sh.dim:(off + n) * sh.dim], n, sh.n_heads,
                                      sh.head_dim)
        kr, vr = O.context_kv(ctx[b], w, sh.eps)
        parity(k, kr, f"ctx_k stream {b}")
        parity(v, vr, f"ctx_v stream {b}")
        off += n


# --------------------------------------------------------------- kv append
# rows of 2304 (> 2048) take the two-launch append path, the tiny block the fused one
WIDE = BlockShape(dim=2304, n_heads=18, head_dim=128, ffn_dim=256, frames=2, lat_h=4, lat_w=8)


@pytest.mark.parametrize("sh", [TINY, WIDE], ids=["tiny", "wide"])
def test_kv_append_placement(A, sh):
    """q~ and k~ match the oracle; values land bit-exactly in the oracle's slot
    map through a shuffled page table; nothing else of the pool changes."""
    import torch
    rng = make_rng(43)
    caches = [2 * sh.chunk_tokens, 0, sh.chunk_tokens]
    pos0 = [6, 0, 4]
    B = len(caches)
    T = sh.tokens_per_frame
    frames = [c // T + sh.frames for c in caches]
    perm = np.random.default_rng(1).permutation(sum(frames) + 3)
    ids, nxt = [], 0
    for f in frames:
        ids.append([int(p) for p in perm[nxt:nxt + f]])
        nxt += f
    pc = PagedCache(sh, ids, len(perm))
    pc.upload()
    before_k, before_v = pc.device_bits()
    qkv = normal_bf16(rng, (B * sh.chunk_tokens, 3 * sh.dim))
    g_q = normal_bf16(rng, (sh.dim,), 0.02, 1.0)
    g_k = normal_bf16(rng, (sh.dim,), 0.02, 1.0)
    dims = A.dims_from_shape(sh)
    batch = A.Batch([sh.chunk_tokens] * B, caches, pos0)
    q_out = torch.empty((B * sh.chunk_tokens, sh.dim), dtype=torch.bfloat16, device="cuda")
    A.ardit_kv_append(None, dims, batch, dev_bf16(qkv), dev_bf16(g_q), dev_bf16(g_k), pc.kv(A),
                      q_out)
    _sync()
    qg = host_f32(q_out)
    after_k, after_v = pc.device_bits()
    touched_k = np.zeros(after_k.shape, bool)
    touched_v = np.zeros(after_v.shape, bool)
    L, D, H, d = sh.chunk_tokens, sh.dim, sh.n_heads, sh.head_dim
    for b in range(B):
        rows = qkv[b * L:(b + 1) * L]
        pos = O.chunk_positions(sh.frames, sh.lat_h, sh.lat_w, pos0[b])
        qr = O.rope3d(O.rms_norm(rows[:, :D], sh.eps, g_q).reshape(L, H, d), pos, sh.theta)
        kr = O.rope3d(O.rms_norm(rows[:, D:2 * D], sh.eps, g_k).reshape(L, H, d), pos, sh.theta)
        parity(qg[b * L:(b + 1) * L], qr.reshape(L, D), f"q~ stream {b}", quantum=qr)
        vbits = np.ascontiguousarray(rows[:, 2 * D:]).view(np.uint32) >> 16
        for n in range(L):
            j = caches[b] + n
            p, off = ids[b][j // T], j % T
            touched_k[p, :, off, :] = True
            touched_v[p, :, :, off] = True
        kk, vv = pc.read_stream(b, caches[b] + L)
        from workloads import bits_to_f32
        parity(bits_to_f32(kk[caches[b]:]).reshape(L, D), kr.reshape(L, D), f"k~ stream {b}",
               quantum=kr)
        assert np.array_equal(vv[caches[b]:].reshape(L, D), vbits.astype(np.uint16)), \
            f"value placement stream {b}"
    assert np.array_equal(after_k[~touched_k], before_k[~touched_k]), "keys written outside slots"
    assert np.array_equal(after_v[~touched_v], before_v[~touched_v]), "values written outside slots"


# ---------------------------------------------------------------- attention
def _attn_case(A, sh, q_lens, caches, seed, shuffle=True, fill_bits=NAN_BITS, qzero=False):
    import torch
    rng = make_rng(seed)
    H, d, T = sh.n_heads, sh.head_dim, sh.tokens_per_frame
    kvl = [c + q for c, q in zip(caches, q_lens)]
    frames = [(k + T - 1) // T for k in kvl]
    n_pages = sum(frames) + 2
    perm = np.random.default_rng(seed).permutation(n_pages) if shuffle else np.arange(n_pages)
    ids, nxt = [], 0
    for f in frames:
        ids.append([int(p) for p in perm[nxt:nxt + f]])
        nxt += f
    pc = PagedCache(sh, ids, n_pages, fill_bits=fill_bits)
    ks, vs, qs = [], [], []
    for b in range(len(q_lens)):
        k = normal_bf16(rng, (kvl[b], H, d))
        v = normal_bf16(rng, (kvl[b], H, d))
        q = np.zeros((q_lens[b], H, d), np.float32) if qzero else normal_bf16(rng, (q_lens[b], H, d))
        pc.fill_stream(b, k, v)
        ks.append(k); vs.append(v); qs.append(q)
    pc.upload()
    dims = A.dims_from_shape(sh)
    batch = A.Batch(q_lens, caches)
    q = dev_bf16(np.concatenate(qs).reshape(-1, H * d))
    o = torch.empty_like(q)
    return pc, dims, batch, q, o, qs, ks, vs


def _attn(A, dims, batch, q, kv, o):
    """ardit_attn_fwd with a workspace of the size the library reports."""
    import torch
    n = A.ardit_workspace_size(dims, batch)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    A.ardit_attn_fwd(None, dims, batch, q, kv, o, ws, n)
    return ws


@pytest.mark.parametrize("hd", [64, 128])
def test_attn_ragged_small(A, hd):
    sh = BlockShape(dim=4 * hd, n_heads=4, head_dim=hd, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    q_lens, caches = [192, 100, 7, 130], [384, 0, 128, 64]
    pc, dims, batch, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 50)
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = 0
    for b, n in enumerate(q_lens):
        ref = O.attention(qs[b], ks[b], vs[b]).reshape(n, -1)
        parity(og[off:off + n], ref, f"attn hd={hd} stream {b}", quantum=ref)
        off += n


def test_attn_max_streams(A):
    """The largest batch the ABI takes, 64 streams of ragged queries and caches
    (some empty), against the oracle stream by stream."""
    sh = BlockShape(dim=256, n_heads=2, head_dim=128, ffn_dim=512, frames=1, lat_h=4, lat_w=8)
    assert A.ARDIT_MAX_STREAMS == 64
    rng = np.random.default_rng(82)
    q_lens = [int(v) for v in rng.integers(0, 90, 64)]
    caches = [32 * int(v) for v in rng.integers(0, 5, 64)]
    pc, dims, batch, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 82)
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = 0
    for b, n in enumerate(q_lens):
        if n:
            ref = O.attention(qs[b], ks[b], vs[b]).reshape(n, -1)
            parity(og[off:off + n], ref, f"stream {b}", quantum=ref)
        off += n


@pytest.mark.parametrize("mode", ["dense", "sparse", "fp8"])
def test_attn_empty_streams_change_nothing(A, mode):
    """Streams with no queries (their caches still paged) leave every other
    stream's output bit-identical to a call without them, dense, block-sparse
    and FP8 alike; a batch of empty streams only is accepted and writes
    nothing."""
    import torch
    from harness import dev_i32
    sh = BlockShape(dim=512, n_heads=4, head_dim=128, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    q_lens, caches = [0, 300, 0, 70], [640, 128, 0, 192]
    pc, dims, _, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 81)
    extra = {"dense": {}, "sparse": {"sparsity": [0.6] * 4}, "fp8": {"quant": [1] * 4}}[mode]
    _attn(A, dims, A.Batch(q_lens, caches, **extra), q, pc.kv(A), o)
    keep = [1, 3]
    sub = {k: [v[b] for b in keep] for k, v in extra.items()}
    table = dev_i32(np.ascontiguousarray(pc.table_host[keep]))
    kv = A.kv_paged(pc.k, pc.v, table, pc.n_pages, pc.max_frames)
    o2 = torch.full_like(o, float("nan"))
    _attn(A, dims, A.Batch([q_lens[b] for b in keep], [caches[b] for b in keep], **sub), q, kv,
          o2)
    _sync()
    assert np.array_equal(host_bits(o), host_bits(o2))
    # empty streams only: nothing to compute, nothing written
    o3 = torch.full_like(o, float("nan"))
    _attn(A, dims, A.Batch([0, 0], [640, 0], **{k: v[:2] for k, v in extra.items()}), q,
          pc.kv(A), o3)
    _sync()
    assert np.isnan(host_f32(o3)).all()


def test_attn_visibility_nan_poison(A):
    """q = 0 gives the mean of exactly the visible values; every page slot
    outside [0, kv_len) holds NaN, so reading one would poison the output."""
    sh = TINY
    q_lens, caches = [100, 33], [64, 0]
    pc, dims, batch, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 51, qzero=True)
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = 0
    for b, n in enumerate(q_lens):
        assert np.isfinite(og[off:off + n]).all()
        mean = vs[b].astype(np.float64).mean(axis=0).reshape(-1)
        ref = np.broadcast_to(mean, (n, mean.size))
        parity(og[off:off + n], ref, f"mean of visible {b}", quantum=ref)
        off += n


def test_attn_page_permutation_bit_identical(A):
    sh = TINY
    outs = []
    for shuffle in (False, True):
        pc, dims, batch, q, o, *_ = _attn_case(A, sh, [192, 50], [320, 128], 52, shuffle=shuffle)
        _attn(A, dims, batch, q, pc.kv(A), o)
        _sync()
        outs.append(host_bits(o))
    assert np.array_equal(outs[0], outs[1])


def test_attn_split_schedule_ragged(A):
    """Three streams, 8 heads of 64: 144 (stream, head, 256-query) items for
    256 CUs, so the key ranges are split between workgroups (ranges cross item
    and stream boundaries) and merged; sampled rows of every stream, including
    the ragged last query tile."""
    sh = BlockShape(dim=512, n_heads=8, head_dim=64, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    q_lens, caches = [1500, 700, 2300], [3008, 0, 1216]
    pc, dims, batch, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 53)
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = 0
    for b, n in enumerate(q_lens):
        rows = sample_rows(n, seed=b)
        ref = O.attention(qs[b][rows], ks[b], vs[b]).reshape(len(rows), -1)
        parity(og[off:off + n][rows], ref, f"split attn stream {b}", quantum=ref)
        off += n


def test_attn_chunk_over_cache_4680x14040(A):
    """4680 queries (3 frames of 30x52) over 9360 cached + 4680 own keys, 12
    heads of 128, QK-RMSNorm applied to Q and K; sampled query rows."""
    import torch
    wl = WORKLOADS["attn"]
    sh = wl.shape
    rng = make_rng(wl.wid)
    L, c = sh.chunk_tokens, 2 * sh.chunk_tokens
    H, d, D = sh.n_heads, sh.head_dim, sh.dim
    q = bf16_round(O.rms_norm(rng.standard_normal((L, D), dtype=np.float32), sh.eps))
    k = bf16_round(O.rms_norm(rng.standard_normal((c + L, D), dtype=np.float32), sh.eps))
    v = normal_bf16(rng, (c + L, H, d))
    T = sh.tokens_per_frame
    pc = PagedCache(sh, [list(range((c + L) // T))], (c + L) // T)
    pc.fill_stream(0, k.reshape(-1, H, d), v)
    pc.upload()
    qd = dev_bf16(q)
    o = torch.empty_like(qd)
    _attn(A, A.dims_from_shape(sh), A.Batch([L], [c]), qd, pc.kv(A), o)
    _sync()
    rows = sample_rows(L, seed=2)
    ref = O.attention(q[rows].reshape(-1, H, d), k.reshape(-1, H, d), v).reshape(len(rows), D)
    parity(host_f32(o)[rows], ref, "attn 4680x14040")


@pytest.mark.parametrize("name", ["block13b", "large"])
def test_attn_sp2_share_full_keys(A, name):
    """One GPU's share of Ulysses SP2 (Appendix C): after the all-to-all a GPU
    holds every query of the chunk for half the heads and attends over the
    head-partitioned pages at the full key length -- the 1.3B-class block's 6
    of 12 heads over 32760 keys (114 items, so the split schedule and its
    merge run at full length) and the large block's 20 of 40 heads over 37440
    keys through its wrapped ring.  Q and K RMS-normalised over the share's
    width, V ~ N(0, 1); sampled query rows against the oracle."""
    import torch
    from workloads import stream_page_ids
    wl = WORKLOADS[name]
    full = wl.shape
    hs = full.n_heads // 2
    sh = BlockShape(dim=hs * full.head_dim, n_heads=hs, head_dim=full.head_dim,
                    ffn_dim=full.ffn_dim, frames=full.frames, lat_h=full.lat_h, lat_w=full.lat_w)
    H, d, D, L = sh.n_heads, sh.head_dim, sh.dim, sh.chunk_tokens
    cache = wl.cache_chunks[0] * L
    rng = make_rng(60 + wl.wid)
    q = bf16_round(O.rms_norm(rng.standard_normal((L, D), dtype=np.float32), sh.eps))
    k = bf16_round(O.rms_norm(rng.standard_normal((cache + L, D), dtype=np.float32), sh.eps))
    v = normal_bf16(rng, (cache + L, H, d))
    ids, n_pages = stream_page_ids(wl)
    pc = PagedCache(sh, ids[:1], n_pages)
    pc.fill_stream(0, k.reshape(-1, H, d), v)
    pc.upload()
    qd = dev_bf16(q)
    o = torch.empty_like(qd)
    _attn(A, A.dims_from_shape(sh), A.Batch([L], [cache]), qd, pc.kv(A), o)
    _sync()
    rows = sample_rows(L, seed=3)
    ref = O.attention(q[rows].reshape(-1, H, d), k.reshape(-1, H, d), v).reshape(len(rows), D)
    parity(host_f32(o)[rows], ref, f"SP2 share {name}", quantum=ref)


# -------------------------------------------------------------------- block
def _check_block(run, b, rows=None, tag=""):
    ref = run.reference(b, rows=rows)
    L, D = run.shape.chunk_tokens, run.shape.dim
    out = host_f32(run.out)[b * L:(b + 1) * L]
    x = run.case.x[b]
    sel = ref["rows"]
    parity(out[sel], ref["out"], f"{tag} out stream {b}")
    parity(out[sel] - x[sel], ref["out"] - x[sel], f"{tag} out-x stream {b}", tol=5e-2,
           quantum=ref["out"], cos_ref=bf16_round(ref["out"]) - x[sel])
    from workloads import bits_to_f32
    kk, vv = run.pages.read_stream(b, run.case.cache_len[b] + L)
    c = run.case.cache_len[b]
    parity(bits_to_f32(kk[c:]).reshape(L, D), ref["k_new"].reshape(L, D), f"{tag} k pages {b}",
           quantum=ref["k_new"])
    parity(bits_to_f32(vv[c:]).reshape(L, D), ref["v_new"].reshape(L, D), f"{tag} v pages {b}",
           quantum=ref["v_new"])
    if c:
        assert np.array_equal(kk[:c], np.asarray(
            (run.case.cache_k[b].view(np.uint32) >> 16).astype(np.uint16))), "cache keys changed"
    return ref


def _check_self_attention(A, dims, batch, kv, k_pages, v_pages, page_ids, cache_len, L, refs,
                          ws, ws_bytes, tag, fp8=()):
    """The block's self-attention output at its real size.  The block call
    reuses its attention buffer for the text cross-attention, so the output is
    recomputed by ardit_attn_fwd -- the same kernels and schedule as in the
    block -- over the pages the block call left (the chunk's keys and values
    as the GPU appended them), fed the oracle's rotated queries rounded to
    bf16.  For every stream b in refs (an oracle block result on sampled rows)
    the sampled rows are compared (a) with the oracle attention of those very
    queries over the keys and values read back from the pages, at the bar
    plus half a bf16 ulp (the kernel's own arithmetic), and (b) with the
    oracle block's own o at 5e-2 of its RMS plus half an ulp and the 0.9995
    cosine (the whole path: the keys in the pages come from the bf16-stored
    adaLN output through the QKV GEMM and are stored bf16 themselves, which
    moves a peaked softmax by up to 3e-2 of the RMS, measured on the
    ragged batch's stream with no cache).  Streams in fp8 run FP8 attention
    and take the FP8 criterion against (a)."""
    import torch
    from workloads import bf16_round
    D = dims.dim
    H, d = dims.n_heads, dims.head_dim
    n = len(cache_len)
    qh = np.zeros((n * L, D), np.float32)
    for b, ref in refs.items():
        qh[b * L:(b + 1) * L] = bf16_round(ref["q"].reshape(L, D))
    qd = dev_bf16(qh)
    o = torch.empty_like(qd)
    A.ardit_attn_fwd(None, dims, batch, qd, kv, o, ws, ws_bytes)
    _sync()
    og = host_f32(o)
    from harness import read_stream_pages
    for b, ref in refs.items():
        sel = ref["rows"]
        K, V = read_stream_pages(k_pages, v_pages, page_ids[b], cache_len[b] + L)
        got = og[b * L + sel]
        qb = qh[b * L:(b + 1) * L].reshape(L, H, d)
        if b in fp8:
            _fp8_check(got, qb, K, V, f"{tag} fp8 o stream {b}", rows=sel)
            continue
        on_pages = O.attention(qb[sel], K, V).reshape(len(sel), D)
        parity(got, on_pages, f"{tag} o stream {b} (pages)", quantum=on_pages)
        parity(got, ref["o"], f"{tag} o stream {b} (block)", tol=5e-2, quantum=ref["o"])


def _run_self_attention_check(A, run, refs, tag):
    c = run.case
    _check_self_attention(A, run.dims, run.batch, run.pages.kv(A), run.pages.k, run.pages.v,
                          run.pages.page_ids, c.cache_len, run.shape.chunk_tokens, refs, run.ws,
                          run.ws_bytes, tag)


def test_block_tiny(A):
    run = BlockRun(WORKLOADS["tiny"], A, shuffle_pages_seed=3)
    run.run()
    _sync()
    _check_block(run, 0, tag="tiny")


def test_block_half_tile_widths(A):
    """dim, 3 dim and ffn_dim that are multiples of 128 but not of 256,
    a chunk of 144 tokens that ends inside a row tile, and two streams."""
    import dataclasses
    sh = BlockShape(dim=384, n_heads=3, head_dim=128, ffn_dim=640, frames=3, lat_h=6, lat_w=8)
    wl = dataclasses.replace(WORKLOADS["tiny"], shape=sh, cache_chunks=(1, 0),
                             frame_pos0=(3, 0), timesteps=(750, 250), ctx_len=40)
    run = BlockRun(wl, A, shuffle_pages_seed=5)
    run.run()
    _sync()
    for b in range(2):
        _check_block(run, b, tag="half-tile")


def test_block_tiny_strong_branches(A):
    """Same shapes with gates near 1 and larger output projections, so every
    branch moves `out` well beyond the bf16 rounding of the residual."""
    case = draw_block_case(WORKLOADS["tiny"])
    w = case.block_w
    w["mod_table"] = w["mod_table"].copy()
    w["mod_table"][2] += 1.0
    w["mod_table"][5] += 1.0
    for k in ("w_o", "w_co"):
        w[k] = w[k] * 8.0
    w["w_2"] = w["w_2"] * 4.0
    run = BlockRun(WORKLOADS["tiny"], A, case=case)
    run.run()
    _sync()
    ref = _check_block(run, 0, tag="strong")
    assert np.abs(ref["x1"] - case.x[0]).std() > 0.05      # self-attention branch visible
    assert np.abs(ref["x2"] - ref["x1"]).std() > 0.05      # cross-attention branch visible


def test_block_deterministic_and_page_order_invariant(A):
    outs = []
    for seed in (None, 11, 11):
        run = BlockRun(WORKLOADS["tiny"], A, shuffle_pages_seed=seed)
        run.run()
        _sync()
        outs.append(host_bits(run.out))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[1], outs[2])


def test_ragged_batch_equals_single_calls(A):
    import torch
    wl = WORKLOADS["tiny"]
    base = draw_block_case(wl)
    sh = wl.shape
    rng = make_rng(60)
    caches = [0, 2 * sh.chunk_tokens, sh.chunk_tokens]
    case = draw_block_case(wl)
    case.x, case.cache_k, case.cache_v, case.ctx = [], [], [], []
    case.cache_len, case.frame_pos0, case.t = [], [], []
    for i, c in enumerate(caches):
        case.x.append(normal_bf16(rng, (sh.chunk_tokens, sh.dim)))
        case.cache_k.append(normal_bf16(rng, (c, sh.n_heads, sh.head_dim)))
        case.cache_v.append(normal_bf16(rng, (c, sh.n_heads, sh.head_dim)))
        case.ctx.append(normal_bf16(rng, (8 + 8 * i, sh.dim)))
        case.cache_len.append(c)
        case.frame_pos0.append(c // sh.tokens_per_frame + 5)
        case.t.append([1000.0, 500.0, 250.0][i])
    run = BlockRun(wl, A, case=case, shuffle_pages_seed=5)
    run.run()
    _sync()
    batched = host_bits(run.out).reshape(3, sh.chunk_tokens, sh.dim)
    for i in range(3):
        single = draw_block_case(wl)
        single.block_w, single.time_w = case.block_w, case.time_w
        for f in ("x", "cache_k", "cache_v", "ctx", "cache_len", "frame_pos0", "t"):
            setattr(single, f, [getattr(case, f)[i]])
        r1 = BlockRun(wl, A, case=single)
        r1.run()
        _sync()
        assert np.array_equal(host_bits(r1.out).reshape(sh.chunk_tokens, sh.dim), batched[i]), i
        ref = run.reference(i)
        parity(host_f32(run.out)[i * sh.chunk_tokens:(i + 1) * sh.chunk_tokens], ref["out"],
               f"ragged stream {i}")


def test_block_varlen_max_streams(A):
    """64 streams (the ABI's maximum) of the tiny block in one varlen call:
    caches of 0-2 chunks, different timesteps, text lengths and frame
    positions; stream-indexed work (modulation rows, RoPE positions, page
    slots, text blocks) checked against the oracle on eight streams."""
    wl = WORKLOADS["tiny"]
    sh = wl.shape
    rng = make_rng(61)
    pick = np.random.default_rng(61)
    case = draw_block_case(wl)
    case.x, case.cache_k, case.cache_v, case.ctx = [], [], [], []
    case.cache_len, case.frame_pos0, case.t = [], [], []
    for i in range(64):
        c = int(pick.integers(0, 3)) * sh.chunk_tokens
        case.x.append(normal_bf16(rng, (sh.chunk_tokens, sh.dim)))
        case.cache_k.append(normal_bf16(rng, (c, sh.n_heads, sh.head_dim)))
        case.cache_v.append(normal_bf16(rng, (c, sh.n_heads, sh.head_dim)))
        case.ctx.append(normal_bf16(rng, (int(pick.integers(1, 40)), sh.dim)))
        case.cache_len.append(c)
        case.frame_pos0.append(c // sh.tokens_per_frame + int(pick.integers(0, 9)))
        case.t.append(float(pick.choice([1000.0, 750.0, 500.0, 250.0])))
    run = BlockRun(wl, A, case=case, shuffle_pages_seed=7)
    assert run.B == 64
    run.run()
    _sync()
    for b in (0, 1, 17, 31, 32, 45, 62, 63):
        _check_block(run, b, rows=sample_rows(sh.chunk_tokens, seed=b, n_random=24),
                     tag="64 streams")


def test_stack_equals_repeated_blocks_and_tracks_oracle(A):
    """A 30-layer stack of the tiny block equals 30 single-block calls bit for
    bit, and stays within the parity bar of a 30-layer float64 oracle run."""
    import torch
    wl = WORKLOADS["tiny"]
    sh = wl.shape
    n_layers = 30
    case = draw_block_case(wl)
    rng = make_rng(70)
    layer_w = [draw_block_weights(rng, sh) for _ in range(n_layers)]
    caches_k = [normal_bf16(rng, (case.cache_len[0], sh.n_heads, sh.head_dim)) for _ in range(n_layers)]
    caches_v = [normal_bf16(rng, (case.cache_len[0], sh.n_heads, sh.head_dim)) for _ in range(n_layers)]
    runs = []
    for l in range(n_layers):
        c = draw_block_case(wl)
        c.block_w = layer_w[l]
        c.cache_k, c.cache_v = [caches_k[l]], [caches_v[l]]
        runs.append(BlockRun(wl, A, case=c))
    r0 = runs[0]
    r0.run()      # time modulation and layer-0 text K/V
    for r in runs[1:]:
        A.ardit_ctx_kv(None, r.dims, r.batch, r.ctx, A.block_weights(r.w_dev), r.ctx_k, r.ctx_v,
                       r.ws, r.ws_bytes)
    out = torch.empty_like(r0.x)
    A.ardit_stack_fwd(None, r0.dims, r0.batch, r0.x, [r.pages.kv(A) for r in runs], r0.mod,
                      [r.ctx_k for r in runs], [r.ctx_v for r in runs],
                      [A.block_weights(r.w_dev) for r in runs], out, r0.ws, r0.ws_bytes)
    _sync()
    stack_bits = host_bits(out)
    # same layers one call at a time (the pages see identical writes)
    cur = r0.x
    for l, r in enumerate(runs):
        nxt = torch.empty_like(cur)
        A.ardit_block_fwd_varlen(None, r.dims, r.batch, cur, r.pages.kv(A), r0.mod, r.ctx_k,
                                 r.ctx_v, A.block_weights(r.w_dev), nxt, r0.ws, r0.ws_bytes)
        cur = nxt
    _sync()
    assert np.array_equal(host_bits(cur), stack_bits)
    # float64 oracle through the 30 layers
    m_t = O.time_modulation(case.t[0], case.time_w, sh.dim)
    x = case.x[0].astype(np.float64)
    for l in range(n_layers):
        kc, vc = O.context_kv(runs[l].case.ctx[0], layer_w[l], sh.eps)
        # the residual stream is bf16 between blocks, on both sides
        x = bf16_round(O.block_forward(x, caches_k[l], caches_v[l], case.frame_pos0[0], m_t, kc,
                                       vc, layer_w[l], sh)["out"]).astype(np.float64)
    parity(host_f32(out), x, "30-layer stack", quantum=x, half_ulps=2.0 * np.sqrt(n_layers))


def test_block_192_row_gemm_tiles(A):
    """A 4680-row chunk whose QKV and FFN-up widths (3 * 1152 = 3456) are
    multiples of 128 but not of 256: the GEMMs take 192-row tiles there (25
    row tiles, the last holding 72 rows, and a half tile of columns), and
    128-row tiles for the 1152-wide products; checked against the oracle on
    sampled rows of two streams."""
    import dataclasses
    sh = BlockShape(dim=1152, n_heads=9, head_dim=128, ffn_dim=3456, frames=3, lat_h=30, lat_w=52)
    wl = dataclasses.replace(WORKLOADS["tiny"], shape=sh, cache_chunks=(1, 0),
                             frame_pos0=(3, 0), timesteps=(750, 1000), ctx_len=64)
    run = BlockRun(wl, A, shuffle_pages_seed=11)
    run.run()
    _sync()
    for b in range(2):
        _check_block(run, b, rows=sample_rows(sh.chunk_tokens, seed=20 + b), tag="gemm-192")


@pytest.mark.parametrize("name", ["block13b", "ragged", "large"])
def test_block_full_size_sampled_rows(A, name):
    """Full-size block step (one layer) of the 1.3B-class, ragged 8-stream and
    large ring-buffer workloads, checked on sampled query rows of every
    stream: out, out - x, the appended keys/values and the self-attention
    output o (which the residual would hide in out)."""
    wl = WORKLOADS[name]
    sh = wl.shape
    page_ids = None
    n_pages = None
    if wl.ring_slots:
        page_ids = [ring_page_ids(sh, wl.frame_pos0[0] // sh.frames, wl.cache_chunks[0],
                                  wl.ring_slots)]
        n_pages = wl.ring_slots * sh.frames
        assert page_ids[0] != sorted(page_ids[0])     # the ring has wrapped
    run = BlockRun(wl, A, page_ids=page_ids, n_pages=n_pages,
                   shuffle_pages_seed=None if wl.ring_slots else 9)
    run.run()
    _sync()
    refs = {b: _check_block(run, b, rows=sample_rows(sh.chunk_tokens, seed=b), tag=name)
            for b in range(run.B)}
    # the self-attention output of every stream (every cache length of the
    # ragged batch; through the wrapped ring of the large one)
    _run_self_attention_check(A, run, refs, name)
    streams = sorted({int(np.argmin(run.case.cache_len)), int(np.argmax(run.case.cache_len))})
    if name == "ragged":
        # One stream of the 37440-row batch, run alone: every kernel computes a
        # row (and a query's attention) the same way whatever else is in the
        # launch, so the stream's whole output agrees bit for bit.
        b = streams[0]
        single = copy.copy(run.case)
        for f in ("x", "cache_k", "cache_v", "ctx", "cache_len", "frame_pos0", "t"):
            setattr(single, f, [getattr(run.case, f)[b]])
        r1 = BlockRun(wl, A, case=single)
        r1.run()
        _sync()
        T = sh.chunk_tokens
        assert np.array_equal(host_bits(r1.out), host_bits(run.out)[b * T:(b + 1) * T])


@pytest.mark.parametrize("name", ["block13b", "large"])
def test_stack_teacher_forced_layers(A, name):
    """The full 30-layer 1.3B-class and 40-layer large stacks (weights, caches
    and text drawn on the device): layer-by-layer block calls equal one
    ardit_stack_fwd bit for bit, and layers 0, L/2 and L-1 each match the
    oracle block fed that layer's GPU input (teacher forcing) on sampled
    rows: out, out - x, the appended keys/values and the self-attention
    output through the layer's pages (the large stack's ring has wrapped)."""
    import torch
    from harness import DeviceStack, read_stream_pages
    wl = WORKLOADS[name]
    n_layers = wl.layers
    st = DeviceStack(wl, A, n_layers, seed=15319 + 50 * wl.wid)
    sh = st.shape
    L, D = sh.chunk_tokens, sh.dim
    check = (0, n_layers // 2, n_layers - 1)
    ins, outs = {}, {}
    cur = st.x
    for l in range(n_layers):
        nxt = torch.empty_like(cur)
        A.ardit_block_fwd_varlen(None, st.dims, st.batch, cur, st.kv[l], st.mod, st.ctx_k[l],
                                 st.ctx_v[l], st.w[l], nxt, st.ws, st.ws_bytes)
        if l in check:
            ins[l], outs[l] = cur, nxt
        cur = nxt
    out = torch.empty_like(st.x)
    A.ardit_stack_fwd(None, st.dims, st.batch, st.x, st.kv, st.mod, st.ctx_k, st.ctx_v, st.w,
                      out, st.ws, st.ws_bytes)
    _sync()
    assert np.array_equal(host_bits(out), host_bits(cur)), "stack != layer-by-layer calls"
    tw = st.time_weights_host()
    m_t = O.time_modulation(st.t[0], tw, D)
    for l in check:
        w, ck, cv, ctx = st.host_layer(l)
        x = host_f32(ins[l])
        kc, vc = O.context_kv(ctx, w, sh.eps)
        rows = sample_rows(L, seed=l, n_random=32)
        ref = O.block_forward(x, ck, cv, st.frame_pos0[0], m_t, kc, vc, w, sh, rows=rows)
        tag = f"{name} layer {l}"
        got = host_f32(outs[l])[rows]
        # out is stored bf16: deep in the stack the residual stream has grown
        # (RMS 2.3 at layer 39 of the large stack, elements past 8) and half an
        # ulp of its largest elements is 1.3e-2 of the RMS, so the rounding of
        # the stored output is added to the bar as for every stored tensor
        parity(got, ref["out"], f"{tag} out", quantum=ref["out"])
        parity(got - x[rows], ref["out"] - x[rows], f"{tag} out-x", tol=5e-2, quantum=ref["out"],
               cos_ref=bf16_round(ref["out"]) - x[rows])
        c = st.cache_len[0]
        K, V = read_stream_pages(st.k[l], st.v[l], st.page_ids[0], c + L)
        parity(K[c:].reshape(L, D), ref["k_new"].reshape(L, D), f"{tag} k pages",
               quantum=ref["k_new"])
        parity(V[c:].reshape(L, D), ref["v_new"].reshape(L, D), f"{tag} v pages",
               quantum=ref["v_new"])
        assert np.array_equal(K[:c], ck), f"{tag}: cached keys changed"
        _check_self_attention(A, st.dims, st.batch, st.kv[l], st.k[l], st.v[l], st.page_ids,
                              st.cache_len, L, {0: ref}, st.ws, st.ws_bytes, tag)


# ----------------------------------------------------- block-sparse attention
S = O.sparse_ref


def _sparse_rows(A, dims, batch, q, kv, row_stride):
    """ardit_sparse_select into a fresh [rows][row_stride] int32 buffer."""
    import torch
    n = A.ardit_workspace_size(dims, batch)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    H = dims.n_heads
    rows = H * sum((n + 255) // 256 for n in batch.q_lens)
    blocks = torch.full((rows, row_stride), -7, dtype=torch.int32, device="cuda")
    A.ardit_sparse_select(None, dims, batch, q, kv, blocks, row_stride, ws, n)
    _sync()
    return blocks.cpu().numpy()


def _check_selection(got, qs, ks, rho, H, tag, rel_tol=1e-5):
    """got: [H * n_qtiles, stride] rows of one stream.  Equal to the oracle's
    fp32 selection, except that a tile may trade places with one whose float64
    score is within rel_tol of it (rounding order); -1 padding after n_keep.
    Returns the lists [H, n_qtiles, n_keep]."""
    n_k = (ks.shape[0] + S.K_BLOCK - 1) // S.K_BLOCK
    nk = S.keep_count(n_k, rho)
    nq = (qs.shape[0] + S.Q_BLOCK - 1) // S.Q_BLOCK
    got = got.reshape(H, nq, -1)
    assert (got[:, :, nk:] == -1).all(), f"{tag}: padding"
    lists = got[:, :, :nk]
    ref = S.select_blocks(S.block_scores(qs, ks), nk)
    s64 = S.block_scores(qs, ks, dtype=np.float64)
    n_diff = 0
    for h in range(H):
        for i in range(nq):
            g = lists[h, i]
            assert (np.diff(g) > 0).all() and g[0] >= 0 and g[-1] < n_k, f"{tag}: list {g}"
            if not np.array_equal(g, ref[h, i]):
                n_diff += 1
                sc = s64[h, i]
                tol = rel_tol * np.abs(sc).max()
                dropped = np.setdiff1d(np.arange(n_k), g)
                assert sc[g].min() >= sc[dropped].max() - tol, f"{tag}: wrong tiles h={h} i={i}"
    assert n_diff <= max(1, H * nq // 50), f"{tag}: {n_diff} rows differ from the oracle"
    return lists


@pytest.mark.parametrize("hd", [64, 128])
def test_sparse_select_and_attention_ragged(A, hd):
    """Four streams with rho 0.8, 0 (every tile), 0.6 and 1 (one tile), ragged
    query and key tiles, pages shuffled: the lists match the oracle's selection
    (ascending, -1 padded to the row stride) and the attention over them
    matches the oracle's masked attention on every row."""
    sh = BlockShape(dim=4 * hd, n_heads=4, head_dim=hd, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    q_lens, caches, rho = [600, 256, 300, 70], [1280, 0, 640, 192], [0.8, 0.0, 0.6, 1.0]
    pc, dims, _, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 60)
    batch = A.Batch(q_lens, caches, sparsity=rho)
    H = sh.n_heads
    rows = _sparse_rows(A, dims, batch, q, pc.kv(A), row_stride=9)
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = r0 = 0
    for b, n in enumerate(q_lens):
        nq = (n + 255) // 256
        lists = _check_selection(rows[r0:r0 + H * nq], qs[b], ks[b], rho[b], H, f"stream {b}")
        if rho[b] == 0.0:
            assert (lists == np.arange(lists.shape[-1])).all()
        ref = S.sparse_attention(qs[b], ks[b], vs[b], lists).reshape(n, -1)
        parity(og[off:off + n], ref, f"sparse attn hd={hd} stream {b}", quantum=ref)
        off += n
        r0 += H * nq


@pytest.mark.parametrize("rho", [0.6, 0.9])
def test_sparse_attention_4680x14040(A, rho):
    """4680 queries over 14040 keys, 12 heads of 128, QK-RMSNorm applied: every
    item's list against the oracle's selection, sampled rows of the attention."""
    import torch
    wl = WORKLOADS["attn"]
    sh = wl.shape
    rng = make_rng(wl.wid)
    L, c = sh.chunk_tokens, 2 * sh.chunk_tokens
    H, d, D = sh.n_heads, sh.head_dim, sh.dim
    q = bf16_round(O.rms_norm(rng.standard_normal((L, D), dtype=np.float32), sh.eps))
    k = bf16_round(O.rms_norm(rng.standard_normal((c + L, D), dtype=np.float32), sh.eps))
    v = normal_bf16(rng, (c + L, H, d))
    T = sh.tokens_per_frame
    pc = PagedCache(sh, [list(range((c + L) // T))], (c + L) // T)
    pc.fill_stream(0, k.reshape(-1, H, d), v)
    pc.upload()
    qd = dev_bf16(q)
    o = torch.empty_like(qd)
    dims = A.dims_from_shape(sh)
    batch = A.Batch([L], [c], sparsity=[rho])
    nk = S.keep_count((c + L + 63) // 64, rho)
    rows = _sparse_rows(A, dims, batch, qd, pc.kv(A), row_stride=nk)
    lists = _check_selection(rows, q.reshape(L, H, d), k.reshape(-1, H, d), rho, H, f"rho={rho}")
    _attn(A, dims, batch, qd, pc.kv(A), o)
    _sync()
    sel = sample_rows(L, seed=3)
    ref = S.sparse_attention(q.reshape(L, H, d), k.reshape(-1, H, d), v, lists,
                             rows=sel).reshape(len(sel), D)
    parity(host_f32(o)[sel], ref, f"sparse attn 4680x14040 rho={rho}", quantum=ref)


def test_sparse_block_varlen(A):
    """A ragged batch of four tiny-shape streams at rho 0.6 / 0.9 / 0.7 / 0.8
    through the block call.  The oracle selects from its bf16-rounded q and k;
    the kernels score their own bf16 values, so a stream is compared only when
    no item of it has two tiles at its keep boundary closer than 1% of the
    row's largest score (at least two of the four must qualify)."""
    from workloads.gen import Workload
    wl = Workload(11, "sparse_tiny", WORKLOADS["tiny"].shape, cache_chunks=(2, 4, 0, 6),
                  frame_pos0=(6, 12, 0, 18), ctx_len=32, timesteps=(750, 500, 1000, 250))
    rho = [0.6, 0.9, 0.7, 0.8]
    run = BlockRun(wl, A)
    c = run.case
    import torch
    run.batch = A.Batch([run.shape.chunk_tokens] * 4, c.cache_len, c.frame_pos0,
                        [a.shape[0] for a in c.ctx], sparsity=rho)
    run.ws_bytes = A.ardit_workspace_size(run.dims, run.batch)
    run.ws = torch.empty(run.ws_bytes, dtype=torch.uint8, device="cuda")
    run.run()
    _sync()
    sh = run.shape
    L = sh.chunk_tokens
    out = host_f32(run.out)
    checked = 0
    for b in range(4):
        m_t = O.time_modulation(c.t[b], c.time_w, sh.dim)
        kc, vc = O.context_kv(c.ctx[b], c.block_w, sh.eps)
        ref = O.block_forward(c.x[b], c.cache_k[b], c.cache_v[b], c.frame_pos0[b], m_t, kc, vc,
                              c.block_w, sh, rho=rho[b])
        K = np.concatenate([c.cache_k[b], ref["k_new"]])
        sc = S.block_scores(bf16_round(ref["q"]), bf16_round(K), dtype=np.float64)
        nk = ref["blocks"].shape[-1]
        srt = -np.sort(-sc, axis=-1)
        if nk < sc.shape[-1]:
            margin = srt[..., nk - 1] - srt[..., nk]
            if (margin < 1e-2 * np.abs(sc).max(axis=-1)).any():
                continue
        checked += 1
        parity(out[b * L:(b + 1) * L], ref["out"], f"sparse block out stream {b}")
        parity(out[b * L:(b + 1) * L] - c.x[b], ref["out"] - c.x[b], f"sparse out-x stream {b}",
               tol=5e-2, quantum=ref["out"], cos_ref=bf16_round(ref["out"]) - c.x[b])
    assert checked >= 2, f"only {checked} streams had an unambiguous selection"


def test_sparse_long_cache_more_than_1024_tiles(A):
    """A 66860-key stream (1045 key tiles, past the 1024 the selection keeps in
    registers) next to a short one: the lists of both match the oracle's and
    the attention matches on sampled rows."""
    sh = BlockShape(dim=128, n_heads=2, head_dim=64, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    q_lens, caches, rho = [300, 129], [66560, 128], [0.9, 0.7]
    pc, dims, _, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 61)
    batch = A.Batch(q_lens, caches, sparsity=rho)
    H = sh.n_heads
    rows = _sparse_rows(A, dims, batch, q, pc.kv(A), row_stride=S.keep_count(1045, 0.9))
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = r0 = 0
    for b, n in enumerate(q_lens):
        nq = (n + 255) // 256
        lists = _check_selection(rows[r0:r0 + H * nq], qs[b], ks[b], rho[b], H, f"stream {b}")
        sel = sample_rows(n, seed=b)
        ref = S.sparse_attention(qs[b], ks[b], vs[b], lists, rows=sel).reshape(len(sel), -1)
        parity(og[off:off + n][sel], ref, f"long sparse attn stream {b}", quantum=ref)
        off += n
        r0 += H * nq


# ---------------------------------------------------------- FP8 attention
F8 = O.fp8_ref


def test_mx_quantize_bit_exact(A):
    """E4M3 codes and E8M0 scales of the block quantisation equal the oracle's
    on rows spanning magnitudes 2^-30 .. 2^30, with zero and single-element
    blocks."""
    import torch
    rng = make_rng(70)
    rows, cols = 64, 384
    x = rng.standard_normal((rows, cols)).astype(np.float32)
    x *= np.exp2(rng.integers(-30, 30, size=(rows, 1))).astype(np.float32)
    x[3, 32:64] = 0.0                     # an all-zero block
    x[5, 64:96] = 0.0
    x[5, 70] = -3.0e-3                    # a block with one non-zero element
    x = bf16_round(x)
    xd = dev_bf16(x)
    codes = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    scales = torch.empty((rows, cols // 32), dtype=torch.uint8, device="cuda")
    A.ardit_mx_quantize(None, xd, rows, cols, cols, codes, scales)
    _sync()
    ref_codes, ref_e = F8.mx_quantize(x, axis=1)
    table = np.zeros(256)                  # E4M3 decode (codes 0x7f / 0xff are NaN)
    for code in range(256):
        sign = -1.0 if code & 0x80 else 1.0
        ex, m = (code >> 3) & 0xF, code & 7
        mag = m / 8 * 2.0 ** -6 if ex == 0 else (1 + m / 8) * 2.0 ** (ex - 7)
        table[code] = np.nan if code & 0x7F == 0x7F else sign * mag
    got = table[codes.cpu().numpy()]
    np.testing.assert_array_equal(np.where(got == 0, 0.0, got), np.where(ref_codes == 0, 0.0, ref_codes))
    np.testing.assert_array_equal(scales.cpu().numpy().astype(np.int64), ref_e[:, ::32] + 127)


def _fp8_check(og, qs, ks, vs, tag, mask=None, rows=None):
    """FP8 attention output og ([rows][H d]) against the oracle's FP8 attention
    of the same bf16 inputs: the statistical criterion of harness.fp8_parity
    (error spread of the E4M3 weight rounding, no scale error, cosine), and
    every element within the oracle's worst-case bound.  rows: the query rows
    og holds (the query blocks quantise per row, so a row subset is exact)."""
    q_in = qs if rows is None else qs[rows]
    if mask is not None and rows is not None:
        mask = mask[:, rows]
    o_ref, bound, sig = F8.fp8_attention(q_in, ks, vs, mask=mask, sigma=True)
    n = len(q_in)
    o_ref = o_ref.reshape(n, -1)
    bound = bound.reshape(n, -1)
    print(fp8_parity(og, o_ref, sig.reshape(n, -1), tag))
    err = np.abs(og - o_ref)
    lim = bound + half_ulp(o_ref) + 1e-6
    assert np.all(err <= lim), f"{tag}: max err/bound {float((err / lim).max()):.3f}"
    return float((err / lim).max())


def half_ulp(ref):
    from harness import half_ulp_bf16
    return half_ulp_bf16(ref)


def test_fp8_attention_mixed_batch(A):
    """Four streams, FP8 / bf16 / FP8 / FP8, ragged query and key tiles, pages
    shuffled and NaN-filled outside the streams: FP8 outputs within the
    oracle's weight-quantisation bound of FP8 attention on the same bf16
    inputs, the bf16 stream at the bf16 bar."""
    sh = BlockShape(dim=512, n_heads=4, head_dim=128, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    q_lens, caches, quant = [600, 256, 300, 70], [1280, 0, 640, 192], [1, 0, 1, 1]
    pc, dims, _, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 71)
    batch = A.Batch(q_lens, caches, quant=quant)
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = 0
    worst = 0.0
    for b, n in enumerate(q_lens):
        if quant[b]:
            worst = max(worst, _fp8_check(og[off:off + n].reshape(n, -1), qs[b], ks[b], vs[b],
                                          f"fp8 stream {b}"))
            exact = O.attention(qs[b], ks[b], vs[b]).reshape(n, -1)
            rel = np.sqrt(np.mean((og[off:off + n] - exact) ** 2) / np.mean(exact ** 2))
            assert 1e-3 < rel < 0.1, rel     # quantised, and by a few percent only
        else:
            ref = O.attention(qs[b], ks[b], vs[b]).reshape(n, -1)
            parity(og[off:off + n], ref, f"bf16 stream {b}", quantum=ref)
        off += n
    print(f"fp8 worst err / bound {worst:.3f}")


def test_fp8_block_sparse(A):
    """FP8 together with block-sparse attention (rho 0.8 and 0.6): the kept
    tiles of the lists, FP8 arithmetic on them."""
    sh = BlockShape(dim=512, n_heads=4, head_dim=128, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    q_lens, caches, rho, quant = [600, 300], [1280, 640], [0.8, 0.6], [1, 1]
    pc, dims, _, q, o, qs, ks, vs = _attn_case(A, sh, q_lens, caches, 72)
    batch = A.Batch(q_lens, caches, sparsity=rho, quant=quant)
    H = sh.n_heads
    rows = _sparse_rows(A, dims, batch, q, pc.kv(A), row_stride=16)
    _attn(A, dims, batch, q, pc.kv(A), o)
    _sync()
    og = host_f32(o)
    off = r0 = 0
    for b, n in enumerate(q_lens):
        nq = (n + 255) // 256
        lists = _check_selection(rows[r0:r0 + H * nq], qs[b], ks[b], rho[b], H, f"stream {b}")
        mask = np.stack([S.block_mask(lists[h], n, ks[b].shape[0]) for h in range(H)])
        _fp8_check(og[off:off + n].reshape(n, -1), qs[b], ks[b], vs[b], f"fp8 sparse {b}", mask=mask)
        off += n
        r0 += H * nq


@pytest.mark.parametrize("cache_chunks", [2, 6], ids=["4680x14040", "4680x32760"])
def test_fp8_attention_full_size(A, cache_chunks):
    """The attention workload's shape (4680 queries, 12 heads of 128,
    QK-RMSNorm) in FP8 over 2 cached chunks (14040 keys) and over the
    1.3B-class block's 6 (32760 keys), sampled rows against the FP8 oracle
    with the statistical criterion (which an all-zero, halved or 2%-scaled
    output fails at these lengths, see the CPU pins)."""
    import torch
    wl = WORKLOADS["attn"]
    sh = wl.shape
    rng = make_rng(wl.wid + 10 * cache_chunks)
    L, c = sh.chunk_tokens, cache_chunks * sh.chunk_tokens
    H, d, D = sh.n_heads, sh.head_dim, sh.dim
    q = bf16_round(O.rms_norm(rng.standard_normal((L, D), dtype=np.float32), sh.eps))
    k = bf16_round(O.rms_norm(rng.standard_normal((c + L, D), dtype=np.float32), sh.eps))
    v = normal_bf16(rng, (c + L, H, d))
    T = sh.tokens_per_frame
    pc = PagedCache(sh, [list(range((c + L) // T))], (c + L) // T)
    pc.fill_stream(0, k.reshape(-1, H, d), v)
    pc.upload()
    qd = dev_bf16(q)
    o = torch.empty_like(qd)
    _attn(A, A.dims_from_shape(sh), A.Batch([L], [c], quant=[1]), qd, pc.kv(A), o)
    _sync()
    sel = sample_rows(L, seed=4)
    _fp8_check(host_f32(o)[sel], q.reshape(L, H, d), k.reshape(-1, H, d), v,
               f"fp8 4680x{c + L}", rows=sel)


def _run_self_attention_check_fp8(A, run, refs):
    c = run.case
    _check_self_attention(A, run.dims, run.batch, run.pages.kv(A), run.pages.k, run.pages.v,
                          run.pages.page_ids, c.cache_len, run.shape.chunk_tokens,
                          {b: dict(r, rows=np.arange(run.shape.chunk_tokens)) for b, r in
                           refs.items()}, run.ws, run.ws_bytes, "fp8 block", fp8=(0,))


def test_fp8_block_varlen(A):
    """The 1.3B-class block shape (12 heads of 128) with two streams, FP8 and
    bf16 attention, through the block call: the FP8 stream's output against the
    oracle's block with FP8 attention (the two sides quantise slightly
    different bf16 roundings of q and k, so the bar is the block bar at 3x the
    max-error tolerance), the bf16 stream at the block bar."""
    from workloads.gen import Workload
    sh = BlockShape(dim=1536, n_heads=12, head_dim=128, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)
    wl = Workload(12, "fp8_block", sh, cache_chunks=(2, 1), frame_pos0=(6, 3), ctx_len=32,
                  timesteps=(750, 500))
    run = BlockRun(wl, A)
    c = run.case
    import torch
    run.batch = A.Batch([sh.chunk_tokens] * 2, c.cache_len, c.frame_pos0,
                        [a.shape[0] for a in c.ctx], quant=[1, 0])
    run.ws_bytes = A.ardit_workspace_size(run.dims, run.batch)
    run.ws = torch.empty(run.ws_bytes, dtype=torch.uint8, device="cuda")
    run.run()
    _sync()
    L = sh.chunk_tokens
    out = host_f32(run.out)
    refs = {}
    for b, fp8 in enumerate((True, False)):
        m_t = O.time_modulation(c.t[b], c.time_w, sh.dim)
        kc, vc = O.context_kv(c.ctx[b], c.block_w, sh.eps)
        ref = O.block_forward(c.x[b], c.cache_k[b], c.cache_v[b], c.frame_pos0[b], m_t, kc, vc,
                              c.block_w, sh, fp8=fp8)
        parity(out[b * L:(b + 1) * L], ref["out"], f"{'fp8' if fp8 else 'bf16'} block out {b}",
               tol=6e-2 if fp8 else 2e-2)
        refs[b] = ref
    # the residual hides the attention: its output checked on its own, the FP8
    # stream with the FP8 criterion over the pages the block left
    _run_self_attention_check_fp8(A, run, refs)
