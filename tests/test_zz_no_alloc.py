"""The allocation-free paged attention (ardit_attn_fwd_noalloc) against
ardit_attn_fwd with a caller workspace, through the C ABI, on two calls in a
row: a dense batch whose few work items take the split schedule (its partial
results live in the library's static scratch), then a smaller block-sparse
batch (its selection's means, scores and lists in the same scratch, over what
the first call left there).  Same kernels and schedule on both sides, so the
outputs must agree bit for bit; one stream of each call is also checked
against the float64 oracle at the bar plus half a bf16 ulp."""
import numpy as np
import pytest

import oracle as O
from harness import NAN_BITS, PagedCache, dev_bf16, host_bits, host_f32, parity
from workloads import BlockShape, make_rng, normal_bf16

pytestmark = pytest.mark.gpu

SH = BlockShape(dim=512, n_heads=4, head_dim=128, ffn_dim=1024, frames=3, lat_h=8, lat_w=8)


@pytest.fixture(scope="module")
def A(gpu):
    from paper_2606_15319_amd import ardit
    return ardit


def _case(A, q_lens, caches, seed, rho=None):
    import torch
    rng = make_rng(seed)
    H, d, T = SH.n_heads, SH.head_dim, SH.tokens_per_frame
    kvl = [c + q for c, q in zip(caches, q_lens)]
    frames = [(k + T - 1) // T for k in kvl]
    n_pages = sum(frames) + 2
    perm = np.random.default_rng(seed).permutation(n_pages)
    ids, nxt = [], 0
    for f in frames:
        ids.append([int(p) for p in perm[nxt:nxt + f]])
        nxt += f
    pc = PagedCache(SH, ids, n_pages, fill_bits=NAN_BITS)
    qs, ks, vs = [], [], []
    for b in range(len(q_lens)):
        k = normal_bf16(rng, (kvl[b], H, d))
        v = normal_bf16(rng, (kvl[b], H, d))
        qs.append(normal_bf16(rng, (q_lens[b], H, d)))
        pc.fill_stream(b, k, v)
        ks.append(k)
        vs.append(v)
    pc.upload()
    batch = A.Batch(q_lens, caches, sparsity=rho)
    q = dev_bf16(np.concatenate(qs).reshape(-1, H * d))
    return pc, batch, q, qs, ks, vs


def _both(A, pc, batch, q):
    import torch
    dims = A.dims_from_shape(SH)
    n = A.ardit_workspace_size(dims, batch)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    o_ws = torch.full_like(q, float("nan"))
    o_na = torch.full_like(q, float("nan"))
    A.ardit_attn_fwd(None, dims, batch, q, pc.kv(A), o_ws, ws, n)
    A.ardit_attn_fwd_noalloc(None, dims, batch, q, pc.kv(A), o_na)
    torch.cuda.synchronize()
    return host_bits(o_ws), host_bits(o_na), host_f32(o_na)


def test_noalloc_equals_workspace_call_twice(A):
    # call 1: two dense streams, 12 + 4 items over 12800 / 5120 keys: the
    # items fill few CUs, so the key ranges are split and merged via scratch
    q1, c1 = [600, 150], [12288, 4992]
    pc, batch, q, qs, ks, vs = _case(A, q1, c1, 301)
    ws_bits, na_bits, og = _both(A, pc, batch, q)
    assert np.array_equal(ws_bits, na_bits), "dense: no-alloc output differs"
    ref = O.attention(qs[1], ks[1], vs[1]).reshape(q1[1], -1)
    parity(og[q1[0]:], ref, "no-alloc dense stream 1", quantum=ref)
    # call 2, smaller: one block-sparse stream (rho 0.8) and one dense in the
    # same sparse batch, whose selection reuses the scratch the first call wrote
    q2, c2 = [300, 70], [2560, 448]
    pc, batch, q, qs, ks, vs = _case(A, q2, c2, 302, rho=[0.8, 0.0])
    ws_bits, na_bits, og = _both(A, pc, batch, q)
    assert np.array_equal(ws_bits, na_bits), "sparse: no-alloc output differs"
    ref = O.attention(qs[1], ks[1], vs[1]).reshape(q2[1], -1)
    parity(og[q2[0]:], ref, "no-alloc rho=0 stream 1", quantum=ref)


def test_noalloc_rejections_enqueue_nothing(A):
    """FP8 streams and batches beyond the scratch are refused before any
    launch, leaving the output untouched."""
    import torch
    dims = A.dims_from_shape(SH)
    pc, batch, q, _, _, _ = _case(A, [64], [256], 303)
    o = torch.full_like(q, float("nan"))
    with pytest.raises(A.ArditError) as e:
        A.ardit_attn_fwd_noalloc(None, dims, A.Batch([64], [256], quant=[1]), q, pc.kv(A), o)
    assert e.value.status == -5
    torch.cuda.synchronize()
    assert np.isnan(host_f32(o)).all()
