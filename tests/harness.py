"""Test harness: seeded cases on the device, oracle references, parity metric.

Parity bar (from the target contract): max |gpu - ref| <= 2e-2 * RMS(ref) and
cosine(gpu, ref) >= 0.9995, with ref the float64 oracle on the same bf16
inputs.  The block output is held to exactly that bar.

Intermediate tensors that the library stores in bf16 (attention outputs,
cached keys/values, the branch delta out - x) are compared with the same bar
plus the unavoidable rounding of a bf16 result: half a bf16 ulp of the
reference value, 2^(floor(log2 |ref|) - 8).  Without it the bar cannot be met
by any bf16-output implementation on heavy-tailed tensors: a small attention
test has max |o| / RMS(o) ~ 10, so rounding alone reaches 10 * 2^-9 ~ 2e-2
of the RMS (reproduced exactly by a CPU emulation of the kernel's arithmetic).

The branch delta out - x of a block is ~4% of x, so its comparison is
dominated by the bf16 rounding of `out` itself (a CPU emulation of the
kernels' storage precisions reproduces the GPU's errors exactly and shows the
final rounding alone caps cos(delta) near 0.999).  The delta is therefore
compared, for its cosine, with the delta of the bf16-rounded reference (a
wrong branch then shows up as extra rounding flips), and for its max with
5e-2 * RMS(delta) + half an ulp of out: the 2e-2 of the output bar plus the
bf16 storage of the FFN input and hidden activations, measured at ~1.7e-2 of
RMS(delta) by the same emulation.

A stack of L blocks carries a bf16 residual between blocks on both sides; a
rounding decision that differs once persists, so its max bound grows by
sqrt(L) ulps (a random walk of single-ulp flips) while the cosine keeps the
0.9995 bar.
"""
from __future__ import annotations

import numpy as np

import oracle as O
from workloads import bf16_bits, bits_to_f32
from workloads.gen import draw_block_case, ring_page_ids  # noqa: F401

TOL = 2e-2
COS_MIN = 0.9995
NAN_BITS = 0x7FC0


# ----------------------------------------------------------------- device io
def dev_bf16(a, device="cuda"):
    import torch
    bits = bf16_bits(np.asarray(a, dtype=np.float32))
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(device)


def dev_f32(a, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def dev_i32(a, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)


def host_f32(t) -> np.ndarray:
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.float().cpu().numpy()


def host_bits(t) -> np.ndarray:
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def upload_block_weights(w: dict, device="cuda"):
    out = {}
    for k, v in w.items():
        out[k] = dev_f32(v, device) if k == "mod_table" else dev_bf16(v, device)
    return out


# ------------------------------------------------------------------- metric
def half_ulp_bf16(ref):
    """Half a bf16 ulp at each |ref| (0 where ref == 0)."""
    r = np.abs(np.asarray(ref, np.float64))
    _, ex = np.frexp(r)                 # r = m 2^ex, m in [0.5, 1)
    return np.where(r > 0, np.ldexp(1.0, ex - 9), 0.0)


def parity(gpu, ref, name, tol=TOL, cos_min=COS_MIN, quantum=None, half_ulps=1.0,
           cos_ref=None):
    """Assert the parity bar.  quantum: optional array whose bf16 half-ulps
    (times half_ulps) are added to the max-abs bound (the reference of a
    bf16-stored tensor); cos_ref: optional reference for the cosine only."""
    g = np.asarray(gpu, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    assert np.isfinite(g).all(), f"{name}: non-finite GPU values"
    rms = float(np.sqrt(np.mean(r * r)))
    err = np.abs(g - r)
    bound = tol * rms
    if quantum is not None:
        bound = bound + half_ulps * half_ulp_bf16(np.asarray(quantum, np.float64).ravel())
    c = r if cos_ref is None else np.asarray(cos_ref, dtype=np.float64).ravel()
    cos = float(np.dot(g, c) / (np.linalg.norm(g) * np.linalg.norm(c) + 1e-300))
    worst = float(np.max(err - bound)) if err.size else 0.0
    msg = (f"{name}: max|d|={float(err.max()) if err.size else 0:.3e} rms(ref)={rms:.3e} "
           f"ratio={float(err.max()) / rms if rms else 0:.3e} cos={cos:.6f}")
    assert worst <= 0.0 and cos >= cos_min, msg
    return msg


# -------------------------------------------------------------------- pages
class PagedCache:
    """A device page pool for one layer plus the host view of its contents."""

    def __init__(self, shape, page_ids_per_stream, n_pages, device="cuda", fill_bits=NAN_BITS):
        import torch
        T = shape.tokens_per_frame
        H, d = shape.n_heads, shape.head_dim
        self.T, self.H, self.d = T, H, d
        self.n_pages = n_pages
        self.page_ids = [list(p) for p in page_ids_per_stream]
        self.max_frames = max(len(p) for p in self.page_ids)
        self.k_host = np.full((n_pages, H, T, d), fill_bits, dtype=np.uint16)
        self.v_host = np.full((n_pages, H, d, T), fill_bits, dtype=np.uint16)
        table = np.zeros((len(self.page_ids), self.max_frames), dtype=np.int32)
        for b, p in enumerate(self.page_ids):
            table[b, :len(p)] = p
        self.table_host = table
        self.device = device
        self.table = dev_i32(table, device)
        self.k = None
        self.v = None

    def fill_stream(self, b, k_tokens, v_tokens):
        from paper_2606_15319_amd.layout import pack_pages
        pack_pages(bf16_bits(k_tokens), bf16_bits(v_tokens), self.page_ids[b], self.k_host,
                   self.v_host)

    def upload(self):
        import torch
        self.k = torch.from_numpy(self.k_host.view(np.int16)).view(torch.bfloat16).to(self.device)
        self.v = torch.from_numpy(self.v_host.view(np.int16)).view(torch.bfloat16).to(self.device)

    def kv(self, A):
        return A.kv_paged(self.k, self.v, self.table, self.n_pages, self.max_frames)

    def read_stream(self, b, n_tokens):
        """Logical [n, H, d] bf16 bits of stream b read back from the device."""
        from paper_2606_15319_amd.layout import unpack_pages
        k = host_bits(self.k).reshape(self.k_host.shape)
        v = host_bits(self.v).reshape(self.v_host.shape)
        return unpack_pages(k, v, self.page_ids[b], n_tokens)

    def device_bits(self):
        return (host_bits(self.k).reshape(self.k_host.shape),
                host_bits(self.v).reshape(self.v_host.shape))


def frames_needed(shape, cache_len):
    return cache_len // shape.tokens_per_frame + shape.frames


# -------------------------------------------------------------- block runs
class BlockRun:
    """Inputs of one block step for a batch of streams, on host and device."""

    def __init__(self, wl, A, device="cuda", page_ids=None, n_pages=None, ctx_lens=None,
                 case=None, shuffle_pages_seed=None):
        self.wl = wl
        self.A = A
        sh = wl.shape
        self.shape = sh
        self.case = case if case is not None else draw_block_case(wl, ctx_lens=ctx_lens)
        c = self.case
        B = len(c.x)
        self.B = B
        if page_ids is None:
            page_ids, nxt = [], 0
            for b in range(B):
                nf = frames_needed(sh, c.cache_len[b])
                page_ids.append(list(range(nxt, nxt + nf)))
                nxt += nf
            n_pages = nxt
            if shuffle_pages_seed is not None:
                perm = np.random.default_rng(shuffle_pages_seed).permutation(n_pages)
                page_ids = [[int(perm[p]) for p in ids] for ids in page_ids]
        self.pages = PagedCache(sh, page_ids, n_pages, device)
        for b in range(B):
            if c.cache_len[b]:
                self.pages.fill_stream(b, c.cache_k[b], c.cache_v[b])
        self.pages.upload()
        self.dims = A.dims_from_shape(sh)
        self.batch = A.Batch([sh.chunk_tokens] * B, c.cache_len, c.frame_pos0,
                             [a.shape[0] for a in c.ctx])
        self.x = dev_bf16(np.concatenate(c.x), device)
        self.ctx = dev_bf16(np.concatenate(c.ctx), device)
        self.w_dev = upload_block_weights(c.block_w, device)
        self.tw_dev = {k: dev_bf16(v, device) for k, v in c.time_w.items()}
        import torch
        self.ws_bytes = A.ardit_workspace_size(self.dims, self.batch)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.mod = torch.empty((B, 6, sh.dim), dtype=torch.float32, device=device)
        nctx = sum(a.shape[0] for a in c.ctx)
        self.ctx_k = torch.empty((nctx * sh.dim,), dtype=torch.bfloat16, device=device)
        self.ctx_v = torch.empty((nctx * sh.dim,), dtype=torch.bfloat16, device=device)
        self.out = torch.empty((B * sh.chunk_tokens, sh.dim), dtype=torch.bfloat16, device=device)

    def run(self, stream=None):
        A = self.A
        wts = A.block_weights(self.w_dev)
        A.ardit_time_mod(stream, self.dims, self.case.t, A.time_weights(self.tw_dev), self.mod,
                         self.ws, self.ws_bytes)
        A.ardit_ctx_kv(stream, self.dims, self.batch, self.ctx, wts, self.ctx_k, self.ctx_v,
                       self.ws, self.ws_bytes)
        A.ardit_block_fwd_varlen(stream, self.dims, self.batch, self.x, self.pages.kv(A), self.mod,
                                 self.ctx_k, self.ctx_v, wts, self.out, self.ws, self.ws_bytes)

    def reference(self, b, rows=None):
        """Float64 oracle of stream b (optionally only some query rows)."""
        c, sh = self.case, self.shape
        m_t = O.time_modulation(c.t[b], c.time_w, sh.dim)
        kc, vc = O.context_kv(c.ctx[b], c.block_w, sh.eps)
        return O.block_forward(c.x[b], c.cache_k[b], c.cache_v[b], c.frame_pos0[b], m_t, kc, vc,
                               c.block_w, sh, rows=rows)


def sample_rows(L, seed=0, n_random=48):
    """First rows, a random spread, and the ragged last tile of a chunk."""
    rng = np.random.default_rng(seed)
    last = (L // 128) * 128
    rows = set(range(0, min(L, 40))) | set(range(max(0, last - 8), L))
    rows |= set(int(r) for r in rng.choice(L, size=min(L, n_random), replace=False))
    return np.array(sorted(rows))
