"""Benchmark: ms per chunk-denoise-step per block on one MI355X.

Default workload: the large AR-DiT block (hidden 5120, 40 heads x 128, FFN
13824), one stream at chunk index 11 (frames 33..35, 3 latent frames of
30 x 52 = 4680 tokens) over a rolling window of the 7 previous chunks (32760
cached tokens) held in a ring of 8 chunk slots that has wrapped (physical
pages not in logical order), 512 text tokens, 40 layers, t = 1000.  One bench
step is one denoising step of the chunk: the time modulation for t followed
by all 40 blocks through ardit_stack_fwd; value = ms per step / 40.  Inputs
are synthetic (seeded normal draws on the device), resident in HBM before
timing starts.

--workload block13b runs the 1.3B-class block instead (hidden 1536, 12 x 128,
FFN 8960, 4680 tokens over a 28080-token cache, 30 layers, t cycling
1000/750/500/250); --workload ragged the 8-stream batch of that block (caches
of 0..7 chunks, per-stream t, 4 layers by default).

The JSON line also carries the roofline of the dominant kernel (paged
self-attention: 4 L_q L_k D flops per launch, timed with HIP events around
each launch on the stream it runs on) and the float64 CPU oracle timed on
one block step of layer 0 (cpu_baseline; on the large block a bounded sample
of it, see cpu_baseline).  roofline.traffic is the HBM bytes per attention
launch measured with rocprofv3 counters (FETCH_SIZE and WRITE_SIZE,
FETCH_SIZE scaled by what it reads for a plain copy of known size, see
--copy-probe), taken from the workload's profile summary under profiles/ when
that summary was made from the current attention sources, else null.

--sparsity RHO runs the same workload with block-sparse self-attention at
sparsity RHO (the fidelity knob; every 256-query tile keeps
ceil((1 - RHO) n) of its n key tiles of 64): the step then also runs the
block selection, and the roofline counts the attention kernel's kept keys,
4 L_q (n_keep 64) D flops per launch.

--quant fp8 runs the self-attention of every stream in FP8 (the quantisation
knob): the timed kernel is the FP8 attention, priced against the 5.0 PFLOP/s
dense fp8 peak; its quantisation pre-pass is in `value` only.

--chunk times whole-chunk generation instead (1.3B-class stack): one bench
step is one ardit_chunk_generate of the same chunk (4 denoising steps at
1000/750/500/250 with the sampler update between them, then the commit pass
at t = 0), the cache being chunks 0..5 of a window of W = 7 chunks (no sink)
while chunk 6 is generated; value = ms per chunk.

--micro only runs the measurement kernels (include/ardit_micro.h): MFMA
throughput in bf16 and fp8 with register operands, and a 1 GiB device copy;
the default run also measures them (a few ms) and reports each roofline
against the measured peak besides the published one.

--workload ragged --cold times every elementwise launch of one step of the
8-stream batch twice: after a 512 MiB buffer is read (neither L2 nor the
256 MB last-level cache holds the operands, and neither holds dirty lines) and
back to back, per kernel."""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0       # MI355X dense fp8 MFMA
TIMESTEPS = (1000.0, 750.0, 500.0, 250.0)
DEFAULT_LAYERS = {"large": 40, "block13b": 30, "ragged": 4}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--layers", type=int, default=None,
                   help="layers of the stack (default: 40 large, 30 block13b, 4 ragged)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--sparsity", type=float, default=0.0, metavar="RHO",
                   help="attention sparsity rho of every stream (0: dense)")
    p.add_argument("--quant", choices=("bf16", "fp8"), default="bf16",
                   help="self-attention precision of every stream (the quantisation knob)")
    p.add_argument("--workload", choices=("large", "block13b", "ragged"), default="large",
                   help="large: the 5120-wide block over a wrapped ring of 7 cached chunks "
                        "(default); block13b: the 1.3B-class block; ragged: the 8-stream "
                        "batch of 1.3B-class blocks (elementwise kernels at 37440 rows)")
    p.add_argument("--chunk", action="store_true",
                   help="time whole-chunk generation (4 steps + commit) of the 1.3B-class stack")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only copy MIB MiB on the device 5 times with one kernel (counter calibration)")
    p.add_argument("--micro", action="store_true",
                   help="only run the measurement kernels: MFMA throughput (bf16, fp8) and "
                        "the HBM copy, and print one line with the measured peaks")
    p.add_argument("--sp2", action="store_true",
                   help="time one GPU's share of Ulysses SP2: every query of the chunk for half "
                        "the heads over the full keys (paged self-attention alone)")
    p.add_argument("--cold", action="store_true",
                   help="with --workload ragged: time every elementwise launch of one step "
                        "after a 512 MiB write (cold caches) and warm, per kernel")
    return p.parse_args()


def traffic_summary(workload):
    return os.path.join(ROOT, "profiles", f"attn_paged_{workload}_hbm_traffic.md")


ATTN_SOURCES = ("paper_2606_15319_amd/csrc/k_attn.hip", "paper_2606_15319_amd/csrc/launch.h",
                "paper_2606_15319_amd/csrc/common.h")


def attn_source_hash():
    import hashlib
    h = hashlib.sha256()
    for rel in ATTN_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per attention launch from the workload's counter summary, or
    None when the summary is missing or was made from other attention sources."""
    try:
        fields = {}
        with open(traffic_summary(workload)) as f:
            for line in f:
                if ":" in line and line.startswith("- "):
                    k, v = line[2:].split(":", 1)
                    fields[k.strip()] = v.strip().strip("`")
        if fields.get("attention sources sha256") != attn_source_hash():
            return None
        return int(fields["HBM bytes per launch"])
    except (OSError, KeyError, ValueError):
        return None


def copy_probe(mib):
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        torch.mul(src, 1.0, out=dst)   # one elementwise kernel: reads and writes mib MiB
    torch.cuda.synchronize()
    log(f"copied {mib} MiB 5 times ({mib * (1 << 20)} bytes read and written per copy)")


def measured_peaks(A, reps=3):
    """Measured MFMA throughput (bf16, fp8; TFLOP/s) and HBM copy bandwidth
    (TB/s, bytes read + written) with the library's measurement kernels, best
    of `reps` launches each."""
    import torch
    wgs = 256 * 2 * 4        # 2 workgroups of 4 waves per CU, four rounds
    sink = torch.empty(wgs * 256, dtype=torch.float32, device="cuda")
    out = {}
    for name, dtype, iters in (("mfma_bf16", 0, 2000), ("mfma_fp8", 1, 2000)):
        best = 0.0
        for r in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            flops = A.ardit_micro_mfma(None, dtype, wgs, iters, sink)
            e1.record()
            torch.cuda.synchronize()
            if r:
                best = max(best, flops / (e0.elapsed_time(e1) * 1e-3) / 1e12)
        out[name + "_tflops"] = round(best, 1)
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    A.ardit_micro_fill(None, src, nbytes, 0x3f800000)
    best = 0.0
    for r in range(reps + 2):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        A.ardit_micro_copy(None, src, dst, nbytes)
        e1.record()
        torch.cuda.synchronize()
        if r:
            best = max(best, 2 * nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e12)
    out["copy_tbps"] = round(best, 3)
    sink = torch.empty(32 << 10, dtype=torch.uint8, device="cuda")
    best = 0.0
    for r in range(reps + 2):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        A.ardit_micro_read(None, src, nbytes, sink, sink.numel())
        e1.record()
        torch.cuda.synchronize()
        if r:
            best = max(best, nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e12)
    out["read_tbps"] = round(best, 3)
    del src, dst
    torch.cuda.synchronize()
    return out


def micro_main():
    import torch
    from paper_2606_15319_amd import ardit as A
    torch.cuda.set_device(0)
    m = measured_peaks(A, reps=5)
    m.update({"probe": "measurement kernels",
              "note": "MFMA: 2048 workgroups x 4 waves, 2000 iterations of independent register "
                      "chains (bf16 8 x v_mfma_f32_16x16x32_bf16, fp8 4 x "
                      "v_mfma_scale_f32_32x32x64_f8f6f4); copy: 1 GiB read + 1 GiB written, "
                      "read: 1 GiB read, 16-byte accesses four in flight per thread; best of 5",
              "published": {"mfma_bf16_tflops": PEAK_BF16_TFLOPS, "mfma_fp8_tflops": PEAK_FP8_TFLOPS,
                            "hbm_tbps": 8.0}})
    print(json.dumps(m), flush=True)


def sp2_share_shape(sh):
    """The block shape one GPU sees under Ulysses SP2 (Appendix C): after the
    all-to-all it holds every token of the chunk for half the heads, and the
    head-partitioned pages hold those heads only."""
    from workloads import BlockShape
    hs = sh.n_heads // 2
    return BlockShape(dim=hs * sh.head_dim, n_heads=hs, head_dim=sh.head_dim, ffn_dim=sh.ffn_dim,
                      frames=sh.frames, lat_h=sh.lat_h, lat_w=sh.lat_w, eps=sh.eps,
                      theta=sh.theta, time_freq_dim=sh.time_freq_dim)


def sp2_main(args):
    """One GPU's share of Ulysses SP2: 4680 queries of half the heads over the
    stream's full key length through its (head-partitioned) pages; the paged
    self-attention launch timed alone with the library's events."""
    import torch
    from paper_2606_15319_amd import ardit as A
    from workloads import WORKLOADS, stream_page_ids
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = WORKLOADS[args.workload]
    sh = sp2_share_shape(wl.shape)
    H, d, T, L = sh.n_heads, sh.head_dim, sh.tokens_per_frame, sh.chunk_tokens
    cache = wl.cache_chunks[0] * L
    ids, n_pages = stream_page_ids(wl)
    ids = ids[:1]
    g = torch.Generator(device=dev)
    g.manual_seed(15319 + wl.wid)
    kp = torch.randn((n_pages, H, T, d), generator=g, device=dev).to(torch.bfloat16)
    vp = torch.randn((n_pages, H, d, T), generator=g, device=dev).to(torch.bfloat16)
    q = torch.randn((L, H * d), generator=g, device=dev).to(torch.bfloat16)
    o = torch.empty_like(q)
    table = torch.tensor([ids[0]], dtype=torch.int32, device=dev)
    kv = A.kv_paged(kp, vp, table, n_pages, len(ids[0]))
    dims = A.dims_from_shape(sh)
    batch = A.Batch([L], [cache])
    nws = A.ardit_workspace_size(dims, batch)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    for _ in range(max(args.warmup, 1)):
        A.ardit_attn_fwd(None, dims, batch, q, kv, o, ws, nws)
    torch.cuda.synchronize()
    A.ardit_timing_collect()
    A.ardit_timing_enable(True)
    for _ in range(args.steps):
        A.ardit_attn_fwd(None, dims, batch, q, kv, o, ws, nws)
    torch.cuda.synchronize()
    A.ardit_timing_enable(False)
    n, ms = A.ardit_timing_collect()
    avg = ms / max(n, 1)
    L_k = cache + L
    flops = 4.0 * L * L_k * H * d
    items = H * ((L + 255) // 256)
    meas = measured_peaks(A)
    tf = flops / (avg * 1e-3) / 1e12
    print(json.dumps({
        "probe": "one GPU's share of Ulysses SP2",
        "workload": f"{wl.name}: {H} of {wl.shape.n_heads} heads of {d}, {L} queries over {L_k} "
                    f"keys through the stream's pages", "items": items,
        "split_schedule": items * 4 < 3 * 256,
        "ms_per_launch": round(avg, 4), "launches": n, "gflop": round(flops / 1e9, 1),
        "tflops": round(tf, 1), "frac": round(tf / PEAK_BF16_TFLOPS, 4),
        "frac_of_measured": round(tf / meas["mfma_bf16_tflops"], 4)}), flush=True)


# bytes each elementwise launch of a block moves per token row and hidden
# unit: inputs read once, outputs written once (bf16 2 bytes, fp32 4)
ELEMENTWISE_BYTES_PER_ND = {"adaln_norm": 4, "qk_norm_rope / kv append": 12, "cross pre-norm": 6,
                            "cross q-norm": 4, "adaln_norm 2": 6}


def cold_elementwise(A, model, sh, n_rows):
    """Every elementwise launch of one step, cold (a 512 MiB read before each)
    and warm (back to back), grouped by kernel: median ms and TB/s."""
    import statistics
    import torch
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    res = {}
    for mode in ("cold", "warm"):
        A.ardit_timing_flush(flush if mode == "cold" else None, flush.numel() if mode == "cold" else 0)
        A.ardit_timing_enable(1 << A.TIME_ELEMENTWISE)
        model.step(0)
        torch.cuda.synchronize()
        A.ardit_timing_enable(False)
        A.ardit_timing_flush(None, 0)
        recs = A.ardit_timing_records(A.TIME_ELEMENTWISE)
        by = {}
        for name, ms in recs:
            by.setdefault(name, []).append(ms)
        for name, v in by.items():
            ms = statistics.median(v)
            nbytes = ELEMENTWISE_BYTES_PER_ND[name] * n_rows * sh.dim
            res.setdefault(name, {"bytes": nbytes, "launches": len(v)})
            res[name][mode + "_ms"] = round(ms, 4)
            res[name][mode + "_TBps"] = round(nbytes / (ms * 1e-3) / 1e12, 3)
    for r in res.values():
        r["cold_frac_of_8TBps"] = round(r["cold_TBps"] / 8.0, 3)
    return res


class Model:
    """Weights, pages and text K/V of every layer for a batch of streams (one
    chunk each, stream b over cache_lens[b] cached tokens in pages page_ids[b],
    logical order), drawn on the device."""

    def __init__(self, A, wl, n_layers, dev, rho=0.0, timesteps=None, fp8=False):
        import torch
        from workloads import stream_page_ids
        sh = wl.shape
        self.A, self.sh, self.n_layers = A, sh, n_layers
        D, H, d = sh.dim, sh.n_heads, sh.head_dim
        T = sh.tokens_per_frame
        cache_lens = [c * sh.chunk_tokens for c in wl.cache_chunks]
        B = len(cache_lens)
        self.B = B
        self.cache_lens, self.ctx_len = list(cache_lens), wl.ctx_len
        self.cache_len = cache_lens[0]
        self.frame_pos0 = list(wl.frame_pos0)
        page_ids, n_pages = stream_page_ids(wl)
        self.page_ids, self.n_pages = page_ids, n_pages
        max_frames = max(len(p) for p in page_ids)
        self.dims = A.dims_from_shape(sh)
        self.rho = rho
        self.timesteps = timesteps
        self.fp8 = fp8
        self.batch = A.Batch([sh.chunk_tokens] * B, cache_lens, self.frame_pos0,
                             [wl.ctx_len] * B, sparsity=[rho] * B, quant=[1 if fp8 else 0] * B)
        self.ws_bytes = A.ardit_workspace_size(self.dims, self.batch)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        from workloads.gen import block_weight_shapes, GAIN_NAMES
        shapes = block_weight_shapes(sh)
        self.w, self.kv, self.ctx_k, self.ctx_v, self.keep = [], [], [], [], []
        table = torch.zeros((B, max_frames), dtype=torch.int32)
        for b, ids in enumerate(page_ids):
            table[b, :len(ids)] = torch.tensor(ids, dtype=torch.int32)
        self.table = table.to(dev)
        ctx_len = wl.ctx_len
        for layer in range(n_layers):
            g = torch.Generator(device=dev)
            g.manual_seed(15319 + wl.wid + 1000 * layer)
            wd = {}
            for name, shp in shapes.items():
                t = torch.randn(shp, generator=g, device=dev, dtype=torch.float32) * 0.02
                if name in GAIN_NAMES:
                    t += 1.0
                wd[name] = t if name == "mod_table" else t.to(torch.bfloat16)
                del t
            kp = torch.randn((n_pages, H, T, d), generator=g, device=dev).to(torch.bfloat16)
            vp = torch.randn((n_pages, H, d, T), generator=g, device=dev).to(torch.bfloat16)
            ctx = torch.randn((B * ctx_len, D), generator=g, device=dev).to(torch.bfloat16)
            ck = torch.empty(B * ctx_len * D, dtype=torch.bfloat16, device=dev)
            cv = torch.empty_like(ck)
            w = A.block_weights(wd)
            A.ardit_ctx_kv(None, self.dims, self.batch, ctx, w, ck, cv, self.ws, self.ws_bytes)
            self.w.append(w)
            self.kv.append(A.kv_paged(kp, vp, self.table, n_pages, max_frames))
            self.ctx_k.append(ck)
            self.ctx_v.append(cv)
            self.keep.append((wd, kp, vp, ctx))
        g = torch.Generator(device=dev)
        g.manual_seed(15319 + wl.wid)
        tshapes = {"w_t1": (D, 256), "b_t1": (D,), "w_t2": (D, D), "b_t2": (D,),
                   "w_m": (6 * D, D), "b_m": (6 * D,)}
        self.tw_dev = {k: (torch.randn(s, generator=g, device=dev) * 0.02).to(torch.bfloat16)
                       for k, s in tshapes.items()}
        self.tw = A.time_weights(self.tw_dev)
        self.step_ts = TIMESTEPS if wl.name == "block13b" else (float(wl.timesteps[0]),)
        self.xs = [torch.randn((B * sh.chunk_tokens, D), generator=g, device=dev).to(torch.bfloat16)
                   for _ in self.step_ts]
        self.mod = torch.empty((B, 6, D), dtype=torch.float32, device=dev)
        self.out = torch.empty_like(self.xs[0])

    def setup_chunk(self, timesteps, window):
        """Whole-chunk generation of chunk c = cache / L_q of stream 0 under a
        window of `window` chunks: its page table is the one set up above."""
        import torch
        A, sh = self.A, self.sh
        c = self.cache_len // sh.chunk_tokens
        ids, cached = A.ardit_window_pages(c, 0, window, sh.frames)
        assert self.B == 1 and cached * sh.tokens_per_frame == self.cache_len
        assert ids == self.table[0].tolist()[:len(ids)], "window pages differ from the pool layout"
        self.gen_ts = list(timesteps)
        g = torch.Generator(device=self.xs[0].device)
        g.manual_seed(15319 + 6)
        self.noise = torch.randn((len(timesteps) - 1,) + tuple(self.xs[0].shape), generator=g,
                                 device=self.xs[0].device).to(torch.bfloat16)
        self.x0 = torch.empty_like(self.xs[0])

    def generate(self):
        A = self.A
        A.ardit_chunk_generate(None, self.dims, self.batch, [len(self.gen_ts)], [self.gen_ts],
                               self.xs[0], self.noise, self.kv, self.tw, self.ctx_k, self.ctx_v,
                               self.w, self.x0, self.ws, self.ws_bytes)

    def step(self, k):
        A = self.A
        ts = self.timesteps or [self.step_ts[k % len(self.step_ts)]] * self.B
        A.ardit_time_mod(None, self.dims, ts, self.tw, self.mod, self.ws, self.ws_bytes)
        A.ardit_stack_fwd(None, self.dims, self.batch, self.xs[k % len(self.xs)], self.kv,
                          self.mod, self.ctx_k, self.ctx_v, self.w, self.out, self.ws,
                          self.ws_bytes)


def cpu_baseline(model, sample_every=1):
    """The float64 oracle on one block step (layer 0, the first timestep) of
    the same workload, on the host cores, with the layer's own inputs copied
    back.  sample_every > 1 bounds the CPU time: the oracle always computes the
    keys and values of the whole chunk, then the rest of the block only for the
    rows it is asked for, so it is timed twice -- on query row 0 alone (t1) and
    on every sample_every-th row (n rows, tn) -- and the full step is
    extrapolated linearly in the rows, t1 + (tn - t1) (L_q - 1) / (n - 1)."""
    import numpy as np
    import torch

    import oracle as O
    from workloads import bits_to_f32

    def host(t):
        if t.dtype == torch.bfloat16:
            return bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
        return t.float().cpu().numpy()

    sh = model.sh
    wd, kp, vp, ctx = model.keep[0]
    w = {k: host(v) for k, v in wd.items()}
    tw = {k: host(v) for k, v in model.tw_dev.items()}
    H, d, T, Lq = sh.n_heads, sh.head_dim, sh.tokens_per_frame, sh.chunk_tokens
    nf = model.cache_len // T
    pages = torch.tensor(model.page_ids[0][:nf], dtype=torch.long, device=kp.device)
    ck = np.transpose(host(kp.index_select(0, pages)), (0, 2, 1, 3)).reshape(-1, H, d)
    cv = np.transpose(host(vp.index_select(0, pages)), (0, 3, 1, 2)).reshape(-1, H, d)
    x = host(model.xs[0])[:Lq]
    ctxh = host(ctx)[:model.ctx_len]
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    m_t = O.time_modulation(model.step_ts[0], tw, sh.dim)
    kc, vc = O.context_kv(ctxh, w, sh.eps)
    t_ctx = time.perf_counter()

    def run(rows):
        a = time.perf_counter()
        O.block_forward(x, ck, cv, model.frame_pos0[0], m_t, kc, vc, w, sh, rows=rows,
                        rho=model.rho, fp8=model.fp8)
        return time.perf_counter() - a

    what = (f"one block step (layer 0, t={model.step_ts[0]:g}) of the same workload: "
            f"{Lq} queries over {model.cache_len + Lq} keys"
            f"{' at sparsity %g' % model.rho if model.rho else ''}"
            f"{' with FP8 attention' if model.fp8 else ''}, float64 numpy; text K/V and time "
            f"modulation ({(t_ctx - t0) * 1e3:.0f} ms) excluded as on the GPU path")
    if sample_every <= 1:
        ms = run(None) * 1e3
        sample = "measured: " + what
    else:
        rows = np.arange(0, Lq, sample_every)
        t1 = run(np.array([0]))
        tn = run(rows)
        ms = (t1 + (tn - t1) * (Lq - 1) / (len(rows) - 1)) * 1e3
        sample = (f"extrapolated from a sample of {what}: the oracle timed on query row 0 "
                  f"({t1 * 1e3:.0f} ms) and on every {sample_every}th row ({len(rows)} rows, "
                  f"{tn * 1e3:.0f} ms; keys and values of the whole chunk in both), linear in "
                  f"the rows to all {Lq}")
    return {"value": round(ms, 1), "unit": "ms per chunk-denoise-step per block",
            "cores": int(threads), "kind": "oracle", "sample": sample}


def kernel_breakdown(A, model, args, sh, cache_lens):
    """One more step, outside the timed region, with events around every GEMM
    and elementwise launch: their rates against the MFMA and HBM peaks.
    GEMM work per block 2 N D (6 D + 2 F) flops (QKV, O, cross-Q, cross-O,
    FFN up and down); elementwise bytes per block 32 N D (each input read once,
    each output written once, bf16 2 bytes and fp32 4: adaLN from bf16 4ND,
    QK-norm/RoPE/key append 8ND, value append 4ND, cross pre-norm from fp32
    6ND, cross q-norm 4ND, adaLN from fp32 6ND)."""
    import torch
    A.ardit_timing_enable((1 << A.TIME_GEMM) | (1 << A.TIME_ELEMENTWISE))
    model.step(args.steps)
    torch.cuda.synchronize()
    A.ardit_timing_enable(False)
    ng, gms = A.ardit_timing_collect_kind(A.TIME_GEMM)
    ne, ems = A.ardit_timing_collect_kind(A.TIME_ELEMENTWISE)
    N, D, F = sh.chunk_tokens * len(cache_lens), sh.dim, sh.ffn_dim
    blocks = args.layers
    gflop = 2.0 * N * D * (6 * D + 2 * F) * blocks / 1e9
    ebytes = 32.0 * N * D * blocks
    g_tf = gflop / (gms * 1e-3) / 1e3
    e_tb = ebytes / (ems * 1e-3) / 1e12
    log(f"GEMMs {gms / blocks:.3f} ms/block ({g_tf:.0f} TFLOP/s over {ng} launches), "
        f"elementwise {ems / blocks:.3f} ms/block ({e_tb:.2f} TB/s over {ne} launches)")
    return {"gemm": {"ms_per_block": round(gms / blocks, 4), "achieved": round(g_tf, 1),
                     "unit": "TFLOP/s", "peak": PEAK_BF16_TFLOPS,
                     "frac": round(g_tf / PEAK_BF16_TFLOPS, 4), "launches": ng},
            "elementwise": {"ms_per_block": round(ems / blocks, 4), "achieved": round(e_tb, 3),
                            "unit": "TB/s", "peak": 8.0, "frac": round(e_tb / 8.0, 4),
                            "launches": ne},
            "note": "one extra step with events around each GEMM and elementwise launch, "
                    "outside the timed region"}


def workload_name(wl, args):
    sh = wl.shape
    if args.chunk:
        return ("whole-chunk generation, 1.3B-class AR-DiT stack: D=1536, 12x128 heads, "
                f"FFN 8960, {args.layers} layers, chunk 6 of a stream (4680 tokens, "
                "3x30x52) over a window of W=7 chunks holding chunks 0..5 (28080 "
                "tokens), 512 text tokens, 4 denoising steps at t=1000/750/500/250 "
                "with the sampler update, then the commit pass at t=0")
    if wl.name == "ragged":
        return ("ragged batch of 8 streams of the 1.3B-class block (D=1536, 12x128 "
                "heads, FFN 8960), one 4680-token chunk each over caches of "
                f"{'/'.join(str(c) for c in wl.cache_chunks)} chunks, 512 text tokens "
                f"each, {args.layers} layers, per-stream t")
    if wl.name == "large":
        return (f"large AR-DiT block: D={sh.dim}, {sh.n_heads}x{sh.head_dim} heads, FFN "
                f"{sh.ffn_dim}, chunk 11 of a stream (4680 tokens, 3x30x52, frames 33-35) over "
                "a rolling window of the 7 previous chunks (32760 tokens) in a wrapped ring of "
                f"8 chunk slots, 512 text tokens, {args.layers} layers, one denoising step at "
                "t=1000")
    return ("1.3B-class AR-DiT block: D=1536, 12x128 heads, FFN 8960, chunk 4680 "
            "tokens (3x30x52) over a 28080-token cache, 512 text tokens, "
            f"{args.layers} layers, t=1000/750/500/250")


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the block's hot path is a one-GPU kernel "
              "pipeline; run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.micro:
        micro_main()
        return
    if args.sp2:
        if args.workload not in ("large", "block13b"):
            print("--sp2 takes the large or block13b workload", file=sys.stderr)
            sys.exit(2)
        sp2_main(args)
        return
    if args.cold and args.workload != "ragged":
        print("--cold times the elementwise kernels of the ragged workload only", file=sys.stderr)
        sys.exit(2)
    if args.chunk and args.workload == "large":
        args.workload = "block13b"
    if args.chunk and (args.workload != "block13b" or args.sparsity or args.quant != "bf16"):
        print("--chunk runs the dense bf16 block13b workload only", file=sys.stderr)
        sys.exit(2)
    if args.layers is None:
        args.layers = DEFAULT_LAYERS[args.workload]
    import torch
    from paper_2606_15319_amd import ardit as A
    from workloads import WORKLOADS

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = WORKLOADS[args.workload]
    sh = wl.shape
    cache_lens = [c * sh.chunk_tokens for c in wl.cache_chunks]
    ragged = args.workload == "ragged"
    log(f"drawing {args.layers} layers of the {args.workload} workload on the device")
    model = Model(A, wl, args.layers, dev, rho=args.sparsity,
                  timesteps=[float(t) for t in wl.timesteps] if ragged else None,
                  fp8=args.quant == "fp8")
    if args.cold:
        model.step(0)
        torch.cuda.synchronize()
        res = cold_elementwise(A, model, sh, sh.chunk_tokens * len(cache_lens))
        print(json.dumps({"probe": "elementwise kernels, cold and warm",
                          "workload": workload_name(wl, args), "rows": sh.chunk_tokens * len(cache_lens),
                          "flush": "512 MiB read before each cold launch",
                          "kernels": res}), flush=True)
        return
    if args.chunk:
        model.setup_chunk(TIMESTEPS, window=7)
        run = lambda k: model.generate()   # noqa: E731
    else:
        run = model.step
    torch.cuda.synchronize()
    log("warmup")
    for k in range(args.warmup):
        run(k)
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    A.ardit_timing_collect()
    A.ardit_timing_enable(True)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for k in range(args.steps):
        run(k)
    stop.record()
    torch.cuda.synchronize()
    A.ardit_timing_enable(False)
    total_ms = start.elapsed_time(stop)
    n_attn, attn_ms = A.ardit_timing_collect()
    ms_step = total_ms / args.steps
    passes = len(TIMESTEPS) + 1 if args.chunk else 1
    ms_block = ms_step / (args.layers * passes)
    L_q, D = sh.chunk_tokens, sh.dim
    L_k = cache_lens[0] + L_q
    attn_flops = 0.0
    keys = L_k
    for c in cache_lens:
        n_tiles = (c + L_q + 63) // 64
        keys = c + L_q
        if args.sparsity > 0:
            n_keep = max(1, min(n_tiles, math.ceil((1.0 - args.sparsity) * n_tiles - 1e-3)))
            keys = min(c + L_q, 64 * n_keep)
        attn_flops += 4.0 * L_q * keys * D
    attn_avg_ms = attn_ms / max(n_attn, 1)
    achieved = attn_flops / (attn_avg_ms * 1e-3) / 1e12
    log(f"{ms_step:.3f} ms/step, {ms_block:.4f} ms/block pass, attention {attn_avg_ms:.4f} ms "
        f"({achieved:.1f} TFLOP/s) over {n_attn} launches")
    breakdown = None
    if not args.chunk:
        breakdown = kernel_breakdown(A, model, args, sh, cache_lens)
    cpu = None
    if not args.no_cpu_baseline and not ragged:
        log("timing the CPU oracle on one block step")
        cpu = cpu_baseline(model, sample_every=4 if args.workload == "large" else 1)
        if args.chunk:
            # one block pass, scaled to the chunk's layers x passes
            cpu["value"] = round(cpu["value"] * args.layers * passes, 1)
            cpu["unit"] = "ms per chunk"
            cpu["sample"] += (f"; scaled by {args.layers} layers x {passes} passes to a chunk "
                              "(extrapolated)")
        log(f"oracle: {cpu['value']} ms on {cpu['cores']} threads")
    peak = PEAK_FP8_TFLOPS if args.quant == "fp8" else PEAK_BF16_TFLOPS
    log("measuring the MFMA and copy peaks")
    meas = measured_peaks(A)
    meas_peak = meas["mfma_fp8_tflops" if args.quant == "fp8" else "mfma_bf16_tflops"]
    if breakdown:
        breakdown["gemm"]["frac_of_measured"] = round(
            breakdown["gemm"]["achieved"] / meas["mfma_bf16_tflops"], 4)
        breakdown["elementwise"]["frac_of_measured"] = round(
            breakdown["elementwise"]["achieved"] / meas["copy_tbps"], 4)
    line = {
        "metric": "ms per chunk" if args.chunk else "ms per chunk-denoise-step per block",
        "value": round(ms_step if args.chunk else ms_block, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "ms_per_block_pass": round(ms_block, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if args.quant == "bf16" else "bf16 (attention fp8 e4m3)",
        "data": "synthetic (seeded normal draws, random-init weights)",
        "config": {"workload": workload_name(wl, args),
                   "layers": args.layers, "chunk_tokens": L_q,
                   "kv_tokens": L_k if not ragged else [c + L_q for c in cache_lens],
                   "ctx_tokens": wl.ctx_len, "sparsity": args.sparsity,
                   "attention_quant": args.quant,
                   "attended_keys": keys if not ragged else None},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": (None if (args.sparsity or ragged or args.quant == "fp8"
                                          or args.chunk)
                                 else measured_traffic(args.workload)),
                     "kernel": (("FP8 " if args.quant == "fp8" else "")
                                + ("block-sparse " if args.sparsity else "")
                                + "paged self-attention"),
                     "avg_launch_ms": round(attn_avg_ms, 4), "launches": n_attn,
                     "measured_peak": meas_peak,
                     "frac_of_measured": round(achieved / meas_peak, 4) if meas_peak else None},
        "measured_peaks": meas,
        "breakdown": breakdown,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
