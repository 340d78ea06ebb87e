"""Offline latency profiler of the fidelity-configuration space on one GPU.

The controller routes each chunk to a point of an empirical latency-quality
Pareto frontier profiled offline over the 90 configurations (S, rho, W, Q)
(paper, Section 5.2 and Appendix A; the offline profiler of Section 6).  This
module measures the latency side on the device it runs on: for every
configuration, ms per chunk of ardit_chunk_generate for one stream of an
L-layer stack in steady state (the window full: W cached chunks, chunk index
W), S steps at timesteps 1000 (1 - i / S), block-sparse attention at rho,
FP8 attention when Q is FP8, then the commit pass.

The quality side is VBench in the paper and cannot be measured here (no
trained weights, no benchmark).  The score recorded in its place is a
numerical placeholder: minus the relative L2 distance between the
configuration's clean chunk and the reference configuration's (4, 0, 7,
FP16) on the same starting noise, weights and cache -- how far the
configuration moves the output, not how good it looks.

Run: python -m paper_2606_15319_amd.profiler --out result.json [--md summary.md]
"""
from __future__ import annotations

import argparse
import itertools
import json
import sys
import time

STEPS = (2, 3, 4)
SPARSITY = (0.0, 0.6, 0.7, 0.8, 0.9)
WINDOWS = (1, 3, 7)
QUANTS = (0, 1)                  # ardit_quant: FP16/bf16, FP8
REFERENCE = (4, 0.0, 7, 0)


def timesteps(S):
    return [1000.0 * (1.0 - i / S) for i in range(S)]


def log(msg):
    print(f"[profiler] {msg}", file=sys.stderr, flush=True)


class Stack:
    """An L-layer 1.3B-class stack (D 1536, 12 x 128 heads, FFN 8960, chunks of
    3 x 30 x 52 tokens, 512 text tokens), weights and pages drawn on the device,
    a pool of (max W + 1) chunk slots per layer."""

    def __init__(self, A, n_layers, seed=15319, dev="cuda"):
        import torch
        self.A = A
        D, F, H, d = 1536, 8960, 12, 128
        self.lat_h, self.lat_w, self.frames = 30, 52, 3
        T = self.lat_h * self.lat_w
        self.T, self.Lq, self.D = T, self.frames * T, D
        self.dims = A.make_dims(D, H, d, F, self.frames, self.lat_h, self.lat_w)
        self.ctx_len = 512
        slots = max(WINDOWS) + 1
        self.n_pages = slots * self.frames
        shapes = {"w_qkv": (3 * D, D), "b_qkv": (3 * D,), "g_q": (D,), "g_k": (D,),
                  "w_o": (D, D), "b_o": (D,), "g_n3": (D,), "w_cq": (D, D), "b_cq": (D,),
                  "g_cq": (D,), "w_ck": (D, D), "b_ck": (D,), "g_ck": (D,), "w_cv": (D, D),
                  "b_cv": (D,), "w_co": (D, D), "b_co": (D,), "w_1": (F, D), "b_1": (F,),
                  "w_2": (D, F), "b_2": (D,), "mod_table": (6, D)}
        gains = ("g_q", "g_k", "g_n3", "g_cq", "g_ck")
        cb = A.Batch(ctx_lens=[self.ctx_len])
        ws_bytes = A.ardit_workspace_size(self.dims, cb)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        self.keep, self.w, self.pages, self.ctx_k, self.ctx_v = [], [], [], [], []
        for layer in range(n_layers):
            g = torch.Generator(device=dev)
            g.manual_seed(seed + 1000 * layer)
            wd = {}
            for name, shp in shapes.items():
                t = torch.randn(shp, generator=g, device=dev) * 0.02
                if name in gains:
                    t += 1.0
                wd[name] = t if name == "mod_table" else t.to(torch.bfloat16)
            kp = torch.randn((self.n_pages, H, T, d), generator=g, device=dev).to(torch.bfloat16)
            vp = torch.randn((self.n_pages, H, d, T), generator=g, device=dev).to(torch.bfloat16)
            ctx = torch.randn((self.ctx_len, D), generator=g, device=dev).to(torch.bfloat16)
            ck = torch.empty(self.ctx_len * D, dtype=torch.bfloat16, device=dev)
            cv = torch.empty_like(ck)
            w = A.block_weights(wd)
            A.ardit_ctx_kv(None, self.dims, cb, ctx, w, ck, cv, ws, ws_bytes)
            self.keep.append((wd, ctx))
            self.w.append(w)
            self.pages.append((kp, vp))
            self.ctx_k.append(ck)
            self.ctx_v.append(cv)
        g = torch.Generator(device=dev)
        g.manual_seed(seed + 7)
        tshapes = {"w_t1": (D, 256), "b_t1": (D,), "w_t2": (D, D), "b_t2": (D,),
                   "w_m": (6 * D, D), "b_m": (6 * D,)}
        self.tw_dev = {k: (torch.randn(s, generator=g, device=dev) * 0.02).to(torch.bfloat16)
                       for k, s in tshapes.items()}
        self.tw = A.time_weights(self.tw_dev)
        self.x_init = torch.randn((self.Lq, D), generator=g, device=dev).to(torch.bfloat16)
        self.noise = torch.randn((max(STEPS) - 1, self.Lq, D), generator=g,
                                 device=dev).to(torch.bfloat16)
        self.dev = dev

    def setup(self, S, rho, W, Q):
        """Batch, page tables and workspace of one configuration (chunk W of a
        stream under a window of W chunks, no sink)."""
        import torch
        A = self.A
        ids, cached = A.ardit_window_pages(W, 0, W, self.frames)
        table = torch.tensor([ids], dtype=torch.int32, device=self.dev)
        batch = A.Batch([self.Lq], [cached * self.T], [W * self.frames], [self.ctx_len],
                        sparsity=[rho], quant=[Q])
        kvs = [A.kv_paged(kp, vp, table, self.n_pages, len(ids)) for kp, vp in self.pages]
        ws_bytes = A.ardit_workspace_size(self.dims, batch)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=self.dev)
        x0 = torch.empty_like(self.x_init)
        return dict(batch=batch, kvs=kvs, ws=ws, ws_bytes=ws_bytes, x0=x0, table=table, S=S)

    def generate(self, c):
        self.A.ardit_chunk_generate(None, self.dims, c["batch"], [c["S"]], [timesteps(c["S"])],
                                    self.x_init, self.noise, c["kvs"], self.tw, self.ctx_k,
                                    self.ctx_v, self.w, c["x0"], c["ws"], c["ws_bytes"])


def profile(n_layers=30, reps=2):
    import torch
    from paper_2606_15319_amd import ardit as A
    torch.cuda.set_device(0)
    log(f"drawing a {n_layers}-layer stack on the device")
    st = Stack(A, n_layers)
    torch.cuda.synchronize()
    space = list(itertools.product(STEPS, SPARSITY, WINDOWS, QUANTS))
    space.remove(REFERENCE)
    space.insert(0, REFERENCE)
    rows = []
    ref = None
    for k, (S, rho, W, Q) in enumerate(space):
        c = st.setup(S, rho, W, Q)
        st.generate(c)                                  # warm-up (and the output)
        torch.cuda.synchronize()
        out = c["x0"].float()
        if ref is None:
            ref = out.clone()
        dist = float(torch.linalg.vector_norm(out - ref) / torch.linalg.vector_norm(ref))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            st.generate(c)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        rows.append(dict(steps=S, sparsity=rho, window=W, quant=Q, latency_ms=round(ms, 3),
                         quality=-round(dist, 6)))
        log(f"{k + 1}/{len(space)} S={S} rho={rho} W={W} Q={'FP8' if Q else 'FP16'}: "
            f"{ms:.1f} ms/chunk, distance to reference {dist:.4f}")
    cfgs = [(r["steps"], r["sparsity"], r["window"], r["quant"], r["latency_ms"], r["quality"])
            for r in rows]
    frontier, floor = A.ardit_pareto_frontier(cfgs)
    return dict(layers=n_layers, reps=reps, device=torch.cuda.get_device_name(0), configs=rows,
                frontier=frontier, quality_floor=floor)


def markdown(res, command):
    rows = res["configs"]
    fr = set(res["frontier"])
    lines = ["# Fidelity configurations: latency per chunk on one MI355X", "",
             "Command (from the repository root, on the GPU):", "", "```", command, "```", "",
             f"One stream of the 1.3B-class stack ({res['layers']} layers, D 1536, 12 x 128 "
             "heads, FFN 8960, chunk 4680 tokens, 512 text tokens) in steady state: W cached "
             "chunks (W x 4680 keys) plus the chunk; S steps at 1000 (1 - i/S), then the "
             f"commit pass; mean of {res['reps']} timed generations after one warm-up, HIP "
             "events.  quality = minus the relative L2 distance of the clean chunk to the "
             "reference configuration's (4, 0, 7, FP16) on the same inputs: a numerical "
             "placeholder for the VBench score the paper profiles (random weights).  "
             f"Frontier: {len(fr)} of {len(rows)} configurations (marked *), quality floor "
             f"(median) {res['quality_floor']:.4f}.", "",
             "| S | rho | W | Q | ms/chunk | quality | frontier |", "|---:|---:|---:|---|---:|---:|:-:|"]
    order = sorted(range(len(rows)), key=lambda i: rows[i]["latency_ms"])
    for i in order:
        r = rows[i]
        lines.append(f"| {r['steps']} | {r['sparsity']} | {r['window']} | "
                     f"{'FP8' if r['quant'] else 'FP16'} | {r['latency_ms']:.3f} | "
                     f"{r['quality']:.6f} | {'*' if i in fr else ''} |")
    return "\n".join(lines) + "\n"


def read_profile(path):
    """(S, rho, W, Q, ms per chunk, quality) rows from a profile: the JSON this
    module writes, or the table of its markdown summary."""
    if path.endswith(".json"):
        with open(path) as f:
            return [(r["steps"], r["sparsity"], r["window"], r["quant"], r["latency_ms"],
                     r["quality"]) for r in json.load(f)["configs"]]
    import re
    rows = []
    pat = re.compile(r"\| (\d) \| ([0-9.]+) \| (\d) \| (FP16|FP8) \| ([0-9.]+) \| (-?[0-9.]+) \|")
    with open(path) as f:
        for line in f:
            m = pat.match(line)
            if m:
                rows.append((int(m[1]), float(m[2]), int(m[3]), int(m[4] == "FP8"), float(m[5]),
                             float(m[6])))
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--layers", type=int, default=30)
    ap.add_argument("--reps", type=int, default=2)
    ap.add_argument("--out", default=None)
    ap.add_argument("--md", default=None)
    a = ap.parse_args()
    if not a.out:
        ap.error("--out is required")
    t0 = time.time()
    res = profile(a.layers, a.reps)
    with open(a.out, "w") as f:
        json.dump(res, f, indent=1)
    if a.md:
        cmd = "python -m paper_2606_15319_amd.profiler " + " ".join(sys.argv[1:])
        with open(a.md, "w") as f:
            f.write(markdown(res, cmd))
    log(f"done in {time.time() - t0:.0f} s; frontier {len(res['frontier'])} configurations")


if __name__ == "__main__":
    main()
