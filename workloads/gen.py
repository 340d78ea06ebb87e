"""Shapes, seeds and draws of the synthetic workloads.

Shapes follow the paper's setting: a chunk is three latent frames at 480p
(Evaluation, experimental setup), the KV window W counts at most 7 earlier
chunks and denoising uses S <= 4 steps (Appendix A, fidelity-configuration
space).  The paper fixes no model sizes; the two model shapes below (a
1.3B-class and a large one) and the 30 x 52 latent grid per frame (480 x 832
pixels at a 16x spatial reduction) are assumptions made here.

Every value is drawn in fp32 from numpy's PCG64 seeded with 15319 + the
workload id, then rounded to bf16 with round-to-nearest-even, so the oracle
and the GPU path see bit-identical inputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 15319


# --------------------------------------------------------------------------
# bf16 <-> fp32 (bit manipulation only)
# --------------------------------------------------------------------------
def bf16_bits(a) -> np.ndarray:
    """fp32 values -> bf16 bit patterns (uint16), round to nearest even."""
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    u = a32.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    with np.errstate(over="ignore"):
        r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    bits = r.astype(np.uint16)
    nan = np.isnan(a32)
    if nan.any():
        bits[nan] = np.uint16(0x7FC0)
    return bits


def bits_to_f32(b) -> np.ndarray:
    """bf16 bit patterns (uint16) -> fp32 values (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(a) -> np.ndarray:
    """fp32 values rounded to the nearest bf16, returned as fp32."""
    return bits_to_f32(bf16_bits(a))


def make_rng(workload_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(SEED_BASE + int(workload_id)))


def normal_bf16(rng: np.random.Generator, shape, std: float = 1.0,
                mean: float = 0.0) -> np.ndarray:
    """N(mean, std^2) drawn in fp32, rounded to bf16, returned as fp32."""
    z = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        z *= np.float32(std)
    if mean != 0.0:
        z += np.float32(mean)
    return bf16_round(z)


# --------------------------------------------------------------------------
# shapes
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class BlockShape:
    """Geometry of one AR-DiT block and of one chunk of latent tokens."""
    dim: int
    n_heads: int
    head_dim: int
    ffn_dim: int
    frames: int          # latent frames per chunk
    lat_h: int
    lat_w: int
    eps: float = 1e-6
    theta: float = 10000.0
    time_freq_dim: int = 256

    @property
    def tokens_per_frame(self) -> int:
        return self.lat_h * self.lat_w

    @property
    def chunk_tokens(self) -> int:
        return self.frames * self.tokens_per_frame


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: a block shape plus stream/cache geometry."""
    wid: int
    name: str
    shape: BlockShape
    cache_chunks: tuple = (0,)      # earlier chunks held in each stream's cache
    frame_pos0: tuple = (0,)        # absolute latent-frame index of each chunk's first frame
    ctx_len: int = 512
    timesteps: tuple = (1000,)
    layers: int = 1
    ring_slots: int = 0             # >0: the cache is a ring of this many chunk slots
    attention_only: bool = False
    notes: str = ""

    @property
    def n_streams(self) -> int:
        return len(self.cache_chunks)


SHAPE_TINY = BlockShape(dim=256, n_heads=4, head_dim=64, ffn_dim=1024,
                        frames=3, lat_h=8, lat_w=8)
SHAPE_1P3B = BlockShape(dim=1536, n_heads=12, head_dim=128, ffn_dim=8960,
                        frames=3, lat_h=30, lat_w=52)
SHAPE_LARGE = BlockShape(dim=5120, n_heads=40, head_dim=128, ffn_dim=13824,
                         frames=3, lat_h=30, lat_w=52)


def _ragged_draw():
    # cache lengths U{0..7} chunks and timesteps from {1000,750,500,250},
    # drawn from the ragged workload's own generator before anything else.
    rng = make_rng(4)
    chunks = tuple(int(c) for c in rng.integers(0, 8, size=8))
    ts = tuple(int(t) for t in rng.choice(np.array([1000, 750, 500, 250]), size=8))
    return chunks, ts


_RAGGED_CHUNKS, _RAGGED_TS = _ragged_draw()

WORKLOADS = {
    "tiny": Workload(1, "tiny", SHAPE_TINY, cache_chunks=(2,), frame_pos0=(6,),
                     ctx_len=32, timesteps=(750,), layers=1,
                     notes="single block, one stream, parity case"),
    "attn": Workload(2, "attn", BlockShape(dim=1536, n_heads=12, head_dim=128,
                                           ffn_dim=8960, frames=3, lat_h=30, lat_w=52),
                     cache_chunks=(2,), frame_pos0=(6,), attention_only=True,
                     notes="attention only: 4680 queries over 9360 cached + 4680 own keys"),
    "block13b": Workload(3, "block13b", SHAPE_1P3B, cache_chunks=(6,),
                         frame_pos0=(18,), ctx_len=512,
                         timesteps=(1000, 750, 500, 250), layers=30,
                         notes="1.3B-class block, one stream, 30 layers x 4 steps"),
    "ragged": Workload(4, "ragged", SHAPE_1P3B, cache_chunks=_RAGGED_CHUNKS,
                       frame_pos0=tuple(3 * c for c in _RAGGED_CHUNKS), ctx_len=512,
                       timesteps=_RAGGED_TS, layers=1,
                       notes="8 streams, per-stream cache 0..7 chunks"),
    "large": Workload(5, "large", SHAPE_LARGE, cache_chunks=(7,), frame_pos0=(33,),
                      ctx_len=512, timesteps=(1000,), layers=40, ring_slots=8,
                      notes="rolling window of 7 chunks in a ring of 8 slots, wrapped"),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def ring_page_ids(shape: BlockShape, chunk_index: int, cache_chunks: int, ring_slots: int):
    """Physical pages, in logical order, of a stream whose cache is a ring of
    ring_slots chunk slots (chunk c in slot c % ring_slots, frame f of slot s in
    page s * frames + f), holding chunks chunk_index - cache_chunks .. chunk_index."""
    ids = []
    for c in range(chunk_index - cache_chunks, chunk_index + 1):
        slot = c % ring_slots
        ids += [slot * shape.frames + f for f in range(shape.frames)]
    return ids


def stream_page_ids(wl: Workload):
    """(page ids per stream in logical order, pool size) of a workload's caches:
    the ring layout when the workload has ring slots, else consecutive pages
    per stream (each stream's cache frames plus its chunk's)."""
    sh = wl.shape
    if wl.ring_slots:
        ids = [ring_page_ids(sh, p // sh.frames, c, wl.ring_slots)
               for c, p in zip(wl.cache_chunks, wl.frame_pos0)]
        return [[i + s * wl.ring_slots * sh.frames for i in r] for s, r in enumerate(ids)], \
            len(ids) * wl.ring_slots * sh.frames
    ids, nxt = [], 0
    for c in wl.cache_chunks:
        nf = (c + 1) * sh.frames
        ids.append(list(range(nxt, nxt + nf)))
        nxt += nf
    return ids, nxt


# --------------------------------------------------------------------------
# weight draws
# --------------------------------------------------------------------------
TIME_WEIGHT_ORDER = ("w_t1", "b_t1", "w_t2", "b_t2", "w_m", "b_m")
BLOCK_WEIGHT_ORDER = ("w_qkv", "b_qkv", "g_q", "g_k", "w_o", "b_o", "g_n3",
                      "w_cq", "b_cq", "g_cq", "w_ck", "b_ck", "g_ck",
                      "w_cv", "b_cv", "w_co", "b_co", "w_1", "b_1", "w_2", "b_2",
                      "mod_table")
GAIN_NAMES = ("g_q", "g_k", "g_n3", "g_cq", "g_ck")


def _time_weight_shapes(dim: int, fdim: int = 256):
    return {"w_t1": (dim, fdim), "b_t1": (dim,), "w_t2": (dim, dim),
            "b_t2": (dim,), "w_m": (6 * dim, dim), "b_m": (6 * dim,)}


def block_weight_shapes(shape: BlockShape):
    D, F = shape.dim, shape.ffn_dim
    s = {"w_qkv": (3 * D, D), "b_qkv": (3 * D,), "g_q": (D,), "g_k": (D,),
         "w_o": (D, D), "b_o": (D,), "g_n3": (D,),
         "w_cq": (D, D), "b_cq": (D,), "g_cq": (D,),
         "w_ck": (D, D), "b_ck": (D,), "g_ck": (D,),
         "w_cv": (D, D), "b_cv": (D,), "w_co": (D, D), "b_co": (D,),
         "w_1": (F, D), "b_1": (F,), "w_2": (D, F), "b_2": (D,),
         "mod_table": (6, D)}
    return s


def draw_time_weights(rng: np.random.Generator, dim: int, fdim: int = 256,
                      std: float = 0.02) -> dict:
    shapes = _time_weight_shapes(dim, fdim)
    return {k: normal_bf16(rng, shapes[k], std) for k in TIME_WEIGHT_ORDER}


def draw_block_weights(rng: np.random.Generator, shape: BlockShape,
                       std: float = 0.02) -> dict:
    """Matrices, biases and mod_table ~ N(0, std^2); norm gains ~ 1 + N(0, std^2)."""
    shapes = block_weight_shapes(shape)
    out = {}
    for k in BLOCK_WEIGHT_ORDER:
        if k in GAIN_NAMES:
            out[k] = normal_bf16(rng, shapes[k], std, mean=1.0)
        else:
            out[k] = normal_bf16(rng, shapes[k], std)
    return out


def draw_ragged_streams(wl: Workload):
    """Per-stream (cache_tokens, frame_pos0, timestep) of a workload."""
    T = wl.shape.chunk_tokens
    return [(c * T, p, t) for c, p, t in zip(wl.cache_chunks, wl.frame_pos0,
                                               _cycle(wl.timesteps, wl.n_streams))]


def _cycle(seq, n):
    return [seq[i % len(seq)] for i in range(n)]


@dataclass
class BlockCase:
    """All inputs of one block call for a set of streams (fp32, bf16-exact)."""
    shape: BlockShape
    time_w: dict
    block_w: dict
    x: list = field(default_factory=list)          # per stream [L_q, D]
    cache_k: list = field(default_factory=list)    # per stream [c, H, d]
    cache_v: list = field(default_factory=list)
    ctx: list = field(default_factory=list)        # per stream [L_x, D]
    cache_len: list = field(default_factory=list)
    frame_pos0: list = field(default_factory=list)
    t: list = field(default_factory=list)


def draw_block_case(wl: Workload, ctx_lens=None) -> BlockCase:
    """Draw one block-step case in the documented order: time-MLP weights, the
    block's weights, then per stream its text context, cache K, cache V and
    chunk activations."""
    sh = wl.shape
    rng = make_rng(wl.wid)
    if wl.name == "ragged":
        _ = rng.integers(0, 8, size=8), rng.choice(np.array([1000, 750, 500, 250]), size=8)
    tw = draw_time_weights(rng, sh.dim, sh.time_freq_dim)
    bw = draw_block_weights(rng, sh)
    case = BlockCase(shape=sh, time_w=tw, block_w=bw)
    for i, (c, p, t) in enumerate(draw_ragged_streams(wl)):
        lx = wl.ctx_len if ctx_lens is None else ctx_lens[i]
        case.ctx.append(normal_bf16(rng, (lx, sh.dim)))
        case.cache_k.append(normal_bf16(rng, (c, sh.n_heads, sh.head_dim)))
        case.cache_v.append(normal_bf16(rng, (c, sh.n_heads, sh.head_dim)))
        case.x.append(normal_bf16(rng, (sh.chunk_tokens, sh.dim)))
        case.cache_len.append(c)
        case.frame_pos0.append(p)
        case.t.append(float(t))
    return case
