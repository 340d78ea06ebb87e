"""C-ABI checks that need no GPU: the library loads, exports every function
include/ardit.h declares, and host validation returns the documented status
before anything is enqueued (the fake device addresses below are never
dereferenced because every call fails a host check first)."""
import os
import re

import numpy as np
import pytest

A = pytest.importorskip("paper_2606_15319_amd.ardit",
                        reason="libardit.so not built (python -m paper_2606_15319_amd.build)")

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADERS = [os.path.join(INCLUDE, f) for f in sorted(os.listdir(INCLUDE)) if f.endswith(".h")]
FAKE = 1 << 20   # 16-byte aligned stand-in address, never dereferenced


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ardit_[a-z_]+)\s*\(", text)))


def test_every_declared_function_is_exported():
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert A.has_symbol(n), n
    assert set(names) == set(A.exported_symbols())


def test_status_strings_and_version():
    for code, name in A.STATUS.items():
        assert A.ardit_status_str(code) == name
    assert A.ardit_status_str(123) == "ARDIT_UNKNOWN"
    assert A.ardit_version() == 502


def _dims(**kw):
    d = dict(dim=256, n_heads=4, head_dim=64, ffn_dim=1024, frames_per_chunk=3, lat_h=8, lat_w=8)
    d.update(kw)
    return A.make_dims(**d)


def _weights():
    return A.block_weights({k: FAKE for k in A._BLOCK_FIELDS})


def _kv(max_frames=9, n_pages=9):
    return A.kv_paged(FAKE, FAKE, FAKE, n_pages, max_frames)


def _status(fn, *args):
    with pytest.raises(A.ArditError) as e:
        fn(*args)
    return e.value.status


def _block(dims=None, cache_len=384, pos=6, ctx_len=32, kv=None, ws_bytes=None, x=FAKE, w=None):
    dims = dims or _dims()
    b = A.Batch([192], [cache_len], [pos], [ctx_len])
    need = A.ardit_workspace_size(dims, b) if ws_bytes is None else ws_bytes
    A.ardit_block_fwd(FAKE, dims, x, kv or _kv(), cache_len, pos, FAKE, FAKE, FAKE, ctx_len,
                      w or _weights(), FAKE, FAKE, need)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96, n_heads=2, dim=192), -5),     # head_dim outside {64, 128}
    (dict(n_heads=3), -2),                           # D != H * d
    (dict(dim=320, n_heads=5), -5),                  # D not a multiple of 128
    (dict(ffn_dim=1000), -5),
    (dict(lat_h=3, lat_w=3), -5),                    # T not a multiple of 8
    (dict(lat_h=3, lat_w=8), -5),                    # T = 24: a 64-key tile spans 4 frames
    (dict(lat_h=5, lat_w=8), -5),                    # T = 40: 3 frames
    (dict(lat_h=2, lat_w=8), -5),                    # T = 16
    (dict(lat_w=0), -2),
])
def test_dims_rejected(kw, code):
    assert _status(_block, _dims(**kw)) == code


def test_cache_len_not_frame_multiple():
    assert _status(_block, None, 100) == -2


def test_cache_overflow_is_capacity():
    assert _status(_block, None, 384, 6, 32, _kv(max_frames=8)) == -3


def test_workspace_too_small():
    assert _status(_block, None, 384, 6, 32, None, 1024) == -4


def test_null_and_misaligned_pointers():
    assert _status(_block, None, 384, 6, 32, None, None, 0) == -1
    assert _status(_block, None, 384, 6, 32, None, None, FAKE + 2) == -1
    w = {k: FAKE for k in A._BLOCK_FIELDS}
    w["w_o"] = 0
    assert _status(_block, None, 384, 6, 32, None, None, FAKE, A.block_weights(w)) == -1


def test_ctx_len_zero_rejected():
    assert _status(_block, None, 384, 6, 0) == -2


def test_varlen_wrong_chunk_length():
    d = _dims()
    b = A.Batch([192, 100], [0, 0], [0, 0], [8, 8])
    assert _status(A.ardit_block_fwd_varlen, FAKE, d, b, FAKE, _kv(), FAKE, FAKE, FAKE,
                   _weights(), FAKE, FAKE, 1 << 30) == -2


def test_too_many_streams():
    d = _dims()
    b = A.Batch([192] * 65, [0] * 65, [0] * 65, [8] * 65)
    assert _status(A.ardit_workspace_size, d, b) == -1


def test_cache_beyond_2_30_rejected():
    d = _dims()
    T = d.lat_h * d.lat_w
    assert _status(A.ardit_workspace_size, d, A.Batch([100], [(1 << 30) + T])) == -3
    assert A.ardit_workspace_size(d, A.Batch([100], [1 << 30])) > 0


def test_attn_fwd_validation():
    d = _dims()
    b = A.Batch([100], [64])
    need = A.ardit_workspace_size(d, b)
    assert _status(A.ardit_attn_fwd, FAKE, d, b, FAKE, _kv(max_frames=2), FAKE, FAKE, need) == -3
    assert _status(A.ardit_attn_fwd, FAKE, d, A.Batch([100], [10]), FAKE, _kv(), FAKE, FAKE,
                   need) == -2
    # the workspace carries the partial results of a split schedule
    assert _status(A.ardit_attn_fwd, FAKE, d, b, FAKE, _kv(), FAKE, FAKE, need - 1) == -4
    assert _status(A.ardit_attn_fwd, FAKE, d, b, FAKE, _kv(), FAKE, 0, need) == -1


def test_time_mod_validation():
    d = _dims()
    tw = A.time_weights({k: FAKE for k in A._TIME_FIELDS})
    assert _status(A.ardit_time_mod, FAKE, d, [], tw, FAKE, FAKE, 1 << 20) == -1
    assert _status(A.ardit_time_mod, FAKE, d, [1.0], tw, FAKE, FAKE, 16) == -4


def test_stack_rejects_aliasing_and_bad_layers():
    d = _dims()
    b = A.Batch([192], [384], [6], [32])
    need = A.ardit_workspace_size(d, b)
    assert _status(A.ardit_stack_fwd, FAKE, d, b, FAKE, [], FAKE, [], [], [], FAKE, FAKE,
                   need) == -1
    assert _status(A.ardit_stack_fwd, FAKE, d, b, FAKE, [_kv()], FAKE, [FAKE], [FAKE],
                   [_weights()], FAKE, FAKE, need) == -1


def test_workspace_size_grows_with_tokens():
    d = _dims()
    s1 = A.ardit_workspace_size(d, A.Batch([192], [0], [0], [32]))
    s2 = A.ardit_workspace_size(d, A.Batch([192, 192], [0, 0], [0, 0], [32, 32]))
    assert s2 > s1 > 0 and s1 % 256 == 0


def test_last_error_names_the_problem():
    with pytest.raises(A.ArditError):
        _block(_dims(n_heads=3))
    assert "n_heads" in A.ardit_last_error()


def test_layout_round_trip():
    from paper_2606_15319_amd.layout import (pack_pages, unpack_pages, ctx_to_device_layout,
                                             ctx_from_device_layout)
    rng = np.random.default_rng(0)
    H, d, T = 3, 8, 16
    n = 40
    k = rng.standard_normal((n, H, d)).astype(np.float32)
    v = rng.standard_normal((n, H, d)).astype(np.float32)
    kp = np.zeros((5, H, T, d), np.float32)
    vp = np.zeros((5, H, d, T), np.float32)
    ids = [4, 0, 2]
    pack_pages(k, v, ids, kp, vp)
    assert kp[4, 1, 3, 5] == k[3, 1, 5] and vp[0, 2, 6, 1] == v[17, 2, 6]
    k2, v2 = unpack_pages(kp, vp, ids, n)
    assert np.array_equal(k2, k) and np.array_equal(v2, v)
    kc = rng.standard_normal((7, H * d))
    vc = rng.standard_normal((7, H * d))
    kf, vf = ctx_to_device_layout(kc, vc, H)
    kc2, vc2 = ctx_from_device_layout(kf, vf, 7, H, d)
    assert np.array_equal(kc, kc2) and np.array_equal(vc, vc2)


def test_sparsity_validation():
    d = _dims()
    for bad in (1.5, -0.1, float("nan")):
        assert _status(A.ardit_workspace_size, d, A.Batch([100], [64], sparsity=[bad])) == -1
        assert "sparsity" in A.ardit_last_error()
    # more key tiles than the selection ranks (16384 tiles of 64 keys)
    big = A.Batch([192], [64 * 16384], sparsity=[0.5])
    assert _status(A.ardit_workspace_size, d, big) == -5
    # the same length is fine when dense
    assert A.ardit_workspace_size(d, A.Batch([192], [64 * 16384], sparsity=[0.0])) > 0


def test_sparse_workspace_holds_means_scores_and_lists():
    """Extra workspace of a sparse batch: the fp32 mean query of every item
    (H x query tiles x d), its fp32 score per key tile and the kept-tile lists
    (H x query tiles x n_keep int32), each rounded up to 256 bytes; n_keep
    from the oracle's rule."""
    from oracle.sparse_ref import keep_count
    d = _dims()
    q, c = 768, 6336                       # 3 query tiles; 7104 keys = 111 tiles
    dense = A.ardit_workspace_size(d, A.Batch([q], [c]))
    assert A.ardit_workspace_size(d, A.Batch([q], [c], sparsity=[0.0])) == dense
    up = lambda n: (n + 255) // 256 * 256
    items = 4 * 3
    for rho in (0.6, 0.7, 0.8, 0.9, 1.0):
        nk = keep_count(111, rho)
        want = dense + up(items * 64 * 4) + up(items * 111 * 4) + up(items * nk * 4)
        assert A.ardit_workspace_size(d, A.Batch([q], [c], sparsity=[rho])) == want, rho


def test_sparse_select_validation():
    d = _dims()
    b = A.Batch([600, 70], [1280, 192], sparsity=[0.8, 1.0])
    need = A.ardit_workspace_size(d, b)
    # stream 0 keeps ceil(0.2 * 30) = 6 of its 30 tiles
    assert _status(A.ardit_sparse_select, FAKE, d, b, FAKE, _kv(max_frames=40), FAKE, 5, FAKE,
                   need) == -1
    assert "row_stride" in A.ardit_last_error()
    assert _status(A.ardit_sparse_select, FAKE, d, b, FAKE, _kv(max_frames=40), 0, 6, FAKE,
                   need) == -1
    assert _status(A.ardit_sparse_select, FAKE, d, b, FAKE, _kv(max_frames=40), FAKE, 6, FAKE,
                   need - 1) == -4
    assert _status(A.ardit_sparse_select, FAKE, d, b, FAKE, _kv(max_frames=4), FAKE, 6, FAKE,
                   need) == -3


def test_quant_validation():
    d = _dims()   # head_dim 64
    assert _status(A.ardit_workspace_size, d, A.Batch([100], [64], quant=[2])) == -1
    assert "quant" in A.ardit_last_error()
    # FP8 attention is built for head_dim 128
    assert _status(A.ardit_workspace_size, d, A.Batch([100], [64], quant=[1])) == -5
    d128 = _dims(dim=512, n_heads=4, head_dim=128)
    dense = A.ardit_workspace_size(d128, A.Batch([100], [64]))
    f8 = A.ardit_workspace_size(d128, A.Batch([100], [64], quant=[1]))
    up = lambda n: (n + 255) // 256 * 256
    # query codes + scales for every row, keys and values of the FP8 stream padded to 64-key tiles
    keys = 192
    want = dense + up(100 * 512) + up(100 * 512 // 32) + 2 * (up(4 * keys * 128) + up(4 * keys * 128 // 32))
    assert f8 == want


def test_mx_quantize_validation():
    assert _status(A.ardit_mx_quantize, FAKE, FAKE, 4, 48, 48, FAKE, FAKE) == -2
    assert _status(A.ardit_mx_quantize, FAKE, FAKE, 4, 64, 60, FAKE, FAKE) == -2
    assert _status(A.ardit_mx_quantize, FAKE, 0, 4, 64, 64, FAKE, FAKE) == -1


# ------------------------------------------------ chunk generation (host side)
def test_window_pages_match_oracle_listing():
    """The C page-table policy equals the oracle's window listing and slot map
    for every small (chunk, sink, window, frames) case, bit for bit."""
    import itertools
    import oracle as O
    for c, sink, win, f in itertools.product(range(14), range(4), range(6), (1, 3)):
        ids, cached = A.ardit_window_pages(c, sink, win, f, page_base=5)
        ref, ref_cached = O.chunk_ref.window_page_table(c, sink, win, f)
        assert cached == ref_cached and ids == [5 + int(v) for v in ref], (c, sink, win, f)
        # slots of held chunks and of the chunk itself are distinct pages
        assert len(set(ids)) == len(ids)
        assert max(ids) < 5 + (sink + win + 1) * f


def test_window_pages_rejections():
    assert _status(A.ardit_window_pages, -1, 0, 1, 3) == -1
    assert _status(A.ardit_window_pages, 0, 0, -1, 3) == -1
    assert _status(A.ardit_window_pages, 0, 0, 1, 0) == -1
    # table too short for 1 sink + 2 window chunks + the chunk (12 frames)
    assert _status(A.ardit_window_pages, 5, 1, 2, 3, 0, 11) == -3
    assert _status(A.ardit_window_pages, 5, 1, 2, 3, 2**31 - 10) == -3


def _gen(n_steps=(2,), ts=((1000.0, 500.0),), x0=FAKE + (1 << 30), noise=FAKE, ws_bytes=None,
         x_init=FAKE, dims=None, layers=2):
    dims = dims or _dims()
    B = len(n_steps)
    b = A.Batch([192] * B, [384] * B, [6] * B, [32] * B)
    need = A.ardit_workspace_size(dims, b) if ws_bytes is None else ws_bytes
    A.ardit_chunk_generate(FAKE, dims, b, list(n_steps), [list(t) for t in ts], x_init, noise,
                           [_kv()] * layers, A.time_weights({k: FAKE for k in A._TIME_FIELDS}),
                           [FAKE] * layers, [FAKE] * layers, [_weights()] * layers, x0,
                           FAKE + (1 << 34), need)


@pytest.mark.parametrize("kw,code", [
    (dict(n_steps=(1, 2), ts=((1000.0,), (1000.0, 500.0))), -1),   # steps increase along the batch
    (dict(n_steps=(0,), ts=((),)), -1),                              # no step
    (dict(n_steps=(17,), ts=((500.0,) * 17,)), -1),                  # above ARDIT_MAX_STEPS
    (dict(ts=((1000.0, 1001.0),)), -1),                              # timestep outside [0, 1000]
    (dict(ts=((float("nan"), 500.0),)), -1),
    (dict(noise=None), -1),                                          # two steps need noise
    (dict(x0=FAKE), -1),                                             # x0_out overlaps x_init
    (dict(x0=FAKE + (1 << 34)), -1),                                 # x0_out overlaps the workspace
    (dict(ws_bytes=1 << 20), -4),
    (dict(layers=0), -1),
])
def test_chunk_generate_rejections(kw, code):
    assert _status(lambda: _gen(**kw)) == code


def test_workspace_holds_generation_buffers():
    """The workspace grows by the velocity buffer and the modulation of the batch."""
    d = _dims()
    one = A.ardit_workspace_size(d, A.Batch([192], [384], [6], [32]))
    two = A.ardit_workspace_size(d, A.Batch([192] * 2, [384] * 2, [6] * 2, [32] * 2))
    assert two - one >= 2 * 192 * 256 * 2 + 6 * 256 * 4


def test_timing_masks_and_kinds():
    """Host-side checks of the timing facility (no launch is recorded here)."""
    assert _status(A.ardit_timing_enable, 8) == -1
    assert _status(A.ardit_timing_enable, -1) == -1
    assert _status(A.ardit_timing_collect_kind, 3) == -1
    A.ardit_timing_enable(7)
    A.ardit_timing_enable(False)
    for k in (A.TIME_ATTENTION, A.TIME_GEMM, A.TIME_ELEMENTWISE):
        assert A.ardit_timing_collect_kind(k) == (0, 0.0)
    assert A.ardit_timing_collect() == (0, 0.0)


def test_text_offsets_beyond_2_31_rejected():
    """Text keys/values are addressed by a 32-bit element offset: a batch whose
    text tokens times the width reach 2^31 is refused before any launch."""
    d = _dims(dim=8192, n_heads=64, head_dim=128)
    at_limit = A.Batch(ctx_lens=[4096] * 64)              # 2^18 tokens * 2^13 = 2^31
    assert _status(A.ardit_workspace_size, d, at_limit) == -3
    assert "2^31" in A.ardit_last_error()
    below = A.Batch(ctx_lens=[4096] * 63 + [4095])
    assert A.ardit_workspace_size(d, below) > 0


def test_debug_checks_switch():
    assert _status(A.ardit_debug_checks, 2) == -1
    assert _status(A.ardit_debug_checks, -1) == -1
    A.ardit_debug_checks(1)
    A.ardit_debug_checks(0)


def test_noalloc_attention_host_rejections():
    """The allocation-free attention refuses, before touching the device, FP8
    streams and batches whose scratch exceeds its 72 MiB."""
    d = _dims(dim=512, n_heads=4, head_dim=128)
    assert _status(A.ardit_attn_fwd_noalloc, FAKE, d, A.Batch([64], [256], quant=[1]), FAKE,
                   _kv(max_frames=9), FAKE) == -5
    # 2048 items x 10048 key tiles of fp32 scores alone are 82 MB
    big = A.Batch([131072], [512000], sparsity=[0.9])
    assert _status(A.ardit_attn_fwd_noalloc, FAKE, d, big, FAKE, _kv(max_frames=10048),
                   FAKE) == -4
    assert "72" in A.ardit_last_error() or "scratch" in A.ardit_last_error()
    assert _status(A.ardit_attn_fwd_noalloc, FAKE, d, A.Batch([64], [256]), 0,
                   _kv(max_frames=9), FAKE) == -1


def test_timing_flush_records_and_micro_host_checks():
    """Host-side checks of the cold-timing flush, the per-launch records and
    the measurement kernels (nothing is launched here)."""
    assert _status(A.ardit_timing_flush, FAKE, 0) == -1          # buffer without size
    assert _status(A.ardit_timing_flush, None, 64) == -1         # size without buffer
    assert _status(A.ardit_timing_flush, FAKE + 8, 64) == -1     # misaligned
    assert _status(A.ardit_timing_flush, FAKE, 24) == -1         # not a multiple of 16
    A.ardit_timing_flush(FAKE, 1 << 20)
    A.ardit_timing_flush(None, 0)
    assert _status(A.ardit_timing_records, 3) == -1
    assert A.ardit_timing_records(A.TIME_ELEMENTWISE) == []
    assert _status(A.ardit_micro_mfma, FAKE, 2, 4, 10, FAKE) == -1
    assert _status(A.ardit_micro_mfma, FAKE, 0, 0, 10, FAKE) == -1
    assert _status(A.ardit_micro_mfma, FAKE, 0, 4, 10, 0) == -1
    assert _status(A.ardit_micro_copy, FAKE, FAKE, FAKE + 4096, 20) == -1
    assert _status(A.ardit_micro_copy, FAKE, FAKE, FAKE + 16, 4096) == -1   # overlap
    assert _status(A.ardit_micro_fill, FAKE, FAKE + 4, 64) == -1
    assert _status(A.ardit_micro_read, FAKE, FAKE, 1 << 20, FAKE, 16) == -1   # sink too small
    assert _status(A.ardit_micro_read, FAKE, FAKE + 8, 1 << 20, FAKE, 1 << 15) == -1
    assert _status(A.ardit_timing_flush, FAKE, 64 * 1024) == -1             # below 128 KiB
