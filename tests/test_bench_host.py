"""Host-side contract of bench.py, checked without a GPU: it refuses more than
one GPU and conflicting modes before touching the device, and it reports the
counter-measured attention traffic only while the summary's recorded source
hash matches the attention sources."""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench_module():
    spec = importlib.util.spec_from_file_location("bench_host", os.path.join(ROOT, "bench.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=120)


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = _run("--gpus", n)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_chunk_mode_conflicts_are_refused():
    for extra in (["--quant", "fp8"], ["--sparsity", "0.9"], ["--workload", "ragged"]):
        r = _run("--chunk", *extra)
        assert r.returncode == 2, extra
        assert "--chunk" in r.stderr


def test_traffic_reported_only_for_matching_sources(tmp_path):
    m = _bench_module()
    good = tmp_path / "good.md"
    good.write_text("text\n\n- HBM bytes per launch: 12345\n"
                    f"- attention sources sha256: `{m.attn_source_hash()}`\n")
    stale = tmp_path / "stale.md"
    stale.write_text("- HBM bytes per launch: 12345\n- attention sources sha256: `00`\n")
    broken = tmp_path / "broken.md"
    broken.write_text(f"- attention sources sha256: `{m.attn_source_hash()}`\n")
    for name, want in (("good", 12345), ("stale", None), ("broken", None), ("missing", None)):
        m.traffic_summary = lambda wl, n=name: str(tmp_path / f"{n}.md")
        assert m.measured_traffic("large") == want, name


def test_default_workload_is_the_large_ring():
    m = _bench_module()
    import sys as _s
    argv = _s.argv
    try:
        _s.argv = ["bench.py"]
        args = m.parse()
    finally:
        _s.argv = argv
    assert args.workload == "large" and args.layers is None
    assert m.DEFAULT_LAYERS["large"] == 40
    from workloads import WORKLOADS, stream_page_ids
    wl = WORKLOADS["large"]
    ids, n = stream_page_ids(wl)
    assert n == 24 and sorted(ids[0]) == list(range(24))
    assert ids[0] != sorted(ids[0])          # the ring has wrapped
    assert ids[0][-3:] == [9, 10, 11]       # chunk 11 sits in slot 3
