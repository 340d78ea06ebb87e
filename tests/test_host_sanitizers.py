"""The library's host code -- argument validation, workspace layout,
attention planning (XCD split, split schedule, sparse and FP8 planning), the
page-table policy, timing records and the controller -- built with
AddressSanitizer and UndefinedBehaviorSanitizer and driven by the ABI and
controller tests on the CPU, with no sanitizer report.

api.cpp and control.cpp are compiled for the host with
-fsanitize=address,undefined (no recovery: the first report ends the run),
linked with the kernel objects of the regular build into a copy of the
package, and tests/test_abi.py and tests/test_control.py run against that
copy in a subprocess with the ASan runtime preloaded.  CPU only: nothing here
touches a GPU."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_15319_amd")

# host-only sanitizer flags: each -fsanitize= right after -Xarch_host, so the
# device code is built exactly as in the regular library
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _runtime_dir():
    for d in sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux")):
        if os.path.exists(os.path.join(d, "libclang_rt.asan-x86_64.so")):
            return d
    return None


def test_host_code_clean_under_asan_and_ubsan(tmp_path):
    from paper_2606_15319_amd import build as B
    hipcc = B.hipcc()
    rt = _runtime_dir()
    if not shutil.which(hipcc) and not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    if rt is None:
        pytest.skip("no ASan runtime in the ROCm toolchain")
    kernel_objs = [os.path.join(PKG, "_build", os.path.splitext(s)[0] + ".o") for s in B.SOURCES
                   if s.endswith(".hip")]
    if not all(os.path.exists(o) for o in kernel_objs):
        B.build()
    obj_dir = tmp_path / "obj"
    obj_dir.mkdir()
    host_objs = []
    for src in ("api.cpp", "control.cpp"):
        o = str(obj_dir / (os.path.splitext(src)[0] + ".o"))
        flags = [f for f in B.FLAGS if f != "-O3"] + ["-O1", "-g"] + SAN
        r = subprocess.run([hipcc, *flags, "-x", "hip", "-c", os.path.join(B.CSRC, src), "-o", o],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        host_objs.append(o)
    repo = tmp_path / "repo"
    for d in ("tests", "oracle", "workloads", "include", "profiles"):
        shutil.copytree(os.path.join(ROOT, d), repo / d,
                        ignore=shutil.ignore_patterns("__pycache__", "*.pyc"))
    (repo / "paper_2606_15319_amd").mkdir(parents=True)
    for f in glob.glob(os.path.join(PKG, "*.py")):
        shutil.copy(f, repo / "paper_2606_15319_amd")
    lib = str(repo / "paper_2606_15319_amd" / "libardit.so")
    r = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libasan",
                        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                        "-o", lib, *host_objs, *kernel_objs], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    # the host code really is instrumented
    syms = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True,
                          text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms
    env = dict(os.environ)
    env.update({"LD_PRELOAD": os.path.join(rt, "libclang_rt.asan-x86_64.so"),
                "LD_LIBRARY_PATH": rt + (":" + env["LD_LIBRARY_PATH"]
                                         if env.get("LD_LIBRARY_PATH") else ""),
                "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1",
                "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"})
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_abi.py", "tests/test_control.py"], cwd=str(repo), env=env,
                       capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
