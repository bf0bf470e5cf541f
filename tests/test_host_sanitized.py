"""The host side of libpnn under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only, no GPU).

plan.hip (plan construction, workspace layout, offset arithmetic, argument validation of every entry
point) is compiled with host-side ASan + UBSan (the device code is untouched: each -fsanitize= sits
behind -Xarch_host) and linked with the ordinary kernel objects.  A child Python process with the
ASan runtime preloaded then runs tests/test_abi.py against that library: plans for every workload,
parameter layouts, the inspect walk over every internal tensor, every error and alignment path.
Any sanitizer report aborts the child (-fno-sanitize-recover), so the test fails on the first one.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2103_08802_amd", "csrc")
OUT = os.path.join(ROOT, "_build", "asan")
KERNEL_SOURCES = ["k_conv.hip", "k_gemm.hip", "k_misc.hip", "k_unit.hip", "noalloc.hip"]
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def _asan_runtime():
    r = subprocess.run(["hipcc", "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def _build_sanitized():
    sys.path.insert(0, ROOT)
    import __graft_entry__ as G
    os.makedirs(OUT, exist_ok=True)
    objs = []
    for src in KERNEL_SOURCES:                 # the ordinary objects of the last build, else compile
        obj = os.path.join(G.BUILD, os.path.splitext(src)[0] + ".o")
        objs.append(obj if os.path.exists(obj) else G._compile(src))
    plan_obj = os.path.join(OUT, "plan.o")
    cmd = ["hipcc"] + [f for f in G.HIPCC_FLAGS if f != "-O3"] + ["-O1", "-g"] + HOST_SAN + \
          ["-c", os.path.join(CSRC, "plan.hip"), "-o", plan_obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    lib = os.path.join(OUT, "libpnn_asan.so")
    r = subprocess.run(["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", lib, plan_obj] + objs,
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return lib


CHILD = r"""
import sys
sys.path.insert(0, {root!r})
from paper_2103_08802_amd import binding as B
B.LIB_PATH = {lib!r}
import pytest
rc = pytest.main(["-q", "-x", "-s", "-p", "no:cacheprovider", {tests!r}])
assert B.lib()._name == {lib!r}
sys.exit(rc)
"""


def test_abi_under_asan_and_ubsan():
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("no ASan runtime in this toolchain")
    lib = _build_sanitized()
    env = dict(os.environ)
    env["LD_PRELOAD"] = rt + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    code = CHILD.format(root=ROOT, lib=lib, tests=os.path.join(ROOT, "tests", "test_abi.py"))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out
