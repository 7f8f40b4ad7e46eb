"""The host C++ of the library (argument validation, the Lloyd and uniform
grids, the bits allocation, GPTQ orchestration) under AddressSanitizer and
UndefinedBehaviorSanitizer: the CPU ABI tests run against a build whose host
sources are instrumented (the GPU code is not), with the clang ASan runtime
preloaded into a fresh interpreter. Any sanitizer report aborts that run.

No kernel is launched: the ABI tests only call host entry points and
argument sets that the host rejects.
"""
import glob
import os
import subprocess
import sys

import pytest

from conftest import ROOT


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_abi_tests_pass_under_host_sanitizers(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("clang ASan runtime not found")
    sys.path.insert(0, ROOT)
    from paper_2411_17525_amd import build as B
    lib = B.build_host_sanitized(verbose=False)
    log = str(tmp_path / "san")
    env = dict(os.environ)
    env.update({
        "HIGGS_LIB": lib,
        "LD_PRELOAD": rt,
        "ASAN_OPTIONS": f"detect_leaks=0:abort_on_error=1:log_path={log}",
        "UBSAN_OPTIONS": f"halt_on_error=1:print_stacktrace=1:log_path={log}",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    reports = []
    for path in glob.glob(log + "*"):
        with open(path) as f:
            reports.append(f.read()[:4000])
    assert not reports, "sanitizer report:\n" + "\n".join(reports)
    assert r.returncode == 0, (r.stdout[-3000:] + r.stderr[-3000:])
    assert " passed" in r.stdout
