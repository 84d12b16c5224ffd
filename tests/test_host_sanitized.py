"""The host-side tests (argument validation, launch planning, pool and
optimizer host logic) against a build of libcas with AddressSanitizer and
UndefinedBehaviorSanitizer on its host code. Needs hipcc, no GPU: every call
these tests make fails validation or is a planning query."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not installed")
def test_host_code_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("clang AddressSanitizer runtime not found")
    from paper_2606_04557_amd import build
    lib = build.build(sanitize=True)
    env = dict(os.environ)
    env["CAS_LIB"] = lib
    env["LD_PRELOAD"] = rt + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    log = str(tmp_path / "san")
    env["ASAN_OPTIONS"] = f"detect_leaks=0:abort_on_error=1:log_path={log}"
    env["UBSAN_OPTIONS"] = f"print_stacktrace=1:log_path={log}"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "tests/test_host_lib.py", "tests/test_pool_policy.py"],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    reports = "".join(open(f).read() for f in glob.glob(log + "*"))
    assert r.returncode == 0 and not reports, (r.stdout[-3000:], reports[:3000])
