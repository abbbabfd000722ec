"""The library's host code under AddressSanitizer: the host-only paths
(bandwidth allocation, epoch scheduling, argument and shape validation, the
workspace sizes) run through the C ABI from the CPU tests that cover them,
against a build whose host code is instrumented.  Runs where no preload
library is configured, since the sanitizer runtime must be preloaded."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang++"


def _asan_runtime():
    if not os.path.exists(CLANG):
        return None
    r = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(bool(os.environ.get("LD_PRELOAD")) or os.path.exists("/etc/ld.so.preload"),
                    reason="a preload library is configured; the sanitizer runtime would have to replace it")
def test_host_paths_are_clean_under_address_sanitizer():
    runtime = _asan_runtime()
    if runtime is None or not os.path.exists("/opt/rocm/bin/hipcc"):
        pytest.skip("no hipcc or no AddressSanitizer runtime")
    sys.path.insert(0, ROOT)
    from paper_2605_22850_amd import build
    lib = build.build(asan=True)
    # the build is instrumented: its host code calls the sanitizer's checks
    nm = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report_load" in nm and "__asan_init" in nm
    env = dict(os.environ, LD_PRELOAD=runtime, OC_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1:exitcode=86")
    # and it is the library those tests load
    probe = subprocess.run([sys.executable, "-c", "import paper_2605_22850_amd as oc; oc.oc_abi_version(); "
                            "print(*sorted({l.split()[-1] for l in open('/proc/self/maps') if 'objectcache' in l}))"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert probe.stdout.split() == [lib], probe.stdout + probe.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
                        "tests/test_scheduler.py", "tests/test_abi.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
