"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer:
tests/sanitize/build.sh compiles every source (sanitizers on the host pass
only) with a C++ driver of the ABI's validation, workspace sizing and layout
paths; the driver must finish cleanly.  It never launches a kernel, so it runs
without a GPU (and is skipped where one is visible, since nothing here needs
it)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:  # pragma: no cover
        return False


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc")
@pytest.mark.skipif(_gpu_visible(), reason="host-only check; runs where no GPU is visible")
def test_abi_host_code_under_asan_ubsan(tmp_path):
    exe = tmp_path / "abi_san"
    b = subprocess.run(["bash", os.path.join(HERE, "sanitize", "build.sh"), str(exe)],
                       capture_output=True, text=True, timeout=900)
    assert b.returncode == 0, b.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "abi driver ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
