"""The host library under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

tests/host_sanitize.cpp drives every entry point that needs no device: the
partition and cycle helpers, the threshold update and its binary32 form,
status strings, init's argument errors and its clean failure without a GPU,
and NULL contexts.  The host code is built with the sanitizers (each
-fsanitize= behind -Xarch_host, so no device code is instrumented), the
kernels without; the driver must report nothing and exit 0.  Skipped where a
GPU is present, since init would then succeed and allocate device memory."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2310_00967_amd import build  # noqa: E402

SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _no_gpu():
    try:
        import torch
        return not torch.cuda.is_available()
    except ImportError:
        return True


@pytest.mark.skipif(not _no_gpu(), reason="needs a machine without a GPU (init must fail)")
def test_host_library_is_clean_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    try:
        cc = build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not found")
    csrc = build.CSRC
    objs = []
    for src in build.KERNEL_SOURCES:  # kernels and their launch code: not instrumented
        obj = tmp_path / (src + ".o")
        subprocess.run([cc, *build.COMMON, *build.DEVICE, "-x", "hip", "-c", os.path.join(csrc, src),
                        "-o", str(obj)], check=True, capture_output=True, text=True)
        objs.append(str(obj))
    lib = tmp_path / "micro_sparsify.o"
    subprocess.run([cc, *build.COMMON, "-O1", "-g", *SAN, "-c", os.path.join(csrc, "micro_sparsify.cpp"),
                    "-o", str(lib)], check=True, capture_output=True, text=True)
    drv = tmp_path / "host_sanitize.o"
    subprocess.run([cc, "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror", f"-I{build.INCLUDE}", *SAN,
                    "-c", os.path.join(ROOT, "tests", "host_sanitize.cpp"), "-o", str(drv)],
                   check=True, capture_output=True, text=True)
    exe = tmp_path / "host_sanitize"
    subprocess.run([cc, f"--offload-arch={build.ARCH}", *SAN, str(drv), str(lib), *objs, "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=240, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert r.stdout.strip() == "ok"
    assert "runtime error" not in r.stderr
