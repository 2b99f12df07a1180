"""The host side of the C ABI (argument checks, overlap sweep, gate decision, pool bookkeeping) built with
AddressSanitizer and UndefinedBehaviorSanitizer on the host pass only, and run on the CPU (no GPU call is made)."""
import os
import shutil
import subprocess

import pytest

from paper_2609_34060_amd import build as B

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs the HIP toolchain")
def test_host_abi_under_asan_and_ubsan(tmp_path):
    objs = [os.path.join(B.BUILD_DIR, os.path.splitext(s)[0] + ".o") for s in B.SOURCES if s != "kvc_api.cpp"]
    if not all(os.path.exists(o) for o in objs):
        pytest.skip("libkvc objects not built (run paper_2609_34060_amd/build.py)")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
           "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
    api_o = str(tmp_path / "kvc_api_san.o")
    drv_o = str(tmp_path / "abi_sanitize.o")
    exe = str(tmp_path / "abi_sanitize")
    flags = [*B.DEVICE_FLAGS, "-I", B.INCLUDE, "-I", B.CSRC]
    for cmd in ([B.hipcc(), *flags, *san, "-x", "hip", "-c", os.path.join(B.CSRC, "kvc_api.cpp"), "-o", api_o],
                [B.hipcc(), "-O1", "-std=c++17", "-I", B.INCLUDE, *san, "-c",
                 os.path.join(HERE, "native", "abi_sanitize.cpp"), "-o", drv_o],
                [B.hipcc(), "--offload-arch=gfx950", *san, drv_o, api_o, *objs, "-o", exe]):
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr[-3000:]
    assert "all host checks passed" in res.stdout
