"""The host library (argument validation, sizes, offsets, region layouts) built
with AddressSanitizer and UndefinedBehaviorSanitizer on its host code only
(the device code is compiled as usual), driven by tests/sanitize/host_abi_check.cpp
on the CPU: every query and every validation error path, no kernel launched.
Any sanitizer report aborts the driver."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_32628_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="CPU-only check (the driver expects no device)")
def test_host_library_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "host_abi_check"
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++20", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-Wno-unused-command-line-argument", *san]
    objs = []
    for f in ("host.cpp", "draft.hip", "rank.hip", "prep.hip", "attn.hip"):
        o = tmp_path / (f + ".o")
        r = subprocess.run([HIPCC, *flags, "-x", "hip", "-c", os.path.join(CSRC, f), "-o", str(o)],
                           capture_output=True, text=True, timeout=900)
        assert r.returncode == 0, (f, r.stderr[-3000:])
        objs.append(str(o))
    drv = tmp_path / "host_abi_check.o"
    r = subprocess.run([HIPCC, *flags, "-x", "c++", "-c", os.path.join(ROOT, "tests", "sanitize", "host_abi_check.cpp"),
                        "-o", str(drv)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", *san, *objs, str(drv), "-o", str(exe)],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "host ABI checks passed" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
