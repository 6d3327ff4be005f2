"""Build libda2.so (all HIP kernels and the host library) for gfx950 in-tree.

Run ``python -m paper_2609_32628_amd.build`` (or call ``build()``); the
result is ``paper_2609_32628_amd/libda2.so``.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libda2.so")
BUILD = os.path.join(HERE, "_build")
SOURCES = ["host.cpp", "draft.hip", "rank.hip", "prep.hip", "attn.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++20",
    "-ffp-contract=off",                          # encoders round every operation once
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",         # keep MFMA accumulators in VGPRs (no AGPR copies)
    "-Wno-unused-command-line-argument",
]


# The attention and draft kernels never produce NaN (finite operands, -inf only
# for masked logits and padding), so max/min need no NaN canonicalization there.
EXTRA = {"attn.hip": ["-fno-honor-nans"], "draft.hip": ["-fno-honor-nans"]}


def _compile(src):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


PROBE_SRC = os.path.join(os.path.dirname(HERE), "tests", "probes", "fmt_probe.hip")
PROBE_OUT = os.path.join(os.path.dirname(HERE), "tests", "probes", "libda2_probe.so")


def build_probe():
    """Device format probe used by the GPU tests (test infrastructure)."""
    if not os.path.exists(PROBE_SRC):
        return None
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-shared", PROBE_SRC, "-o", PROBE_OUT + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for the probe:\n{r.stdout}\n{r.stderr}")
    os.replace(PROBE_OUT + ".tmp", PROBE_OUT)
    return PROBE_OUT


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, OUT)
    build_probe()
    if verbose:
        print("built", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
