"""Build libkvx.so (the C-ABI copy engine) for gfx950 with hipcc.

``python -m paper_2606_31093_amd.build_lib`` rebuilds it in place; extra
``-D`` defines (tuning knobs of the kernels) can be passed for experiments,
with a different output path.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libkvx.so")
# The test build: its hash chain gives up after one empty poll, and planned
# transfers of any size take the sweep launch (its launch choice starts as
# KVX_CHOOSE_SWEEP), with at most 2048 workgroups, so that larger cases loop
# over page slots.  These are compile-time options: the product library has
# no switch for them.
TEST_LIBRARY = os.path.join(PKG, "libkvx_test.so")
TEST_DEFINES = ("KVX_HASH_IDLE_POLLS=1", "KVX_SWEEP_MIN_BYTES=0", "KVX_SWEEP_MAX_BLOCKS=2048",
                "KVX_LAUNCH_CHOICE_DEFAULT=1")
SOURCES = [os.path.join(CSRC, "kvx_kernels.hip"), os.path.join(CSRC, "kvx_hash.hip"),
           os.path.join(CSRC, "kvx_api.cpp")]
HEADERS = [os.path.join(INCLUDE, "kvx.h"), os.path.join(CSRC, "kvx_internal.h"),
           os.path.join(CSRC, "kvx_hash.h")]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def command(output: str = LIBRARY, defines=()) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            # no packed-FP32 instructions anywhere (the kernels have no float math)
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-I", INCLUDE, "-I", CSRC,
            *[f"-D{d}" for d in defines], "-o", output, *SOURCES]


def build(output: str = LIBRARY, defines=(), quiet: bool = True) -> str:
    tmp = f"{output}.tmp{os.getpid()}"
    r = subprocess.run(command(tmp, defines), capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed:\n{r.stdout}\n{r.stderr}")
    if not quiet:
        sys.stderr.write(r.stderr)
    os.replace(tmp, output)
    return output


def is_stale(output: str = LIBRARY) -> bool:
    if not os.path.exists(output):
        return True
    t = os.path.getmtime(output)
    return any(os.path.getmtime(s) > t for s in SOURCES + HEADERS)


def build_all() -> list:
    """The library and its test build."""
    return [build(), build(TEST_LIBRARY, TEST_DEFINES)]


if __name__ == "__main__":
    defs = [a[2:] for a in sys.argv[1:] if a.startswith("-D")]
    outs = [a for a in sys.argv[1:] if not a.startswith("-D")]
    print(build(outs[0] if outs else LIBRARY, defs, quiet=False))
