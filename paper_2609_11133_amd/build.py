"""Build the HIP library ``libmoe_decode.so`` for gfx950 with hipcc (in-tree)."""
from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmoe_decode.so")
PROBE = os.path.join(PKG, "stream_probe")
SOURCES = ["route.hip", "expert.hip", "mfma.hip", "nvfp4.hip", "attn.hip", "api.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    "-O3",
    f"--offload-arch={ARCH}",
    "-fPIC",
    "-std=c++17",
    "-Wall",
    "-Wno-unused-function",
    # packed fp32 instructions disabled (v_pk_{add,mul,fma}_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(force: bool = True) -> str:
    """Compile every HIP source for gfx950 and link ``libmoe_decode.so``."""
    if not force and os.path.exists(LIB):
        return LIB
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    r = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


def build_probe() -> str:
    """The HBM streaming reference executable: measurement tooling, not part of the
    library.  Its runs give the streaming ceilings and the copy-kernel scale of the
    FETCH_SIZE / WRITE_SIZE counters that the traffic profiles are normalised by;
    built on request only (``python -m paper_2609_11133_amd.build --probe``)."""
    tmp = PROBE + ".tmp"
    r = subprocess.run([HIPCC, *FLAGS, os.path.join(CSRC, "stream_probe.hip"), "-o", tmp], capture_output=True,
                       text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for stream_probe.hip:\n{r.stderr}")
    os.replace(tmp, PROBE)
    return PROBE


if __name__ == "__main__":
    import sys

    print(build_probe() if "--probe" in sys.argv[1:] else build())
