"""Build the gfx950 decode-attention library in-tree (hipcc, no JIT cache)."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "librl_decode_attn.so")
SOURCES = [os.path.join(CSRC, "rlda_kernels.hip"), os.path.join(CSRC, "rlda_multi.hip"),
           os.path.join(CSRC, "rlda_host.cpp")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Read-bandwidth reference kernels (bench support, not the attention path).
PROBE_SOURCES = [os.path.join(CSRC, "hbm_probe.hip")]
PROBE_LIB = os.path.join(HERE, "libhbm_probe.so")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I", INCLUDE, "-I", CSRC,
]


def build(verbose: bool = False, out: str = LIB, defines=(), sources=None) -> str:
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-D" + d for d in defines] + (sources or SOURCES) + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if noise not in ln]
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), flush=True)
    os.replace(tmp, out)
    return out


def device_asm(out_path: str, source: int = 0) -> str:
    """Write the gfx950 assembly of one kernel source (for register / spill review)."""
    cmd = [HIPCC] + [f for f in FLAGS if f not in ("-shared", "-fPIC")] + [
        "--cuda-device-only", "-S", SOURCES[source], "-o", out_path]
    subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
    return out_path


def build_all(verbose: bool = False) -> None:
    """The attention library and the read-bandwidth probe library."""
    build(verbose=verbose)
    build(verbose=verbose, out=PROBE_LIB, sources=PROBE_SOURCES)


if __name__ == "__main__":
    build_all(verbose="-v" in sys.argv)
    print(LIB)
    print(PROBE_LIB)
