"""Build step: compile the HIP kernels and C-ABI into libspecmoe_verify.so,
and the benchmark's streaming-read probe into its own libspecmoe_probe.so
(not part of the library).

Cross-compiles for gfx950 (MI355X) with hipcc; no GPU is needed to build.
Packed-FP32 instructions are disabled for all device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(HERE, "csrc", "verify_attn.hip"), os.path.join(HERE, "csrc", "accept.hip")]
INCLUDE = os.path.join(ROOT, "include")
OUTPUT = os.path.join(HERE, "libspecmoe_verify.so")
PROBE_SOURCES = [os.path.join(HERE, "csrc", "stream_probe.hip")]
PROBE_OUTPUT = os.path.join(HERE, "libspecmoe_probe.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build_command(output: str = OUTPUT, extra=(), sources=SOURCES):
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            f"-I{INCLUDE}", *extra, *sources, "-o", output]


def build(verbose: bool = False, output: str = OUTPUT) -> str:
    """Compile the library and the probe (always, even if builds are present);
    return the library's path."""
    _compile(SOURCES, output, verbose)
    _compile(PROBE_SOURCES, PROBE_OUTPUT, verbose)
    return output


def _compile(sources, output: str, verbose: bool) -> None:
    tmp = output + ".tmp"
    cmd = build_command(tmp, sources=sources)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    # every symbol must resolve: a kernel template whose host-side stub the
    # compiler silently failed to emit links fine but cannot be loaded
    check = subprocess.run([sys.executable, "-c", f"import ctypes; ctypes.CDLL({tmp!r})"],
                           capture_output=True, text=True)
    if check.returncode != 0:
        raise RuntimeError(f"built library does not load:\n{check.stderr.strip().splitlines()[-1]}")
    os.replace(tmp, output)


if __name__ == "__main__":
    print(build(verbose=True))
