"""Build libspdp.so (HIP for gfx950 + host C++) in-tree with hipcc.

Run ``python -m paper_2607_21985_amd.build`` (or call ``build()``). The
library lands next to this file so that it travels with the source tree.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libspdp.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libspdp)")


PEAK_LIB = os.path.join(HERE, "libspdp_peak.so")


def build(verbose: bool = False) -> str:
    """Compile every source of the library (and the benchmark's read-roof
    kernel, libspdp_peak.so); always rebuilds. Returns the library's path."""
    cc = hipcc()
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    common = ["-O3", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC, "-Wall"]
    # Packed fp32 VALU ops are kept off for all device code.
    device = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    jobs = [
        ([cc, "-x", "c++"] + common + ["-c", os.path.join(CSRC, "host.cpp"),
                                       "-o", os.path.join(objdir, "host.o")]),
        # the 4x4x4 MFMA accumulators of the batched decode stay in VGPRs
        # (the AGPR form would add registers and moves and cost occupancy)
        ([cc] + common + device + ["-mllvm", "-amdgpu-mfma-vgpr-form=true", "-c", os.path.join(CSRC, "spdp.hip"),
                                   "-o", os.path.join(objdir, "spdp.o")]),
        ([cc] + common + device + ["-c", os.path.join(CSRC, "spmm.hip"),
                                   "-o", os.path.join(objdir, "spmm.o")]),
    ]
    # the sources compile concurrently (the decode kernels' instantiations
    # take most of the time)
    procs = []
    for cmd in jobs:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    failed = None
    for cmd, proc in procs:
        text, _ = proc.communicate()
        out = "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)
        if proc.returncode != 0 and failed is None:
            failed = f"compile failed: {' '.join(cmd)}\n{out}"
        if verbose and out.strip():
            print(out, flush=True)
    if failed:
        raise RuntimeError(failed)
    tmp = LIB + ".tmp"
    link = [cc, "-shared", f"--offload-arch={ARCH}", "-o", tmp,
            os.path.join(objdir, "host.o"), os.path.join(objdir, "spdp.o"), os.path.join(objdir, "spmm.o"),
            "-lpthread"]
    res = subprocess.run(link, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(link)}\n{res.stdout}{res.stderr}")
    os.replace(tmp, LIB)
    # the benchmark's streaming-read roof: its own small library
    tmp = PEAK_LIB + ".tmp"
    peak = [cc] + common + device + ["-shared", "-o", tmp, os.path.join(CSRC, "peak.hip")]
    res = subprocess.run(peak, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(peak)}\n{res.stdout}{res.stderr}")
    os.replace(tmp, PEAK_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
