"""Builds libcis.so (the HIP kernels and the C ABI) in-tree for gfx950 with hipcc.

    python -m paper_2609_32444_amd.build      # or: from paper_2609_32444_amd.build import build
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_PATH = os.path.join(HERE, "libcis.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in
           ("cis_kernels.hip", "cis_kernels_ext.hip", "cis_gemm.hip", "cis_api.cpp")]
# bandwidth probes for the roofline (a separate library; not part of the loss)
PROBE_PATH = os.path.join(HERE, "libcis_probe.so")
PROBE_SOURCES = [os.path.join(HERE, "csrc", "bw_probe.hip")]
HEADERS = [os.path.join(ROOT, "include", "cis.h"), os.path.join(HERE, "csrc", "cis_internal.h"),
           os.path.join(HERE, "csrc", "cis_row.h"), os.path.join(HERE, "csrc", "cis_gemm.h")]

# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in device code (the compiler's host pass warns
# that it does not know the feature; that warning is expected).
HIPCC_FLAGS = [
    "-x", "hip", "--offload-arch=gfx950", "-O3", "-std=c++20", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def _report(proc, verbose):
    if proc.returncode != 0:
        sys.stderr.write(proc.stdout + proc.stderr)
        raise RuntimeError(f"hipcc failed with status {proc.returncode}")
    if verbose:
        noise = "'-packed-fp32-ops' is not a recognized feature"
        out = "\n".join(l for l in (proc.stdout + proc.stderr).splitlines() if noise not in l)
        if out.strip():
            print(out)


def _compile(sources, out_path, verbose):
    """Compiles each source to an object file in parallel, then links the shared library."""
    tmp = out_path + ".tmp"
    objs = [f"{out_path}.{i}.o" for i in range(len(sources))]
    procs = [subprocess.Popen([hipcc(), *HIPCC_FLAGS, "-c", src, "-o", obj],
                              stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
             for src, obj in zip(sources, objs)]
    try:
        for p in procs:
            out, err = p.communicate()
            _report(subprocess.CompletedProcess(p.args, p.returncode, out, err), verbose)
        link = subprocess.run([hipcc(), "--offload-arch=gfx950", "-shared", *objs, "-o", tmp],
                              capture_output=True, text=True)
        _report(link, verbose)
    finally:
        for p in procs:
            if p.poll() is None:
                p.kill()
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    os.replace(tmp, out_path)


def build(verbose: bool = False) -> str:
    """Compiles libcis.so and libcis_probe.so; always recompiles. Returns libcis.so's path."""
    _compile(SOURCES, LIB_PATH, verbose)
    _compile(PROBE_SOURCES, PROBE_PATH, verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
