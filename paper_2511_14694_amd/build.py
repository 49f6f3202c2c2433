"""Build libfocus.so (the FOCUS C-ABI library) for gfx950 with hipcc.

    python -m paper_2511_14694_amd.build          # or build() from Python

Every HIP source is compiled to an object under _build/ (in parallel), then the
objects are linked into paper_2511_14694_amd/libfocus.so next to this file.
Always rebuilds: it is the "does it compile" check as well as the build.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libfocus.so")
SOURCES = ["api.hip", "layout.hip", "compact.hip", "window_attn.hip", "decode.hip", "fidelity.hip", "gemm.hip", "adapter.hip"]

ARCH = "gfx950"
# Packed fp32 VALU ops are kept out of all device code (-packed-fp32-ops); the
# host pass warns that it does not know the feature, which is harmless.
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics", f"-I{INCLUDE}", f"-I{CSRC}",
]


# Per-source extra flags.  The attention kernels never see a NaN (finite
# inputs; masked scores are -inf), so their max reductions need no NaN
# canonicalisation (device code only: the host checks test for NaN).
EXTRA_FLAGS = {"window_attn.hip": ["-Xarch_device", "-fno-honor-nans"]}


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the FOCUS library needs ROCm's hipcc")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = [ln for ln in (res.stderr or "").splitlines()
             if "packed-fp32-ops" not in ln and ln.strip()]
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n" + "\n".join(noise))
    if verbose and noise:
        print("\n".join(noise), file=sys.stderr)


def build(verbose: bool = False, save_temps: bool = False) -> str:
    """Compile every HIP source and link libfocus.so; returns its path."""
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    jobs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        for src in SOURCES:
            obj = os.path.join(BUILD, src.replace(".hip", ".o"))
            objs.append(obj)
            cmd = [hipcc, *HIPCC_FLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
            if save_temps:
                cmd.insert(1, "-save-temps=obj")
            jobs.append(ex.submit(_run, cmd, verbose))
        for j in jobs:
            j.result()
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, save_temps="--save-temps" in sys.argv))
