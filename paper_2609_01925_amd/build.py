"""Builds libcrisp.so (the HIP kernels and the C ABI) for gfx950 with hipcc, and
libcrisp_debug.so, built with CRISP_DEBUG: device-side checks of the inputs before
each call's kernels, and the attention's tile pipeline serialised (a race check).

    python -m paper_2609_01925_amd.build

Sources are compiled in parallel into _build/ and linked in-tree next to this
file, so the library travels with the source tree.
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
LIB = os.path.join(PKG, "libcrisp.so")
LIB_DEBUG = os.path.join(PKG, "libcrisp_debug.so")  # CRISP_DEBUG: device-side input checks
# measurement only: MFMA and copy peak-rate microbenchmarks that the benchmark reports
# beside the published peaks (not part of the CRISP path)
PEAKS_SRC = os.path.join(PKG, "peaks", "peaks.hip")
LIB_PEAKS = os.path.join(PKG, "libcrisp_peaks.so")
ARCH = "gfx950"

# Packed fp32 VALU forms are kept out of every kernel: the compiler would
# otherwise form them from ordinary float code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall", "-Wno-unused-function"]
# Per-source device flags.  The attention and estimator kernels keep their MFMA
# results (scores, read by the softmax every tile, and the output accumulators) in
# VGPRs; left to itself the compiler places them in AGPRs and copies every score out
# again.
EXTRA = {"attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"], "estimate.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libcrisp)")


def sources():
    hip = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    cpp = sorted(f for f in os.listdir(CSRC) if f.endswith(".cpp"))
    return hip, cpp


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in p.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in line)
    return p.returncode, " ".join(cmd), out


def build(verbose: bool = False) -> str:
    """Compile every source and link libcrisp.so; returns its path.  Raises on failure."""
    cc = hipcc()
    os.makedirs(BUILD, exist_ok=True)
    hip, cpp = sources()
    jobs = []
    for f in hip:
        obj = os.path.join(BUILD, f[:-4] + ".o")
        jobs.append([cc, f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS, *EXTRA.get(f, []), "-c",
                     os.path.join(CSRC, f), "-o", obj])
    for f in cpp:
        obj = os.path.join(BUILD, f[:-4] + ".o")
        jobs.append([cc, f"--offload-arch={ARCH}", *COMMON, "-c", os.path.join(CSRC, f), "-o", obj])
    # the debug library: host layer with input checks, attention with its tile
    # pipeline serialised (the other kernels are the release objects)
    debug_jobs = [[cc, f"--offload-arch={ARCH}", *COMMON, "-DCRISP_DEBUG=1", "-c", os.path.join(CSRC, f),
                   "-o", os.path.join(BUILD, f[:-4] + "_debug.o")] for f in cpp]
    debug_jobs.append([cc, f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS, *EXTRA.get("attn.hip", []),
                       "-DCRISP_DEBUG=1", "-c", os.path.join(CSRC, "attn.hip"), "-o", os.path.join(BUILD, "attn_debug.o")])
    peaks_job = [cc, f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS, "-c", PEAKS_SRC,
                 "-o", os.path.join(BUILD, "peaks.o")]
    workers = min(len(jobs) + len(debug_jobs) + 1, max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(_run, jobs + debug_jobs + [peaks_job]))
    bad = [(cmd, out) for rc, cmd, out in results if rc != 0]
    if verbose or bad:
        for rc, cmd, out in results:
            if out.strip():
                print(out, file=sys.stderr)
    if bad:
        raise RuntimeError("libcrisp compile failed:\n" + "\n".join(f"$ {c}\n{o}" for c, o in bad))
    objs = [j[-1] for j in jobs]
    replaced = {f[:-4] + ".o" for f in cpp} | {"attn.o"}
    debug_objs = [o for o in objs if os.path.basename(o) not in replaced] + [j[-1] for j in debug_jobs]
    for target, members in ((LIB, objs), (LIB_DEBUG, debug_objs), (LIB_PEAKS, [peaks_job[-1]])):
        tmp = target + ".tmp"
        rc, cmd, out = _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *members, "-o", tmp])
        if rc != 0:
            raise RuntimeError(f"libcrisp link failed:\n$ {cmd}\n{out}")
        os.replace(tmp, target)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
