"""Build libgtp.so (HIP kernels for gfx950 + fp64 host table builder + C ABI).

    python -m paper_2401_10216_amd.build [-v]

Objects go to ``_build/`` at the repository root; the library is written
in-tree as ``paper_2401_10216_amd/libgtp.so`` so it travels with the source
tree.  Always recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import time

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libgtp.so")

HIP_SOURCES = ["gtp_api.hip", "gtp_small.hip", "gtp_wave.hip", "gtp_generic.hip", "gtp_escn.hip", "gtp_escn_wave.hip",
               "gtp_mix.hip",
               "gtp_probe.hip", "gtp_wgrad.hip"]
CPP_SOURCES = ["gtp_tables.cpp", "gtp_escn_tables.cpp"]
ARCH = "gfx950"
# Packed fp32 VALU forms stay off: plain fp32 FMAs only.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-Wno-unused-command-line-argument", f"-I{os.path.join(ROOT, 'include')}"]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


GEN = os.path.join(BUILD, "gen")


def generate_constants(verbose: bool = False) -> None:
    """Compile and run the generator of the compile-time tables of the
    thread-per-product kernels (from the library's own fp64 table builders)."""
    os.makedirs(GEN, exist_ok=True)
    exe = os.path.join(BUILD, "gen_small_consts")
    cmd = ["g++", *CXX_FLAGS, "-o", exe, os.path.join(CSRC, "gen_small_consts.cpp"),
           os.path.join(CSRC, "gtp_tables.cpp"), os.path.join(CSRC, "gtp_escn_tables.cpp")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if verbose or r.returncode:
        print(" ".join(cmd))
        print(r.stdout, r.stderr)
    if r.returncode:
        raise RuntimeError("generator build failed")
    out = os.path.join(GEN, "gtp_small_consts.inc")
    out_e = os.path.join(GEN, "gtp_escn_consts.inc")
    r = subprocess.run([exe, out + ".tmp", out_e + ".tmp"], capture_output=True, text=True)
    if r.returncode:
        print(r.stdout, r.stderr)
        raise RuntimeError("generator failed")
    os.replace(out + ".tmp", out)
    os.replace(out_e + ".tmp", out_e)


POISON_BUILD = os.path.join(ROOT, "_build_poison")
POISON_LIB = os.path.join(PKG, "libgtp_poison.so")


def build(verbose: bool = False, poison: bool = True) -> str:
    """Compile and link libgtp.so and, with poison=True, the poisoned-LDS
    debug build libgtp_poison.so (-DGTP_POISON_LDS: every kernel fills its
    LDS with NaN before first use; the tests compare it with the regular
    build).  Both always recompile; at most 8 compilers run at once."""
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    generate_constants(verbose)
    variants = [(BUILD, LIB, [])] + ([(POISON_BUILD, POISON_LIB, ["-DGTP_POISON_LDS"])] if poison else [])
    jobs = []  # (cmd, obj, variant index)
    for vi, (bdir, _, extra) in enumerate(variants):
        os.makedirs(bdir, exist_ok=True)
        for s in HIP_SOURCES:
            obj = os.path.join(bdir, s.replace(".hip", ".o"))
            jobs.append(([hipcc, *HIP_FLAGS, *extra, f"-I{GEN}", "-c", os.path.join(CSRC, s), "-o", obj], obj, vi))
        for s in CPP_SOURCES:
            obj = os.path.join(bdir, s.replace(".cpp", ".o"))
            jobs.append((["g++", *CXX_FLAGS, "-c", os.path.join(CSRC, s), "-o", obj], obj, vi))
    t0 = time.time()
    failed = []
    running = []
    pending = sorted(jobs, key=lambda j: 0 if "gtp_small" in j[1] else 1)  # the longest first
    while pending or running:
        while pending and len(running) < 8:
            cmd, obj, vi = pending.pop(0)
            running.append((subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True), cmd,
                            obj))
        p, cmd, obj = running.pop(0)
        out, _ = p.communicate()
        if verbose or p.returncode:
            print(" ".join(cmd))
            if out:
                print(out)
        if p.returncode:
            failed.append(obj)
    if failed:
        raise RuntimeError(f"compilation failed: {failed}")
    for vi, (bdir, lib, _) in enumerate(variants):
        tmp = lib + ".tmp"
        link = [hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *[o for _, o, v in jobs if v == vi]]
        r = subprocess.run(link, capture_output=True, text=True)
        if r.returncode:
            print(" ".join(link))
            print(r.stdout, r.stderr)
            raise RuntimeError("link failed")
        os.replace(tmp, lib)
        if verbose:
            print(f"built {lib} in {time.time() - t0:.1f}s")
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv, poison="--no-poison" not in sys.argv)
