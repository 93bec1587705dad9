"""The radix-2 FFT pieces of the matrix-core kernel's FFT variant, built for
the host from the same header (gtp_fft.hpp) and checked against plain O(N^2)
DFT sums: complex transforms of both signs, the real forward transform and
the twiddle powers.  CPU only (hipcc compiles the host side)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2401_10216_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_register_fft_pieces(tmp_path):
    exe = str(tmp_path / "fft_host")
    cmd = [HIPCC, "-O2", "-std=c++17", "-x", "hip", "--offload-arch=gfx950", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "fft_host_main.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    lines = dict(ln.split() for ln in r.stdout.split("\n") if ln.strip())
    assert len(lines) == 12
