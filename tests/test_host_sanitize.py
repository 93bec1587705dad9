"""AddressSanitizer + UndefinedBehaviorSanitizer build of the host code that
validates nothing on the device: the fp64 table builders (gtp_tables.cpp,
gtp_escn_tables.cpp) and the build-time constant generator
(gen_small_consts.cpp), each run under the sanitizers.  CPU only (g++)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2401_10216_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1",
       "-std=c++17"]


def _build(tmp_path, name, sources):
    exe = str(tmp_path / name)
    cmd = ["g++", *SAN, f"-I{CSRC}", "-o", exe, *sources]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def _env():
    env = dict(os.environ)
    # a library preloaded by the environment may come before the ASan runtime
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:halt_on_error=1:verify_asan_link_order=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_table_builders_clean_under_sanitizers(tmp_path):
    exe = _build(tmp_path, "host_sanitize", [os.path.join(ROOT, "tests", "host_sanitize_main.cpp"),
                                             os.path.join(CSRC, "gtp_tables.cpp"),
                                             os.path.join(CSRC, "gtp_escn_tables.cpp")])
    r = subprocess.run([exe], capture_output=True, text=True, env=_env(), timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
    assert r.stdout.count("ok ") == 19


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_constant_generator_clean_under_sanitizers(tmp_path):
    exe = _build(tmp_path, "gen_small_consts", [os.path.join(CSRC, "gen_small_consts.cpp"),
                                                os.path.join(CSRC, "gtp_tables.cpp"),
                                                os.path.join(CSRC, "gtp_escn_tables.cpp")])
    out1, out2 = tmp_path / "s.inc", tmp_path / "e.inc"
    r = subprocess.run([exe, str(out1), str(out2)], capture_output=True, text=True, env=_env(), timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr
    # the sanitized generator writes the same constants as the library build's
    built = os.path.join(ROOT, "_build", "gen", "gtp_small_consts.inc")
    if os.path.exists(built):
        assert out1.read_text() == open(built).read()
