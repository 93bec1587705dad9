"""Host-side checks of the C-ABI library (no GPU needed): it loads and exports
every symbol of include/gtp.h, its fp64 tables match closed forms derived from
the paper, its sampled three-step pipeline equals the oracle, and every invalid
argument is rejected before any HIP call."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from oracle import gtp_oracle as O
from paper_2401_10216_amd import gtp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def tri(l, m):
    return l * (l + 1) // 2 + m


@pytest.fixture(scope="module")
def L():
    return gtp.lib()


def test_exports_every_declared_symbol(L):
    header = open(os.path.join(ROOT, "include", "gtp.h")).read()
    names = set(re.findall(r"\b(gtp_[a-z0-9_]+)\s*\(", header))
    assert {"gtp_full", "gtp_sh2fourier", "gtp_fourier_conv", "gtp_fourier2sh", "gtp_selfproduct"} <= names
    for n in sorted(names):
        assert hasattr(L, n), n


def host_plan(L1, L2, Lout):
    return gtp.Plan(L1, L2, Lout, gtp.GTP_PLAN_HOST_ONLY)


def test_t1_closed_forms():
    p = host_plan(2, 2, 2)
    ld = 3  # rows hold u = 0..max(L1, L2, min(Lout, L1 + L2))
    T1 = p.table(0).reshape(-1, ld)
    c1 = math.sqrt(3 / (4 * math.pi))
    # Y_1^0 = c1 cos(t): a_1 = c1;  Y_1^1 theta factor = c1 sin(t): b_1 = c1
    assert abs(T1[tri(1, 0), 1] - c1) < 1e-15 and abs(T1[tri(1, 0), 0]) < 1e-15
    assert abs(T1[tri(1, 1), 1] - c1) < 1e-15
    # Y_0^0 = 1/sqrt(4 pi)
    assert abs(T1[tri(0, 0), 0] - 1 / math.sqrt(4 * math.pi)) < 1e-15
    # Y_2^0 = sqrt(5/(16 pi)) (3 cos^2 - 1) = sqrt(5/(16 pi)) (1/2 + 3/2 cos 2t)
    c2 = math.sqrt(5 / (16 * math.pi))
    assert abs(T1[tri(2, 0), 0] - 0.5 * c2) < 1e-15 and abs(T1[tri(2, 0), 2] - 1.5 * c2) < 1e-15
    # Y_2^2 theta factor = sqrt(15/(16 pi)) sin^2 = sqrt(15/(16 pi)) (1 - cos 2t)/2
    c22 = math.sqrt(15 / (16 * math.pi))
    assert abs(T1[tri(2, 2), 0] - 0.5 * c22) < 1e-15 and abs(T1[tri(2, 2), 2] + 0.5 * c22) < 1e-15


def test_z_tables_match_paper_closed_form():
    """2 pi (Zc + i sgn(u) Zs) for Y_0^0 is z^{0,0}_{u,0} of eq. fs-sh (golden values)."""
    import json
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "closed_forms.json")))["fourier2sh_z00"]["values"]
    p = host_plan(2, 2, 2)
    info = p.info()
    ldz = info["NT"] + 1
    Zc = p.table(1).reshape(-1, ldz)
    Zs = p.table(2).reshape(-1, ldz)
    for u, re_, im_ in g:
        au = abs(u)
        z = 2 * math.pi * (Zc[0, au] + 1j * np.sign(u) * Zs[0, au])
        assert abs(z - (re_ + 1j * im_)) < 1e-13, (u, z)


def test_sampling_tables_parity_and_poles():
    p = host_plan(6, 6, 6)
    info = p.info()
    NT, NJ = info["NT"], info["NT"] + 1
    S = p.table(3).reshape(-1, NJ)
    W = p.table(4).reshape(-1, NJ)
    for l in range(7):
        for m in range(l + 1):
            sg = (-1) ** (l + m)
            assert np.abs(S[tri(l, m)][::-1] - sg * S[tri(l, m)]).max() < 1e-13
            assert np.abs(W[tri(l, m)][::-1] - sg * W[tri(l, m)]).max() < 1e-15
            if m > 0:
                assert S[tri(l, m), 0] == 0 and S[tri(l, m), NT] == 0
    # S is the theta factor of the real SH at the nodes (pinned by the oracle's SH)
    th = np.arange(NJ) * math.pi / NT
    Y = O.real_sh(6, th, np.zeros_like(th))
    for l in range(7):
        assert np.abs(S[tri(l, 0)] - Y[:, l * l + l]).max() < 1e-13
        for m in range(1, l + 1):
            assert np.abs(S[tri(l, m)] - Y[:, l * l + l + m]).max() < 1e-13  # cos(0) = 1 at phi = 0


@pytest.mark.parametrize("L1,L2,Lout", [(0, 0, 0), (1, 0, 1), (2, 2, 2), (1, 3, 2), (3, 2, 6), (6, 6, 6),
                                         (2, 2, 3), (3, 2, 3), (5, 1, 4), (8, 8, 8), (4, 7, 2), (12, 12, 12)])
def test_host_pipeline_equals_oracle(L1, L2, Lout):
    rng = np.random.default_rng(100 + L1 + 13 * L2 + 169 * Lout)
    a = rng.standard_normal((6, O.nsh(L1)))
    b = rng.standard_normal((6, O.nsh(L2)))
    p = host_plan(L1, L2, Lout)
    y = gtp.gtp_debug_host_pipeline(p, a, b)
    ref = O.gtp(a, b, L1, L2, Lout) if max(L1, L2, Lout) <= 8 else O.gtp_grid(a, b, L1, L2, Lout)
    assert O.max_rel_err(y, ref) < 1e-12


def test_plan_info_geometry():
    p = host_plan(6, 6, 6)
    i = p.info()
    assert (i["U"], i["Le"], i["NT"], i["NP"]) == (12, 6, 13, 20)
    p = host_plan(2, 1, 7)
    i = p.info()
    assert (i["U"], i["Le"], i["NT"], i["NP"]) == (3, 3, 4, 8)
    assert p.grid_floats(1) == 2 * 25 and p.grid_floats(2) == 2 * 9 and p.grid_floats(3) == 2 * 49
    assert p.grid_floats(4) == -1


# ---------------------------------------------------------------- validation before any HIP call

def status(fn, *args):
    return fn(*args)


def test_plan_create_rejects_bad_degrees(L):
    h = ctypes.c_void_p()
    for args in [(-1, 2, 2), (2, -1, 2), (2, 2, -1), (65, 2, 2), (2, 65, 2), (2, 2, 65)]:
        assert L.gtp_plan_create(ctypes.byref(h), *args, gtp.GTP_PLAN_HOST_ONLY) == gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_plan_create(None, 1, 1, 1, gtp.GTP_PLAN_HOST_ONLY) == gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_plan_create(ctypes.byref(h), 1, 1, 1, 1 << 5 | 1 << 6) == gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_plan_create(ctypes.byref(h), 1, 1, 1, 1 << 10) == gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_plan_destroy(None) == gtp.GTP_OK


def test_plan_create_without_device_reports_no_device(L):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is visible")
    h = ctypes.c_void_p()
    assert L.gtp_plan_create(ctypes.byref(h), 2, 2, 2, 0) == gtp.GTP_ERR_NO_DEVICE
    assert b"device" in L.gtp_last_error()


def fake(addr):
    return ctypes.c_void_p(addr)


def test_full_validation(L):
    p = host_plan(2, 2, 2)
    H = p.handle
    x1, x2, y = fake(0x100000), fake(0x200000), fake(0x300000)
    S = ctypes.c_void_p(0)
    INV = gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_full(None, x1, x2, 0, 4, 4, y, S) == INV
    assert L.gtp_full(H, x1, x2, 7, 4, 4, y, S) == INV  # bad dtype
    assert L.gtp_full(H, x1, x2, 0, -1, 4, y, S) == INV
    assert L.gtp_full(H, x1, x2, 0, 4, -4, y, S) == INV
    assert L.gtp_full(H, x1, x2, 0, 1 << 40, 1 << 40, y, S) == INV  # B*C overflow
    assert L.gtp_full(H, x1, x2, 0, 1 << 30, 1 << 30, y, S) == INV  # B*C*K overflow
    assert L.gtp_full(H, None, x2, 0, 4, 4, y, S) == INV
    assert L.gtp_full(H, x1, None, 0, 4, 4, y, S) == INV
    assert L.gtp_full(H, x1, x2, 0, 4, 4, None, S) == INV
    assert L.gtp_full(H, x1, x2, 0, 4, 4, fake(0x100000 + 64), S) == INV  # y overlaps x1
    assert L.gtp_full(H, x1, x2, 0, 4, 4, fake(0x200000 - 16), S) == INV  # y overlaps x2 from below
    assert L.gtp_full(H, fake(0x100002), x2, 0, 4, 4, y, S) == INV  # misaligned f32
    assert L.gtp_full(H, x1, x2, 0, 0, 4, y, S) == gtp.GTP_OK  # empty batch is a no-op
    assert L.gtp_full(H, None, None, 0, 4, 0, None, S) == gtp.GTP_OK
    # a valid call on a host-only plan is refused after validation
    assert L.gtp_full(H, x1, x2, 0, 4, 4, y, S) == INV
    assert b"HOST_ONLY" in L.gtp_last_error()


def test_backward_validation(L):
    p = host_plan(2, 3, 4)
    H = p.handle
    x1, x2, dy, d1, d2 = fake(0x100000), fake(0x200000), fake(0x300000), fake(0x400000), fake(0x500000)
    S = ctypes.c_void_p(0)
    INV, OK = gtp.GTP_ERR_INVALID_ARG, gtp.GTP_OK
    f = L.gtp_full_backward
    assert f(None, x1, x2, 0, dy, 4, 4, d1, d2, S) == INV
    assert f(H, x1, x2, 3, dy, 4, 4, d1, d2, S) == INV  # bad dtype
    assert f(H, x1, x2, 0, dy, -1, 4, d1, d2, S) == INV
    assert f(H, x1, x2, 0, dy, 1 << 30, 1 << 30, d1, d2, S) == INV  # size overflow
    assert f(H, x1, x2, 0, None, 4, 4, d1, d2, S) == INV  # dy NULL
    assert f(H, x1, None, 0, dy, 4, 4, d1, None, S) == INV  # dx1 needs x2
    assert f(H, None, x2, 0, dy, 4, 4, None, d2, S) == INV  # dx2 needs x1
    assert f(H, x1, x2, 0, dy, 4, 4, fake(0x300000 + 8), d2, S) == INV  # dx1 overlaps dy
    assert f(H, x1, x2, 0, dy, 4, 4, d1, fake(0x200000 + 4), S) == INV  # dx2 overlaps x2
    assert f(H, x1, x2, 0, dy, 4, 4, d1, fake(0x400000 + 4 * 16 * 9 - 4), S) == INV  # dx1 overlaps dx2
    assert f(H, x1, x2, 0, dy, 4, 4, fake(0x400002), d2, S) == INV  # misaligned
    assert f(H, x1, x2, 0, dy, 0, 4, d1, d2, S) == OK  # empty batch
    assert f(H, x1, x2, 0, dy, 4, 4, None, None, S) == OK  # nothing requested
    assert f(H, None, x2, 0, dy, 4, 4, d1, None, S) == INV  # valid, but the plan is host-only
    assert b"HOST_ONLY" in L.gtp_last_error()


def test_weighted_validation(L):
    p = host_plan(2, 3, 4)
    H = p.handle
    x1, x2, y, w1, w2, wo = (fake(a) for a in (0x100000, 0x200000, 0x300000, 0x400000, 0x500000, 0x600000))
    S = ctypes.c_void_p(0)
    INV, OK = gtp.GTP_ERR_INVALID_ARG, gtp.GTP_OK
    f = L.gtp_full_weighted
    assert f(None, x1, x2, 0, w1, w2, wo, 0, 4, 4, y, S) == INV
    assert f(H, x1, x2, 2, w1, w2, wo, 0, 4, 4, y, S) == INV  # bad dtype
    assert f(H, x1, x2, 0, w1, w2, wo, 2, 4, 4, y, S) == INV  # per_channel not 0/1
    assert f(H, x1, x2, 0, w1, w2, wo, 0, -4, 4, y, S) == INV
    assert f(H, None, x2, 0, w1, w2, wo, 0, 4, 4, y, S) == INV
    assert f(H, x1, x2, 0, w1, w2, wo, 0, 4, 4, None, S) == INV
    assert f(H, x1, x2, 0, fake(0x300000 + 4), w2, wo, 0, 4, 4, y, S) == INV  # y overlaps w1
    assert f(H, x1, x2, 0, w1, w2, fake(0x300000 - 8), 0, 4, 4, y, S) == INV  # wout (5 floats) runs into y
    # wout's 5 floats end exactly where y starts: valid, refused only for the host-only plan
    assert f(H, x1, x2, 0, w1, w2, fake(0x300000 - 20), 0, 4, 4, y, S) == INV
    assert b"HOST_ONLY" in L.gtp_last_error()
    assert f(H, x1, x2, 0, w1, fake(0x500002), wo, 0, 4, 4, y, S) == INV  # misaligned weight
    assert f(H, x1, x2, 0, w1, w2, wo, 1, 0, 4, y, S) == OK  # empty batch
    # valid arguments (NULL weights are ones) on a host-only plan: refused after validation
    assert f(H, x1, x2, 0, None, None, None, 0, 4, 4, y, S) == INV
    assert b"HOST_ONLY" in L.gtp_last_error()


def test_channel_mix_validation(L):
    p = host_plan(2, 2, 2)
    H = p.handle
    x1, x2, W, y = fake(0x100000), fake(0x200000), fake(0x300000), fake(0x400000)
    S = ctypes.c_void_p(0)
    INV, OK = gtp.GTP_ERR_INVALID_ARG, gtp.GTP_OK
    f = L.gtp_channel_mix
    assert f(None, x1, x2, 0, W, 4, 3, 5, 2, y, S) == INV
    assert f(H, x1, x2, 4, W, 4, 3, 5, 2, y, S) == INV  # bad dtype
    assert f(H, x1, x2, 0, W, -1, 3, 5, 2, y, S) == INV
    assert f(H, x1, x2, 0, W, 4, 3, -5, 2, y, S) == INV
    assert f(H, x1, x2, 0, W, 4, 1 << 40, 1 << 40, 2, y, S) == INV  # C1 C2 overflow
    assert f(H, x1, x2, 0, None, 4, 3, 5, 2, y, S) == INV  # W needed when C1 C2 > 0
    assert f(H, None, x2, 0, W, 4, 3, 5, 2, y, S) == INV
    assert f(H, x1, x2, 0, W, 4, 3, 5, 2, None, S) == INV
    assert f(H, x1, x2, 0, W, 4, 3, 5, 2, fake(0x300000 + 8), S) == INV  # y overlaps W
    assert f(H, x1, x2, 0, W, 4, 3, 5, 2, fake(0x100000 + 4), S) == INV  # y overlaps x1
    assert f(H, x1, x2, 0, fake(0x300002), 4, 3, 5, 2, y, S) == INV  # misaligned
    assert f(H, x1, x2, 0, W, 0, 3, 5, 2, y, S) == OK  # empty batch
    assert f(H, x1, x2, 0, W, 4, 3, 5, 0, y, S) == OK  # no output channels
    assert f(H, None, None, 0, None, 4, 0, 5, 2, y, S) == INV  # C1 = 0: zeros, but the plan is host-only
    assert b"HOST_ONLY" in L.gtp_last_error()


def test_stage_validation(L):
    p = host_plan(2, 3, 2)
    H = p.handle
    a, b, c = fake(0x100000), fake(0x200000), fake(0x300000)
    S = ctypes.c_void_p(0)
    INV = gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_sh2fourier(H, 3, a, 0, 4, b, S) == INV
    assert L.gtp_sh2fourier(H, 1, a, 9, 4, b, S) == INV
    assert L.gtp_sh2fourier(H, 1, a, 0, -2, b, S) == INV
    assert L.gtp_sh2fourier(H, 1, a, 0, 4, fake(0x100000 + 8), S) == INV
    assert L.gtp_sh2fourier(H, 1, a, 0, 0, b, S) == gtp.GTP_OK
    assert L.gtp_fourier_conv(H, a, b, -1, c, S) == INV
    assert L.gtp_fourier_conv(H, a, b, 4, fake(0x200000 + 8), S) == INV
    assert L.gtp_fourier_conv(H, None, b, 4, c, S) == INV
    assert L.gtp_fourier2sh(H, a, 4, fake(0x100000 + 4), S) == INV
    assert L.gtp_fourier2sh(H, a, 4, None, S) == INV
    assert L.gtp_fourier2sh(None, a, 4, c, S) == INV


def test_selfproduct_and_filter_validation(L):
    a, c = fake(0x100000), fake(0x300000)
    S = ctypes.c_void_p(0)
    INV = gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_selfproduct(-1, 3, 3, 0, a, 0, 4, 4, c, S) == INV
    assert L.gtp_selfproduct(2, 0, 3, 0, a, 0, 4, 4, c, S) == INV
    assert L.gtp_selfproduct(2, 3, 3, 7, a, 0, 4, 4, c, S) == INV
    assert L.gtp_selfproduct(2, 3, 3, 0, a, 5, 4, 4, c, S) == INV
    assert L.gtp_selfproduct(2, 3, 3, 0, a, 0, 4, 4, fake(0x100000 + 4), S) == INV
    assert L.gtp_selfproduct(2, 3, 3, 0, None, 0, 4, 4, c, S) == INV
    assert L.gtp_selfproduct(22, 3, 3, 1, a, 0, 4, 4, c, S) == gtp.GTP_ERR_UNSUPPORTED
    assert L.gtp_selfproduct(2, 3, 3, 0, a, 0, 0, 4, c, S) == gtp.GTP_OK
    assert L.gtp_sh_filter(-1, a, None, 4, 1, c, S) == INV
    assert L.gtp_sh_filter(65, a, None, 4, 1, c, S) == INV
    assert L.gtp_sh_filter(3, a, None, 4, 2, c, S) == INV  # h NULL needs C == 1
    assert L.gtp_sh_filter(3, None, None, 4, 1, c, S) == INV
    assert L.gtp_sh_filter(3, a, None, 4, 1, fake(0x100000 + 4), S) == INV
    assert L.gtp_sh_filter(3, a, None, 0, 1, c, S) == gtp.GTP_OK


def test_status_strings(L):
    for s, name in gtp._STATUS.items():
        assert L.gtp_status_str(s).decode() == name
    assert L.gtp_status_str(99).decode() == "GTP_ERR_UNKNOWN"


def test_alignment_checked_everywhere(L):
    """Every entry point refuses a pointer that is not a multiple of its
    element size (2 bytes for bf16 inputs, 4 for fp32 data) before any HIP
    call."""
    p = host_plan(2, 3, 2)
    H = p.handle
    a, b, c = fake(0x100000), fake(0x200000), fake(0x300000)
    S = ctypes.c_void_p(0)
    INV = gtp.GTP_ERR_INVALID_ARG

    def misaligned(status):
        return status == INV and b"misaligned" in L.gtp_last_error()

    assert misaligned(L.gtp_sh2fourier(H, 1, fake(0x100002), 0, 4, b, S))  # f32 x
    assert misaligned(L.gtp_sh2fourier(H, 1, fake(0x100001), 1, 4, b, S))  # bf16 x
    assert misaligned(L.gtp_sh2fourier(H, 1, a, 0, 4, fake(0x200002), S))  # grid
    assert not misaligned(L.gtp_sh2fourier(H, 1, fake(0x100002), 1, 4, b, S))  # bf16 at 2 bytes is fine
    assert misaligned(L.gtp_fourier_conv(H, a, fake(0x200001), 4, c, S))
    assert misaligned(L.gtp_fourier_conv(H, a, b, 4, fake(0x300002), S))
    assert misaligned(L.gtp_fourier2sh(H, fake(0x100002), 4, c, S))
    assert misaligned(L.gtp_fourier2sh(H, a, 4, fake(0x300003), S))
    assert misaligned(L.gtp_selfproduct(2, 3, 3, 0, fake(0x100002), 0, 4, 4, c, S))
    assert misaligned(L.gtp_selfproduct(2, 3, 3, 0, fake(0x100001), 1, 4, 4, c, S))
    assert misaligned(L.gtp_selfproduct(2, 3, 3, 0, a, 0, 4, 4, fake(0x300002), S))
    assert misaligned(L.gtp_sh_filter(3, fake(0x100002), None, 4, 1, c, S))
    assert misaligned(L.gtp_sh_filter(3, a, fake(0x200001), 4, 2, c, S))
    assert misaligned(L.gtp_sh_filter(3, a, b, 4, 2, fake(0x300002), S))
    # the input size is bounded like the output size
    assert L.gtp_selfproduct(64, 2, 0, 0, a, 0, 1 << 25, 1 << 25, c, S) == INV


def test_fail_alloc_hook_reports_alloc_error(L, monkeypatch):
    """GTP_TEST_FAIL_ALLOC=host makes the fp64 table build fail as if out of
    memory: plan creation returns GTP_ERR_ALLOC with nothing leaked."""
    h = ctypes.c_void_p()
    monkeypatch.setenv("GTP_TEST_FAIL_ALLOC", "host")
    assert L.gtp_plan_create(ctypes.byref(h), 3, 3, 3, gtp.GTP_PLAN_HOST_ONLY) == gtp.GTP_ERR_ALLOC
    assert h.value is None
    assert b"allocation" in L.gtp_last_error()
    monkeypatch.delenv("GTP_TEST_FAIL_ALLOC")
    assert L.gtp_plan_create(ctypes.byref(h), 3, 3, 3, gtp.GTP_PLAN_HOST_ONLY) == gtp.GTP_OK
    assert L.gtp_plan_destroy(h) == gtp.GTP_OK


def test_noalloc_escn_validation(L):
    """gtp_conv_escn_noalloc shares gtp_conv_escn's checks and refuses, before
    any HIP call, an edge whose scratch needs exceed the static array."""
    x, r, h, y = fake(0x1000000), fake(0x2000000), fake(0x3000000), fake(0x40000000)
    S = ctypes.c_void_p(0)
    INV = gtp.GTP_ERR_INVALID_ARG
    f = L.gtp_conv_escn_noalloc
    p = host_plan(6, 6, 6)
    assert f(None, x, 0, r, h, 4, 4, y, S) == INV
    assert f(p.handle, x, 3, r, h, 4, 4, y, S) == INV
    assert f(p.handle, x, 0, r, h, -1, 4, y, S) == INV
    assert f(p.handle, x, 0, None, h, 4, 4, y, S) == INV
    assert f(p.handle, x, 0, r, h, 4, 4, fake(0x1000000 + 8), S) == INV  # y overlaps x
    assert f(p.handle, x, 0, fake(0x2000002), h, 4, 4, y, S) == INV  # misaligned r
    assert f(p.handle, x, 0, r, h, 0, 4, y, S) == gtp.GTP_OK
    assert f(p.handle, x, 0, r, h, 4, 4, y, S) == INV and b"HOST_ONLY" in L.gtp_last_error()
    q = host_plan(2, 64, 2)  # filter route: C * 65^2 * 4 bytes per edge
    C = (64 << 20) // (4 * 65 * 65) + 1
    assert f(q.handle, x, 0, r, h, 1, C, y, S) == gtp.GTP_ERR_UNSUPPORTED
    assert b"scratch" in L.gtp_last_error()
    # a huge channel count: refused without overflowing on the way
    assert f(q.handle, x, 0, r, fake(1 << 47), 1, 1 << 40, fake(1 << 50), S) == gtp.GTP_ERR_UNSUPPORTED
    assert f(q.handle, x, 0, r, h, 2, C - 1, y, S) == INV and b"HOST_ONLY" in L.gtp_last_error()


def test_compute_probe_validation(L):
    sink = fake(0x100000)
    fl = ctypes.c_double(0.0)
    INV = gtp.GTP_ERR_INVALID_ARG
    S = ctypes.c_void_p(0)
    assert L.gtp_compute_probe(2, 16, sink, ctypes.byref(fl), S) == INV
    assert L.gtp_compute_probe(-1, 16, sink, ctypes.byref(fl), S) == INV
    assert L.gtp_compute_probe(0, 0, sink, ctypes.byref(fl), S) == INV
    assert L.gtp_compute_probe(0, (1 << 30) + 1, sink, ctypes.byref(fl), S) == INV
    assert L.gtp_compute_probe(0, 16, None, ctypes.byref(fl), S) == INV
    assert L.gtp_compute_probe(1, 16, sink, None, S) == INV
    assert L.gtp_compute_probe(1, 16, fake(0x100002), ctypes.byref(fl), S) == INV  # misaligned


def test_stream_probe_validation(L):
    a, b = fake(0x100000), fake(0x200000)
    S = ctypes.c_void_p(0)
    INV = gtp.GTP_ERR_INVALID_ARG
    assert L.gtp_stream_probe(4, a, b, 64, S) == INV
    assert L.gtp_stream_probe(3, a, b, 48, S) == INV  # mode 3: a multiple of 32
    assert L.gtp_stream_probe(0, a, b, 20, S) == INV  # not a multiple of 16
    assert L.gtp_stream_probe(0, a, b, -16, S) == INV
    assert L.gtp_stream_probe(0, None, b, 64, S) == INV
    assert L.gtp_stream_probe(1, None, None, 64, S) == INV
    assert L.gtp_stream_probe(2, a, fake(0x100000 + 32), 64, S) == INV  # overlap
    assert L.gtp_stream_probe(3, a, fake(0x100000 + 32), 64, S) == INV  # dst inside src
    assert L.gtp_stream_probe(2, fake(0x100008), b, 64, S) == INV  # misaligned
    assert L.gtp_stream_probe(2, a, b, 0, S) == gtp.GTP_OK


def test_weighted_backward_validation(L):
    p = host_plan(2, 3, 4)
    H = p.handle
    x1, x2, dy = fake(0x100000), fake(0x200000), fake(0x300000)
    w1, w2, wo = fake(0x400000), fake(0x500000), fake(0x600000)
    d1, d2, g1, g2, go = fake(0x700000), fake(0x800000), fake(0x900000), fake(0xa00000), fake(0xb00000)
    S = ctypes.c_void_p(0)
    INV, OK = gtp.GTP_ERR_INVALID_ARG, gtp.GTP_OK
    f = L.gtp_full_weighted_backward
    assert f(None, x1, x2, 0, w1, w2, wo, 0, dy, 4, 4, d1, d2, g1, g2, go, S) == INV
    assert f(H, x1, x2, 5, w1, w2, wo, 0, dy, 4, 4, d1, d2, g1, g2, go, S) == INV  # dtype
    assert f(H, x1, x2, 0, w1, w2, wo, 2, dy, 4, 4, d1, d2, g1, g2, go, S) == INV  # per_channel
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, -4, 4, d1, d2, g1, g2, go, S) == INV
    assert f(H, None, x2, 0, w1, w2, wo, 0, dy, 4, 4, d1, d2, g1, g2, go, S) == INV
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, 4, 4, fake(0x300000 + 4), d2, g1, g2, go, S) == INV  # dx1 over dy
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, 4, 4, d1, d2, fake(0x400000), g2, go, S) == INV  # dw1 over w1
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, 4, 4, d1, d2, g1, fake(0x900000 + 4), go, S) == INV  # dw2 over dw1
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, 4, 4, d1, d2, g1, g2, fake(0xb00002), S) == INV  # misaligned
    assert f(H, x1, x2, 0, w1, w2, wo, 1, dy, 4, 1 << 17, None, None, g1, None, None, S) == gtp.GTP_ERR_UNSUPPORTED
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, 4, 4, None, None, None, None, None, S) == OK  # nothing requested
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, 0, 4, d1, d2, None, None, None, S) == OK  # empty, no weight grads
    assert f(H, x1, x2, 0, w1, w2, wo, 0, dy, 4, 4, d1, d2, g1, g2, go, S) == INV
    assert b"HOST_ONLY" in L.gtp_last_error()
