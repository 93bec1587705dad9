"""Poisoned-LDS debug build against the regular build.

libgtp_poison.so is the library compiled with -DGTP_POISON_LDS: every kernel
fills its LDS with a quiet NaN before first use, so a kernel that reads LDS
it has not written (a race between waves, a missing barrier or wait, an
index past what was staged) returns NaN or other values than the regular
build.  Every kernel family runs here once through each build on the same
inputs (ragged sizes, both input types, the padded and companion-plan
routes); the outputs must be finite and agree with the regular build's to
1e-6 of the output norm.
"""
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import gtp_oracle as O  # noqa: E402
from paper_2401_10216_amd import gtp  # noqa: E402

pytestmark = pytest.mark.gpu

POISON_LIB = os.path.join(os.path.dirname(gtp.__file__), "libgtp_poison.so")


def _say(msg):
    print(msg, flush=True)


def _dev(a, bf16=False):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    return t.to(torch.bfloat16) if bf16 else t


def _both(run):
    """run() with the regular build, then inside the poisoned-LDS build."""
    a = run()
    torch.cuda.synchronize()
    with gtp.use_library(POISON_LIB):
        b = run()
        torch.cuda.synchronize()
    return a, b


def _agree(a, b, what):
    a = [t.float().cpu().numpy().astype(np.float64) for t in (a if isinstance(a, (tuple, list)) else [a])]
    b = [t.float().cpu().numpy().astype(np.float64) for t in (b if isinstance(b, (tuple, list)) else [b])]
    for u, v in zip(a, b):
        assert np.isfinite(v).all(), f"{what}: non-finite output of the poisoned build"
        err = O.max_rel_err(v.reshape(-1, v.shape[-1]), u.reshape(-1, u.shape[-1]))
        _say(f"  {what}: err={err:.2e}")
        assert err <= 1e-6, (what, err)


FULL = [((1, 1, 1), 0, False), ((2, 2, 2), 0, False), ((3, 3, 3), 0, True), ((5, 5, 5), 0, False),
        ((6, 6, 6), 0, False), ((7, 7, 7), 0, False), ((8, 8, 8), 0, True), ((2, 2, 3), 0, False),
        ((6, 6, 2), 0, False), ((4, 6, 5), 0, False), ((3, 3, 0), 0, False), ((10, 3, 7), 0, False),
        ((12, 12, 12), 0, False), ((16, 16, 16), 0, True), ((32, 32, 32), 0, False), ((64, 64, 64), 0, False),
        ((16, 16, 16), gtp.GTP_CONV_FFT, False), ((32, 32, 32), gtp.GTP_CONV_FFT, False),
        ((64, 64, 64), gtp.GTP_CONV_FFT, False), ((4, 4, 4), gtp.GTP_CONV_DIRECT, False),
        ((5, 5, 5), gtp.GTP_FORCE_GENERIC, False), ((3, 4, 6), 0, False)]


@pytest.mark.skipif(not os.path.exists(POISON_LIB), reason="poisoned-LDS build not built")
@pytest.mark.parametrize("degs,flags,bf16", FULL)
def test_full_poisoned_matches(degs, flags, bf16):
    L1, L2, Lo = degs
    n = 70 if max(degs) < 64 else 9
    rng = np.random.default_rng(200 + L1 + 3 * L2 + 7 * Lo + flags)
    x1 = _dev(rng.standard_normal((n, 1, O.nsh(L1))), bf16)
    x2 = _dev(rng.standard_normal((n, 1, O.nsh(L2))), bf16)
    _say(f"poison full {degs} flags={flags} bf16={bf16}")
    a, b = _both(lambda: gtp.gtp_full(gtp.Plan(L1, L2, Lo, flags), x1, x2))
    _agree(a, b, f"full {degs}")


@pytest.mark.skipif(not os.path.exists(POISON_LIB), reason="poisoned-LDS build not built")
def test_other_entry_points_poisoned_match():
    rng = np.random.default_rng(210)
    # weighted product and its gradients, backward
    for L in (6, 16):
        B, C = 5, 13
        x1 = _dev(rng.standard_normal((B, C, O.nsh(L))))
        x2 = _dev(rng.standard_normal((B, C, O.nsh(L))))
        w1, w2, wo = (_dev(rng.standard_normal((C, L + 1))) for _ in range(3))
        _say(f"poison weighted L={L}")
        a, b = _both(lambda: gtp.gtp_full_weighted(gtp.Plan(L, L, L), x1, x2, w1, w2, wo, per_channel=True))
        _agree(a, b, f"weighted {L}")
        dy = _dev(rng.standard_normal((B, C, O.nsh(L))))
        a, b = _both(lambda: gtp.gtp_full_backward(gtp.Plan(L, L, L), x1, x2, dy))
        _agree(a, b, f"backward {L}")
    L = 4
    x1 = _dev(rng.standard_normal((7, 3, O.nsh(L))))
    x2 = _dev(rng.standard_normal((7, 3, O.nsh(L))))
    w1, w2, wo = (_dev(rng.standard_normal((3, L + 1))) for _ in range(3))
    dy = _dev(rng.standard_normal((7, 3, O.nsh(L))))
    _say("poison weighted backward L=4")

    def wbwd():
        g = gtp.gtp_full_weighted_backward(gtp.Plan(L, L, L), x1, x2, dy, w1, w2, wo, per_channel=True)
        return [g[k] for k in ("dx1", "dx2", "dw1", "dw2", "dwout")]

    a, b = _both(wbwd)
    _agree(a, b, "weighted backward")
    x1 = _dev(rng.standard_normal((9, 2, O.nsh(4))))
    x2 = _dev(rng.standard_normal((9, 2, O.nsh(6))))
    dy = _dev(rng.standard_normal((9, 2, O.nsh(5))))
    a, b = _both(lambda: gtp.gtp_full_backward(gtp.Plan(4, 6, 5), x1, x2, dy))
    _agree(a, b, "backward (4, 6, 5)")
    # rotated-frame convolution: one product per lane (6, 7), matrix cores (16, padded 12)
    for L, C in ((6, 70), (7, 64), (16, 37), (12, 20)):
        B = 6
        x = _dev(rng.standard_normal((B, C, O.nsh(L))))
        r = _dev(rng.standard_normal((B, 3)))
        h = _dev(rng.standard_normal((B, C, L + 1)))
        _say(f"poison conv_escn L={L} C={C}")
        a, b = _both(lambda: gtp.gtp_conv_escn(gtp.Plan(L, L, L), x, r, h))
        _agree(a, b, f"conv_escn {L}")
    # channel mixing (fused kernel; L = 7 odd strides)
    for L, C in ((6, 32), (7, 9)):
        B = 3
        x1 = _dev(rng.standard_normal((B, C, O.nsh(L))))
        x2 = _dev(rng.standard_normal((B, C, O.nsh(L))))
        W = _dev(rng.standard_normal((C, C, C)) / C)
        _say(f"poison channel_mix L={L} C={C}")
        a, b = _both(lambda: gtp.gtp_channel_mix(gtp.Plan(L, L, L), x1, x2, W))
        _agree(a, b, f"channel_mix {L}")
    # many-body products
    x = _dev(rng.standard_normal((11, 5, O.nsh(2))))
    for mode in (gtp.GTP_SELF_STEPWISE, gtp.GTP_SELF_FUSED):
        _say(f"poison selfproduct mode={mode}")
        a, b = _both(lambda: gtp.gtp_selfproduct(x, 2, 3, 3, mode))
        _agree(a, b, f"selfproduct {mode}")
    # the unfused stages
    L = 4
    xa = _dev(rng.standard_normal((6, O.nsh(L))))
    xb = _dev(rng.standard_normal((6, O.nsh(L))))

    def stages():
        p = gtp.Plan(L, L, L)
        g1 = gtp.gtp_sh2fourier(p, 1, xa)
        g2 = gtp.gtp_sh2fourier(p, 2, xb)
        g3 = gtp.gtp_fourier_conv(p, g1, g2)
        return gtp.gtp_fourier2sh(p, g3)

    _say("poison unfused stages")
    a, b = _both(stages)
    _agree(a, b, "unfused stages")
