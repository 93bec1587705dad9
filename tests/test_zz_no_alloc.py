"""gtp_conv_escn_noalloc (static device scratch, no allocation) against
gtp_conv_escn on the same inputs, through the C ABI: two calls in a row, the
second with a smaller input, on the rotated-frame kernels (several scratch
chunks, fp32 and bf16) and on the filter route (degrees without a
rotated-frame kernel, and a direct-convolution plan).  Bar: the fp32 parity
bar of the product, 1e-5 relative per product; the oracle checks a sample."""
import sys

import numpy as np
import pytest

from oracle import gtp_oracle as O
from paper_2401_10216_amd import gtp, inputs

pytestmark = pytest.mark.gpu
TOL = 1e-5
torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gtp.lib()


def _case(seed, B, C, L1, L2, bf16):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, C, O.nsh(L1))).astype(np.float32)
    r = rng.standard_normal((B, 3))
    r[0] = 0.0  # a zero edge vector (taken as the pole)
    r[1] = (0.0, 0.0, -2.0)  # the other pole
    r = r.astype(np.float32)
    h = rng.standard_normal((B, C, L2 + 1)).astype(np.float32)
    if bf16:
        bits, x = inputs.round_to_bf16(x)
        tx = torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)
    else:
        tx = torch.from_numpy(x).cuda()
    return x, r, h, tx, torch.from_numpy(r).cuda(), torch.from_numpy(h).cuda()


# (degrees, flags, bf16, first call (B, C), second call (B, C)); scratch is
# 64 MiB: 2240 B per edge at L = 6 (29959 edges per chunk), 4560 B at L = 8,
# 28560 B at L = 16 (2349 edges per chunk), C * 121 * 4 B on the L = 10
# filter route
CASES = [
    ((6, 6, 6), 0, False, (40000, 64), (1000, 96)),
    ((8, 8, 8), 0, True, (20000, 64), (300, 70)),
    ((10, 10, 10), 0, False, (5000, 64), (100, 3)),
    ((4, 4, 4), gtp.GTP_CONV_DIRECT, False, (3000, 64), (50, 5)),
    ((3, 5, 4), 0, False, (700, 200), (20, 1)),
    ((16, 16, 16), 0, False, (3000, 64), (40, 17)),
]


@pytest.mark.parametrize("degs,flags,bf16,first,second", CASES)
def test_noalloc_matches_allocating_entry_point(degs, flags, bf16, first, second):
    L1, L2, Lout = degs
    plan = gtp.Plan(L1, L2, Lout, flags)
    for call, (B, C) in enumerate((first, second)):
        _say(f"noalloc L={degs} flags={flags} bf16={bf16} call={call} B={B} C={C}")
        x, r, h, tx, tr, th = _case(100 * call + L1 + 10 * L2, B, C, L1, L2, bf16)
        ref = gtp.gtp_conv_escn(plan, tx, tr, th)
        y = torch.full((B, C, O.nsh(Lout)), float("nan"), device="cuda:0")
        gtp.gtp_conv_escn(plan, tx, tr, th, y=y, noalloc=True)
        torch.cuda.synchronize()
        a = y.cpu().numpy().astype(np.float64)
        b = ref.cpu().numpy().astype(np.float64)
        assert np.isfinite(a).all()
        err = O.max_rel_err(a, b)
        _say(f"  vs gtp_conv_escn: err={err:.3e} identical={np.array_equal(a, b)}")
        assert err <= TOL
        # a sample, including the last edge, against the oracle
        bi = np.unique(np.r_[0, 1, B - 1, np.linspace(0, B - 1, 6).astype(int)])
        ci = np.arange(C) % C
        sel = [(int(e), int(c)) for e in bi for c in ci[:4]]
        eb = np.array([e for e, _ in sel])
        cb = np.array([c for _, c in sel])
        want = O.conv_escn(x[eb, cb][:, None].astype(np.float64), r[eb].astype(np.float64),
                           h[eb, cb][:, None].astype(np.float64), L1, L2, Lout)[:, 0]
        assert O.max_rel_err(a[eb, cb], want) <= TOL


def test_noalloc_rejects_edges_larger_than_scratch():
    """One edge's filter rows above 64 MiB: refused before any launch."""
    plan = gtp.Plan(2, 64, 2)
    C = (64 << 20) // (4 * 65 * 65) + 1
    x = torch.zeros((1, C, 9), device="cuda:0")
    r = torch.zeros((1, 3), device="cuda:0")
    h = torch.zeros((1, C, 65), device="cuda:0")
    with pytest.raises(gtp.GTPError, match="scratch"):
        gtp.gtp_conv_escn(plan, x, r, h, noalloc=True)
