"""The build-time constants of the thread-per-product and rotated-frame
kernels (S, W and the node-pair rows E as instruction literals) are the
plan's own tables rounded once to fp32, value for value.

The generator runs here on the CPU (it is host code); its output is compared
with the fp64 tables a plan exposes through gtp_plan_table.
"""
import os
import re

import numpy as np
import pytest

from paper_2401_10216_amd import build, gtp


def _parse(path, struct):
    """{L: {name: array}} from the generated C++ constants."""
    text = open(path).read()
    out = {}
    for m in re.finditer(struct + r"<(\d+)> \{(.*?)\n\};", text, re.S):
        L, body = int(m.group(1)), m.group(2)
        arrs = {}
        for a in re.finditer(r"static constexpr float (\w+)\[(\d+)\]\[(\d+)\] = \{(.*?)\n  \};", body, re.S):
            name, n0, n1 = a.group(1), int(a.group(2)), int(a.group(3))
            vals = [float.fromhex(v.strip().rstrip("f")) for v in re.findall(r"[-0-9a-fx.p+]+f", a.group(4))]
            arrs[name] = np.array(vals, dtype=np.float64).reshape(n0, n1)
        out[L] = arrs
    return out


@pytest.fixture(scope="module")
def consts():
    build.generate_constants()
    gen = build.GEN
    return (_parse(os.path.join(gen, "gtp_small_consts.inc"), "SmallConsts"),
            _parse(os.path.join(gen, "gtp_escn_consts.inc"), "EscnConsts"))


@pytest.mark.parametrize("L", range(1, 9))
def test_small_consts_equal_plan_tables(consts, L):
    small, _ = consts
    p = gtp.Plan(L, L, L, gtp.GTP_PLAN_HOST_ONLY)
    NJ = p.info()["NT"] + 1
    S = p.table(3).reshape(-1, NJ).astype(np.float32).astype(np.float64)
    W = p.table(4).reshape(-1, NJ).astype(np.float32).astype(np.float64)
    assert small[L]["S"].shape == S.T.shape and small[L]["W"].shape == W.T.shape
    assert np.array_equal(small[L]["S"], S.T)
    assert np.array_equal(small[L]["W"], W.T)


@pytest.mark.parametrize("L", range(1, 9))
def test_escn_consts_equal_plan_tables(consts, L):
    _, escn = consts
    p = gtp.Plan(L, L, L, gtp.GTP_PLAN_HOST_ONLY)
    E = p.table(11).astype(np.float32).astype(np.float64)
    got = escn[L]["E"]
    assert got.size == E.size and got.shape[0] == L + 1
    assert np.array_equal(got, E.reshape(got.shape))
