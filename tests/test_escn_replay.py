"""CPU replay (numpy fp64) of the rotated-frame convolution kernel's data flow
from the plan's own tables (J: real-SH matrices of R_x(90 deg); E: theta-node
rows), against the fp64 oracle: checks the tables and the kernel's algorithm
(rotation built as J^T Z(-beta) J Z(-alpha), zonal product over mirror pairs
of theta nodes, rotation back) without a GPU."""
import math

import numpy as np
import pytest

from oracle import gtp_oracle as O
from paper_2401_10216_amd import gtp


def z_rot(l, c, s):
    """Z(-g) on degree l: (c_m, s_m) pairs of order m rotated by -g, c = cos(m g), s = sin(m g) arrays."""
    d = 2 * l + 1
    Z = np.zeros((d, d))
    Z[l, l] = 1.0
    for m in range(1, l + 1):
        Z[l + m, l + m] = c[m]
        Z[l + m, l - m] = s[m]
        Z[l - m, l + m] = -s[m]
        Z[l - m, l - m] = c[m]
    return Z


def pad4(n):
    return (n + 3) // 4 * 4


def row_layout(L):
    """Offsets of the m-major node-table row: filter, then Theta chunks, then W chunks."""
    os_, ow = [], []
    o = pad4(L + 1)
    for m in range(L + 1):
        os_.append(o)
        o += pad4(L + 1 - m)
    for m in range(L + 1):
        ow.append(o)
        o += pad4(L + 1 - m)
    return os_, ow, o


def replay(plan, x, r, h, L):
    info = plan.info()
    J = plan.table(10)
    E = plan.table(11)
    NT, K = info["NT"], (L + 1) ** 2
    OS, OW, ERL = row_layout(L)
    NPAIR = (NT + 1) // 2
    E = E.reshape(NPAIR, ERL)
    y = np.zeros((x.shape[0], x.shape[1], K))
    for b in range(x.shape[0]):
        rx, ry, rz = r[b]
        rho = math.hypot(rx, ry)
        nr = math.hypot(rho, rz)
        ca, sa, cb, sb = 1.0, 0.0, 1.0, 0.0
        if nr > 0:
            cb, sb = rz / nr, rho / nr
            if rho > 0:
                ca, sa = rx / rho, ry / rho
        al, be = math.atan2(sa, ca), math.atan2(sb, cb)
        cam = [math.cos(m * al) for m in range(L + 1)]
        sam = [math.sin(m * al) for m in range(L + 1)]
        cbm = [math.cos(m * be) for m in range(L + 1)]
        sbm = [math.sin(m * be) for m in range(L + 1)]
        D = np.zeros((K, K))
        off = 0
        for l in range(L + 1):
            d = 2 * l + 1
            Jl = J[off:off + d * d].reshape(d, d)
            off += d * d
            D[l * l:(l + 1) ** 2, l * l:(l + 1) ** 2] = Jl.T @ z_rot(l, cbm, sbm) @ Jl @ z_rot(l, cam, sam)
        for c in range(x.shape[1]):
            xp = D @ x[b, c]
            acc = np.zeros(K)
            for j in range(NPAIR):
                row = E[j]
                fe = sum(row[l] * h[b, c, l] for l in range(0, L + 1, 2))
                fo = sum(row[l] * h[b, c, l] for l in range(1, L + 1, 2))
                fj, fm = fe + fo, fe - fo
                for m in range(L + 1):
                    for sg in ((0,) if m == 0 else (0, 1)):
                        ls = range(m, L + 1)
                        idx = [l * l + l + (-m if sg else m) for l in ls]
                        ae = sum(row[OS[m] + l - m] * xp[i] for l, i in zip(ls, idx) if (l + m) % 2 == 0)
                        ao = sum(row[OS[m] + l - m] * xp[i] for l, i in zip(ls, idx) if (l + m) % 2 == 1)
                        pj, pm = fj * (ae + ao), fm * (ae - ao)
                        for l, i in zip(ls, idx):
                            acc[i] += row[OW[m] + l - m] * (pj + pm if (l + m) % 2 == 0 else pj - pm)
            y[b, c] = D.T @ acc
    return y


@pytest.mark.parametrize("L", [1, 2, 4, 6])
def test_escn_replay_equals_oracle(L):
    rng = np.random.default_rng(200 + L)
    B, C = 5, 2
    x = rng.standard_normal((B, C, (L + 1) ** 2))
    r = rng.standard_normal((B, 3))
    r[0] = 0.0
    r[1] = [0.0, 0.0, -1.5]
    r[2] = [1e-3, 0.0, 2.0]
    h = rng.standard_normal((B, C, L + 1))
    plan = gtp.Plan(L, L, L, gtp.GTP_PLAN_HOST_ONLY)
    got = replay(plan, x, r, h, L)
    ref = O.conv_escn(x, r, h, L, L, L)
    assert np.abs(got - ref).max() < 1e-12 * max(1.0, np.abs(ref).max())


def test_escn_tables_shapes_and_j_orthogonal():
    for L in (1, 3, 8):
        p = gtp.Plan(L, L, L, gtp.GTP_PLAN_HOST_ONLY)
        J = p.table(10)
        assert J.size == sum((2 * l + 1) ** 2 for l in range(L + 1))
        off = 0
        for l in range(L + 1):
            d = 2 * l + 1
            Jl = J[off:off + d * d].reshape(d, d)
            off += d * d
            assert np.abs(Jl @ Jl.T - np.eye(d)).max() < 1e-13
    # no rotated-frame tables outside L1 = L2 = Lout <= 8
    for args in ((2, 2, 3), (9, 9, 9), (0, 0, 0)):
        p = gtp.Plan(*args, gtp.GTP_PLAN_HOST_ONLY)
        assert p.table(10).size == 0 and p.table(11).size == 0
