"""Host replay of the degree-16 matrix-core rotated-frame convolution.

The kernel's data flow, written out in numpy fp64 with the operand images the
plan exports (tables 12 and 13 of gtp_plan_table) and the 16x16x4 contraction
semantics of the matrix cores (A[i][k] from lane 16 k + i, B[k][j] from lane
16 k + j, register r of lane 16 g + i = row 4 g + r, column i).  It checks the
image layouts and the stage-to-stage register conventions against the oracle's
rotated-frame convolution (Sec. 3.3, eq. sh2fs-escn) on the CPU, and the
images themselves against the plan's theta tables (S, W).
"""
import numpy as np
import pytest

from oracle import gtp_oracle as O
from paper_2401_10216_amd import gtp

L = 16
H = L + 1


def tri(l, m):
    return l * (l + 1) // 2 + m


def steps(m):
    n = L + 1 - m
    ne, no = (n + 1) // 2, n // 2
    return (ne + 3) // 4 + (no + 3) // 4 + 4 + (4 if no > 0 else 0)


def lane_floats(m):
    return (steps(m) + 3) // 4 * 4


def moff(m):
    return sum(64 * lane_floats(k) for k in range(m))


@pytest.fixture(scope="module")
def plan():
    p = gtp.Plan(L, L, L, gtp.GTP_PLAN_HOST_ONLY)
    info = p.info()
    NJ = info["NT"] + 1
    S = p.table(3).reshape(-1, NJ)
    W = p.table(4).reshape(-1, NJ)
    return p, info, S, W, p.table(12), p.table(13)


def test_images_follow_theta_tables(plan):
    """Every entry of the operand images is the theta table value its lane,
    step and order name (layout of the header comment), zero past degree L."""
    p, info, S, W, A, Z = plan
    NP = info["NP"]
    assert A.size == moff(L + 1) and Z.size == 16 * H + 3 * H

    def s(l, m, j):
        return S[tri(l, m), j] if l <= L else 0.0

    def cw(l, m, j):
        return (NP if m == 0 else 0.5 * NP) * W[tri(l, m), j] if l <= L else 0.0

    for m in range(L + 1):
        n = L + 1 - m
        ne, no = (n + 1) // 2, n // 2
        ke, ko = (ne + 3) // 4, (no + 3) // 4
        for lane in range(64):
            k, i = lane // 16, lane % 16
            pj = 4 * (i % 4) + i // 4 + 1
            v = A[moff(m) + lane * lane_floats(m):][:steps(m)]
            want = [s(m + 2 * (4 * q + k), m, pj) for q in range(ke)]
            want += [s(m + 1 + 2 * (4 * q + k), m, pj) for q in range(ko)]
            want += [cw(m + 2 * i, m, 4 * r + k + 1) if i < ne else 0.0 for r in range(4)]
            if no:
                want += [cw(m + 1 + 2 * i, m, 4 * r + k + 1) if i < no else 0.0 for r in range(4)]
            np.testing.assert_array_equal(v, np.array(want))
    for g in range(4):
        for r in range(4):
            j = 4 * r + g + 1
            np.testing.assert_allclose(Z[(4 * g + r) * H:][:H], [S[tri(l, 0), 0] * S[tri(l, 0), j] for l in range(H)],
                                       rtol=1e-12, atol=1e-13)
    zp = Z[16 * H:]
    np.testing.assert_allclose(zp[:H], [S[tri(l, 0), 0] ** 2 for l in range(H)], rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(zp[H:2 * H], [S[tri(l, 0), 0] for l in range(H)])
    np.testing.assert_array_equal(zp[2 * H:], [NP * W[tri(l, 0), 0] for l in range(H)])


def mfma(a_lanes, b_lanes, c):
    """c + A B for 64-lane operands (A[i][k] = a_lanes[16 k + i], B[k][j] = b_lanes[16 k + j])."""
    A = a_lanes.reshape(4, 16).T
    B = b_lanes.reshape(4, 16)
    return c + A @ B


def replay_tile(X, hm, D, A, Z):
    """The kernel's stages on one 16-channel tile X[k][c] (fp64); hm[c][l]."""
    X = X.copy()
    lanes = np.arange(64)
    g_of, i_of = lanes // 16, lanes % 16
    # rotate in
    for l in range(L + 1):
        X[l * l:(l + 1) ** 2] = D[l] @ X[l * l:(l + 1) ** 2]
    # filter at the lane's node pairs: FE[4 g + r][c], FO likewise (rows as the tile's)
    FE = np.zeros((16, 16))
    FO = np.zeros((16, 16))
    for g in range(4):
        for r in range(4):
            z = Z[(4 * g + r) * H:][:H]
            FE[4 * g + r] = (z[0::2] * hm[:, 0::2]).sum(axis=1)
            FO[4 * g + r] = (z[1::2] * hm[:, 1::2]).sum(axis=1)
    zp = Z[16 * H:]
    fe0 = (zp[0:H:2] * hm[:, 0::2]).sum(axis=1)
    fo0 = (zp[1:H:2] * hm[:, 1::2]).sum(axis=1)
    for m in range(L + 1):
        n = L + 1 - m
        ne, no = (n + 1) // 2, n // 2
        ke, ko = (ne + 3) // 4, (no + 3) // 4
        nl = lane_floats(m)
        av = A[moff(m):moff(m) + 64 * nl].reshape(64, nl)
        for sg in ([0] if m == 0 else [0, 1]):
            def row(l):
                return l * l + l + (-m if sg else m)

            def bx(l_of_lane):
                return np.array([X[row(l), c] if l <= L else 0.0 for l, c in zip(l_of_lane, i_of)])

            GE = np.zeros((16, 16))
            GO = np.zeros((16, 16))
            for q in range(ke):
                GE = mfma(av[:, q], bx(m + 2 * (4 * q + g_of)), GE)
            for q in range(ko):
                GO = mfma(av[:, ke + q], bx(m + 1 + 2 * (4 * q + g_of)), GO)
            pj = (FE + FO) * (GE + GO)
            pm = (FE - FO) * (GE - GO)
            PE, PO = pj + pm, pj - pm
            YE = np.zeros((16, 16))
            YO = np.zeros((16, 16))
            for r in range(4):
                # B for K-step r: register r of lane (g, c) = P[4 g + r][c]
                YE = mfma(av[:, ke + ko + r], PE[4 * g_of + r, i_of], YE)
                if no:
                    YO = mfma(av[:, ke + ko + 4 + r], PO[4 * g_of + r, i_of], YO)
            if m == 0:
                xs = np.array([X[l * l + l] for l in range(H)])
                ae = (zp[H:2 * H:2][:, None] * xs[0::2]).sum(axis=0)
                ao = (zp[H + 1:2 * H:2][:, None] * xs[1::2]).sum(axis=0)
                p0 = (fe0 + fo0) * (ae + ao)
                q0 = (fe0 - fo0) * (ae - ao)
                pe0, po0 = p0 + q0, p0 - q0
            for ie in range(ne):
                l = m + 2 * ie
                v = YE[ie].copy()
                if m == 0:
                    v += zp[2 * H + l] * pe0
                X[row(l)] = v
            for io in range(no):
                l = m + 1 + 2 * io
                v = YO[io].copy()
                if m == 0:
                    v += zp[2 * H + l] * po0
                X[row(l)] = v
    for l in range(L + 1):
        X[l * l:(l + 1) ** 2] = D[l].T @ X[l * l:(l + 1) ** 2]
    return X


def test_replay_matches_oracle(plan):
    """The replay equals the oracle's rotated-frame convolution (fp64), with
    the edge's rotation taken from the oracle's Wigner-D builder (any rotation
    taking the edge to the pole gives the same product)."""
    p, info, S, W, A, Z = plan
    rng = np.random.default_rng(1616)
    K = (L + 1) ** 2
    for r in (np.array([0.3, -1.2, 0.7]), np.array([0.0, 0.0, 2.0]), np.array([1e-4, 2e-4, -1.0])):
        x = rng.standard_normal((16, K))
        hm = rng.standard_normal((16, H))
        Dfull = O.wigner_d_real(L, O.edge_rotation(r))
        D = [Dfull[l * l:(l + 1) ** 2, l * l:(l + 1) ** 2] for l in range(L + 1)]
        y = replay_tile(x.T.copy(), hm, D, A, Z).T
        ref = O.conv_escn(x[None], r[None], hm[None], L, L, L)[0]
        err = O.max_rel_err(y, ref)
        assert err < 1e-11, err


CLASS_L = 8


def cls_n(l, c):
    return l // 2 + 1 if c == 0 else (l // 2 if c == 2 else (l + 1) // 2)


def cls_start(l, c):
    return [l, l + 1, l & 1, 1 - (l & 1)][c]


def cls_map(l, c):
    return [3, 1, 2, 0][c] if l & 1 else [0, 2, 1, 3][c]


def jtiles(l):
    return 1 if l < CLASS_L else (3 if cls_n(l, 0) > 8 else 2)


def jtcls(t, par):
    return [[0, 3], [1, 2], [0, -1]][t][par]


def jtfirst(t):
    return 8 if t == 2 else 0


def jtrows(l, t, par):
    c = jtcls(t, par)
    return 0 if c < 0 else min(cls_n(l, c) - jtfirst(t), 8)


def jtcols(l, t, par):
    c = jtcls(t, par)
    return 0 if c < 0 else cls_n(l, cls_map(l, c))


def jsteps(l, t):
    return (2 * l + 1 + 3) // 4 if l < CLASS_L else (max(jtcols(l, t, 0), jtcols(l, t, 1)) + 1) // 2


def jnk4(l, t):
    return (jsteps(l, t) + 3) // 4 * 4


def joff(l, t):
    return sum(64 * jnk4(k, u) for k in range(l) for u in range(jtiles(k))) + sum(64 * jnk4(l, u) for u in range(t))


def jrow(rho):
    """Block row of whole-block tile row rho = 4 g + r: 2 r + (g & 1) + 8 (g >> 1)."""
    g, r = rho // 4, rho % 4
    return 2 * r + (g & 1) + 8 * (g >> 1)


def jtrow(l, t, i):
    """Block-local row of tile row i (-1: padding)."""
    if l < CLASS_L:
        return jrow(i) if jrow(i) < 2 * l + 1 else -1
    g, r = i // 4, i % 4
    par, pp = g & 1, 4 * (g // 2) + r
    return cls_start(l, jtcls(t, par)) + 2 * (jtfirst(t) + pp) if pp < jtrows(l, t, par) else -1


def jtcol(l, t, s, k):
    """Block-local column of tile column 4 s + k (-1: padding)."""
    if l < CLASS_L:
        return 4 * s + k if 4 * s + k < 2 * l + 1 else -1
    par, q = k & 1, 2 * s + k // 2
    return cls_start(l, cls_map(l, jtcls(t, par))) + 2 * q if q < jtcols(l, t, par) else -1


def j_blocks(p):
    J = p.table(10)
    out, o = [], 0
    for l in range(L + 1):
        d = 2 * l + 1
        out.append(J[o:o + d * d].reshape(d, d))
        o += d * d
    return out


def z_rot(l, angle, sign):
    """Rotation about the pole on degree block l: each (cos m, sin m) pair
    turned by m angle; sign = -1 for Z(-angle): c' = c cos + s sin, s' = -c sin + s cos."""
    d = 2 * l + 1
    Zm = np.eye(d)
    for m in range(1, l + 1):
        c, s = np.cos(m * angle), np.sin(m * angle)
        ic, is_ = l + m, l - m
        if sign < 0:
            Zm[ic, ic], Zm[ic, is_], Zm[is_, ic], Zm[is_, is_] = c, s, -s, c
        else:
            Zm[ic, ic], Zm[ic, is_], Zm[is_, ic], Zm[is_, is_] = c, -s, s, c
    return Zm


def test_rotation_images_and_factorization(plan):
    """Table 14 holds J and J^T in the lane-permuted K-step layout of the
    output tiles (whole blocks below degree 8, class sub-blocks from 8 on;
    every non-zero of J in exactly one entry), and the kernel's
    factor-by-factor rotation J^T Z(-beta) J Z(-alpha) (angles from the edge
    vector as the kernel takes them) gives the oracle's product."""
    p, info, S, W, A, Z = plan
    JI = p.table(14)
    Jb = j_blocks(p)
    jt = joff(L + 1, 0)
    assert JI.size == 2 * jt
    for l in range(L + 1):
        covered = np.zeros((2 * l + 1, 2 * l + 1), dtype=int)
        for t in range(jtiles(l)):
            for lane in range(64):
                k, i = lane // 16, lane % 16
                row = jtrow(l, t, i)
                same = l < CLASS_L or ((i // 4) & 1) == (k & 1)
                for s in range(jsteps(l, t)):
                    col = jtcol(l, t, s, k)
                    at = joff(l, t) + lane * jnk4(l, t) + s
                    ok = row >= 0 and col >= 0 and same
                    want = Jb[l][row, col] if ok else 0.0
                    wantt = Jb[l][col, row] if ok else 0.0
                    assert JI[at] == want and JI[jt + at] == wantt
                    if ok:
                        covered[row, col] += 1
        # every non-zero of J is in exactly one tile entry
        assert np.all(covered[np.abs(Jb[l]) > 1e-12] == 1)
        assert covered.max() <= 1
    rng = np.random.default_rng(1717)
    K = (L + 1) ** 2
    for r in (np.array([0.3, -1.2, 0.7]), np.array([0.0, 0.0, -2.0]), np.array([0.0, 0.0, 0.0]),
              np.array([-0.8, 0.1, 0.05])):
        rho = np.hypot(r[0], r[1])
        al = np.arctan2(r[1], r[0]) if rho > 0 else 0.0
        be = np.arctan2(rho, r[2]) if (rho > 0 or r[2] != 0) else 0.0
        D = [Jb[l].T @ z_rot(l, be, -1) @ Jb[l] @ z_rot(l, al, -1) for l in range(L + 1)]
        x = rng.standard_normal((16, K))
        hm = rng.standard_normal((16, H))
        y = replay_tile(x.T.copy(), hm, D, A, Z).T
        ref = O.conv_escn(x[None], r[None], hm[None], L, L, L)[0]
        assert O.max_rel_err(y, ref) < 1e-11


def jpass_replay(T, JI, tr):
    """The degree-16 kernel's pass of J (tr = 0) or J^T (tr = 1) over a tile
    T[row][channel], replayed in the kernel's program order: block pairs
    (2p, 2p + 1) (degree 16 alone), the operands (B values) of pair p + 1
    read before pair p's writes, the addresses the kernel forms.  Whole-block
    tiles (degrees below 8) write the rows past the block as they come (zero
    rows of the product), except degree 1, whose padding goes to the spare
    row 289, as does the padding of the class tiles."""
    img = JI[tr * joff(L + 1, 0):]
    T = T.copy()
    lanes = np.arange(64)
    g_of, i_of = lanes // 16, lanes % 16
    gp, gh = g_of & 1, g_of >> 1

    def start(l, t, par, rows):
        c = jtcls(t, par) if jtcls(t, par) >= 0 else jtcls(t, 0)
        return cls_start(l, c) + 2 * jtfirst(t) if rows else cls_start(l, cls_map(l, c))

    def load(l):
        d, R0 = 2 * l + 1, l * l
        A, B = [], []
        for t in range(jtiles(l)):
            nk = jnk4(l, t)
            A.append(img[joff(l, t):joff(l, t) + 64 * nk].reshape(64, nk))
            Bt = []
            for ks in range(jsteps(l, t)):
                if l < CLASS_L:
                    c = 4 * ks + g_of
                    Bt.append(np.where(c < d, T[R0 + c, i_of], 0.0))
                else:
                    cb = 2 * gh + np.where(gp == 1, start(l, t, 1, False), start(l, t, 0, False))
                    v = T[R0 + cb + 4 * ks, i_of]
                    ok = 2 * ks + gh < np.where(gp == 1, jtcols(l, t, 1), jtcols(l, t, 0))
                    Bt.append(np.where(ok, v, 0.0))
            B.append(Bt)
        return A, B

    def mma(l, A, B):
        return [sum(mfma(A[t][:, ks], B[t][ks], np.zeros((16, 16))) for ks in range(len(B[t])))
                for t in range(jtiles(l))]

    def store(l, acc):
        d, R0 = 2 * l + 1, l * l
        for t in range(jtiles(l)):
            for r in range(4):
                v = acc[t][4 * g_of + r, i_of]
                if l < CLASS_L:
                    row = np.array([jrow(4 * g + r) for g in g_of])
                    tgt = np.where(row < d, R0 + row, 289) if l == 1 else R0 + row
                else:
                    rb = 8 * gh + np.where(gp == 1, start(l, t, 1, True), start(l, t, 0, True))
                    ok = 4 * gh + r < np.where(gp == 1, jtrows(l, t, 1), jtrows(l, t, 0))
                    tgt = np.where(ok, R0 + rb + 2 * r, 289)
                assert tgt.max() <= 289
                T[tgt, i_of] = v

    pairs = [(2 * p, 2 * p + 1) for p in range(L // 2)] + [(L,)]
    ops = {l: load(l) for l in pairs[0]}
    for p, pr in enumerate(pairs):
        acc = {l: mma(l, *ops[l]) for l in pr}
        if p + 1 < len(pairs):
            ops = {l: load(l) for l in pairs[p + 1]}
        for l in pr:
            store(l, acc[l])
    return T


def test_jpass_replay_padded_writes(plan):
    """The J and J^T passes as the kernel orders them equal the block-wise
    products on every degree block (so no padded write lands on a row that is
    read or kept afterwards), and rows 290, 291 (the next channel's) are
    never written."""
    p = plan[0]
    JI = p.table(14)
    Jb = j_blocks(p)
    rng = np.random.default_rng(1818)
    T0 = rng.standard_normal((292, 16))
    for tr in (0, 1):
        T = jpass_replay(T0, JI, tr)
        for l in range(L + 1):
            blk = Jb[l].T if tr else Jb[l]
            np.testing.assert_allclose(T[l * l:(l + 1) ** 2], blk @ T0[l * l:(l + 1) ** 2], rtol=1e-12, atol=1e-12)
        np.testing.assert_array_equal(T[290:], T0[290:])
