"""CPU checks of the lane-permuted tables of the matrix-core wave kernel
(L1 = L2 = Lout = L in {16, 32, 64}).

The tables are host logic: test_replay_matches_oracle replays the kernel's
data flow in numpy from the plan's own tables -- lane layout, the 16x16x4
matrix-core operand layout (A[i][k] from lane 16k + i, B[k][j] from lane
16k + j, D[4g + r][j] in register r of lane 16g + j), the rotation
recurrences, the mirror exchange between lanes i and i ^ 8 and the pole
terms -- and compares the result with the oracle (Sec. 3.2 pipeline vs the
quadrature-defined product).  The GPU parity tests then check that the
kernel computes what this replay computes.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2401_10216_amd import gtp

HOST_ONLY = 16


def _geo(L, NP):
    Q = NP // 4
    G = dict(L=L, NP=NP, Q=Q, NMB=(Q + 16) // 16, NKS=L // 8, PASSES=L // 8, K=(L + 1) ** 2, NMP2=2 * L + 2)
    G["NMBP"] = (G["NMB"] + 1) // 2 * 2
    G["NMR"] = L // 32 if L > 32 else 1
    G["ASD"] = 6 * G["NMBP"]
    G["AST"] = G["ASD"] + 4 * G["NMR"] * G["NMBP"]
    G["TWRN"] = G["AST"] + 4 * G["NMR"]
    G["NTH"] = 256 if L > 32 else 64
    G["NROW"] = (L + 1) * (L + 2) // 2 - (L + 1)
    G["NIT"] = (G["NROW"] + G["NTH"] - 1) // G["NTH"]
    G["NV0"] = (L + 1 + 7) // 8
    G["NV0P"] = (G["NV0"] + 3) // 4 * 4
    nu = lambda s: L // 2 - 4 * s
    G["nu"] = nu
    G["u2off"] = lambda s: sum(nu(q) // 2 for q in range(s))
    G["TU2"] = G["u2off"](G["NKS"])

    def xb(c):
        # pair blocks hold the nu(s) - g u-steps that have a coefficient, + 1 pad
        return (L + 1) + sum(4 * (nu(q // 4) - q % 4) + 1 for q in range(c))

    G["xb"] = xb
    # the image also covers every group's reads of all nu(s) u-steps
    G["XQ"] = max([xb(L // 2)] + [xb(c) + 4 * nu(c // 4) for c in range(L // 2)])
    return G


def _mfma(a, b, c):
    """16x16x4 fp32 matrix-core step on 64 lanes: returns c + A @ B in the D layout."""
    A = a.reshape(4, 16).T      # A[i][k] = a[16k + i]
    B = b.reshape(4, 16)        # B[k][j] = b[16k + j]
    D = A @ B
    lane = np.arange(64)
    out = c.copy()
    for r in range(4):
        out[:, r] += D[4 * (lane // 16) + r, lane % 16]
    return out


def _xor(v, m):
    return v[np.arange(64) ^ m]


def _rot(c, s, cr, sr):
    return c * cr - s * sr, s * cr + c * sr


def replay(plan, L, x1, x2):
    NP = plan.info()["NP"]
    G = _geo(L, NP)
    Q, NMB, NMBP, NKS, PASSES = G["Q"], G["NMB"], G["NMBP"], G["NKS"], G["PASSES"]
    NMP2, NIT, NROW, NTH = G["NMP2"], G["NIT"], G["NROW"], G["NTH"]
    NT = 2 * L + 1
    TWR = plan.table(5).reshape(64, G["TWRN"])
    SMP = plan.table(6).reshape(PASSES, G["TU2"], 64, 4)
    SM0P = plan.table(7).reshape(PASSES + 1, 64, G["NV0P"])
    XMAPP = plan.table(9).astype(np.int64).reshape(NTH, -1)
    W = plan.table(4).reshape(-1, NT + 1)
    lane = np.arange(64)
    g, i = lane // 16, lane % 16
    h, pi = i // 8, i % 8

    # LDS image of the inputs, staged by NTH threads
    xs = np.zeros(G["XQ"] * 4)
    tid = np.arange(NTH)
    for k in range(XMAPP.shape[1]):
        idx = tid + NTH * k
        ok = (idx < G["K"]) & (XMAPP[:, k] >= 0)
        xs[XMAPP[ok, k]] = x1[idx[ok]]
        xs[XMAPP[ok, k] + 2] = x2[idx[ok]]
    xq = xs.reshape(-1, 4)

    def m0(pass_):
        s1 = np.zeros(64)
        s2 = np.zeros(64)
        for v in range(G["NV0"]):
            l = 8 * v + g + 4 * h
            ok = l <= L
            sv = SM0P[pass_, :, v]
            s1[ok] += sv[ok] * xq[l[ok], 0]
            s2[ok] += sv[ok] * xq[l[ok], 2]
        out = []
        for a in (s1, s2):
            a = a + _xor(a, 8)
            t = _xor(a, 16)
            sm, dif = a + t, np.where(g & 1, t - a, a - t)
            node, mirror = sm + _xor(sm, 32), dif + _xor(dif, 32)
            out.append(np.where(h == 1, mirror, node))
        return out

    def one_pass(p):
        """Moments eo[parity][pi][slot] of pass p, as one wave computes them."""
        c1, c2 = m0(p)
        acc = np.zeros((2, NMB, 4, 64, 4))
        acc[0, :, 0] = c1[:, None]
        acc[1, :, 0] = c2[:, None]
        twc = np.zeros((4, NMB, 64))
        r8 = np.zeros((2, NMB, 64))
        for mb in range(NMB):
            twc[0, mb], twc[2, mb], twc[1, mb], twc[3, mb] = (TWR[:, 6 * mb + e] for e in range(4))
            r8[0, mb], r8[1, mb] = TWR[:, 6 * mb + 4], TWR[:, 6 * mb + 5]
        for s in range(NKS):
            c = 4 * s + g
            xa = np.array([G["xb"](cc) for cc in c]) + h
            xe = np.array([G["xb"](cc) for cc in c]) + 3 - h
            Vo = np.zeros((64, 4))
            Ve = np.zeros((64, 4))
            for u2 in range(G["nu"](s) // 2):
                sv = SMP[p, G["u2off"](s) + u2]
                for e in range(2):
                    u = 2 * u2 + e
                    Vo += sv[:, 2 * e, None] * xq[xa + 4 * u]
                    Ve += sv[:, 2 * e + 1, None] * xq[xe + 4 * u]
            Bo = np.where(h[:, None] == 1, _xor(Vo, 8) - Vo, _xor(Vo, 8) + Vo)
            Be = np.where(h[:, None] == 1, _xor(Ve, 8) - Ve, _xor(Ve, 8) + Ve)
            for mb in range(NMB):
                for ti in range(2):
                    acc[ti, mb, 0] = _mfma(twc[0, mb], Be[:, 2 * ti], acc[ti, mb, 0])
                    acc[ti, mb, 1] = _mfma(twc[1, mb], Bo[:, 2 * ti], acc[ti, mb, 1])
                    acc[ti, mb, 2] = _mfma(twc[2, mb], Be[:, 2 * ti + 1], acc[ti, mb, 2])
                    acc[ti, mb, 3] = _mfma(twc[3, mb], Bo[:, 2 * ti + 1], acc[ti, mb, 3])
            for mb in range(NMB):
                twc[0, mb], twc[2, mb] = _rot(twc[0, mb], twc[2, mb], r8[0, mb], r8[1, mb])
                twc[1, mb], twc[3, mb] = _rot(twc[1, mb], twc[3, mb], r8[0, mb], r8[1, mb])
        for mb in range(NMB):
            pe1, po1, qe1, qo1 = acc[0, mb]
            pe2, po2, qe2, qo2 = acc[1, mb]
            if L < 64:
                # class sums: a quarter of the four sample products (the seeds carry the 4)
                acc[0, mb] = np.stack([pe1 * pe2 + po1 * po2 + qe1 * qe2 + qo1 * qo2,
                                       pe1 * po2 + po1 * pe2 + qe1 * qo2 + qo1 * qe2,
                                       pe1 * qe2 + po1 * qo2 + qe1 * pe2 + qo1 * po2,
                                       pe1 * qo2 + po1 * qe2 + qe1 * po2 + qo1 * pe2])
                continue
            s1, d1, s2, d2 = pe1 + po1, pe1 - po1, qe1 + qo1, qe1 - qo1
            t1, u1, t2, u2_ = pe2 + po2, pe2 - po2, qe2 + qo2, qe2 - qo2
            hk, hmk = (s1 + s2) * (t1 + t2), (s1 - s2) * (t1 - t2)
            hpk, hpmk = (d1 + d2) * (u1 + u2_), (d1 - d2) * (u1 - u2_)
            a, b, dd, ee = hk + hmk, hpk + hpmk, hk - hmk, hpk - hpmk
            acc[0, mb] = np.stack([a + b, a - b, dd + ee, dd - ee])
        fold = 4.0 if L < 64 else 1.0
        NMR, ASD, AST = G["NMR"], G["ASD"], G["AST"]
        o = np.zeros((NMR, 4, 64, 4))
        zz = np.zeros(64)
        for mr in range(NMR):
            st = TWR[:, AST + 4 * mr:AST + 4 * mr + 4]
            for mb in range(NMB):
                ce, se, co, so = (TWR[:, ASD + 4 * (mr * NMBP + mb) + e].copy() for e in range(4))
                for r in range(4):
                    if 16 * mb + 4 * r > Q:
                        break  # all four samples past Q: the kernel skips the contraction
                    if r:
                        ce, se = _rot(ce, se, st[:, 0], st[:, 1])
                        co, so = _rot(co, so, st[:, 2], st[:, 3])
                    k = 16 * mb + 4 * r + g  # register r of lane group g holds this sample
                    w = np.where(k > Q, 0.0, np.where((k == 0) | (k == Q), 0.5, 1.0))
                    for ty, opnd in enumerate((ce, co, se, so)):
                        o[mr, ty] = _mfma(w * opnd, acc[0, mb, ty][:, r], o[mr, ty])
                    if mr == 0:
                        zz += w * fold * acc[0, mb, 0][:, r]
        zz = zz + _xor(zz, 16)
        zz = zz + _xor(zz, 32)
        eo = np.zeros(2 * 8 * NMP2)
        base = (h * 8 + pi) * NMP2
        for mr in range(NMR):
            for odd in range(2):
                for r in range(4):
                    m = 2 * (16 * mr + 4 * g + r) + (1 if odd else 2)
                    oc, os_ = o[mr, odd][:, r], o[mr, odd + 2][:, r]
                    pc, ps = _xor(oc, 8), _xor(os_, 8)
                    vc = np.where(h == 1, pc - oc, pc + oc)
                    vs = np.where(h == 1, ps - os_, ps + os_)
                    ok = m <= L
                    eo[(base + 2 * m)[ok]] = vc[ok]
                    eo[(base + 2 * m + 1)[ok]] = vs[ok]
        pz = _xor(zz, 8)
        ok = g == 0
        eo[base[ok]] = np.where(h == 1, pz - zz, pz + zz)[ok]
        return eo

    eos = [one_pass(p) for p in range(PASSES)]
    # theta analysis: thread tid owns row tri(tid, 0) (tid <= L) and the rows
    # with m > 0 numbered q = tid + NTH it
    WPf = plan.table(8)
    if NTH == 64:
        WPr = WPf.reshape(PASSES, NIT + 1, 64, 8)
        wrow = lambda it, t_: np.concatenate([WPr[p, it, t_] for p in range(PASSES)], axis=-1)
    else:
        WPr = WPf.reshape(NIT + 1, NTH, L)
        wrow = lambda it, t_: WPr[it, t_]
    eo_all = np.stack(eos)  # [pass][slots]
    y = np.zeros(G["K"])
    p1, p2 = m0(PASSES)
    f = p1 * p2 * NP
    fN, fS = f[0], f[8]
    for l in range(L + 1):
        wv = wrow(NIT, l)
        acc0 = sum(wv[8 * p + jj] * eo_all[p, (l & 1) * 8 * NMP2 + jj * NMP2] for p in range(PASSES) for jj in range(8))
        y[l * l + l] = acc0 + W[l * (l + 1) // 2, 0] * (fN + (-fS if l & 1 else fS))
    for it in range(NIT):
        for t_ in range(NTH):
            q = t_ + NTH * it
            if q >= NROW:
                continue
            l = int((math.sqrt(8 * q + 1) + 1) // 2)
            l -= (l * (l - 1) // 2 > q)
            l += ((l + 1) * l // 2 <= q)
            m = q - l * (l - 1) // 2 + 1
            er = ((l + m) & 1) * 8 * NMP2 + 2 * m
            wv = wrow(it, t_)
            ac = as_ = 0.0
            for p in range(PASSES):
                for jj in range(8):
                    ac += wv[8 * p + jj] * eo_all[p, er + jj * NMP2]
                    as_ += wv[8 * p + jj] * eo_all[p, er + jj * NMP2 + 1]
            y[l * l + l + m] = ac
            y[l * l + l - m] = as_
    return y


@pytest.mark.parametrize("L", [16, 32, 64])
def test_replay_matches_oracle(L):
    plan = gtp.Plan(L, L, L, flags=HOST_ONLY)
    rng = np.random.default_rng(700 + L)
    x1 = rng.standard_normal((L + 1) ** 2)
    x2 = rng.standard_normal((L + 1) ** 2)
    y = replay(plan, L, x1, x2)
    ref = oracle.gtp_grid(x1[None], x2[None], L, L, L)[0]
    assert np.abs(y - ref).max() <= 1e-12 * np.linalg.norm(ref)


def test_replay_matches_dense_oracle_L16():
    L = 16
    plan = gtp.Plan(L, L, L, flags=HOST_ONLY)
    rng = np.random.default_rng(716)
    x1 = rng.standard_normal((L + 1) ** 2)
    x2 = rng.standard_normal((L + 1) ** 2)
    ref = oracle.gtp(x1[None], x2[None], L, L, L)[0]
    assert np.abs(replay(plan, L, x1, x2) - ref).max() <= 1e-12 * np.linalg.norm(ref)


@pytest.mark.parametrize("L", [16, 32, 64])
def test_seed_table_angles(L):
    """TWR holds cos/sin of the stated multiples of phi_k = 2 pi k / NP."""
    plan = gtp.Plan(L, L, L, flags=HOST_ONLY)
    NP = plan.info()["NP"]
    G = _geo(L, NP)
    Q, NMBP = G["Q"], G["NMBP"]
    TWR = plan.table(5).reshape(64, G["TWRN"])
    cs = lambda m, k: (math.cos(2 * math.pi * (m * k % NP) / NP), math.sin(2 * math.pi * (m * k % NP) / NP))
    for lane in range(64):
        g, i = lane // 16, lane % 16
        for mb in range(G["NMB"]):
            # synthesis row i computes sample 16 mb + 4 (i mod 4) + i // 4
            k = 16 * mb + 4 * (i % 4) + i // 4
            want = [*cs(2 * g + 2, k), *cs(2 * g + 1, k), *cs(8, k)] if k <= Q else [0.0] * 6
            assert np.allclose(TWR[lane, 6 * mb:6 * mb + 6], want, atol=1e-14)
            k0 = 16 * mb + g
            fold = 4.0 if L < 64 else 1.0  # the weight all analysis samples share
            for mr in range(G["NMR"]):
                me = 2 * (16 * mr + i) + 2
                want = [fold * v for v in (*cs(me, k0), *cs(me - 1, k0))]
                want = [v if (me - e // 2) <= L else 0.0 for e, v in enumerate(want)]
                a = G["ASD"] + 4 * (mr * NMBP + mb)
                assert np.allclose(TWR[lane, a:a + 4], want, atol=1e-14)
        for mr in range(G["NMR"]):
            # rotation from register r to r + 1: four samples on
            me = 2 * (16 * mr + i) + 2
            want = [*cs(me, 4), *cs(me - 1, 4)]
            want = [v if (me - e // 2) <= L else 0.0 for e, v in enumerate(want)]
            a = G["AST"] + 4 * mr
            assert np.allclose(TWR[lane, a:a + 4], want, atol=1e-14)


@pytest.mark.parametrize("L", [16, 32, 64])
def test_scatter_map_is_a_bijection_into_the_image(L):
    """Every input coefficient gets its own LDS slot; sine slots are odd, m = 0 cos slots are quad starts."""
    plan = gtp.Plan(L, L, L, flags=HOST_ONLY)
    G = _geo(L, plan.info()["NP"])
    NTH = G["NTH"]
    xm = plan.table(9).astype(np.int64).reshape(NTH, -1)
    slots = {}
    for lane in range(NTH):
        for k in range(xm.shape[1]):
            idx = lane + NTH * k
            if idx < G["K"]:
                slots[idx] = xm[lane, k]
            else:
                assert xm[lane, k] == -1
    vals = np.array(list(slots.values()))
    assert len(set(vals.tolist())) == G["K"]
    assert vals.min() >= 0 and vals.max() < 4 * G["XQ"]
    for idx, sl in slots.items():
        l = int(math.isqrt(idx))
        ms = idx - l * l - l
        assert (sl % 4 == 1) == (ms < 0) and sl % 4 in (0, 1)


def test_no_wave_tables_for_other_degrees():
    for (a, b, c) in [(16, 16, 8), (8, 8, 8), (32, 16, 32), (64, 64, 32), (48, 48, 48)]:
        plan = gtp.Plan(a, b, c, flags=HOST_ONLY)
        for which in range(5, 10):
            assert plan.table(which).size == 0
