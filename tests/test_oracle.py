"""Pins for the fp64 oracle: everything here is checked against something other
than the oracle itself (closed forms, library routines, the Racah formula,
brute force, symmetry and equivariance), so that a dropped term, a wrong sign or
index, or a transposed operand anywhere in it fails at least one test."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import gtp_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def idx(l, m):
    return l * l + l + m


# --------------------------------------------------------------------------- quadrature

@pytest.mark.parametrize("n", [1, 2, 3, 7, 16, 33, 64])
def test_gauss_legendre_matches_numpy(n):
    x, w = O.gauss_legendre(n)
    xr, wr = np.polynomial.legendre.leggauss(n)
    assert np.allclose(x, xr, atol=1e-14, rtol=0)
    assert np.allclose(w, wr, atol=1e-14, rtol=0)


def test_gauss_legendre_exactness():
    n = 9
    x, w = O.gauss_legendre(n)
    for k in range(2 * n):
        exact = 0.0 if k % 2 else 2.0 / (k + 1)
        assert abs(np.dot(w, x ** k) - exact) < 1e-14
    # and not beyond: degree 2n is not integrated exactly
    assert abs(np.dot(w, x ** (2 * n)) - 2.0 / (2 * n + 1)) > 1e-8


def test_sphere_quadrature_area_and_monomials():
    th, ph, w = O.sphere_quadrature(6)
    assert abs(w.sum() - 4 * math.pi) < 1e-13
    z = np.cos(th)
    x = np.sin(th) * np.cos(ph)
    # int z^2 = 4pi/3, int x^2 z^2 = 4pi/15, int x^4 = 4pi/5 (textbook moments)
    assert abs(np.dot(w, z * z) - 4 * math.pi / 3) < 1e-13
    assert abs(np.dot(w, x * x * z * z) - 4 * math.pi / 15) < 1e-13
    assert abs(np.dot(w, x ** 4) - 4 * math.pi / 5) < 1e-13


# --------------------------------------------------------------------------- real SH

def test_real_sh_degree1_closed_form():
    rng = np.random.default_rng(1)
    r = rng.standard_normal((50, 3))
    r /= np.linalg.norm(r, axis=1, keepdims=True)
    Y = O.real_sh_xyz(1, r)
    c = math.sqrt(3 / (4 * math.pi))
    assert np.allclose(Y[:, 0], 1 / math.sqrt(4 * math.pi), atol=1e-15)
    assert np.allclose(Y[:, 1:4], c * r[:, [1, 2, 0]], atol=1e-14)


def test_real_sh_degree2_closed_form():
    rng = np.random.default_rng(2)
    r = rng.standard_normal((50, 3))
    r /= np.linalg.norm(r, axis=1, keepdims=True)
    x, y, z = r.T
    Y = O.real_sh_xyz(2, r)
    c = 0.5 * math.sqrt(15 / math.pi)
    want = np.stack([c * x * y, c * y * z, 0.25 * math.sqrt(5 / math.pi) * (3 * z * z - 1),
                     c * x * z, 0.5 * c * (x * x - y * y)], axis=1)
    assert np.allclose(Y[:, 4:9], want, atol=1e-14)


def test_real_sh_matches_scipy_complex_sh():
    """Real SH from scipy's complex SH (Condon-Shortley phase) by the unitary map
    Y_l^m = sqrt2 (-1)^m Re Yc_l^m, Y_l^-m = sqrt2 (-1)^m Im Yc_l^m."""
    from scipy.special import sph_harm_y
    rng = np.random.default_rng(3)
    th = np.arccos(rng.uniform(-1, 1, 40))
    ph = rng.uniform(0, 2 * math.pi, 40)
    L = 12
    Y = O.real_sh(L, th, ph)
    for l in range(L + 1):
        assert np.allclose(Y[:, idx(l, 0)], sph_harm_y(l, 0, th, ph).real, atol=1e-12)
        for m in range(1, l + 1):
            yc = sph_harm_y(l, m, th, ph)
            s = math.sqrt(2) * (-1) ** m
            assert np.allclose(Y[:, idx(l, m)], s * yc.real, atol=1e-12)
            assert np.allclose(Y[:, idx(l, -m)], s * yc.imag, atol=1e-12)


def test_real_sh_orthonormal():
    L = 10
    th, ph, w = O.sphere_quadrature(2 * L)
    Y = O.real_sh(L, th, ph)
    gram = (Y * w[:, None]).T @ Y
    assert np.abs(gram - np.eye(O.nsh(L))).max() < 1e-13


def test_real_sh_parity():
    rng = np.random.default_rng(4)
    r = rng.standard_normal((20, 3))
    Y = O.real_sh_xyz(6, r)
    Yn = O.real_sh_xyz(6, -r)
    sign = np.concatenate([np.full(2 * l + 1, (-1.0) ** l) for l in range(7)])
    assert np.allclose(Yn, Y * sign, atol=1e-13)


# --------------------------------------------------------------------------- Gaunt coefficients

def _fact(n):
    return math.factorial(n) if n >= 0 else None


def racah_3j(l1, l2, l3, m1, m2, m3):
    """Wigner 3j symbol by the Racah formula (Appendix, 3j closed form), exact
    rational arithmetic then a single square root."""
    if m1 + m2 + m3 != 0:
        return 0.0
    if l3 < abs(l1 - l2) or l3 > l1 + l2 or abs(m1) > l1 or abs(m2) > l2 or abs(m3) > l3:
        return 0.0
    tri = Fraction(_fact(l1 + l2 - l3) * _fact(l1 - l2 + l3) * _fact(-l1 + l2 + l3), _fact(l1 + l2 + l3 + 1))
    fac = (_fact(l1 - m1) * _fact(l1 + m1) * _fact(l2 - m2) * _fact(l2 + m2) * _fact(l3 - m3) * _fact(l3 + m3))
    kmin = max(0, l2 - l3 - m1, l1 - l3 + m2)
    kmax = min(l1 + l2 - l3, l1 - m1, l2 + m2)
    s = Fraction(0)
    for k in range(kmin, kmax + 1):
        s += Fraction((-1) ** k, _fact(k) * _fact(l1 + l2 - l3 - k) * _fact(l1 - m1 - k) * _fact(l2 + m2 - k)
                      * _fact(l3 - l2 + m1 + k) * _fact(l3 - l1 - m2 + k))
    val = math.sqrt(tri * fac) * float(s)
    return (-1) ** (l1 - l2 - m3) * val


def complex_gaunt(l1, l2, l3, m1, m2, m3):
    """int Yc Yc Yc dOmega for complex SH (Appendix Gaunt-3j relation)."""
    return (math.sqrt((2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1) / (4 * math.pi))
            * racah_3j(l1, l2, l3, 0, 0, 0) * racah_3j(l1, l2, l3, m1, m2, m3))


def real_from_complex(l):
    """U with Y_real[m] = sum_mu U[m, mu] Yc[mu] for our real convention
    (no CS phase in the real functions; Yc carries it)."""
    U = np.zeros((2 * l + 1, 2 * l + 1), dtype=complex)
    U[l, l] = 1.0
    for m in range(1, l + 1):
        # sqrt2 Q cos = ((-1)^m Yc^m + Yc^-m)/sqrt2 ; sqrt2 Q sin = ((-1)^m Yc^m - Yc^-m)/(i sqrt2)
        U[l + m, l + m] = (-1) ** m / math.sqrt(2)
        U[l + m, l - m] = 1 / math.sqrt(2)
        U[l - m, l + m] = (-1) ** m / (1j * math.sqrt(2))
        U[l - m, l - m] = -1 / (1j * math.sqrt(2))
    return U


def test_gaunt_matches_racah_formula():
    L = 3
    G = O.gaunt_tensor(L, L, L)
    for l1 in range(L + 1):
        for l2 in range(L + 1):
            for l3 in range(L + 1):
                Gc = np.zeros((2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1))
                for a in range(-l1, l1 + 1):
                    for b in range(-l2, l2 + 1):
                        for c in range(-l3, l3 + 1):
                            Gc[a + l1, b + l2, c + l3] = complex_gaunt(l1, l2, l3, a, b, c)
                U1, U2, U3 = real_from_complex(l1), real_from_complex(l2), real_from_complex(l3)
                Gr = np.einsum("ia,jb,kc,abc->ijk", U1, U2, U3, Gc)
                assert np.abs(Gr.imag).max() < 1e-13
                blk = G[l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2, l3 * l3:(l3 + 1) ** 2]
                assert np.abs(blk - Gr.real).max() < 1e-13, (l1, l2, l3)


def test_gaunt_matches_sympy_real_gaunt():
    """sympy builds its real SH from Condon-Shortley complex SH, so they differ
    from ours by a sign per function: (-1)^mu for mu > 0 and (-1)^(mu+1) for
    mu < 0.  With that map every entry up to degree 3 must agree."""
    from sympy.physics.wigner import real_gaunt
    L = 3
    G = O.gaunt_tensor(L, L, L)

    def sgn(l, mu):
        return (-1) ** mu if mu > 0 else ((-1) ** (mu + 1) if mu < 0 else 1)

    checked = 0
    for l1 in range(L + 1):
        for l2 in range(l1, L + 1):
            for l3 in range(l2, L + 1):
                if (l1 + l2 + l3) % 2 or l3 > l1 + l2:
                    continue
                for a in range(-l1, l1 + 1):
                    for b in range(-l2, l2 + 1):
                        for c in range(-l3, l3 + 1):
                            ref = float(real_gaunt(l1, l2, l3, a, b, c))
                            mine = G[idx(l1, a), idx(l2, b), idx(l3, c)]
                            s = sgn(l1, a) * sgn(l2, b) * sgn(l3, c)
                            assert abs(mine - s * ref) < 1e-13, (l1, l2, l3, a, b, c, mine, ref)
                            checked += 1
    assert checked > 200


def test_gaunt_closed_forms(golden):
    G = O.gaunt_tensor(2, 2, 2)
    for e in golden["gaunt"]:
        (l1, l2, l3), (m1, m2, m3) = e["l"], e["m"]
        assert abs(G[idx(l1, m1), idx(l2, m2), idx(l3, m3)] - e["value"]) < 1e-15


def test_gaunt_selection_rules_and_symmetry():
    L = 4
    G = O.gaunt_tensor(L, L, L)
    ls = np.array([l for l in range(L + 1) for _ in range(2 * l + 1)])
    ms = np.array([m for l in range(L + 1) for m in range(-l, l + 1)])
    l1, l2, l3 = np.meshgrid(ls, ls, ls, indexing="ij")
    m1, m2, m3 = np.meshgrid(ms, ms, ms, indexing="ij")
    parity = (l1 + l2 + l3) % 2 == 1
    triangle = (l3 > l1 + l2) | (l3 < np.abs(l1 - l2))
    a1, a2, a3 = np.abs(m1), np.abs(m2), np.abs(m3)
    mrule = ~((a3 == a1 + a2) | (a3 == np.abs(a1 - a2)))
    nsin = (m1 < 0).astype(int) + (m2 < 0) + (m3 < 0)
    sinrule = nsin % 2 == 1
    forbidden = parity | triangle | mrule | sinrule
    assert np.abs(G[forbidden]).max() < 1e-15
    assert (np.abs(G[~forbidden]) > 1e-12).sum() > 0.5 * (~forbidden).sum()
    for perm in [(1, 0, 2), (0, 2, 1), (2, 1, 0), (1, 2, 0), (2, 0, 1)]:
        assert np.abs(G - G.transpose(perm)).max() < 1e-15


# --------------------------------------------------------------------------- Gaunt tensor product

def test_worked_example(golden):
    e = golden["worked_example"]
    x = np.zeros(O.nsh(1))
    x[e["x_index"]] = e["x_value"]
    assert abs(e["x_value"] - math.sqrt(4 * math.pi / 3)) < 1e-15
    y = O.gtp(x, x, 1, 1, 2)
    want = np.zeros(9)
    for k, v in e["y"].items():
        want[int(k)] = v
    assert np.abs(y - want).max() < 1e-14
    assert np.abs(O.gtp_grid(x, x, 1, 1, 2) - want).max() < 1e-14


def test_scalar_channel_and_invariant():
    rng = np.random.default_rng(5)
    x1 = rng.standard_normal((7, O.nsh(3)))
    x2 = rng.standard_normal((7, O.nsh(2)))
    y = O.gtp(x1, x2, 3, 2, 4)
    # y_00 = <x1, x2>_{l <= min} / sqrt(4 pi): integrate F1 F2 against the constant Y_0^0
    assert np.allclose(y[:, 0], np.einsum("nk,nk->n", x1[:, :9], x2) / math.sqrt(4 * math.pi), atol=1e-13)
    # product with a constant function c*Y_0^0 scales by c/sqrt(4 pi)
    e0 = np.zeros((7, O.nsh(2)))
    e0[:, 0] = 2.5
    y = O.gtp(x1, e0, 3, 2, 3)
    assert np.allclose(y, 2.5 / math.sqrt(4 * math.pi) * x1, atol=1e-13)


def test_commutative_and_parity():
    rng = np.random.default_rng(6)
    a = rng.standard_normal((5, O.nsh(3)))
    b = rng.standard_normal((5, O.nsh(3)))
    assert np.allclose(O.gtp(a, b, 3, 3, 5), O.gtp(b, a, 3, 3, 5), atol=1e-13)
    s = np.concatenate([np.full(2 * l + 1, (-1.0) ** l) for l in range(6)])
    # inversion: x -> (-1)^l x on both inputs leaves F1 F2 even => y -> (-1)^l y
    assert np.allclose(O.gtp(a * s[:16], b * s[:16], 3, 3, 5), O.gtp(a, b, 3, 3, 5) * s, atol=1e-13)
    # odd x odd -> even only
    ao = a * (s[:16] < 0)
    bo = b * (s[:16] < 0)
    y = O.gtp(ao, bo, 3, 3, 5)
    assert np.abs(y * (s < 0)).max() < 1e-14


def test_mode_a_equals_brute_force_grid():
    """Pointwise multiplication on a dense 200 x 400 GL x uniform grid."""
    rng = np.random.default_rng(7)
    L1, L2, Lout = 3, 4, 4
    a = rng.standard_normal((4, O.nsh(L1)))
    b = rng.standard_normal((4, O.nsh(L2)))
    t, wt = O.gauss_legendre(200)
    ph = 2 * math.pi * np.arange(400) / 400
    TH, PH = np.meshgrid(np.arccos(t), ph, indexing="ij")
    W = np.outer(wt, np.full(400, 2 * math.pi / 400))
    Y = O.real_sh(4, TH, PH)
    F = np.einsum("nk,tpk->ntp", a, Y[..., :O.nsh(L1)]) * np.einsum("nk,tpk->ntp", b, Y[..., :O.nsh(L2)])
    ybf = np.einsum("ntp,tpk->nk", F * W, Y[..., :O.nsh(Lout)])
    assert np.abs(O.gtp(a, b, L1, L2, Lout) - ybf).max() < 1e-12
    assert np.abs(O.gtp_grid(a, b, L1, L2, Lout) - ybf).max() < 1e-12


def test_truncation_and_zero_fill():
    rng = np.random.default_rng(8)
    a = rng.standard_normal((3, O.nsh(2)))
    b = rng.standard_normal((3, O.nsh(1)))
    y = O.gtp(a, b, 2, 1, 5)
    assert np.abs(y[:, O.nsh(3):]).max() < 1e-14
    assert np.abs(O.gtp(a, b, 2, 1, 2) - y[:, :9]).max() < 1e-14


def test_equivariance_random_rotation():
    rng = np.random.default_rng(9)
    L1, L2, Lout = 2, 3, 4
    R = O.random_rotation(rng)
    assert abs(np.linalg.det(R) - 1) < 1e-12
    D = O.wigner_d_real(max(L1, L2, Lout), R)
    D1, D2, D3 = D[:O.nsh(L1), :O.nsh(L1)], D[:O.nsh(L2), :O.nsh(L2)], D[:O.nsh(Lout), :O.nsh(Lout)]
    assert np.abs(D3 @ D3.T - np.eye(O.nsh(Lout))).max() < 1e-12
    a = rng.standard_normal((5, O.nsh(L1)))
    b = rng.standard_normal((5, O.nsh(L2)))
    y = O.gtp(a, b, L1, L2, Lout)
    yr = O.gtp(a @ D1.T, b @ D2.T, L1, L2, Lout)
    assert np.abs(yr - y @ D3.T).max() < 1e-12


def test_wigner_d_degree1_is_rotation():
    rng = np.random.default_rng(10)
    R = O.random_rotation(rng)
    D = O.wigner_d_real(1, R)
    P = np.array([[0, 1, 0], [0, 0, 1], [1, 0, 0]])  # (x,y,z) -> (y,z,x) ordering of Y_1
    assert np.abs(D[1:4, 1:4] - P @ R @ P.T).max() < 1e-13


# --------------------------------------------------------------------------- the three stages

def test_sh2fourier_closed_forms(golden):
    for key in ("Y1_0", "Y1_1"):
        e = golden["sh2fourier"][key]
        L = e["L"]
        x = np.zeros(O.nsh(L))
        x[e["index"]] = 1.0
        g = O.sh2fourier(x, L)
        want = np.zeros_like(g)
        for u, v, re, im in e["nonzero"]:
            want[u + L, v + L] = re + 1j * im
        assert np.abs(g - want).max() < 1e-15


def test_sh2fourier_sparsity_hermitian_and_pointwise():
    rng = np.random.default_rng(11)
    L = 5
    for l in range(L + 1):
        for m in range(-l, l + 1):
            x = np.zeros(O.nsh(L))
            x[idx(l, m)] = 1.0
            g = O.sh2fourier(x, L)
            v = np.arange(-L, L + 1)
            off = np.abs(v) != abs(m)
            assert np.abs(g[:, off]).max() < 1e-14  # nonzero only for m = +-v (Sec. 3.2)
            uu = np.arange(-L, L + 1)
            if l < L:
                assert np.abs(g[np.abs(uu) > l, :]).max() < 1e-14  # theta degree <= l
    x = rng.standard_normal((3, O.nsh(L)))
    g = O.sh2fourier(x, L)
    assert np.abs(g - np.conj(g[:, ::-1, ::-1])).max() < 1e-14  # real function
    th = np.arccos(rng.uniform(-1, 1, 30))
    ph = rng.uniform(0, 2 * math.pi, 30)
    u = np.arange(-L, L + 1)
    E = np.exp(1j * (u[None, :, None] * th[:, None, None] + u[None, None, :] * ph[:, None, None]))
    Fs = np.einsum("nuv,puv->np", g, E)
    F = x @ O.real_sh(L, th, ph).T
    assert np.abs(Fs.imag).max() < 1e-13
    assert np.abs(Fs.real - F).max() < 1e-12


def test_fourier_conv_matches_scipy():
    from scipy.signal import convolve2d
    rng = np.random.default_rng(12)
    g1 = rng.standard_normal((5, 5)) + 1j * rng.standard_normal((5, 5))
    g2 = rng.standard_normal((7, 7)) + 1j * rng.standard_normal((7, 7))
    assert np.abs(O.fourier_conv(g1, g2) - convolve2d(g1, g2, mode="full")).max() < 1e-13


def test_fourier_conv_is_pointwise_product():
    rng = np.random.default_rng(13)
    a = rng.standard_normal(O.nsh(2))
    b = rng.standard_normal(O.nsh(3))
    g3 = O.fourier_conv(O.sh2fourier(a, 2), O.sh2fourier(b, 3))
    th = rng.uniform(0, math.pi, 20)
    ph = rng.uniform(0, 2 * math.pi, 20)
    u = np.arange(-5, 6)
    E = np.exp(1j * (u[None, :, None] * th[:, None, None] + u[None, None, :] * ph[:, None, None]))
    F3 = np.einsum("uv,puv->p", g3, E)
    Y = O.real_sh(3, th, ph)
    assert np.abs(F3 - (Y[:, :9] @ a) * (Y @ b)).max() < 1e-12


def test_fourier2sh_z00_closed_form(golden):
    L3 = 4
    for u, re, im in golden["fourier2sh_z00"]["values"]:
        g = np.zeros((2 * L3 + 1, 2 * L3 + 1), dtype=complex)
        g[u + L3, L3] = 1.0
        y = O.fourier2sh(g, L3, 0)
        assert abs(y[0] - (re + 1j * im)) < 1e-13, (u, y[0])


def test_fourier2sh_converged_and_round_trip():
    rng = np.random.default_rng(14)
    L = 4
    x = rng.standard_normal((3, O.nsh(L)))
    g = O.sh2fourier(x, L)
    y = O.fourier2sh(g, L, 6)
    assert np.abs(y.imag).max() < 1e-13
    assert np.abs(y.real[:, :O.nsh(L)] - x).max() < 1e-13
    assert np.abs(y.real[:, O.nsh(L):]).max() < 1e-13
    y2 = O.fourier2sh(g, L, 6, n_theta=2 * (2 * (L + 6) + 48))
    assert np.abs(y2 - y).max() < 1e-14


@pytest.mark.parametrize("L1,L2,Lout", [(2, 2, 2), (1, 3, 2), (3, 2, 6), (0, 2, 2), (2, 0, 1), (3, 3, 1)])
def test_three_stages_equal_gaunt_contraction(L1, L2, Lout):
    rng = np.random.default_rng(15 + L1 + 7 * L2 + 49 * Lout)
    a = rng.standard_normal((4, O.nsh(L1)))
    b = rng.standard_normal((4, O.nsh(L2)))
    g3 = O.fourier_conv(O.sh2fourier(a, L1), O.sh2fourier(b, L2))
    y = O.fourier2sh(g3, L1 + L2, Lout)
    assert np.abs(y.imag).max() < 1e-13
    assert np.abs(y.real - O.gtp(a, b, L1, L2, Lout)).max() < 1e-12


# --------------------------------------------------------------------------- many-body

def test_selfproduct_modes():
    rng = np.random.default_rng(16)
    L, Lout = 2, 3
    x = rng.standard_normal((6, O.nsh(L)))
    # nu = 2: both modes are the plain product
    y2 = O.gtp(x, x, L, L, Lout)
    assert np.abs(O.selfproduct(x, L, 2, Lout, "stepwise") - y2).max() < 1e-13
    assert np.abs(O.selfproduct(x, L, 2, Lout, "fused") - y2).max() < 1e-13
    # nu = 3 stepwise is the literal chain with truncation to Lout
    y3s = O.gtp(y2, x, Lout, L, Lout)
    assert np.abs(O.selfproduct(x, L, 3, Lout, "stepwise") - y3s).max() < 1e-13
    # nu = 3 fused is the chain without truncation (generalized Gaunt)
    yfull = O.gtp(O.gtp(x, x, L, L, 2 * L), x, 2 * L, L, Lout)
    assert np.abs(O.selfproduct(x, L, 3, Lout, "fused") - yfull).max() < 1e-12
    # the two differ when the intermediate is truncated (Lout < 2L) ...
    assert np.abs(yfull - y3s).max() > 1e-3
    # ... and agree when it is not
    assert np.abs(O.selfproduct(x, L, 3, 2 * L, "fused") - O.selfproduct(x, L, 3, 2 * L, "stepwise")).max() < 1e-12
    # nu = 1 is the (zero-padded) input
    assert np.abs(O.selfproduct(x, L, 1, Lout, "stepwise")[:, :9] - x).max() == 0


# --------------------------------------------------------------------------- gradients (VJP)

@pytest.mark.parametrize("L1,L2,Lout", [(2, 2, 2), (1, 2, 3), (3, 1, 2), (2, 2, 1)])
def test_vjp_brute_force_basis(L1, L2, Lout):
    """y is linear in x1: dx1[i] = <dy, gtp(e_i, x2)> for every basis vector e_i (and likewise for x2)."""
    rng = np.random.default_rng(40 + L1 + 5 * L2 + 25 * Lout)
    x1 = rng.standard_normal((3, O.nsh(L1)))
    x2 = rng.standard_normal((3, O.nsh(L2)))
    dy = rng.standard_normal((3, O.nsh(Lout)))
    dx1, dx2 = O.gtp_vjp(x1, x2, dy, L1, L2, Lout)
    for i in range(O.nsh(L1)):
        e = np.zeros_like(x1)
        e[:, i] = 1.0
        assert np.abs(dx1[:, i] - np.einsum("nk,nk->n", dy, O.gtp(e, x2, L1, L2, Lout))).max() < 1e-13
    for j in range(O.nsh(L2)):
        e = np.zeros_like(x2)
        e[:, j] = 1.0
        assert np.abs(dx2[:, j] - np.einsum("nk,nk->n", dy, O.gtp(x1, e, L1, L2, Lout))).max() < 1e-13


@pytest.mark.parametrize("L1,L2,Lout", [(6, 6, 6), (3, 5, 4), (4, 2, 9), (16, 16, 16)])
def test_vjp_adjoint_identity(L1, L2, Lout):
    """Euler's identity for a bilinear form: <dx1, x1> = <dy, y> = <dx2, x2>."""
    rng = np.random.default_rng(50 + L1)
    x1 = rng.standard_normal((4, O.nsh(L1)))
    x2 = rng.standard_normal((4, O.nsh(L2)))
    dy = rng.standard_normal((4, O.nsh(Lout)))
    dx1, dx2 = O.gtp_vjp(x1, x2, dy, L1, L2, Lout)
    s = np.einsum("nk,nk->n", dy, O.gtp_grid(x1, x2, L1, L2, Lout))
    assert np.abs(np.einsum("ni,ni->n", dx1, x1) - s).max() < 1e-11 * (1 + np.abs(s).max())
    assert np.abs(np.einsum("nj,nj->n", dx2, x2) - s).max() < 1e-11 * (1 + np.abs(s).max())


def test_vjp_gaunt_and_grid_modes_agree():
    rng = np.random.default_rng(52)
    L1, L2, Lout = 5, 4, 6
    x1 = rng.standard_normal((5, O.nsh(L1)))
    x2 = rng.standard_normal((5, O.nsh(L2)))
    dy = rng.standard_normal((5, O.nsh(Lout)))
    a1, a2 = O.gtp_vjp(x1, x2, dy, L1, L2, Lout, mode="gaunt")
    b1, b2 = O.gtp_vjp(x1, x2, dy, L1, L2, Lout, mode="grid")
    assert np.abs(a1 - b1).max() < 1e-12 and np.abs(a2 - b2).max() < 1e-12


def test_vjp_closed_forms():
    """Gradients that follow from Legendre algebra by hand.

    F2 = z (x2 = sqrt(4 pi / 3) e_(1,0)) and dy = e_(2,0): dx1 = P_L1(z Y_2^0),
    and z P_2 = (3/5) P_3 + (2/5) P_1 gives dx1 = (2/sqrt 15) Y_1^0 + (3/sqrt 35) Y_3^0.
    dy = e_(0,0): dx1 = x2 / sqrt(4 pi) (the gradient of y_00 = <x1, x2> / sqrt(4 pi)).
    A constant F2 = 1 (x2 = sqrt(4 pi) e_0) makes y = P_Lout(x1): dx1 = P_L1(dy), and
    dx2[0] = <x1, dy> / sqrt(4 pi) over the common degrees."""
    L1, L2, Lout = 4, 1, 2
    x2 = np.zeros(O.nsh(L2))
    x2[idx(1, 0)] = math.sqrt(4 * math.pi / 3)
    x1 = np.random.default_rng(53).standard_normal(O.nsh(L1))
    dy = np.zeros(O.nsh(Lout))
    dy[idx(2, 0)] = 1.0
    dx1, _ = O.gtp_vjp(x1, x2, dy, L1, L2, Lout)
    want = np.zeros(O.nsh(L1))
    want[idx(1, 0)] = 2 / math.sqrt(15)
    want[idx(3, 0)] = 3 / math.sqrt(35)
    assert np.abs(dx1 - want).max() < 1e-14
    dy = np.zeros(O.nsh(Lout))
    dy[0] = 1.0
    dx1, _ = O.gtp_vjp(x1, x2, dy, L1, L2, Lout)
    want = np.zeros(O.nsh(L1))
    want[: O.nsh(L2)] = x2 / math.sqrt(4 * math.pi)
    assert np.abs(dx1 - want).max() < 1e-14
    rng = np.random.default_rng(54)
    for (L1, L2, Lout) in [(3, 0, 5), (5, 2, 3)]:
        x1 = rng.standard_normal(O.nsh(L1))
        x2 = np.zeros(O.nsh(L2))
        x2[0] = math.sqrt(4 * math.pi)
        dy = rng.standard_normal(O.nsh(Lout))
        dx1, dx2 = O.gtp_vjp(x1, x2, dy, L1, L2, Lout)
        k = min(O.nsh(L1), O.nsh(Lout))
        want = np.zeros(O.nsh(L1))
        want[:k] = dy[:k]
        assert np.abs(dx1 - want).max() < 1e-13
        assert abs(dx2[0] - x1[:k] @ dy[:k] / math.sqrt(4 * math.pi)) < 1e-13


def test_vjp_is_a_truncated_product():
    """G is symmetric in its three (l, m) pairs: dx1 = P_L1(gtp(dy, x2)), dx2 = P_L2(gtp(dy, x1))."""
    rng = np.random.default_rng(55)
    L1, L2, Lout = 3, 5, 4
    x1 = rng.standard_normal((6, O.nsh(L1)))
    x2 = rng.standard_normal((6, O.nsh(L2)))
    dy = rng.standard_normal((6, O.nsh(Lout)))
    dx1, dx2 = O.gtp_vjp(x1, x2, dy, L1, L2, Lout)
    assert np.abs(dx1 - O.gtp(dy, x2, Lout, L2, L1)).max() < 1e-13
    assert np.abs(dx2 - O.gtp(dy, x1, Lout, L1, L2)).max() < 1e-13


# --------------------------------------------------------------------------- weighted products

def test_weighted_ones_and_constants():
    rng = np.random.default_rng(60)
    L1, L2, Lout = 3, 2, 4
    a = rng.standard_normal((5, O.nsh(L1)))
    b = rng.standard_normal((5, O.nsh(L2)))
    y = O.gtp(a, b, L1, L2, Lout)
    assert np.abs(O.gtp_weighted(a, b, np.ones(L1 + 1), np.ones(L2 + 1), np.ones(Lout + 1), L1, L2, Lout) - y).max() < 1e-13
    # constant weights s1, s2, so multiply the product by s1 s2 so
    yw = O.gtp_weighted(a, b, np.full(L1 + 1, 2.0), np.full(L2 + 1, -0.5), np.full(Lout + 1, 3.0), L1, L2, Lout)
    assert np.abs(yw - (-3.0) * y).max() < 1e-13


def test_weighted_degree_mask_closed_form():
    """Keeping only degree 0 of x1 (F1 = x1_00 / sqrt(4 pi)): y = x1_00 / sqrt(4 pi) * P_Lout(x2);
    an output mask keeps exactly the unmasked degrees of the plain product."""
    rng = np.random.default_rng(61)
    L1, L2, Lout = 4, 3, 5
    a = rng.standard_normal((4, O.nsh(L1)))
    b = rng.standard_normal((4, O.nsh(L2)))
    m1 = np.zeros(L1 + 1)
    m1[0] = 1.0
    y = O.gtp_weighted(a, b, m1, np.ones(L2 + 1), np.ones(Lout + 1), L1, L2, Lout)
    want = np.zeros((4, O.nsh(Lout)))
    want[:, : O.nsh(L2)] = a[:, :1] / math.sqrt(4 * math.pi) * b
    assert np.abs(y - want).max() < 1e-13
    mo = np.array([0.0, 1.0, 0.0, 1.0, 0.0, 1.0])
    y = O.gtp_weighted(a, b, np.ones(L1 + 1), np.ones(L2 + 1), mo, L1, L2, Lout)
    keep = np.concatenate([np.full(2 * l + 1, mo[l]) for l in range(Lout + 1)])
    assert np.abs(y - O.gtp(a, b, L1, L2, Lout) * keep).max() < 1e-13


def test_weighted_degree_blocks_partition_the_product():
    """Summing the single-block products (w1 = e_l1, w2 = e_l2) over all degree pairs gives the plain product."""
    rng = np.random.default_rng(62)
    L1, L2, Lout = 2, 3, 3
    a = rng.standard_normal((3, O.nsh(L1)))
    b = rng.standard_normal((3, O.nsh(L2)))
    tot = np.zeros((3, O.nsh(Lout)))
    for l1 in range(L1 + 1):
        for l2 in range(L2 + 1):
            e1 = np.eye(L1 + 1)[l1]
            e2 = np.eye(L2 + 1)[l2]
            part = O.gtp_weighted(a, b, e1, e2, np.ones(Lout + 1), L1, L2, Lout)
            # triangle rule: the (l1, l2) block reaches only |l1 - l2| <= l <= l1 + l2 with l1 + l2 + l even
            for l in range(Lout + 1):
                if l < abs(l1 - l2) or l > l1 + l2 or (l1 + l2 + l) % 2:
                    assert np.abs(part[:, l * l:(l + 1) ** 2]).max() < 1e-13
            tot += part
    assert np.abs(tot - O.gtp(a, b, L1, L2, Lout)).max() < 1e-13


def test_weighted_sum_equals_scaled_route():
    """The paper's equivalence: the double sum over degree pairs equals the
    product of the weighted inputs' functions, scaled per output degree."""
    rng = np.random.default_rng(63)
    L1, L2, Lout = 5, 4, 6
    a = rng.standard_normal((6, O.nsh(L1)))
    b = rng.standard_normal((6, O.nsh(L2)))
    w1 = rng.standard_normal((6, L1 + 1))
    w2 = rng.standard_normal((6, L2 + 1))
    wo = rng.standard_normal((6, Lout + 1))
    ys = O.gtp_weighted(a, b, w1, w2, wo, L1, L2, Lout, mode="sum")
    yc = O.gtp_weighted(a, b, w1, w2, wo, L1, L2, Lout, mode="scaled")
    assert np.abs(ys - yc).max() < 1e-12


# --------------------------------------------------------------------------- channel mixing

def test_channel_mix_diagonal_weights_are_channel_wise():
    """W[co, c1, c2] = d(co, c1) d(co, c2) reduces to the channel-wise product."""
    rng = np.random.default_rng(80)
    B, C, L = 3, 4, 2
    x1 = rng.standard_normal((B, C, O.nsh(L)))
    x2 = rng.standard_normal((B, C, O.nsh(L)))
    W = np.zeros((C, C, C))
    for c in range(C):
        W[c, c, c] = 1.0
    assert np.abs(O.channel_mix(x1, x2, W, L, L, L) - O.gtp(x1, x2, L, L, L)).max() < 1e-13


def test_channel_mix_rank_one_weights():
    """W = u (x) v (x) w: y[co] = u[co] GTP(sum_c1 v[c1] x1[c1], sum_c2 w[c2] x2[c2]) (bilinearity)."""
    rng = np.random.default_rng(81)
    B, C1, C2, Co, L1, L2, Lo = 2, 3, 5, 4, 2, 3, 3
    x1 = rng.standard_normal((B, C1, O.nsh(L1)))
    x2 = rng.standard_normal((B, C2, O.nsh(L2)))
    u, v, w = rng.standard_normal(Co), rng.standard_normal(C1), rng.standard_normal(C2)
    W = np.einsum("o,i,j->oij", u, v, w)
    a = np.einsum("i,bik->bk", v, x1)
    b = np.einsum("j,bjk->bk", w, x2)
    want = u[None, :, None] * O.gtp(a, b, L1, L2, Lo)[:, None, :]
    assert np.abs(O.channel_mix(x1, x2, W, L1, L2, Lo) - want).max() < 1e-12


def test_channel_mix_single_pair_picks_one_product():
    rng = np.random.default_rng(82)
    B, C1, C2, Co, L = 2, 3, 2, 2, 3
    x1 = rng.standard_normal((B, C1, O.nsh(L)))
    x2 = rng.standard_normal((B, C2, O.nsh(L)))
    W = np.zeros((Co, C1, C2))
    W[1, 2, 0] = -2.5
    y = O.channel_mix(x1, x2, W, L, L, L)
    assert np.abs(y[:, 0]).max() == 0.0
    assert np.abs(y[:, 1] + 2.5 * O.gtp(x1[:, 2], x2[:, 0], L, L, L)).max() < 1e-13


# --------------------------------------------------------------------------- rotated-frame convolution

def _filter(h, r, L2):
    """x2[b, c, (l, m)] = h[b, c, l] Y_l^m(r_b / |r_b|)."""
    rr = np.asarray(r, dtype=np.float64)
    n = np.linalg.norm(rr, axis=1, keepdims=True)
    u = np.where(n > 0, rr / np.where(n > 0, n, 1.0), np.array([0.0, 0.0, 1.0]))
    Y = O.real_sh_xyz(L2, u)
    deg = np.concatenate([np.full(2 * l + 1, l) for l in range(L2 + 1)])
    return h[:, :, deg] * Y[:, None, :]


def test_edge_rotation_maps_direction_to_pole():
    rng = np.random.default_rng(70)
    for _ in range(20):
        r = rng.standard_normal(3) * rng.uniform(0.1, 5.0)
        R = O.edge_rotation(r)
        assert np.allclose(R @ R.T, np.eye(3), atol=1e-14) and abs(np.linalg.det(R) - 1) < 1e-13
        assert np.allclose(R @ (r / np.linalg.norm(r)), [0, 0, 1], atol=1e-14)
    assert np.allclose(O.edge_rotation(np.zeros(3)), np.eye(3))


def test_rotated_filter_has_only_m0():
    """The premise of eq. sh2fs-escn: in the edge frame the SH filter is h_l Y_l^0(pole) at m = 0 only."""
    rng = np.random.default_rng(71)
    L = 5
    for _ in range(5):
        r = rng.standard_normal(3)
        h = rng.standard_normal(L + 1)
        f = _filter(h[None, None, :], r[None, :], L)[0, 0]
        D = O.wigner_d_real(L, O.edge_rotation(r))
        fr = D @ f
        for l in range(L + 1):
            want = np.zeros(2 * l + 1)
            want[l] = h[l] * math.sqrt((2 * l + 1) / (4 * math.pi))
            assert np.abs(fr[l * l:(l + 1) ** 2] - want).max() < 1e-12


@pytest.mark.parametrize("L1,L2,Lout", [(1, 1, 1), (3, 3, 3), (6, 6, 6), (3, 2, 4), (2, 4, 3)])
def test_conv_escn_equals_plain_product(L1, L2, Lout):
    """GTP commutes with rotations: the edge-frame result equals the plain product with the filter."""
    rng = np.random.default_rng(72 + L1 + L2)
    B, C = 4, 3
    x = rng.standard_normal((B, C, O.nsh(L1)))
    r = rng.standard_normal((B, 3))
    r[0] = [0.0, 0.0, 0.0]  # zero vector: direction (0, 0, 1)
    r[1] = [0.0, 0.0, -2.0]  # south pole
    h = rng.standard_normal((B, C, L2 + 1))
    y = O.conv_escn(x, r, h, L1, L2, Lout)
    want = O.gtp(x, _filter(h, r, L2), L1, L2, Lout)
    assert np.abs(y - want).max() < 1e-12


def test_conv_escn_independent_of_the_rotation_chosen():
    """Any rotation taking the edge to the pole gives the same result (here R_z(g) R_b)."""
    rng = np.random.default_rng(73)
    L = 4
    x = rng.standard_normal((3, 2, O.nsh(L)))
    r = rng.standard_normal((3, 3))
    h = rng.standard_normal((3, 2, L + 1))

    def spun(rv):
        g = 0.7
        Rz = np.array([[math.cos(g), -math.sin(g), 0], [math.sin(g), math.cos(g), 0], [0, 0, 1]])
        return Rz @ O.edge_rotation(rv)

    a = O.conv_escn(x, r, h, L, L, L)
    b = O.conv_escn(x, r, h, L, L, L, rotation=spun)
    assert np.abs(a - b).max() < 1e-12


def test_max_rel_err():
    y = np.array([[3.0, 4.0], [0.0, 0.0]])
    assert O.max_rel_err(y, y) == 0
    assert abs(O.max_rel_err(y + [[0.5, 0], [0, 0]], y) - 0.1) < 1e-15
    assert abs(O.max_rel_err(y + [[0, 0], [0, 1e-3]], y) - 1e-3) < 1e-15


@pytest.mark.parametrize("L1,L2,Lout", [(2, 2, 2), (3, 1, 4), (2, 3, 1), (12, 10, 12)])
def test_weighted_vjp_pins(L1, L2, Lout):
    """gtp_weighted_vjp against what the definition fixes: s = <dy, y> is
    linear in each weight row, so a unit step of one weight changes s by
    exactly that weight's gradient (finite difference, exact); s is
    homogeneous of degree one in each of w1, w2, wo and x1, x2, so
    sum_l w[l] dw[l] = s = <dx1, x1> = <dx2, x2> (Euler); with unit weights
    the input gradients are the plain product's (gtp_vjp); weights that are
    zero outside one degree pick that degree's block."""
    rng = np.random.default_rng(L1 + 10 * L2 + 100 * Lout)
    n = 5
    x1 = rng.standard_normal((n, O.nsh(L1)))
    x2 = rng.standard_normal((n, O.nsh(L2)))
    dy = rng.standard_normal((n, O.nsh(Lout)))
    w1 = rng.standard_normal(L1 + 1)
    w2 = rng.standard_normal(L2 + 1)
    wo = rng.standard_normal(Lout + 1)

    def s_of(a, b, c):
        return np.sum(dy * O.gtp_weighted(x1, x2, a, b, c, L1, L2, Lout), axis=1)

    dx1, dx2, dw1, dw2, dwo = O.gtp_weighted_vjp(x1, x2, w1, w2, wo, dy, L1, L2, Lout)
    s0 = s_of(w1, w2, wo)
    scale = np.abs(s0).max() + 1.0
    for l in range(L1 + 1):
        e = np.zeros(L1 + 1)
        e[l] = 1.0
        assert np.abs(s_of(w1 + e, w2, wo) - s0 - dw1[:, l]).max() < 1e-10 * scale
    for l in range(L2 + 1):
        e = np.zeros(L2 + 1)
        e[l] = 1.0
        assert np.abs(s_of(w1, w2 + e, wo) - s0 - dw2[:, l]).max() < 1e-10 * scale
    for l in range(Lout + 1):
        e = np.zeros(Lout + 1)
        e[l] = 1.0
        assert np.abs(s_of(w1, w2, wo + e) - s0 - dwo[:, l]).max() < 1e-10 * scale
    for g in (dw1 @ w1, dw2 @ w2, dwo @ wo, np.sum(dx1 * x1, 1), np.sum(dx2 * x2, 1)):
        assert np.abs(g - s0).max() < 1e-10 * scale
    p1, p2 = O.gtp_vjp(x1, x2, dy, L1, L2, Lout)
    u1, u2, *_ = O.gtp_weighted_vjp(x1, x2, np.ones(L1 + 1), np.ones(L2 + 1), np.ones(Lout + 1), dy, L1, L2, Lout)
    assert np.abs(u1 - p1).max() < 1e-12 * scale and np.abs(u2 - p2).max() < 1e-12 * scale
    # a degree mask on x1 keeps only that degree's block of dx1
    m = np.zeros(L1 + 1)
    m[1] = 1.0
    q1, *_ = O.gtp_weighted_vjp(x1, x2, m, w2, wo, dy, L1, L2, Lout)
    assert np.abs(np.delete(q1, np.arange(1, 4), axis=1)).max() == 0.0
