"""Plain fp64 CPU oracle for the Gaunt Tensor Product (Luo et al., ICLR 2024,
"Enabling efficient equivariant operations in the Fourier basis via Gaunt
Tensor Products").

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, table or
constant generator with the HIP library; the only thing both sides consume is
the seeded input generator in ``paper_2401_10216_amd/inputs.py`` (which does no
arithmetic of the method).

Everything is numpy float64 and written to be checked against the paper by eye:

* real spherical harmonics (Appendix "Spherical Harmonics"), z polar axis, no
  Condon-Shortley phase, index ``i = l*l + l + m``;
* real Gaunt coefficients (Sec. 3.1, eq. ``equivalence-wigner-eckart``) by
  Gauss-Legendre (in cos theta) x uniform-phi quadrature, which is exact for the
  polynomial degree of a triple product;
* the Gaunt tensor product itself (Sec. 3.1, eq. ``tp-eq-mul``) as a dense
  contraction of the Gaunt tensor ("mode A"), and as the pointwise product of
  the two spherical functions on an exact quadrature grid ("mode B");
* its gradients (the vector-Jacobian product of the bilinear map), from the
  same Gaunt tensor or the same quadrature;
* the weighted product with per-degree weights (Sec. 3.1, eq.
  ``tp-eq-mul-weight``) as the double sum over degree pairs;
* the equivariant convolution in the edge frame (Sec. 3.3, eq.
  ``sh2fs-escn``): rotate, multiply by the m = 0 filter, rotate back;
* channel mixing: every pair product of two channel sets, combined with a
  weight tensor;
* the three stages of Sec. 3.2 individually: SH -> 2D Fourier (eq. ``sh-fs``),
  the 2D convolution (eq. ``2D-conv``) and Fourier -> SH (eq. ``fs-sh``), each
  from its plain definition;
* the many-body self product (Sec. 3.3 and Appendix "Implementation
  Details", generalized Gaunt coefficients), stepwise and fused;
* real Wigner-D matrices by quadrature, for the equivariance pin (Appendix D).

Every function is pinned by ``tests/test_oracle.py`` against closed forms,
library routines (scipy spherical harmonics, sympy real Gaunt, numpy
Gauss-Legendre, scipy convolve2d), the Racah formula, brute force and
equivariance.  Nothing here is "parity unpinned".
"""
from __future__ import annotations

import math

import numpy as np

FOUR_PI = 4.0 * math.pi


def nsh(L: int) -> int:
    """Number of real SH coefficients up to degree L: (L+1)^2 (Sec. 2)."""
    return (L + 1) * (L + 1)


# ---------------------------------------------------------------------------
# Quadrature
# ---------------------------------------------------------------------------

def gauss_legendre(n: int):
    """Gauss-Legendre nodes/weights on [-1, 1] by Newton iteration on P_n.

    Textbook construction (Golub & Welsch give the same rule); exact for
    polynomials of degree <= 2n-1.
    """
    if n < 1:
        raise ValueError("n >= 1")
    k = np.arange(1, n + 1, dtype=np.float64)
    x = np.cos(math.pi * (k - 0.25) / (n + 0.5))  # Tricomi initial guess
    for _ in range(100):
        p0 = np.ones_like(x)
        p1 = x.copy()
        for j in range(2, n + 1):
            p0, p1 = p1, ((2 * j - 1) * x * p1 - (j - 1) * p0) / j
        if n == 1:
            p0, p1 = np.ones_like(x), x.copy()
        # derivative of P_n from P_n and P_{n-1}
        dp = n * (x * p1 - p0) / (x * x - 1.0)
        dx = p1 / dp
        x = x - dx
        if np.max(np.abs(dx)) < 1e-16:
            break
    p0 = np.ones_like(x)
    p1 = x.copy()
    for j in range(2, n + 1):
        p0, p1 = p1, ((2 * j - 1) * x * p1 - (j - 1) * p0) / j
    if n == 1:
        p0 = np.ones_like(x)
    dp = n * (x * p1 - p0) / (x * x - 1.0)
    w = 2.0 / ((1.0 - x * x) * dp * dp)
    order = np.argsort(x)
    return x[order], w[order]


def sphere_quadrature(degree: int):
    """Product rule on S^2 exact for every polynomial of total degree <= degree.

    Gauss-Legendre in t = cos(theta) with ceil((degree+1)/2) nodes and a
    uniform phi grid with degree+1 points.  Returns flat (theta, phi, weight)
    arrays whose weights sum to 4*pi.
    """
    nt = max(1, (degree + 2) // 2)
    npf = degree + 1
    t, wt = gauss_legendre(nt)
    phi = 2.0 * math.pi * np.arange(npf) / npf
    th = np.arccos(t)
    TH, PH = np.meshgrid(th, phi, indexing="ij")
    W = np.outer(wt, np.full(npf, 2.0 * math.pi / npf))
    return TH.ravel(), PH.ravel(), W.ravel()


# ---------------------------------------------------------------------------
# Real spherical harmonics
# ---------------------------------------------------------------------------

def real_sh(lmax: int, theta, phi) -> np.ndarray:
    """Orthonormal real spherical harmonics Y_l^m(theta, phi), l <= lmax.

    Convention (the paper leaves it open, Appendix "Spherical Harmonics"):
    z is the polar axis, no Condon-Shortley phase,
      Y_l^0  = Q_l^0(cos th),
      Y_l^m  = sqrt(2) Q_l^m(cos th) cos(m phi),  m > 0,
      Y_l^-m = sqrt(2) Q_l^m(cos th) sin(m phi),  m > 0,
    with Q_l^m = sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!) P_l^m the normalised
    associated Legendre function.  So Y_1 = sqrt(3/(4 pi)) (y, z, x).
    Output index i = l*l + l + m (m = -l..l), last axis.
    """
    theta = np.asarray(theta, dtype=np.float64)
    phi = np.asarray(phi, dtype=np.float64)
    shape = np.broadcast(theta, phi).shape
    theta = np.broadcast_to(theta, shape)
    phi = np.broadcast_to(phi, shape)
    t = np.cos(theta)
    s = np.sin(theta)
    out = np.zeros(shape + (nsh(lmax),), dtype=np.float64)
    sqrt2 = math.sqrt(2.0)

    def store(l, m, q):
        if m == 0:
            out[..., l * l + l] = q
        else:
            out[..., l * l + l + m] = sqrt2 * q * np.cos(m * phi)
            out[..., l * l + l - m] = sqrt2 * q * np.sin(m * phi)

    qmm = np.full(shape, math.sqrt(1.0 / FOUR_PI))
    for m in range(lmax + 1):
        if m > 0:
            qmm = qmm * math.sqrt((2.0 * m + 1.0) / (2.0 * m)) * s
        store(m, m, qmm)
        if m + 1 > lmax:
            continue
        q_prev2 = qmm
        q_prev1 = math.sqrt(2.0 * m + 3.0) * t * qmm
        store(m + 1, m, q_prev1)
        for l in range(m + 2, lmax + 1):
            a = math.sqrt((4.0 * l * l - 1.0) / (l * l - m * m))
            b = math.sqrt(((l - 1.0) ** 2 - m * m) / (4.0 * (l - 1.0) ** 2 - 1.0))
            q = a * (t * q_prev1 - b * q_prev2)
            store(l, m, q)
            q_prev2, q_prev1 = q_prev1, q
    return out


def real_sh_xyz(lmax: int, r) -> np.ndarray:
    """Real SH of unit vectors r[..., 3] (x, y, z) in the convention above."""
    r = np.asarray(r, dtype=np.float64)
    n = np.linalg.norm(r, axis=-1)
    z = np.clip(r[..., 2] / n, -1.0, 1.0)
    theta = np.arccos(z)
    phi = np.arctan2(r[..., 1], r[..., 0])
    return real_sh(lmax, theta, phi)


# ---------------------------------------------------------------------------
# Gaunt coefficients and the Gaunt tensor product (Sec. 3.1)
# ---------------------------------------------------------------------------

def gaunt_tensor(L1: int, L2: int, L3: int) -> np.ndarray:
    """Dense real Gaunt tensor G[i, j, k] = int Y_i Y_j Y_k dOmega.

    i runs over degree <= L1, j over <= L2, k over <= L3.  The quadrature of
    ``sphere_quadrature(L1+L2+L3)`` is exact: a triple product of real SH with
    a non-vanishing phi integral is a polynomial of degree l1+l2+l3 in (x,y,z).
    """
    th, ph, w = sphere_quadrature(L1 + L2 + L3)
    Y = real_sh(max(L1, L2, L3), th, ph)
    Y1 = Y[:, : nsh(L1)]
    Y2 = Y[:, : nsh(L2)]
    Y3w = Y[:, : nsh(L3)] * w[:, None]
    G = np.empty((nsh(L1), nsh(L2), nsh(L3)), dtype=np.float64)
    for i in range(nsh(L1)):
        G[i] = (Y1[:, i : i + 1] * Y2).T @ Y3w
    return G


_GAUNT_CACHE: dict = {}


def _gaunt_cached(L1, L2, L3):
    key = (L1, L2, L3)
    if key not in _GAUNT_CACHE:
        _GAUNT_CACHE[key] = gaunt_tensor(L1, L2, L3)
    return _GAUNT_CACHE[key]


def gtp(x1, x2, L1: int, L2: int, Lout: int, chunk: int = 2048) -> np.ndarray:
    """Gaunt tensor product, mode A (eq. tp-eq-mul, second line).

    y[n, k] = sum_{i,j} G[i, j, k] x1[n, i] x2[n, j], contracted densely over
    every (i, j, k) of the Gaunt tensor.  x1[..., (L1+1)^2], x2[..., (L2+1)^2]
    with identical leading shape; returns y[..., (Lout+1)^2] in float64.
    Output degrees above L1+L2 come out as (quadrature-exact) zeros.
    """
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    lead = x1.shape[:-1]
    assert x1.shape[-1] == nsh(L1) and x2.shape[-1] == nsh(L2)
    assert x2.shape[:-1] == lead
    a = x1.reshape(-1, nsh(L1))
    b = x2.reshape(-1, nsh(L2))
    G = _gaunt_cached(L1, L2, Lout)
    Gm = G.reshape(nsh(L1), nsh(L2) * nsh(Lout))
    y = np.empty((a.shape[0], nsh(Lout)), dtype=np.float64)
    for s in range(0, a.shape[0], chunk):
        T = (a[s : s + chunk] @ Gm).reshape(-1, nsh(L2), nsh(Lout))
        y[s : s + chunk] = np.einsum("nj,njk->nk", b[s : s + chunk], T)
    return y.reshape(lead + (nsh(Lout),))


def gtp_grid(x1, x2, L1: int, L2: int, Lout: int, chunk: int = 4096) -> np.ndarray:
    """Gaunt tensor product, mode B (eq. tp-eq-mul, last line).

    Evaluates F1 = sum x1 Y and F2 = sum x2 Y on a quadrature grid exact for
    degree L1+L2+Lout, multiplies them pointwise and projects onto Y_l^m,
    l <= Lout.  Exact (up to rounding) and cheaper than mode A at large L.
    """
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    lead = x1.shape[:-1]
    a = x1.reshape(-1, nsh(L1))
    b = x2.reshape(-1, nsh(L2))
    th, ph, w = sphere_quadrature(L1 + L2 + Lout)
    Y = real_sh(max(L1, L2, Lout), th, ph)
    Y1 = Y[:, : nsh(L1)]
    Y2 = Y[:, : nsh(L2)]
    Y3w = Y[:, : nsh(Lout)] * w[:, None]
    y = np.empty((a.shape[0], nsh(Lout)), dtype=np.float64)
    for s in range(0, a.shape[0], chunk):
        F = (a[s : s + chunk] @ Y1.T) * (b[s : s + chunk] @ Y2.T)
        y[s : s + chunk] = F @ Y3w
    return y.reshape(lead + (nsh(Lout),))


def gtp_weighted(x1, x2, w1, w2, wo, L1: int, L2: int, Lout: int, mode: str = "auto") -> np.ndarray:
    """Weighted Gaunt tensor product (Sec. 3.1, eq. tp-eq-mul-weight):

        y^(l) = sum_{l1 <= L1} sum_{l2 <= L2} w1[l1] w2[l2] wo[l] (x1^(l1) (x) x2^(l2))^(l),

    the learnable weights w^l_{l1,l2} of the feature-interaction layer in the
    reparameterized form w_{l1} w_{l2} w_l.  x1[n, (L1+1)^2], x2[n, (L2+1)^2];
    w1[n, L1+1], w2[n, L2+1], wo[n, Lout+1] hold the weights of each product
    (rows broadcast).  Mode "sum" (default for max degree <= 8) evaluates the
    double sum over degree pairs with the (l1, l2) blocks of the Gaunt tensor;
    mode "scaled" evaluates the paper's equivalent route (Appendix, weighted
    combinations): the product of the functions of w1 x1 and w2 x2, projected
    and scaled by wo.
    """
    x1 = np.asarray(x1, dtype=np.float64).reshape(-1, nsh(L1))
    x2 = np.asarray(x2, dtype=np.float64).reshape(-1, nsh(L2))
    n = x1.shape[0]
    w1 = np.broadcast_to(np.asarray(w1, dtype=np.float64), (n, L1 + 1))
    w2 = np.broadcast_to(np.asarray(w2, dtype=np.float64), (n, L2 + 1))
    wo = np.broadcast_to(np.asarray(wo, dtype=np.float64), (n, Lout + 1))
    deg = lambda L: np.concatenate([np.full(2 * l + 1, l) for l in range(L + 1)])
    if mode == "auto":
        mode = "sum" if max(L1, L2, Lout) <= 8 else "scaled"
    if mode == "sum":
        G = _gaunt_cached(L1, L2, Lout)
        y = np.zeros((n, nsh(Lout)))
        for l1 in range(L1 + 1):
            b1 = slice(l1 * l1, (l1 + 1) ** 2)
            for l2 in range(L2 + 1):
                b2 = slice(l2 * l2, (l2 + 1) ** 2)
                part = np.einsum("ni,nj,ijk->nk", x1[:, b1], x2[:, b2], G[b1, b2, :])
                y += (w1[:, l1] * w2[:, l2])[:, None] * part
        return y * wo[:, deg(Lout)]
    if mode == "scaled":
        y = gtp_grid(x1 * w1[:, deg(L1)], x2 * w2[:, deg(L2)], L1, L2, Lout)
        return y * wo[:, deg(Lout)]
    raise ValueError(mode)


def gtp_weighted_vjp(x1, x2, w1, w2, wo, dy, L1: int, L2: int, Lout: int):
    """Gradients of s = sum_k dy[k] y[k] with y = gtp_weighted(x1, x2, w1, w2,
    wo) (Sec. 3.1, eq. tp-eq-mul-weight), from the definition

        y_k = wo[l(k)] sum_{i,j} w1[l(i)] w2[l(j)] G[i, j, k] x1_i x2_j

    (l(.) the degree of a coefficient index):
      dx1_i     = w1[l(i)] sum_{j,k} G[i, j, k] (w2 x2)_j (wo dy)_k,
      dw1[l1]   = sum_{i of degree l1} x1_i sum_{j,k} G[i, j, k] (w2 x2)_j (wo dy)_k,
      (x2 and w2 alike), and
      dwo[l]    = sum_{k of degree l} dy_k sum_{i,j} G[i, j, k] (w1 x1)_i (w2 x2)_j.
    The contractions over G are gtp_vjp and gtp of the weighted inputs.
    Weight gradients are per product ([n, L + 1]); summing them over the
    products that share a weight row gives that row's gradient.
    Returns (dx1, dx2, dw1, dw2, dwo) in float64."""
    x1 = np.asarray(x1, dtype=np.float64).reshape(-1, nsh(L1))
    x2 = np.asarray(x2, dtype=np.float64).reshape(-1, nsh(L2))
    dy = np.asarray(dy, dtype=np.float64).reshape(-1, nsh(Lout))
    n = x1.shape[0]
    w1 = np.broadcast_to(np.asarray(w1, dtype=np.float64), (n, L1 + 1))
    w2 = np.broadcast_to(np.asarray(w2, dtype=np.float64), (n, L2 + 1))
    wo = np.broadcast_to(np.asarray(wo, dtype=np.float64), (n, Lout + 1))
    d1, d2, do = degree_index(L1), degree_index(L2), degree_index(Lout)
    u1, u2 = gtp_vjp(x1 * w1[:, d1], x2 * w2[:, d2], dy * wo[:, do], L1, L2, Lout)
    z = gtp(x1 * w1[:, d1], x2 * w2[:, d2], L1, L2, Lout) if max(L1, L2, Lout) <= 8 else \
        gtp_grid(x1 * w1[:, d1], x2 * w2[:, d2], L1, L2, Lout)

    def per_degree(a, b, L):
        return np.stack([(a[:, l * l:(l + 1) ** 2] * b[:, l * l:(l + 1) ** 2]).sum(1) for l in range(L + 1)], 1)
    return (w1[:, d1] * u1, w2[:, d2] * u2, per_degree(x1, u1, L1), per_degree(x2, u2, L2), per_degree(dy, z, Lout))


def degree_index(L: int) -> np.ndarray:
    """Degree l of every coefficient index i = l*l + l + m, i < (L+1)^2."""
    return np.concatenate([np.full(2 * l + 1, l) for l in range(L + 1)])


def gtp_vjp(x1, x2, dy, L1: int, L2: int, Lout: int, chunk: int = 2048, mode: str = "auto"):
    """Gradients of s = sum_k dy[k] y[k], y = gtp(x1, x2, L1, L2, Lout).

    y is bilinear in (x1, x2) with coefficients G[i, j, k] (eq. tp-eq-mul), so
      dx1[n, i] = sum_{j,k} G[i, j, k] x2[n, j] dy[n, k],
      dx2[n, j] = sum_{i,k} G[i, j, k] x1[n, i] dy[n, k].
    For max degree <= 8 this contracts the dense Gaunt tensor; above, the same
    sums are the integrals  int Y_i F2 F_dy dOmega  and  int Y_j F1 F_dy dOmega
    (G is an integral of three real SH), taken on a quadrature grid exact for
    degree L1 + L2 + Lout (mode "gaunt" / "grid" forces one).  Returns
    (dx1, dx2) in float64.
    """
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    lead = x1.shape[:-1]
    a = x1.reshape(-1, nsh(L1))
    b = x2.reshape(-1, nsh(L2))
    d = dy.reshape(-1, nsh(Lout))
    assert a.shape[0] == b.shape[0] == d.shape[0]
    dx1 = np.empty_like(a)
    dx2 = np.empty_like(b)
    if mode == "auto":
        mode = "gaunt" if max(L1, L2, Lout) <= 8 else "grid"
    if mode == "gaunt":
        G = _gaunt_cached(L1, L2, Lout)
        for s in range(0, a.shape[0], chunk):
            e = slice(s, s + chunk)
            Gd = np.einsum("ijk,nk->nij", G, d[e])
            dx1[e] = np.einsum("nij,nj->ni", Gd, b[e])
            dx2[e] = np.einsum("nij,ni->nj", Gd, a[e])
    elif mode == "grid":
        th, ph, w = sphere_quadrature(L1 + L2 + Lout)
        Y = real_sh(max(L1, L2, Lout), th, ph)
        Y1 = Y[:, : nsh(L1)]
        Y2 = Y[:, : nsh(L2)]
        Y3 = Y[:, : nsh(Lout)]
        for s in range(0, a.shape[0], chunk):
            e = slice(s, s + chunk)
            Fd = (d[e] @ Y3.T) * w
            dx1[e] = ((b[e] @ Y2.T) * Fd) @ Y1
            dx2[e] = ((a[e] @ Y1.T) * Fd) @ Y2
    else:
        raise ValueError(mode)
    return dx1.reshape(lead + (nsh(L1),)), dx2.reshape(lead + (nsh(L2),))


# ---------------------------------------------------------------------------
# The three stages of Sec. 3.2, each from its plain definition
# ---------------------------------------------------------------------------

def sh2fourier(x, L: int) -> np.ndarray:
    """SH coefficients -> 2D Fourier coefficients x*_{u,v} (eq. sh-fs).

    The function F = sum x Y is extended from theta in [0, pi] to the torus
    theta in [-pi, pi) by F(-theta, phi) := F(theta, phi + pi) (the double
    Fourier sphere; the paper leaves the theta range open).  The extension is a
    trigonometric polynomial with |u|, |v| <= L, so the 2D DFT of its samples on
    a (2L+2) x (2L+2) torus grid returns its Fourier coefficients exactly.

    x[..., (L+1)^2] -> complex grid[..., 2L+1, 2L+1], grid[..., u+L, v+L].
    """
    x = np.asarray(x, dtype=np.float64)
    lead = x.shape[:-1]
    a = x.reshape(-1, nsh(L))
    N = 2 * L + 2
    th = -math.pi + 2.0 * math.pi * np.arange(N) / N
    ph = 2.0 * math.pi * np.arange(N) / N
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    neg = TH < 0
    Y = real_sh(L, np.abs(TH), np.where(neg, PH + math.pi, PH))  # [N, N, K]
    F = np.einsum("nk,abk->nab", a, Y)  # samples on the torus
    u = np.arange(-L, L + 1)
    Eth = np.exp(-1j * np.outer(u, th)) / N  # [2L+1, N]
    Eph = np.exp(-1j * np.outer(ph, u)) / N  # [N, 2L+1]
    g = np.einsum("ua,nab,bv->nuv", Eth, F, Eph)
    return g.reshape(lead + (2 * L + 1, 2 * L + 1))


def fourier_conv(g1, g2) -> np.ndarray:
    """2D convolution of Fourier grids (eq. 2D-conv), written out literally:
    f3[u1+u2, v1+v2] += f1[u1, v1] * f2[u2, v2].

    g1[..., 2A+1, 2A+1], g2[..., 2B+1, 2B+1] -> g3[..., 2(A+B)+1, 2(A+B)+1],
    all indexed with the centre at the middle.
    """
    g1 = np.asarray(g1, dtype=np.complex128)
    g2 = np.asarray(g2, dtype=np.complex128)
    n1 = g1.shape[-1]
    n2 = g2.shape[-1]
    n3 = n1 + n2 - 1
    g3 = np.zeros(np.broadcast_shapes(g1.shape[:-2], g2.shape[:-2]) + (n3, n3), dtype=np.complex128)
    for a in range(n1):
        for b in range(n1):
            g3[..., a : a + n2, b : b + n2] += g1[..., a, b, None, None] * g2
    return g3


def fourier2sh(g3, L3: int, Lout: int, n_theta: int | None = None) -> np.ndarray:
    """2D Fourier coefficients -> SH coefficients (eq. fs-sh).

    The printed equation claims each Fourier basis function is a finite SH sum,
    which it is not; the reading used here is the projection
        y_l^m = int_{S^2} F(theta, phi) Y_l^m dOmega,
        F = sum_{u,v} g3[u, v] exp(i (u theta + v phi)),  theta in [0, pi].
    The phi integral uses a uniform rule with L3+Lout+1 points (exact for the
    trigonometric polynomial in phi); the theta integral uses Gauss-Legendre in
    theta itself on [0, pi], which converges geometrically for these entire
    integrands (the default node count is far past convergence, see tests).

    g3[..., 2*L3+1, 2*L3+1] -> complex y[..., (Lout+1)^2].  For grids of real
    functions (e.g. made by sh2fourier and fourier_conv) the imaginary part is
    zero up to rounding.
    """
    g3 = np.asarray(g3, dtype=np.complex128)
    lead = g3.shape[:-2]
    a = g3.reshape(-1, 2 * L3 + 1, 2 * L3 + 1)
    if n_theta is None:
        n_theta = 2 * (L3 + Lout) + 48
    xg, wg = gauss_legendre(n_theta)
    th = 0.5 * math.pi * (xg + 1.0)
    wth = 0.5 * math.pi * wg * np.sin(th)  # includes the sin(theta) measure
    npf = L3 + Lout + 1
    ph = 2.0 * math.pi * np.arange(npf) / npf
    wph = 2.0 * math.pi / npf
    u = np.arange(-L3, L3 + 1)
    Eth = np.exp(1j * np.outer(th, u))  # [T, 2L3+1]
    Eph = np.exp(1j * np.outer(u, ph))  # [2L3+1, P]
    F = np.einsum("tu,nuv,vp->ntp", Eth, a, Eph)  # samples of F on the grid
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    Y = real_sh(Lout, TH, PH)  # [T, P, K]
    W = wth[:, None] * wph
    y = np.einsum("ntp,tpk->nk", F * W[None], Y)
    return y.reshape(lead + (nsh(Lout),))


# ---------------------------------------------------------------------------
# Many-body self product (Sec. 3.3; Appendix "Implementation Details")
# ---------------------------------------------------------------------------

def selfproduct(x, L: int, nu: int, Lout: int, mode: str = "stepwise") -> np.ndarray:
    """nu-fold Gaunt product of A = x with itself.

    mode "stepwise": B_1 = P_Lout(A); B_{k+1} = P_Lout(B_k * A), i.e. each of
      the nu-1 products is truncated to degree Lout before the next one.
    mode "fused": P_Lout(F_A^nu), the generalized Gaunt coefficients of the
      appendix with no intermediate truncation; evaluated exactly on a
      quadrature grid of degree nu*L + Lout.
    """
    x = np.asarray(x, dtype=np.float64)
    if nu < 1:
        raise ValueError("nu >= 1")
    lead = x.shape[:-1]
    a = x.reshape(-1, nsh(L))
    if mode == "stepwise":
        if nu == 1:
            y = np.zeros((a.shape[0], nsh(Lout)))
            k = min(nsh(L), nsh(Lout))
            y[:, :k] = a[:, :k]
            return y.reshape(lead + (nsh(Lout),))
        B, LB = a, L
        for _ in range(nu - 1):
            B = gtp(B, a, LB, L, Lout) if max(LB, L, Lout) <= 8 else gtp_grid(B, a, LB, L, Lout)
            LB = Lout
        return B.reshape(lead + (nsh(Lout),))
    if mode == "fused":
        th, ph, w = sphere_quadrature(nu * L + Lout)
        Y = real_sh(max(L, Lout), th, ph)
        F = a @ Y[:, : nsh(L)].T
        y = (F ** nu) @ (Y[:, : nsh(Lout)] * w[:, None])
        return y.reshape(lead + (nsh(Lout),))
    raise ValueError(mode)


# ---------------------------------------------------------------------------
# Rotations (Appendix D, equivariance)
# ---------------------------------------------------------------------------

def random_rotation(rng: np.random.Generator) -> np.ndarray:
    """Uniformly random rotation matrix from a normalised Gaussian quaternion."""
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


def wigner_d_real(L: int, R: np.ndarray) -> np.ndarray:
    """Block-diagonal real Wigner-D for degrees 0..L, by exact quadrature.

    D[i, j] = int Y_i(R r) Y_j(r) dOmega (same-degree blocks only), so that
    Y(R r) = D Y(r), and coefficients of F(R^-1 r) are D x.
    """
    th, ph, w = sphere_quadrature(2 * L)
    r = np.stack([np.sin(th) * np.cos(ph), np.sin(th) * np.sin(ph), np.cos(th)], axis=-1)
    Y = real_sh(L, th, ph)
    YR = real_sh_xyz(L, r @ R.T)
    D = (YR * w[:, None]).T @ Y
    mask = np.zeros_like(D, dtype=bool)
    for l in range(L + 1):
        mask[l * l : (l + 1) ** 2, l * l : (l + 1) ** 2] = True
    return np.where(mask, D, 0.0)


# ---------------------------------------------------------------------------
# Channel mixing (Appendix, combination rules of features in different channels)
# ---------------------------------------------------------------------------

def channel_mix(x1, x2, W, L1: int, L2: int, Lout: int) -> np.ndarray:
    """Channel-mixing combination of two multi-channel features:

        y[b, co] = sum_{c1, c2} W[co, c1, c2] GTP(x1[b, c1], x2[b, c2]),

    the O(C^2)-products rule of the appendix's discussion of channels.
    x1[B, C1, (L1+1)^2], x2[B, C2, (L2+1)^2], W[Co, C1, C2]; returns
    y[B, Co, (Lout+1)^2].  Every pair product is taken by ``gtp`` (or
    ``gtp_grid`` above degree 8) and combined with its weight.
    """
    x1 = np.asarray(x1, dtype=np.float64)
    x2 = np.asarray(x2, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    B, C1, _ = x1.shape
    C2 = x2.shape[1]
    prod = gtp if max(L1, L2, Lout) <= 8 else gtp_grid
    T = np.empty((B, C1, C2, nsh(Lout)))
    for c1 in range(C1):
        a = np.repeat(x1[:, c1:c1 + 1, :], C2, axis=1)
        T[:, c1] = prod(a, x2, L1, L2, Lout)
    return np.einsum("oij,bijk->bok", W, T)


# ---------------------------------------------------------------------------
# Equivariant convolution in the edge frame (Sec. 3.3; Appendix, eq. sh2fs-escn)
# ---------------------------------------------------------------------------

def edge_rotation(r) -> np.ndarray:
    """A rotation taking the direction of r to the pole (0, 0, 1).

    With r / |r| = (sin b cos a, sin b sin a, cos b): R = R_y(-b) R_z(-a).
    A zero vector gives the identity (its direction is taken as (0, 0, 1)).
    """
    r = np.asarray(r, dtype=np.float64)
    n = np.linalg.norm(r)
    if n == 0.0:
        return np.eye(3)
    a = math.atan2(r[1], r[0])
    b = math.acos(max(-1.0, min(1.0, r[2] / n)))
    ca, sa, cb, sb = math.cos(a), math.sin(a), math.cos(b), math.sin(b)
    Rz = np.array([[ca, sa, 0.0], [-sa, ca, 0.0], [0.0, 0.0, 1.0]])   # R_z(-a)
    Ry = np.array([[cb, 0.0, -sb], [0.0, 1.0, 0.0], [sb, 0.0, cb]])   # R_y(-b)
    return Ry @ Rz


def conv_escn(x, r, h, L1: int, L2: int, Lout: int, rotation=edge_rotation) -> np.ndarray:
    """Gaunt product of x[b, c] with the SH filter h[b, c, l] Y_l(r_b / |r_b|),
    in the steps of the rotated-frame construction (Sec. 3.3, eq. sh2fs-escn):

    1. a rotation R_b taking the edge direction to the pole;
    2. its real Wigner-D matrix D_b (degrees <= max(L1, Lout));
    3. x' = D_b x;
    4. the filter in the rotated frame, which has only m = 0 coefficients:
       f[(l, 0)] = h_l Y_l^0(pole);
    5. y' = GTP(x', f) truncated to Lout;
    6. y = D_b^T y'.
    x[B, C, (L1+1)^2], r[B, 3], h[B, C, L2+1]; returns y[B, C, (Lout+1)^2].
    """
    x = np.asarray(x, dtype=np.float64)
    h = np.asarray(h, dtype=np.float64)
    B, C = x.shape[:2]
    LM = max(L1, Lout)
    pole = real_sh(L2, np.array([0.0]), np.array([0.0]))[0]
    y = np.empty((B, C, nsh(Lout)))
    for b in range(B):
        D = wigner_d_real(LM, rotation(r[b]))
        xp = x[b] @ D[: nsh(L1), : nsh(L1)].T
        f = np.zeros((C, nsh(L2)))
        for l in range(L2 + 1):
            f[:, l * l + l] = h[b, :, l] * pole[l * l + l]
        yp = gtp(xp, f, L1, L2, Lout)
        y[b] = yp @ D[: nsh(Lout), : nsh(Lout)]
    return y


# ---------------------------------------------------------------------------
# Error metric
# ---------------------------------------------------------------------------

def max_rel_err(y, yref) -> float:
    """max over products of max_i |y - yref| / ||yref||_2 (per product).

    Products whose reference norm is below 1e-30 are measured in absolute
    error.  The last axis is the coefficient axis.
    """
    y = np.asarray(y, dtype=np.float64)
    yref = np.asarray(yref, dtype=np.float64)
    d = np.abs(y - yref).reshape(-1, y.shape[-1]).max(axis=1)
    nrm = np.linalg.norm(yref.reshape(-1, yref.shape[-1]), axis=1)
    nrm = np.where(nrm < 1e-30, 1.0, nrm)
    return float((d / nrm).max()) if d.size else 0.0
