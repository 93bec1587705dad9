"""CPU check of the direct-convolution path (Sec. 3.2, eq. 2D-conv without
the convolution theorem) as the fused direct kernel computes it: the real-form
theta series from the plan's T1 table, the gathered product-to-sum
convolution, the projection with Zc / Zs -- replayed in numpy from the plan's
fp64 tables and compared with the oracle."""
import math

import numpy as np
import pytest

import oracle
from paper_2401_10216_amd import gtp

HOST_ONLY = 16


def theta_coef(odd1, odd2, is_sum, u1, u2):
    if not odd1 and not odd2:
        return 0.5
    if odd1 and odd2:
        return -0.5 if is_sum else 0.5
    if is_sum:
        return 0.5
    d = u1 - u2 if odd1 else u2 - u1
    return 0.5 if d > 0 else (-0.5 if d < 0 else 0.0)


def direct_replay(plan, x1, x2):
    info = plan.info()
    L1, L2, Lout, U, Le = info["L1"], info["L2"], info["Lout"], info["U"], info["Le"]
    Lt = max(L1, L2, Le)
    T1 = plan.table(0).reshape(-1, Lt + 1)
    NZ = U + 2
    Zc = plan.table(1).reshape(-1, NZ)
    Zs = plan.table(2).reshape(-1, NZ)
    tri = lambda l, m: l * (l + 1) // 2 + m

    def series(x, L):
        g = np.zeros((L + 1, L + 1), complex)
        for m in range(L + 1):
            for u in range(L + 1):
                for l in range(max(m, u), L + 1):
                    if (l - u) % 2:
                        continue
                    c = T1[tri(l, m), u]
                    g[m, u] += c * (x[l * l + l + m] - (1j * x[l * l + l - m] if m else 0))
        return g

    g1, g2 = series(x1, L1), series(x2, L2)
    c3 = np.zeros((Le + 1, U + 1), complex)
    for m3 in range(Le + 1):
        for u3 in range(U + 1):
            acc = 0j
            for m1 in range(L1 + 1):
                for kind in range(3):
                    m2 = (m3 - m1, m1 - m3, m1 + m3)[kind]
                    if m2 < 0 or m2 > L2 or (kind == 2 and m3 == 0):
                        continue
                    s = 0j
                    for u1 in range(L1 + 1):
                        for tk in range(3):
                            u2 = (u3 - u1, u1 - u3, u1 + u3)[tk]
                            if u2 < 0 or u2 > L2 or (tk == 2 and u3 == 0):
                                continue
                            w = theta_coef(m1 & 1, m2 & 1, tk == 0, u1, u2)
                            a, b = g1[m1, u1], g2[m2, u2]
                            s += w * (a * b if kind == 0 else (a * np.conj(b) if kind == 1 else np.conj(a) * b))
                    acc += 0.5 * s
            c3[m3, u3] = acc
    y = np.zeros((Lout + 1) ** 2)
    for l in range(min(Le, Lout) + 1):
        for ms in range(-l, l + 1):
            m = abs(ms)
            Z = (Zs if m & 1 else Zc)[tri(l, m)]
            v = sum(Z[u] * (-c3[m, u].imag if ms < 0 else c3[m, u].real) for u in range(U + 1))
            y[l * l + l + ms] = v * (2 * math.pi if m == 0 else math.pi)
    return y


@pytest.mark.parametrize("L1,L2,Lout", [(1, 1, 2), (2, 2, 2), (3, 2, 4), (2, 3, 1), (4, 4, 4), (3, 3, 7)])
def test_direct_replay_matches_oracle(L1, L2, Lout):
    plan = gtp.Plan(L1, L2, Lout, flags=HOST_ONLY)
    rng = np.random.default_rng(900 + 10 * L1 + L2)
    x1 = rng.standard_normal((L1 + 1) ** 2)
    x2 = rng.standard_normal((L2 + 1) ** 2)
    ref = oracle.gtp(x1[None], x2[None], L1, L2, Lout)[0]
    y = direct_replay(plan, x1, x2)
    assert np.abs(y - ref).max() <= 1e-12 * max(np.linalg.norm(ref), 1e-30)
