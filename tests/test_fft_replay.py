"""numpy replay of the data flow of the matrix-core kernel's radix-FFT phi
stage (the four-step split of a length-NF transform into column DFTs of
length N1 and row DFTs of length N2, the packed two-input spectrum, the real
forward row transform, the twiddles, the pruned outputs and the moment layout
of the theta analysis), step for step in the kernel's index order, against
the phi moments sum_k f1 f2 {cos, sin}(m p_k) of the plan's NP-point grid
computed directly.  Pins the index bookkeeping of that stage on the CPU."""
import numpy as np
import pytest


def fgeo(L):
    NF = 64 if L <= 16 else (128 if L <= 32 else 256)
    N1 = 8 if L <= 32 else 16
    return NF, N1, NF // N1


def replay(L, NP, a1, b1, a2, b2):
    """a*, b*: [16, L+1] cos / sin coefficients of the 16 column nodes' phi
    functions (b[:, 0] unused).  Returns eo[2, 8, 2L+2] as the kernel writes it."""
    NF, N1, N2 = fgeo(L)
    NS = 2 * L + 1
    # packed spectra, twice d_m = c1_m + i c2_m
    sp = np.zeros((16, NS), complex)
    sp[:, 0] = 2 * a1[:, 0] + 2j * a2[:, 0]
    for m in range(1, L + 1):
        sp[:, m] = (a1[:, m] + b2[:, m]) + 1j * (a2[:, m] - b1[:, m])
        sp[:, NS - m] = (a1[:, m] - b2[:, m]) + 1j * (a2[:, m] + b1[:, m])
    T = np.zeros((16, N1, N2), complex)
    for ci in range(16):
        for n2 in range(N2):
            a = np.zeros(N1, complex)
            for m1 in range(N1):
                n = N2 * m1 + n2
                if n <= L:
                    a[m1] = sp[ci, n]
                elif n >= NF - L:
                    a[m1] = sp[ci, NS - NF + n]
            a = np.fft.ifft(a) * N1  # sign +1
            w = np.exp(2j * np.pi * n2 * np.arange(N1) / NF)
            T[ci, :, n2] = a * w
    H2 = N2 // 2 + 1
    T2 = np.zeros((16, H2, N1), complex)
    for ci in range(16):
        for k1 in range(N1):
            z = np.fft.ifft(T[ci, k1, :]) * N2
            g = z.real * z.imag
            X2 = 2 * np.fft.fft(g)[:H2]
            T2[ci, :, k1] = X2 * np.exp(-2j * np.pi * np.arange(H2) * k1 / NF)
    eo = np.full((2, 8, 2 * L + 2), np.nan)
    scale = NP / (8.0 * NF)
    for pp in range(8):
        for m2 in list(range(N2 // 2)) + [N2 // 2]:
            bn = np.fft.fft(T2[pp, m2, :])
            bm = np.fft.fft(T2[8 + pp, m2, :])

            def emit(m, xn, xm):
                eo[0, pp, 2 * m] = (xn.real + xm.real) * scale
                eo[1, pp, 2 * m] = (xn.real - xm.real) * scale
                if m > 0:
                    eo[0, pp, 2 * m + 1] = -(xn.imag + xm.imag) * scale
                    eo[1, pp, 2 * m + 1] = -(xn.imag - xm.imag) * scale
            for m1 in range(N1):
                m = N2 * m1 + m2
                if m <= L:
                    emit(m, bn[m1], bm[m1])
            if m2 != 0 and 2 * m2 != N2:
                for aa in range(1, N1):
                    m = N2 * aa - m2
                    if m <= L:
                        emit(m, np.conj(bn[N1 - aa]), np.conj(bm[N1 - aa]))
    return eo


def direct(L, NP, a1, b1, a2, b2):
    p = 2 * np.pi * np.arange(NP) / NP
    m = np.arange(L + 1)
    C, S = np.cos(np.outer(m, p)), np.sin(np.outer(m, p))
    f1 = a1 @ C + b1 @ S
    f2 = a2 @ C + b2 @ S
    g = f1 * f2
    mc, ms = g @ C.T, g @ S.T  # [16, L+1]
    eo = np.full((2, 8, 2 * L + 2), np.nan)
    for par, sgn in ((0, 1.0), (1, -1.0)):
        eo[par, :, 0::2] = mc[:8] + sgn * mc[8:]
        eo[par, :, 3::2] = (ms[:8] + sgn * ms[8:])[:, 1:]
    return eo


@pytest.mark.parametrize("L,NP", [(16, 52), (32, 100), (64, 196)])
def test_fft_phi_stage_replay(L, NP):
    rng = np.random.default_rng(L)
    a1, b1, a2, b2 = (rng.standard_normal((16, L + 1)) for _ in range(4))
    for b in (b1, b2):
        b[:, 0] = 0.0
    got = replay(L, NP, a1, b1, a2, b2)
    want = direct(L, NP, a1, b1, a2, b2)
    written = ~np.isnan(got)
    # every slot the theta analysis reads is written: cos 0..L, sin 1..L
    assert written[:, :, 0::2].all() and written[:, :, 3::2].all() and not written[:, :, 1].any()
    err = np.abs(got[written] - want[written]).max() / np.abs(want[written]).max()
    assert err < 1e-12, err
