"""Host-side checks of bench.py's bookkeeping (no GPU): the oracle baseline
gathers the device rows of exactly the sampled products, once, for the
forward and the backward step; the formulation flop count is consistent."""
import types

import numpy as np
import pytest
import torch

import bench
from oracle import gtp_oracle as O
from paper_2401_10216_amd import inputs


class _Args:
    def __init__(self, backward):
        self.backward = backward


class _Plan:
    L1 = L2 = Lout = 2


@pytest.mark.parametrize("backward", [False, True])
def test_cpu_baseline_gathers_sampled_rows_once(backward):
    B, C = 700, 3
    rng = np.random.default_rng(1)
    a = rng.standard_normal((B, C, 9)).astype(np.float32)
    b = rng.standard_normal((B, C, 9)).astype(np.float32)
    t1, t2 = torch.from_numpy(a), torch.from_numpy(b)
    y = torch.zeros(B, C, 9)
    lib = types.SimpleNamespace(gtp_full_backward=None)
    step, rows, oracle_of, outs = bench.pair_step(_Args(backward), torch, lib, inputs, _Plan, t1, t2, y, 1)
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    # stand-in for the device results: the oracle's values for every product
    if backward:
        d = inputs.output_gradient(1, (B, C, 9)).astype(np.float64)
        vals = O.gtp_vjp(a64, b64, d, 2, 2, 2)
    else:
        vals = (O.gtp(a64, b64, 2, 2, 2),)
    assert len(outs) == len(vals)
    for buf, v in zip(outs, vals):
        buf.copy_(torch.from_numpy(v.astype(np.float32)))

    def oracle_sample(O_, idx):
        bi = idx
        return oracle_of(O_, idx, a.reshape(B * C, -1)[bi].astype(np.float64),
                         b.reshape(B * C, -1)[bi].astype(np.float64)), rows

    out = bench.cpu_baseline(O, inputs, oracle_sample, B * C, 1, budget_s=0.0)
    assert out["sample"].startswith("1024 ")  # a strict subsample: indices are not the identity
    assert out["max_rel_err_gpu_vs_oracle"] < 1e-6


def test_formulation_flops_values():
    assert [bench.formulation_flops(L, L, L) for L in (2, 4, 6, 8, 16, 32, 64)] == \
        [852, 3996, 9660, 20940, 130572, 910860, 6779916]
    # never above the FFT-based counts the targets were set with
    for L in (4, 6, 8, 16, 32, 64):
        assert bench.formulation_flops(L, L, L) < bench.FFT_FORMULATION_FLOPS[L]


def test_fused_backward_bookkeeping():
    """The backward step is one launch exactly where gtp_full_backward takes the
    one-launch kernel: equal degrees 1..7 on the thread-per-product path."""
    for L in range(1, 8):
        assert bench.fused_backward((L, L, L))
        assert bench.fused_backward((L, L, L), "fft") and bench.fused_backward((L, L, L), "dft")
        assert not bench.fused_backward((L, L, L), "generic") and not bench.fused_backward((L, L, L), "direct")
    for degs in ((8, 8, 8), (16, 16, 16), (0, 0, 0), (6, 6, 2), (4, 6, 5), (2, 2, 3)):
        assert not bench.fused_backward(degs)
    assert not bench.fused_backward(None)
