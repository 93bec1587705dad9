"""The Python binding validates every caller-supplied tensor before the C ABI
is called: wrong shapes, dtypes or devices raise ValueError / TypeError on the
host, so no launch can read or write past a tensor the caller passed.  CPU
only: host-only plans and CPU tensors (which reach the device check last)."""
import pytest

from paper_2401_10216_amd import gtp

torch = pytest.importorskip("torch")

F32, BF16 = torch.float32, torch.bfloat16


def plan(L1, L2, Lout):
    return gtp.Plan(L1, L2, Lout, gtp.GTP_PLAN_HOST_ONLY)


def z(*shape, dtype=F32):
    return torch.zeros(shape, dtype=dtype)


def test_full_checks_y_and_inputs():
    p = plan(2, 2, 3)
    x = z(4, 2, 9)
    with pytest.raises(ValueError, match="y has shape"):
        gtp.gtp_full(p, x, x, y=z(4, 2, 9))  # needs (Lout+1)^2 = 16
    with pytest.raises(TypeError, match="y has dtype"):
        gtp.gtp_full(p, x, x, y=z(4, 2, 16, dtype=BF16))
    with pytest.raises(ValueError, match="coefficient dimension"):
        gtp.gtp_full(p, z(4, 2, 16), x)
    with pytest.raises(TypeError):
        gtp.gtp_full(p, x.double(), x.double())
    with pytest.raises(ValueError, match="contiguous"):
        gtp.gtp_full(p, x, x, y=z(4, 2, 32)[:, :, ::2])
    # every shape right: only the device check is left
    with pytest.raises(ValueError, match="device tensor"):
        gtp.gtp_full(p, x, x, y=z(4, 2, 16))


def test_weighted_checks_weights_and_y():
    p = plan(2, 2, 2)
    x = z(3, 5, 9)
    with pytest.raises(ValueError, match="w1 has shape"):
        gtp.gtp_full_weighted(p, x, x, w1=z(1, 2))
    with pytest.raises(ValueError, match="wout has shape"):
        gtp.gtp_full_weighted(p, x, x, wout=z(1, 3), per_channel=True)  # needs [5, 3]
    with pytest.raises(TypeError, match="w2 has dtype"):
        gtp.gtp_full_weighted(p, x, x, w2=z(1, 3, dtype=BF16))
    with pytest.raises(ValueError, match="y has shape"):
        gtp.gtp_full_weighted(p, x, x, y=z(3, 5, 4))


def test_backward_checks_gradients():
    p = plan(2, 1, 2)
    x1, x2, dy = z(2, 3, 9), z(2, 3, 4), z(2, 3, 9)
    with pytest.raises(ValueError, match="dx1 has shape"):
        gtp.gtp_full_backward(p, x1, x2, dy, dx1=z(2, 3, 4))
    with pytest.raises(ValueError, match="dx2 has shape"):
        gtp.gtp_full_backward(p, x1, x2, dy, dx2=z(2, 3, 9))
    with pytest.raises(TypeError, match="dy must be float32"):
        gtp.gtp_full_backward(p, x1, x2, dy.to(BF16))
    with pytest.raises(ValueError, match="device tensor"):
        gtp.gtp_full_backward(p, x1, x2, dy)


def test_channel_mix_and_escn_check_everything():
    p = plan(2, 2, 2)
    x1, x2 = z(2, 3, 9), z(2, 4, 9)
    with pytest.raises(ValueError, match="W must be"):
        gtp.gtp_channel_mix(p, x1, x2, z(5, 4, 3))
    with pytest.raises(ValueError, match="y has shape"):
        gtp.gtp_channel_mix(p, x1, x2, z(5, 3, 4), y=z(2, 3, 9))
    with pytest.raises(ValueError, match="r must be"):
        gtp.gtp_conv_escn(p, x1, z(2, 4), z(2, 3, 3))
    with pytest.raises(ValueError, match="h must be"):
        gtp.gtp_conv_escn(p, x1, z(2, 3), z(2, 3, 2))
    with pytest.raises(ValueError, match="y has shape"):
        gtp.gtp_conv_escn(p, x1, z(2, 3), z(2, 3, 3), y=z(2, 3, 4))


def test_stage_wrappers_check_grids():
    p = plan(2, 1, 2)
    c64 = torch.complex64
    with pytest.raises(ValueError, match="x has shape"):
        gtp.gtp_sh2fourier(p, 1, z(3, 4))  # L1 = 2 needs 9 coefficients
    with pytest.raises(ValueError, match="which"):
        gtp.gtp_sh2fourier(p, 3, z(3, 9))
    with pytest.raises(ValueError, match="grid has shape"):
        gtp.gtp_sh2fourier(p, 2, z(3, 4), grid=z(3, 5, 5, dtype=c64))
    with pytest.raises(ValueError, match="g2 has shape"):
        gtp.gtp_fourier_conv(p, z(3, 5, 5, dtype=c64), z(3, 5, 5, dtype=c64))
    with pytest.raises(TypeError, match="g1 has dtype"):
        gtp.gtp_fourier_conv(p, z(3, 5, 5), z(3, 3, 3, dtype=c64))
    with pytest.raises(ValueError, match="g3 has shape"):
        gtp.gtp_fourier_conv(p, z(3, 5, 5, dtype=c64), z(3, 3, 3, dtype=c64), g3=z(3, 5, 5, dtype=c64))
    with pytest.raises(ValueError, match="g3 has shape"):
        gtp.gtp_fourier2sh(p, z(3, 5, 5, dtype=c64))
    with pytest.raises(ValueError, match="y has shape"):
        gtp.gtp_fourier2sh(p, z(3, 7, 7, dtype=c64), y=z(3, 4))


def test_selfproduct_and_filter_check_outputs():
    with pytest.raises(ValueError, match="y has shape"):
        gtp.gtp_selfproduct(z(2, 2, 9), 2, 3, 3, y=z(2, 2, 9))
    with pytest.raises(ValueError, match="r must be"):
        gtp.gtp_sh_filter(3, z(4))
    with pytest.raises(ValueError, match="h has shape"):
        gtp.gtp_sh_filter(3, z(4, 3), z(4, 2, 3))
    with pytest.raises(TypeError, match="h has dtype"):
        gtp.gtp_sh_filter(3, z(4, 3), z(4, 2, 4, dtype=BF16))
    with pytest.raises(ValueError, match="out has shape"):
        gtp.gtp_sh_filter(3, z(4, 3), z(4, 2, 4), out=z(4, 2, 9))
