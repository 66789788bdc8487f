"""Pins of the oracle's hidden-state output h = sigmoid(o~) * Norm(h~) (Eq. 6 with Eq. 9):
library forms of LayerNorm / RMSNorm and of the sigmoid, closed forms, and the exact
scale identity that fixes where eps enters."""
import numpy as np
import torch

from oracle import mlstm_ref as R


def _rows(seed, B=2, NH=3, T=5, DV=24, scale=1.5, shift=0.3):
    rng = np.random.default_rng(seed)
    return (rng.normal(shift, scale, (B, NH, T, DV)), rng.normal(0, 2, (B, NH, T, DV)),
            rng.normal(1, 0.2, (NH, DV)), rng.normal(0, 0.2, (NH, DV)))


def test_layer_norm_matches_torch_headwise():
    x, o, w, b = _rows(0)
    got = R.output_gate_norm(x, o, w, b, eps=1e-5, norm="layer")
    xt = torch.from_numpy(x)
    ref = torch.empty_like(xt)
    for hd in range(x.shape[1]):   # the norm's affine parameters belong to the head
        ref[:, hd] = torch.nn.functional.layer_norm(xt[:, hd], (x.shape[3],), torch.from_numpy(w[hd]),
                                                    torch.from_numpy(b[hd]), eps=1e-5)
    ref = torch.sigmoid(torch.from_numpy(o)) * ref
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_rms_norm_matches_torch_headwise():
    x, o, w, _ = _rows(1)
    got = R.output_gate_norm(x, o, w, None, eps=1e-6, norm="rms")
    xt = torch.from_numpy(x)
    ref = torch.empty_like(xt)
    for hd in range(x.shape[1]):
        ref[:, hd] = torch.nn.functional.rms_norm(xt[:, hd], (x.shape[3],), torch.from_numpy(w[hd]), eps=1e-6)
    ref = torch.sigmoid(torch.from_numpy(o)) * ref
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_closed_form_two_valued_row():
    """Row of +a and -a in equal numbers: mean 0 and variance a^2, so both norms give
    +-a / sqrt(a^2 + eps); o~ = 0 halves it."""
    a, eps, DV = 0.7, 1e-3, 8
    x = np.tile(np.array([a, -a]), DV // 2).reshape(1, 1, 1, DV)
    want = x / np.sqrt(a * a + eps) * 0.5
    for norm in ("layer", "rms"):
        np.testing.assert_allclose(R.output_gate_norm(x, np.zeros_like(x), eps=eps, norm=norm), want, rtol=1e-14)


def test_constant_row_layer_norm_is_bias():
    x = np.full((1, 2, 3, 16), 4.25)
    b = np.arange(32, dtype=np.float64).reshape(2, 16) / 7
    got = R.output_gate_norm(x, np.full_like(x, 50.0), None, b, eps=1e-6, norm="layer")
    np.testing.assert_allclose(got, np.broadcast_to(b[None, :, None, :], x.shape), rtol=1e-14, atol=1e-15)


def test_scale_identity_fixes_eps():
    """Norm(alpha x + beta; eps) = Norm(x; eps / alpha^2) for LayerNorm (beta arbitrary) and
    RMSNorm (beta = 0): eps is added to the variance, not to the standard deviation."""
    x, o, w, b = _rows(2)
    alpha, beta, eps = 3.0, -1.25, 1e-2
    for norm, sh in (("layer", beta), ("rms", 0.0)):
        lhs = R.output_gate_norm(alpha * x + sh, o, w, b, eps=eps, norm=norm)
        rhs = R.output_gate_norm(x, o, w, b, eps=eps / alpha ** 2, norm=norm)
        np.testing.assert_allclose(lhs, rhs, rtol=1e-12, atol=1e-13)


def test_sigmoid_is_stable_and_symmetric():
    z = np.array([-800.0, -30.0, -1.0, 0.0, 1.0, 30.0, 800.0])
    s = R.sigmoid(z)
    assert np.isfinite(s).all() and s[0] == 0.0 and s[-1] == 1.0 and s[3] == 0.5
    np.testing.assert_allclose(s + R.sigmoid(-z), 1.0, rtol=0, atol=1e-15)
    np.testing.assert_allclose(s[1:-1], torch.sigmoid(torch.from_numpy(z[1:-1])).numpy(), rtol=1e-15)
