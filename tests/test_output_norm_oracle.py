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


# ---- the layer (Eq. 11) --------------------------------------------------------------------------

def _layer_weights(seed, d, NH, DQK, DV):
    rng = np.random.default_rng(seed)
    N = NH * (2 * DQK + 2 * DV + 2)
    return (rng.normal(0, d ** -0.5, (d, N)), rng.normal(0, (NH * DV) ** -0.5, (NH * DV, d)),
            np.stack([rng.normal(-2.0, 1.0, NH), rng.normal(3.0, 1.0, NH)]), rng.normal(1, 0.1, (NH, DV)))


def test_layer_equals_a_loop_over_heads():
    """Head h uses exactly its own columns of W_in (q, k, v, o head-major; gates one column
    each) and its own rows of W_proj: the layer equals the sum over heads of separate cells."""
    B, T, d, NH, DQK, DV = 2, 7, 12, 3, 4, 5
    Win, Wp, gb, nw = _layer_weights(3, d, NH, DQK, DV)
    x = np.random.default_rng(4).normal(0, 1, (B, T, d))
    y, _ = R.mlstm_layer(x, Win, Wp, gb, nw, NH, DQK, DV, eps=1e-5, cap=15.0)
    off = np.cumsum([0, NH * DQK, NH * DQK, NH * DV, NH, NH, NH * DV])
    acc = np.zeros((B, T, d))
    for hd in range(NH):
        cols = lambda blk, w: Win[:, off[blk] + hd * w: off[blk] + (hd + 1) * w]
        q, k, v, o = x @ cols(0, DQK), x @ cols(1, DQK), x @ cols(2, DV), x @ cols(5, DV)
        ig = 15 * np.tanh((x @ cols(3, 1) + gb[0, hd]) / 15)[..., 0]
        fg = 15 * np.tanh((x @ cols(4, 1) + gb[1, hd]) / 15)[..., 0]
        h, *_ = R.recurrent(q, k, v, ig, fg)
        hn = R.output_gate_norm(h[:, None], o[:, None], nw[hd:hd + 1], None, eps=1e-5)[:, 0]
        acc += hn @ Wp[hd * DV:(hd + 1) * DV]
    np.testing.assert_allclose(y, acc, rtol=1e-12, atol=1e-12)


def test_layer_soft_cap_limits():
    """cap -> infinity is no cap; the capped gates stay inside (-cap, cap)."""
    B, T, d, NH, DQK, DV = 1, 6, 8, 2, 3, 4
    Win, Wp, gb, nw = _layer_weights(5, d, NH, DQK, DV)
    x = np.random.default_rng(6).normal(0, 1, (B, T, d))
    a, _ = R.mlstm_layer(x, Win, Wp, gb, nw, NH, DQK, DV, cap=1e9)
    b, _ = R.mlstm_layer(x, Win, Wp, gb, nw, NH, DQK, DV, cap=None)
    np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-12)
    z = np.linspace(-200, 200, 41)
    assert (np.abs(R.soft_cap(z, 15.0)) < 15.0).all()
    np.testing.assert_allclose(R.soft_cap(1e-3, 15.0), 1e-3, rtol=1e-8)


def test_round_bf16_matches_torch_conversion():
    """The oracle's bf16 rounding against torch's fp32 -> bf16 conversion (round to nearest even)
    on fp32 values spread over the exponent range, exact ties, and subnormals."""
    import torch
    rng = np.random.default_rng(5)
    one = np.float32(1.0)
    ties = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8), 3 * 2.0 ** -9 + 2.0 ** -1,
                     2.0 ** -130 + 2.0 ** -134, 2.0 ** -130 + 3 * 2.0 ** -134], dtype=np.float32)
    vals = np.concatenate([
        (rng.standard_normal(20000) * np.exp2(rng.integers(-140, 120, 20000))).astype(np.float32),
        ties, np.array([0.0, -0.0, one, 2.0 ** -126, 2.0 ** -133, 3.0e38], dtype=np.float32)])
    want = torch.from_numpy(vals).bfloat16().double().numpy()
    got = R.round_bf16(vals.astype(np.float64))
    np.testing.assert_array_equal(got, want)
    assert R.round_bf16(1 + 2.0 ** -8) == 1.0 and R.round_bf16(1 + 3 * 2.0 ** -8) == 1 + 2.0 ** -6


def test_layer_bf16_projections_only_round_q_k_v_o():
    """proj_dtype="bf16" moves a generic output by about bf16 rounding, and leaves it bit for
    bit unchanged when every projection is already a bf16 value (x a one-hot row per step,
    W_in on the bf16 grid): the rounding touches only the projections."""
    rng = np.random.default_rng(6)
    B, T, NH, DQK, DV, d = 1, 5, 2, 4, 4, 8
    x = rng.standard_normal((B, T, d))
    Win = rng.standard_normal((d, NH * (2 * DQK + 2 * DV + 2))) * 0.3
    Wp = rng.standard_normal((NH * DV, d)) * 0.3
    gb = np.array([[-1.0, 0.5], [2.0, 3.0]]); nw = 1 + 0.1 * rng.standard_normal((NH, DV))
    a, _ = R.mlstm_layer(x, Win, Wp, gb, nw, NH, DQK, DV)
    b, _ = R.mlstm_layer(x, Win, Wp, gb, nw, NH, DQK, DV, proj_dtype="bf16")
    assert 0 < np.abs(a - b).max() < 0.05 * np.abs(a).max()
    # a projection already on the bf16 grid is left alone: x = e_j, W_in columns on the grid
    Wg = R.round_bf16(Win)
    xe = np.zeros((B, T, d)); xe[0, np.arange(T), np.arange(T)] = 1.0
    c, _ = R.mlstm_layer(xe, Wg, Wp, gb, nw, NH, DQK, DV)
    e, _ = R.mlstm_layer(xe, Wg, Wp, gb, nw, NH, DQK, DV, proj_dtype="bf16")
    np.testing.assert_array_equal(c, e)


def test_gate_preact_one_hot_rows_and_borders():
    """A one-hot token e_j selects row j of W: i~ = softcap(W[j, :NH] + b_i) exactly; the output
    is head-major; border tokens get f~ = -inf and keep their i~; cap None leaves x W + b."""
    rng = np.random.default_rng(8)
    B, T, d, NH = 2, 5, 7, 3
    W = rng.standard_normal((d, 2 * NH)) * 4
    b = rng.standard_normal((2, NH))
    x = np.zeros((B, T, d))
    js = rng.integers(0, d, (B, T))
    for bb in range(B):
        for t in range(T):
            x[bb, t, js[bb, t]] = 1.0
    border = np.zeros((B, T), bool); border[0, 2] = border[1, 0] = True
    ip, fp = R.gate_preact(x, W, b, cap=15.0, border=border)
    assert ip.shape == (B, NH, T) and fp.shape == (B, NH, T)
    for bb in range(B):
        for t in range(T):
            for h in range(NH):
                assert ip[bb, h, t] == 15.0 * np.tanh((W[js[bb, t], h] + b[0, h]) / 15.0)
                want_f = -np.inf if border[bb, t] else 15.0 * np.tanh((W[js[bb, t], NH + h] + b[1, h]) / 15.0)
                assert fp[bb, h, t] == want_f
    ip0, fp0 = R.gate_preact(x, W, b, cap=None)
    np.testing.assert_allclose(ip0[0, :, 1], W[js[0, 1], :NH] + b[0], rtol=1e-15)
    assert np.abs(ip).max() < 15.0


def test_layer_packed_documents_equal_separate_runs():
    """App. B at the layer level: a sequence of two packed documents with a border at the second
    one's first token gives, token for token, the outputs of the layer run on each document alone
    from the zero state."""
    rng = np.random.default_rng(9)
    NH, DQK, DV = 2, 3, 4
    d = NH * DV
    T1, T2 = 6, 5
    x = rng.standard_normal((1, T1 + T2, d))
    Win = rng.standard_normal((d, NH * (2 * DQK + 2 * DV + 2))) * 0.4
    Wp = rng.standard_normal((NH * DV, d)) * 0.4
    gb = np.array([[-1.0, 0.5], [2.0, 3.0]]); nw = 1 + 0.1 * rng.standard_normal((NH, DV))
    border = np.zeros((1, T1 + T2), bool); border[0, T1] = True
    y, (C, n, m) = R.mlstm_layer(x, Win, Wp, gb, nw, NH, DQK, DV, border=border)
    y1, _ = R.mlstm_layer(x[:, :T1], Win, Wp, gb, nw, NH, DQK, DV)
    y2, (C2, n2, m2) = R.mlstm_layer(x[:, T1:], Win, Wp, gb, nw, NH, DQK, DV)
    np.testing.assert_allclose(y[:, :T1], y1, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(y[:, T1:], y2, rtol=1e-12, atol=1e-13)
    # the state scale-free (the separate run starts from m_0 = 0, the packed one restarts at m = i~)
    np.testing.assert_allclose(C * np.exp(m)[:, None, None], C2 * np.exp(m2)[:, None, None], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(n * np.exp(m)[:, None], n2 * np.exp(m2)[:, None], rtol=1e-12, atol=1e-13)
    y0, _ = R.mlstm_layer(x, Win, Wp, gb, nw, NH, DQK, DV)
    assert np.abs(y0[:, T1:] - y2).max() > 1e-3     # without the border the second document sees the first
