"""Pins of the backward-pass oracle (CPU only).

``recurrent_grad`` (autograd over the step-by-step cell) is tied to central finite differences of
the NumPy recurrent form, an independent implementation; ``parallel_grad`` (the closed form over
the parallel form) is tied to ``recurrent_grad``.  A planted mistake in a copy of the closed form
(a dropped term, a wrong sign) must fail the comparison.
"""
import numpy as np
import pytest

from oracle import mlstm_grad as G
from oracle import mlstm_ref as R


def inputs(seed, S=2, T=7, DQK=3, DV=2, i_mu=0.0, f_mu=3.0, f_sd=1.0):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((S, T, DQK))
    k = rng.standard_normal((S, T, DQK))
    v = rng.standard_normal((S, T, DV))
    ip = rng.normal(i_mu, 1.0, (S, T))
    fp = rng.normal(f_mu, f_sd, (S, T))
    dh = rng.standard_normal((S, T, DV))
    return q, k, v, ip, fp, dh


def loss(q, k, v, ip, fp, dh):
    h, *_ = R.recurrent(q, k, v, ip, fp)
    return float((h * dh).sum())


DISTS = {"standard": dict(), "floor_active": dict(i_mu=-6.0), "short_memory": dict(f_mu=-1.0, f_sd=2.0)}


@pytest.mark.parametrize("dist", list(DISTS))
def test_recurrent_grad_matches_finite_differences(dist):
    q, k, v, ip, fp, dh = inputs(1, **DISTS[dist])
    grads = G.recurrent_grad(q, k, v, ip, fp, dh)
    args = [q, k, v, ip, fp]
    eps = 1e-6
    for j, (x, g) in enumerate(zip(args, grads)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp = x.copy(); xp[idx] += eps
            xm = x.copy(); xm[idx] -= eps
            ap = list(args); ap[j] = xp
            am = list(args); am[j] = xm
            fd[idx] = (loss(*ap, dh) - loss(*am, dh)) / (2 * eps)
        np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-8, err_msg=f"input {j}")


@pytest.mark.parametrize("dist", list(DISTS))
@pytest.mark.parametrize("shape", [(2, 7, 3, 2), (1, 40, 5, 4)])
def test_parallel_grad_matches_recurrent_grad(dist, shape):
    S, T, DQK, DV = shape
    q, k, v, ip, fp, dh = inputs(2, S, T, DQK, DV, **DISTS[dist])
    a = G.recurrent_grad(q, k, v, ip, fp, dh)
    b = G.parallel_grad(q, k, v, ip, fp, dh)
    for j, (x, y) in enumerate(zip(a, b)):
        np.testing.assert_allclose(y, x, rtol=1e-9, atol=1e-11, err_msg=f"input {j}")


def test_v_gradient_is_linear_in_dh_and_closed_form_at_one_token():
    """T = 1 from the zero state: h = (q^.k) v / max(|q^.k|, exp(-i~)) (with the weight e^{i~}
    and m_1 = max(logsig f~, i~) cancelling), so dh/dv is that scalar ratio."""
    q, k, v, ip, fp, dh = inputs(3, S=3, T=1, DQK=4, DV=2)
    dq, dk, dv, di, df = G.parallel_grad(q, k, v, ip, fp, dh)
    qk = (q[:, 0] * k[:, 0]).sum(-1) / 2.0
    m = np.maximum(R.logsigmoid(fp[:, 0]), ip[:, 0])
    w = np.exp(ip[:, 0] - m)
    ratio = w * qk / np.maximum(np.abs(w * qk), np.exp(-m))
    np.testing.assert_allclose(dv[:, 0], ratio[:, None] * dh[:, 0], rtol=1e-12)
    np.testing.assert_allclose(df[:, 0], 0.0, atol=1e-15)   # nothing before the first token to decay


def test_planted_mistakes_fail():
    """A copy of the closed form with the denominator term dropped, or the forget-gate sign
    flipped, no longer matches the definition."""
    q, k, v, ip, fp, dh = inputs(4, S=1, T=9, DQK=3, DV=2)   # |D~| above the floor: dD~ is live
    ref = G.recurrent_grad(q, k, v, ip, fp, dh)
    good = G.parallel_grad(q, k, v, ip, fp, dh)
    assert all(np.allclose(x, y, rtol=1e-9, atol=1e-11) for x, y in zip(ref, good))
    src = open(G.__file__).read()
    ns = {}
    bad1 = src.replace("W = (dN @ v[s].T + dD[:, None]) * Ft", "W = (dN @ v[s].T) * Ft")
    bad2 = src.replace("da = np.cumsum((P - di)[::-1])[::-1]", "da = np.cumsum((P + di)[::-1])[::-1]")
    for bad in (bad1, bad2):
        assert bad != src
        ns = {}
        exec(compile(bad, "planted", "exec"), ns)
        got = ns["parallel_grad"](q, k, v, ip, fp, dh)
        assert not all(np.allclose(x, y, rtol=1e-6, atol=1e-9) for x, y in zip(ref, got))


def _state(seed, S, DQK, DV):
    rng = np.random.default_rng(seed)
    return rng.normal(0, 0.3, (S, DQK, DV)), np.abs(rng.standard_normal((S, DQK))), rng.standard_normal(S)


@pytest.mark.parametrize("dist", list(DISTS))
def test_state_grad_matches_finite_differences(dist):
    """recurrent_grad_state against central differences of the NumPy recurrent form, for every input
    including the initial state (C0, n0, m0)."""
    q, k, v, ip, fp, dh = inputs(3, **DISTS[dist])
    C0, n0, m0 = _state(4, 2, 3, 2)
    grads = G.recurrent_grad_state(q, k, v, ip, fp, C0, n0, m0, dh)
    args = [q, k, v, ip, fp, C0, n0, m0]

    def L(a):
        h, *_ = R.recurrent(*a[:5], a[5], a[6], a[7])
        return float((h * dh).sum())
    eps = 1e-6
    for j, (x, g) in enumerate(zip(args, grads)):
        x = np.asarray(x, dtype=np.float64)
        num = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp = x.copy(); xp[idx] += eps
            xm = x.copy(); xm[idx] -= eps
            ap = list(args); ap[j] = xp
            am = list(args); am[j] = xm
            num[idx] = (L(ap) - L(am)) / (2 * eps)
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-7 * max(1.0, np.abs(num).max()), err_msg=str(j))


def test_state_grad_with_zero_state_is_recurrent_grad():
    """From (C0, n0, m0) = (0, 0, 0) the five input gradients are those of recurrent_grad."""
    q, k, v, ip, fp, dh = inputs(5)
    S, T, DQK = q.shape
    DV = v.shape[2]
    a = G.recurrent_grad_state(q, k, v, ip, fp, np.zeros((S, DQK, DV)), np.zeros((S, DQK)), np.zeros(S), dh)
    b = G.recurrent_grad(q, k, v, ip, fp, dh)
    for x, y in zip(a[:5], b):
        np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-14)


def test_state_grad_with_borders():
    """f~ = -inf (a document border): the gradients stay finite, nothing before the border reaches it
    (with a border on the first token the initial state gets no gradient), and the gradients of the
    tokens after the last border equal those of a fresh run of those tokens from the zero state."""
    q, k, v, ip, fp, dh = inputs(6, S=1, T=9)
    C0, n0, m0 = _state(7, 1, 3, 2)
    fp = fp.copy()
    fp[0, [0, 5]] = -np.inf
    g = G.recurrent_grad_state(q, k, v, ip, fp, C0, n0, m0, dh)
    for x in g:
        assert np.isfinite(x).all()
    assert np.abs(g[5]).max() == 0 and np.abs(g[6]).max() == 0 and g[7][0] == 0
    assert g[4][0, 0] == 0 and g[4][0, 5] == 0
    tail = G.recurrent_grad_state(q[:, 5:], k[:, 5:], v[:, 5:], ip[:, 5:], fp[:, 5:], np.zeros((1, 3, 2)),
                                  np.zeros((1, 3)), np.zeros(1), dh[:, 5:])
    for x, y in zip(g[:5], tail[:5]):
        np.testing.assert_allclose(x[:, 5:], y, rtol=1e-10, atol=1e-12)


def test_term_scales_bound_the_gradients():
    """parallel_grad_scales sums the magnitudes of every term of each element of dq, dk, dv (inner dot
    products included), so it bounds the gradient elementwise (triangle inequality) and is strictly
    larger somewhere."""
    rng = np.random.default_rng(41)
    S, T, DQK, DV = 2, 23, 8, 6
    q, k = rng.standard_normal((S, T, DQK)), rng.standard_normal((S, T, DQK))
    v, dh = rng.standard_normal((S, T, DV)), rng.standard_normal((S, T, DV))
    ip, fp = rng.standard_normal((S, T)), rng.normal(1.0, 2.0, (S, T))
    g = G.parallel_grad(q, k, v, ip, fp, dh)
    sc = G.parallel_grad_scales(q, k, v, ip, fp, dh)
    for x, s in zip(g[:3], sc):
        assert (s >= np.abs(x) - 1e-12 * (1 + np.abs(x))).all()
        assert (s > np.abs(x) * (1 + 1e-6)).any()


def test_term_scales_without_cancellation_are_the_gradient_magnitudes():
    """One token, one dimension, positive q, k, v, dh and the floor active (no denominator term): every
    element of dq, dk, dv is a single product of positive factors, so its scale is its magnitude."""
    rng = np.random.default_rng(42)
    S, T = 4, 1
    q, k = rng.uniform(0.5, 1.0, (S, T, 1)), rng.uniform(0.5, 1.0, (S, T, 1))
    v, dh = rng.uniform(0.5, 1.0, (S, T, 1)), rng.uniform(0.5, 1.0, (S, T, 1))
    ip, fp = np.full((S, T), -5.0), rng.standard_normal((S, T))
    g = G.parallel_grad(q, k, v, ip, fp, dh)
    sc = G.parallel_grad_scales(q, k, v, ip, fp, dh)
    for x, s in zip(g[:3], sc):
        np.testing.assert_allclose(s, np.abs(x), rtol=1e-12)
