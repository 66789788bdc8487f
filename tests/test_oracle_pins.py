"""Pins of the oracle to facts the paper and the mathematics fix (CPU only).

Each oracle form (the C recurrent oracle, and the NumPy recurrent, parallel
and chunkwise forms) is checked against values that do not come from itself:

* a scalar example worked out by hand from Eqs. 2-5, 7-8;
* closed forms: a single token from the zero state; a forget gate of zero
  (state reset every step); a forget gate of one, which reduces the cell to
  causal, exponentially weighted linear attention with a floored normaliser,
  computed here with plain matrix products;
* invariants: h does not depend on the max state m (Eq. 2 only controls the
  magnitude of the exponentials, Sec. 2), and tokens with i~ = -inf and
  f~ = +inf are neutral;
* equivalence of the recurrent, parallel (Eq. 10) and chunkwise forms
  (Sec. 2, "Training Mode") for every chunk size, and state carry;
* a mutation check: plausible mistakes planted in a copy of the recurrence
  fail at least one of these pins.
"""
import math

import numpy as np
import pytest

from oracle import coracle
from oracle import mlstm_ref as R


def _c(q, k, v, ip, fp, C0=None, n0=None, m0=None):
    return coracle.recurrent(q, k, v, ip, fp, C0, n0, m0, nthreads=2)


IMPLS = {
    "c_recurrent": _c,
    "np_recurrent": R.recurrent,
    "np_parallel": R.parallel_quadratic,
    "np_chunkwise_L5": lambda *a, **kw: R.chunkwise(*a, **kw, L=5),
    "np_chunkwise_L64": lambda *a, **kw: R.chunkwise(*a, **kw, L=64),
}
# A forget gate of exactly zero (f~ = -inf, logsig = -inf) is outside the chunkwise form,
# whose decays are differences of in-chunk prefix sums (App. D.1) and turn into -inf - -inf.
IMPLS_RESET = ["c_recurrent", "np_recurrent", "np_parallel"]


def rand_inputs(seed, S=3, T=29, DQK=8, DV=6, i_mu=0.0, i_sd=1.0, f_mu=3.0, f_sd=1.0, state=False):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((S, T, DQK))
    k = rng.standard_normal((S, T, DQK))
    v = rng.standard_normal((S, T, DV))
    ip = rng.normal(i_mu, i_sd, (S, T))
    fp = rng.normal(f_mu, f_sd, (S, T))
    st = (None, None, None)
    if state:
        st = (rng.normal(0, 0.1, (S, DQK, DV)), np.abs(rng.standard_normal((S, DQK))), rng.standard_normal(S))
    return (q, k, v, ip, fp) + st


DISTS = {
    "standard": dict(),
    "floor_active": dict(i_mu=-10.0),           # the input-gate bias init of Sec. 3.2 -> floor branch
    "short_memory": dict(f_mu=-2.0, f_sd=2.0),
    "long_memory_state": dict(f_mu=5.0, f_sd=2.0, state=True),
}


@pytest.mark.parametrize("impl", list(IMPLS))
def test_scalar_example_by_hand(impl):
    """d_qk = d_hv = 1, zero state (m_0 = 0), q = 1 so q^ = 1.

    t=1: f~ = +inf -> logsig = 0; i~ = 0; k = 1, v = 3.
         m_1 = max(0 + 0, 0) = 0, f = i = 1, C_1 = 3, n_1 = 1, h_1 = 3 / max(1, 1) = 3.
    t=2: f~ = 0 -> logsig = -ln 2; i~ = ln 3; k = 2, v = 5.
         m_2 = max(-ln 2, ln 3) = ln 3, f = exp(-ln 2 - ln 3) = 1/6, i = 1,
         C_2 = 3/6 + 2*5 = 10.5, n_2 = 1/6 + 2 = 13/6, h_2 = 10.5 / max(13/6, 1/3) = 63/13.
    t=3: f~ = -inf (forget everything); i~ = -ln 2; k = -1, v = 4.
         m_3 = max(-inf, -ln 2) = -ln 2, f = 0, i = 1, C_3 = -4, n_3 = -1,
         h_3 = -4 / max(1, 2) = -2   (the floor exp(-m_3) = 2 wins).
    """
    q = np.ones((1, 3, 1))
    k = np.array([1.0, 2.0, -1.0]).reshape(1, 3, 1)
    v = np.array([3.0, 5.0, 4.0]).reshape(1, 3, 1)
    ip = np.array([[0.0, math.log(3.0), -math.log(2.0)]])
    fp = np.array([[np.inf, 0.0, -np.inf]])
    T = 3 if impl in IMPLS_RESET else 2
    h, C, n, m = IMPLS[impl](q[:, :T], k[:, :T], v[:, :T], ip[:, :T], fp[:, :T])
    np.testing.assert_allclose(h[0, :, 0], [3.0, 63.0 / 13.0, -2.0][:T], rtol=1e-14)
    np.testing.assert_allclose(C[0, 0, 0], [10.5, -4.0][T - 2], rtol=1e-14)
    np.testing.assert_allclose(n[0, 0], [13.0 / 6.0, -1.0][T - 2], rtol=1e-14)
    np.testing.assert_allclose(m[0], [math.log(3.0), -math.log(2.0)][T - 2], rtol=1e-14)


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("dist", ["standard", "floor_active"])
def test_single_token_closed_form(impl, dist):
    """T = 1 from the zero state: C_1 = i k v^T, n_1 = i k with i = exp(i~ - m_1), so
    h~ = (q^.k) v / max(|q^.k|, exp(-i~)) whatever f~ is (the i factor cancels)."""
    q, k, v, ip, fp, *_ = rand_inputs(1, S=6, T=1, DQK=7, DV=5, **DISTS[dist])
    h, C, n, m = IMPLS[impl](q, k, v, ip, fp)
    qk = np.einsum("sd,sd->s", q[:, 0] / np.sqrt(7), k[:, 0])
    want = qk[:, None] * v[:, 0] / np.maximum(np.abs(qk), np.exp(-ip[:, 0]))[:, None]
    np.testing.assert_allclose(h[:, 0], want, rtol=1e-12, atol=1e-300)
    m_want = np.maximum(R.logsigmoid(fp[:, 0]), ip[:, 0])
    np.testing.assert_allclose(m, m_want, rtol=1e-15)


@pytest.mark.parametrize("impl", IMPLS_RESET)
def test_forget_gate_zero_resets_every_step(impl):
    """f~ = -inf: logsig = -inf, f_t = 0, so each step sees only its own token; with the
    zero-state closed form applied token by token (m_t = i~_t)."""
    q, k, v, ip, fp, *_ = rand_inputs(2, S=2, T=9, DQK=4, DV=3)
    fp[:] = -np.inf
    h, C, n, m = IMPLS[impl](q, k, v, ip, fp)
    qk = np.einsum("std,std->st", q / 2.0, k)
    want = qk[..., None] * v / np.maximum(np.abs(qk), np.exp(-ip))[..., None]
    np.testing.assert_allclose(h, want, rtol=1e-12)
    np.testing.assert_allclose(m, ip[:, -1], rtol=1e-15)


@pytest.mark.parametrize("impl", IMPLS_RESET)
def test_document_border_restarts_from_the_zero_state(impl):
    """App. B (sequence packing): a forget gate of zero at a document border resets the memory
    to the zero matrix.  With restarts at tokens r (an initial state given), h over each
    document and the final state equal a fresh run over that document alone from the zero
    state; h from the zero state does not depend on m_0, so the fresh run's m_0 = 0 is no
    assumption."""
    q, k, v, ip, fp, C0, n0, m0 = rand_inputs(21, S=2, T=31, DQK=5, DV=4, state=True)
    borders = [0, 7, 8, 19, 30]
    fp[:, borders] = -np.inf
    h, C, n, m = IMPLS[impl](q, k, v, ip, fp, C0, n0, m0)
    ends = borders[1:] + [31]
    for r, e in zip(borders, ends):
        hf, Cf, nf, mf = IMPLS[impl](q[:, r:e], k[:, r:e], v[:, r:e], ip[:, r:e], fp[:, r:e])
        np.testing.assert_allclose(h[:, r:e], hf, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(C, Cf, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(n, nf, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(m, mf, rtol=1e-14)


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("i_sd", [0.0, 1.0])
def test_forget_gate_one_is_weighted_linear_attention(impl, i_sd):
    """f~ = +inf: logsig = 0, nothing is forgotten.  From the zero state (m_0 = 0) the cell
    is causal linear attention with token weights exp(i~_j) and the normaliser floored at 1:
    h_t = sum_j w_j (q^_t.k_j) v_j / max(|sum_j w_j q^_t.k_j|, 1)   (i~ = 0: plain weights 1)."""
    q, k, v, ip, fp, *_ = rand_inputs(3, S=2, T=17, DQK=6, DV=4, i_sd=i_sd)
    fp[:] = np.inf
    h, *_ = IMPLS[impl](q, k, v, ip, fp)
    for s in range(2):
        A = np.tril((q[s] / np.sqrt(6)) @ k[s].T) * np.exp(ip[s])[None, :]
        want = (A @ v[s]) / np.maximum(np.abs(A.sum(axis=1)), 1.0)[:, None]
        np.testing.assert_allclose(h[s], want, rtol=1e-11, atol=1e-14)


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("dist", list(DISTS))
def test_h_independent_of_max_state(impl, dist):
    """h does not depend on the stabiliser m: the unstabilised recurrence (no m, floor 1 in
    unscaled units) gives the same h, and its final state equals e^{m_T} C_T."""
    q, k, v, ip, fp, C0, n0, m0 = rand_inputs(4, **DISTS[dist])
    h, C, n, m = IMPLS[impl](q, k, v, ip, fp, C0, n0, m0)
    hu, Cu, nu = R.recurrent_unstabilized(q, k, v, ip, fp, C0, n0, m0)
    np.testing.assert_allclose(h, hu, rtol=1e-9, atol=1e-12 * np.abs(hu).max())
    np.testing.assert_allclose(C * np.exp(m)[:, None, None], Cu, rtol=1e-9, atol=1e-12 * np.abs(Cu).max())
    np.testing.assert_allclose(n * np.exp(m)[:, None], nu, rtol=1e-9, atol=1e-12 * np.abs(nu).max())


@pytest.mark.parametrize("impl", list(IMPLS))
@pytest.mark.parametrize("delta", [-3.0, 2.5])
def test_initial_state_shift_invariance(impl, delta):
    """(C0, n0, m0) and (e^{-delta} C0, e^{-delta} n0, m0 + delta) are the same unscaled state:
    same h and the same scale-free final state e^{m_T} C_T."""
    q, k, v, ip, fp, C0, n0, m0 = rand_inputs(5, state=True)
    h1, C1, n1, m1 = IMPLS[impl](q, k, v, ip, fp, C0, n0, m0)
    h2, C2, n2, m2 = IMPLS[impl](q, k, v, ip, fp, C0 * np.exp(-delta), n0 * np.exp(-delta), m0 + delta)
    np.testing.assert_allclose(h1, h2, rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(C1 * np.exp(m1 - m2)[:, None, None], C2, rtol=1e-10, atol=1e-13)


@pytest.mark.parametrize("impl", list(IMPLS))
def test_neutral_tokens(impl):
    """A token with i~ = -inf (nothing written) and f~ = +inf (nothing forgotten) leaves
    (C, n, m) unchanged, so inserting such tokens changes neither the other outputs nor the
    final state."""
    q, k, v, ip, fp, C0, n0, m0 = rand_inputs(6, T=11, state=True)
    h, C, n, m = IMPLS[impl](q, k, v, ip, fp, C0, n0, m0)
    ins = [0, 4, 4, 11]
    q2 = np.insert(q, ins, 0.7, axis=1)
    k2 = np.insert(k, ins, -1.3, axis=1)
    v2 = np.insert(v, ins, 2.0, axis=1)
    ip2 = np.insert(ip, ins, -np.inf, axis=1)
    fp2 = np.insert(fp, ins, np.inf, axis=1)
    h2, C2, n2, m2 = IMPLS[impl](q2, k2, v2, ip2, fp2, C0, n0, m0)
    keep = np.ones(h2.shape[1], bool)
    keep[np.array(ins) + np.arange(len(ins))] = False
    np.testing.assert_allclose(h2[:, keep], h, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(C2, C, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(m2, m, rtol=1e-15)


@pytest.mark.parametrize("L", [1, 2, 3, 4, 7, 8, 16, 64])
@pytest.mark.parametrize("dist", list(DISTS))
def test_chunkwise_equals_recurrent_any_L(L, dist):
    """The chunkwise form computes the same h and final state for every chunk size,
    including a ragged last chunk (T = 29)."""
    args = rand_inputs(7, T=29, **DISTS[dist])
    h, C, n, m = _c(*args)
    hc, Cc, nc, mc = R.chunkwise(*args, L=L)
    scale = np.abs(h).max()
    np.testing.assert_allclose(hc, h, rtol=1e-11, atol=1e-13 * scale)
    np.testing.assert_allclose(Cc, C, rtol=1e-11, atol=1e-13 * np.abs(C).max())
    np.testing.assert_allclose(nc, n, rtol=1e-11, atol=1e-13 * np.abs(n).max())
    np.testing.assert_allclose(mc, m, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("dist", list(DISTS))
def test_parallel_equals_recurrent(dist):
    args = rand_inputs(8, T=41, DQK=9, DV=7, **DISTS[dist])
    h, C, n, m = _c(*args)
    hp, Cp, np_, mp = R.parallel_quadratic(*args)
    np.testing.assert_allclose(hp, h, rtol=1e-11, atol=1e-13 * np.abs(h).max())
    np.testing.assert_allclose(Cp, C, rtol=1e-11, atol=1e-13 * np.abs(C).max())
    np.testing.assert_allclose(mp, m, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("impl", ["c_recurrent", "np_chunkwise_L5", "np_parallel"])
def test_state_carry(impl):
    """run(T1) then run(T2) from its final state == run(T1 + T2) (the state is the resume point)."""
    q, k, v, ip, fp, C0, n0, m0 = rand_inputs(9, T=30, state=True)
    f = IMPLS[impl]
    h, C, n, m = f(q, k, v, ip, fp, C0, n0, m0)
    ha, Ca, na, ma = f(q[:, :13], k[:, :13], v[:, :13], ip[:, :13], fp[:, :13], C0, n0, m0)
    hb, Cb, nb, mb = f(q[:, 13:], k[:, 13:], v[:, 13:], ip[:, 13:], fp[:, 13:], Ca, na, ma)
    np.testing.assert_allclose(np.concatenate([ha, hb], axis=1), h, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(Cb, C, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(mb, m, rtol=1e-14, atol=1e-14)


def test_empty_sequence_returns_initial_state():
    q, k, v, ip, fp, C0, n0, m0 = rand_inputs(10, T=0, state=True)
    h, C, n, m = _c(q, k, v, ip, fp, C0, n0, m0)
    assert h.shape == (3, 0, 6)
    np.testing.assert_array_equal(C, C0)
    np.testing.assert_array_equal(m, m0)
    h, C, n, m = _c(q, k, v, ip, fp)
    assert not C.any() and not n.any() and not m.any()


def test_c_oracle_rejects_partial_state():
    q, k, v, ip, fp, C0, n0, m0 = rand_inputs(11, T=4, state=True)
    with pytest.raises(ValueError):
        _c(q, k, v, ip, fp, C0, None, None)


def test_c_oracle_threads_do_not_change_results():
    args = rand_inputs(12, S=7, T=33)
    a = coracle.recurrent(*args, nthreads=1)
    b = coracle.recurrent(*args, nthreads=4)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


# ---- mutation check: each planted mistake must fail at least one pin --------------------------

def _mutant_recurrent(mutation):
    def f(q, k, v, ip, fp, C0=None, n0=None, m0=None):
        S, T, DQK = q.shape
        DV = v.shape[2]
        C = np.zeros((S, DQK, DV)) if C0 is None else C0.copy()
        n = np.zeros((S, DQK)) if n0 is None else n0.copy()
        m = np.zeros(S) if m0 is None else m0.copy()
        h = np.empty((S, T, DV))
        sc = 1.0 if mutation == "no_q_scale" else 1.0 / np.sqrt(DQK)
        for t in range(T):
            a = R.logsigmoid(-fp[:, t] if mutation == "sign_logsig" else fp[:, t])
            mn = np.maximum(a + m, ip[:, t])
            fg = np.exp(a + m - mn)
            ig = np.exp(ip[:, t] - mn)
            C = fg[:, None, None] * C + ig[:, None, None] * k[:, t, :, None] * v[:, t, None, :]
            n = fg[:, None] * n + (k[:, t] if mutation == "n_drops_igate" else ig[:, None] * k[:, t])
            m_floor = m if mutation == "floor_old_m" else mn
            m = mn
            qh = q[:, t] * sc
            num = np.einsum("sdv,sd->sv", C, qh) if mutation != "transposed_C" else np.einsum("svd,sd->sv", C, qh)
            den = np.maximum(np.abs(np.einsum("sd,sd->s", n, qh)), np.exp(-m_floor))
            h[:, t] = num / den[:, None]
        return h, C, n, m
    return f


@pytest.mark.parametrize("mutation", ["no_q_scale", "sign_logsig", "n_drops_igate", "floor_old_m",
                                      "transposed_C"])
def test_pins_catch_planted_mistakes(mutation):
    f = _mutant_recurrent(mutation)
    if mutation == "transposed_C":
        # a square head (DQK == DV), where the transposed product is well formed
        q, k, v, ip, fp, *_ = rand_inputs(13, DQK=5, DV=5)
        h, *_ = f(q, k, v, ip, fp)
        hr, *_ = R.parallel_quadratic(q, k, v, ip, fp)
        assert not np.allclose(h, hr, rtol=1e-9)
        return
    failures = 0
    IMPLS["mut"] = f
    try:
        for check, args in [(test_scalar_example_by_hand, ()),
                            (test_single_token_closed_form, ("standard",)),
                            (test_single_token_closed_form, ("floor_active",)),
                            (test_forget_gate_one_is_weighted_linear_attention, (1.0,))] + \
                           [(test_h_independent_of_max_state, (d,)) for d in DISTS]:
            try:
                check("mut", *args)
            except AssertionError:
                failures += 1
    finally:
        IMPLS.pop("mut")
    assert failures > 0, f"no pin detects mutation {mutation}"
