"""mlstm_chunkwise_bwd (the chunkwise training-mode backward pass, bf16 MFMA) against the fp64 gradient
oracle: ``recurrent_grad_state`` (autograd over the step-by-step cell from a given initial state, with
document borders) for a few chunks, and ``parallel_grad`` (its closed form, pinned to it) for the
xLSTM-7B prefill shapes from the zero state.

Bars: dq, dk, dv and dC0 per row (a token's row, a
d-row of C0) at the bf16 bar of 2e-2, a row that is zero in exact arithmetic held to 1e-3 of its
tensor's largest row; dn0 per sequence; the gate gradients, sums of terms of both signs, against
the magnitude of their summands (|err_t| <= tol sum_d |k_td dk_td| for di~, tol sigmoid(-f~_t)
sum_{t' >= t} sum_d (|q dq| + |k dk|) for df~, from the oracle's gradients).  dm0 = <dC0, C0> + dn0 . n0 is a sum of terms of both signs whose total can be far
below the terms: its error is held to the bar times the sum of the terms' magnitudes,
sum |dC0 C0| + sum |dn0 n0| (the error an elementwise relative error of the bar produces)."""
import numpy as np
import pytest
import torch

from oracle import mlstm_grad as G
from paper_2503_13427_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits
from tests.helpers import TOL_BF16, gate_scales, rel_err, row_err

pytestmark = pytest.mark.gpu

DQK, DV, L = 256, 512, 64


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def bf(x):
    return bf16_bits_to_f32(f32_to_bf16_bits(np.asarray(x, np.float32)))


def draw(seed, S, T, i_mu=0.0, f_mu=3.0, f_sd=1.0, state=False, borders=()):
    rng = np.random.default_rng(seed)
    q = bf(rng.standard_normal((S, T, DQK)))
    k = bf(rng.standard_normal((S, T, DQK)) / np.sqrt(DQK) * 4)
    v = bf(rng.standard_normal((S, T, DV)))
    ip = rng.normal(i_mu, 1.0, (S, T)).astype(np.float32)
    fp = rng.normal(f_mu, f_sd, (S, T)).astype(np.float32)
    for t in borders:
        fp[:, t] = -np.inf
    dh = bf(rng.standard_normal((S, T, DV)))
    st = None
    if state:
        C0 = (rng.standard_normal((S, DQK, DV)) * 0.05).astype(np.float32)
        n0 = np.abs(rng.standard_normal((S, DQK)) * 0.3).astype(np.float32)
        m0 = rng.normal(0.5, 1.0, S).astype(np.float32)
        st = (C0, n0, m0)
    return q, k, v, ip, fp, dh, st


def run(B, NH, q, k, v, ip, fp, dh, st, want_state=True):
    """The backward on the GPU; returns the eight gradients as fp64 host arrays [S, T, -1]
    (dC0, dn0, dm0 as [S, ...]) or five when the state gradients are not requested."""
    S, T, _ = q.shape
    mb = _mb()
    d = lambda x, *shape: torch.from_numpy(np.ascontiguousarray(x)).reshape(*shape).cuda()
    qd, kd = d(q, B, NH, T, DQK).bfloat16(), d(k, B, NH, T, DQK).bfloat16()
    vd, dhd = d(v, B, NH, T, DV).bfloat16(), d(dh, B, NH, T, DV).bfloat16()
    ipd, fpd = d(ip, B, NH, T), d(fp, B, NH, T)
    C0 = n0 = m0 = None
    if st is not None:
        C0, n0, m0 = d(st[0], B, NH, DQK, DV), d(st[1], B, NH, DQK), d(st[2], B, NH)
    outs = [torch.full((B, NH, T, DQK), 9.0, device="cuda"), torch.full((B, NH, T, DQK), 9.0, device="cuda"),
            torch.full((B, NH, T, DV), 9.0, device="cuda"), torch.full((B, NH, T), 9.0, device="cuda"),
            torch.full((B, NH, T), 9.0, device="cuda")]
    sg = [None, None, None]
    if want_state:
        sg = [torch.full((B, NH, DQK, DV), 9.0, device="cuda"), torch.full((B, NH, DQK), 9.0, device="cuda"),
              torch.full((B, NH), 9.0, device="cuda")]
    wsb = torch.empty(mb.mlstm_chunkwise_bwd_workspace_bytes(B, NH, T, DQK, DV, L), dtype=torch.uint8, device="cuda")
    mb.mlstm_chunkwise_bwd(qd, kd, vd, ipd, fpd, C0, n0, m0, L, dhd, *outs, *sg, wsb)
    torch.cuda.synchronize()
    got = [o.cpu().numpy().astype(np.float64).reshape(S, T, -1) for o in outs]
    if want_state:
        got += [sg[0].cpu().numpy().astype(np.float64).reshape(S, DQK, DV),
                sg[1].cpu().numpy().astype(np.float64).reshape(S, DQK),
                sg[2].cpu().numpy().astype(np.float64).reshape(S)]
    return got


NAMES = ["dq", "dk", "dv", "di", "df", "dC0", "dn0", "dm0"]


def compare(got, ref, label, tol=TOL_BF16, state=None, q=None, k=None, fp=None):
    errs = {}
    sc = gate_scales(q, k, fp, ref)
    for n, g, r in zip(NAMES, got, ref):
        g = np.asarray(g, np.float64)
        r = np.asarray(r, np.float64).reshape(g.shape)
        assert np.isfinite(g).all(), n
        if n in ("dq", "dk", "dv"):
            errs[n] = row_err(g, r, g.shape[2], f"{label} {n}", floor=1e-3)
        elif n == "dC0":
            errs[n] = row_err(g, r, DV, f"{label} {n}", floor=1e-3)
        elif n == "dm0":
            scale = (np.abs(np.asarray(ref[5]) * np.asarray(state[0], np.float64)).sum(axis=(1, 2)) +
                     np.abs(np.asarray(ref[6]) * np.asarray(state[1], np.float64)).sum(axis=1))
            errs[n] = float((np.abs(g - r) / np.where(scale > 0, scale, 1.0)).max())
        elif n in ("di", "df"):
            scale = sc[0] if n == "di" else sc[1]
            d = np.abs(g.reshape(scale.shape) - r.reshape(scale.shape))
            errs[n] = float((d / np.where(scale > 0, scale, 1.0)).max()) if d.size else 0.0
        else:   # dn0 per sequence
            errs[n] = rel_err(g.reshape(g.shape[0], -1), r.reshape(g.shape[0], -1), 1)
    print(label + " " + " ".join(f"{n} {e:.2e}" for n, e in errs.items()))
    assert max(errs.values()) <= tol, errs


STATE_CASES = [
    # (label, S, T, draw options)
    ("state", 2, 256, dict(state=True)),
    ("state_ragged_borders", 2, 200, dict(state=True, borders=(40, 63, 64, 100, 101, 199))),
    ("zero_state_short_memory", 1, 150, dict(f_mu=-1.0, f_sd=2.0)),
    ("state_floor_active", 1, 130, dict(state=True, i_mu=-6.0)),
    ("state_one_token", 2, 1, dict(state=True)),
    ("state_one_chunk_ragged", 1, 37, dict(state=True, borders=(20,))),
    ("state_border_first_token", 1, 100, dict(state=True, borders=(0, 64))),
]


@pytest.mark.parametrize("case", STATE_CASES, ids=lambda c: c[0])
def test_chunk_bwd_matches_recurrent_oracle(case):
    label, S, T, opts = case
    q, k, v, ip, fp, dh, st = draw(500 + STATE_CASES.index(case), S, T, **opts)
    got = run(1, S, q, k, v, ip, fp, dh, st)
    if st is None:
        st0 = (np.zeros((S, DQK, DV)), np.zeros((S, DQK)), np.zeros(S))
    else:
        st0 = st
    ref = G.recurrent_grad_state(q, k, v, ip, fp, *st0, dh)
    compare(got, ref, label, state=st0, q=q, k=k, fp=fp)


@pytest.mark.parametrize("T", [2048, 8192])
def test_chunk_bwd_prefill_shapes_sampled_heads(T):
    """The prefill shapes (8 heads of 256 x 512, T = 2048; 4 heads at T = 8192) in one call each, from the
    zero state; two heads checked against the closed-form oracle on those heads alone."""
    NH = 8 if T == 2048 else 4
    q, k, v, ip, fp, dh, _ = draw(600 + T, NH, T)
    got = run(1, NH, q, k, v, ip, fp, dh, None, want_state=False)
    for hd in (0, NH - 1):
        sl = slice(hd, hd + 1)
        ref = G.parallel_grad(q[sl], k[sl], v[sl], ip[sl], fp[sl], dh[sl])
        compare([g[sl] for g in got], ref, f"T{T} head {hd}", q=q[sl], k=k[sl], fp=fp[sl])


@pytest.mark.parametrize("fwd_L", [64, 128])
def test_autograd_cell_with_state_and_borders(fwd_L):
    """Gradients through ``mlstm_cell`` (chunkwise forward from a given state, chunkwise backward) for
    the loss sum(h * w), with document borders, against the fp64 oracle with dh = w (bf16)."""
    from paper_2503_13427_amd.cell import mlstm_cell
    S, T = 2, 170
    q, k, v, ip, fp, w, st = draw(640 + fwd_L, S, T, state=True, borders=(30, 64, 129))
    dev = lambda x, *shape: torch.from_numpy(np.ascontiguousarray(x)).reshape(*shape).cuda()
    leaf = lambda x, dt, *shape: dev(x, *shape).to(dt).requires_grad_(True)
    tq, tk = leaf(q, torch.bfloat16, 1, S, T, DQK), leaf(k, torch.bfloat16, 1, S, T, DQK)
    tv = leaf(v, torch.bfloat16, 1, S, T, DV)
    tip, tfp = leaf(ip, torch.float32, 1, S, T), leaf(fp, torch.float32, 1, S, T)
    tC, tn, tm = (leaf(st[0], torch.float32, 1, S, DQK, DV), leaf(st[1], torch.float32, 1, S, DQK),
                  leaf(st[2], torch.float32, 1, S))
    h, (CT, nT, mT) = mlstm_cell(tq, tk, tv, tip, tfp, L=fwd_L, state=(tC, tn, tm), return_state=True)
    assert h.dtype == torch.bfloat16 and not CT.requires_grad
    (h * dev(w, 1, S, T, DV).bfloat16()).sum().backward()
    torch.cuda.synchronize()
    got = [t.grad.float().cpu().numpy().astype(np.float64).reshape(S, T, -1) for t in (tq, tk, tv, tip, tfp)]
    got += [tC.grad.cpu().numpy().astype(np.float64).reshape(S, DQK, DV),
            tn.grad.cpu().numpy().astype(np.float64).reshape(S, DQK), tm.grad.cpu().numpy().astype(np.float64)]
    ref = G.recurrent_grad_state(q, k, v, ip, fp, *st, w)
    # dq, dk, dv come back in bf16 (the dtype of q, k, v): one more rounding of 2^-9 within the bar
    compare(got, ref, f"autograd cell L{fwd_L}", state=st, q=q, k=k, fp=fp)
