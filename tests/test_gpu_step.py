"""mlstm_step on the GPU against the fp64 recurrent oracle (Eqs. 2-5, 7-8).

Parity bar: max relative error per row (each h row of one (batch, head, step), each d-row
of C; see helpers) <= 1e-5 for fp32 q/k/v/h and <= 2e-2 for bf16 q/k/v/h, fp32 state in
both cases.  Few
sequences take the column-split launch (several workgroups per sequence, n' and
m' from a second kernel), many take one workgroup per sequence; both run in
place and out of place.
"""
import os

import numpy as np
import pytest
import torch

from oracle import coracle
from paper_2503_13427_amd import configs
from tests.helpers import TOL_BF16, TOL_F32, dev, host_f64, row_err, state_errs

pytestmark = pytest.mark.gpu


def _mlstm():
    from paper_2503_13427_amd import binding
    return binding


def rand_state(rng, S, DQK, DV):
    C = rng.normal(0, 0.1, (S, DQK, DV)).astype(np.float32)
    n = np.abs(rng.standard_normal((S, DQK))).astype(np.float32)
    m = rng.standard_normal(S).astype(np.float32)
    return C, n, m


def run_steps(q, k, v, ip, fp, C, n, m, dtype, in_place=True):
    """q, k: [S, steps, DQK] host arrays (fp32 or bf16 bits); returns h [S, steps, DV] and the final state."""
    B = 1
    S, steps, DQK = q.shape
    DV = v.shape[2]
    mb = _mlstm()
    tq, tk, tv = dev(q), dev(k), dev(v)
    tip, tfp = dev(ip), dev(fp)
    Cd, nd, md = dev(C).reshape(B, S, DQK, DV), dev(n).reshape(B, S, DQK), dev(m).reshape(B, S)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    h = torch.empty(B, S, steps, DV, dtype=tdt, device="cuda")
    if not in_place:
        C2, n2, m2 = torch.empty_like(Cd), torch.empty_like(nd), torch.empty_like(md)
    for t in range(steps):
        hs = torch.empty(B, S, DV, dtype=tdt, device="cuda")
        # fresh copies: with one sequence a step's slice is contiguous already, and a view of it
        # would start mid-buffer (the library requires 16-byte aligned tensors)
        cp = lambda a: a.clone(memory_format=torch.contiguous_format)
        qt = cp(tq[:, t]).reshape(B, S, DQK)
        kt = cp(tk[:, t]).reshape(B, S, DQK)
        vt = cp(tv[:, t]).reshape(B, S, DV)
        it = cp(tip[:, t]).reshape(B, S)
        ft = cp(tfp[:, t]).reshape(B, S)
        if in_place:
            mb.mlstm_step(qt, kt, vt, it, ft, Cd, nd, md, hs, Cd, nd, md)
        else:
            mb.mlstm_step(qt, kt, vt, it, ft, Cd, nd, md, hs, C2, n2, m2)
            Cd, C2, nd, n2, md, m2 = C2, Cd, n2, nd, m2, md
        h[:, :, t] = hs
    torch.cuda.synchronize()
    return host_f64(h)[0], host_f64(Cd)[0], host_f64(nd)[0], host_f64(md)[0]


def widen(x):
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def check(q, k, v, ip, fp, C, n, m, dtype, tol):
    h, Cg, ng, mg = run_steps(q, k, v, ip, fp, C, n, m, dtype)
    hr, Cr, nr, mr = coracle.recurrent(widen(q), widen(k), widen(v), ip.astype(np.float64), fp.astype(np.float64),
                                       C.astype(np.float64), n.astype(np.float64), m.astype(np.float64))
    eh = row_err(h, hr, v.shape[2], "h")
    eC, en, em = state_errs(Cg, ng, mg, Cr, nr, mr, "state")
    print(f"h {eh:.3e} C {eC:.3e} n {en:.3e} m {em:.3e}")
    assert eh <= tol and eC <= tol and en <= tol and em <= tol, (eh, eC, en, em)
    return h, Cg, ng, mg


def bf16(x):
    from paper_2503_13427_amd.inputs import f32_to_bf16_bits
    return f32_to_bf16_bits(x.astype(np.float32))


@pytest.mark.parametrize("DQK,DV", [(16, 16), (7, 12), (1, 4), (64, 1024), (256, 512), (300, 2048)])
def test_step_fp32_matches_oracle(DQK, DV):
    rng = np.random.default_rng(DQK * 1000 + DV)
    S, steps = 5, 6
    q = rng.standard_normal((S, steps, DQK)).astype(np.float32)
    k = (rng.standard_normal((S, steps, DQK)) / np.sqrt(DQK)).astype(np.float32)
    v = rng.standard_normal((S, steps, DV)).astype(np.float32)
    ip = rng.standard_normal((S, steps)).astype(np.float32)
    fp = rng.normal(3, 1, (S, steps)).astype(np.float32)
    check(q, k, v, ip, fp, *rand_state(rng, S, DQK, DV), "f32", TOL_F32)


@pytest.mark.parametrize("dist", ["standard", "floor_active", "reset_and_neutral"])
def test_step_bf16_xlstm_head_matches_oracle(dist):
    rng = np.random.default_rng(7)
    S, steps, DQK, DV = 24, 8, 256, 512
    q = bf16(rng.standard_normal((S, steps, DQK)))
    k = bf16(rng.standard_normal((S, steps, DQK)))
    v = bf16(rng.standard_normal((S, steps, DV)))
    ip = rng.normal(-10.0 if dist == "floor_active" else 0.0, 1.0, (S, steps)).astype(np.float32)
    fp = rng.normal(3, 1, (S, steps)).astype(np.float32)
    if dist == "reset_and_neutral":
        fp[::3, 2] = -np.inf     # forget gate exactly zero: the state restarts
        ip[1::3, 4] = -np.inf    # nothing written ...
        fp[1::3, 4] = np.inf     # ... and nothing forgotten: a neutral token
    check(q, k, v, ip, fp, *rand_state(rng, S, DQK, DV), "bf16", TOL_BF16)


@pytest.mark.parametrize("S", [1, 8, 300])
def test_step_bf16_head_counts(S):
    """One sequence and B = 1 x 8 heads split each head's columns over many workgroups (n', m'
    from the second kernel); 300 heads keep one workgroup per head.  In place, several steps."""
    rng = np.random.default_rng(100 + S)
    steps, DQK, DV = 4, 256, 512
    q = bf16(rng.standard_normal((S, steps, DQK)))
    k = bf16(rng.standard_normal((S, steps, DQK)))
    v = bf16(rng.standard_normal((S, steps, DV)))
    ip = rng.standard_normal((S, steps)).astype(np.float32)
    fp = rng.normal(3, 1, (S, steps)).astype(np.float32)
    fp[0, 2] = -np.inf
    check(q, k, v, ip, fp, *rand_state(rng, S, DQK, DV), "bf16", TOL_BF16)


def test_step_in_place_equals_out_of_place_and_is_deterministic():
    rng = np.random.default_rng(11)
    S, steps, DQK, DV = 16, 3, 256, 512
    q = bf16(rng.standard_normal((S, steps, DQK)))
    k = bf16(rng.standard_normal((S, steps, DQK)))
    v = bf16(rng.standard_normal((S, steps, DV)))
    ip = rng.standard_normal((S, steps)).astype(np.float32)
    fp = rng.normal(3, 1, (S, steps)).astype(np.float32)
    st = rand_state(rng, S, DQK, DV)
    a = run_steps(q, k, v, ip, fp, *st, "bf16", in_place=True)
    b = run_steps(q, k, v, ip, fp, *st, "bf16", in_place=False)
    c = run_steps(q, k, v, ip, fp, *st, "bf16", in_place=True)
    for x, y, z in zip(a, b, c):
        np.testing.assert_array_equal(x, y)
        np.testing.assert_array_equal(x, z)


def decode_initial_state(heads):
    """State after the decode workload's 128-token prefill, computed by the oracle in fp64 and
    rounded once to fp32 (both sides then start from the same fp32 state)."""
    w = configs.DECODE_B256
    pre = w.prefill_inputs(heads=heads)
    _, C, n, m = coracle.recurrent_inputs(pre)
    return C.astype(np.float32), n.astype(np.float32), m.astype(np.float32)


@pytest.mark.slow
def test_step_decode_workload_full_size_sampled_heads():
    """The decode workload at full size (B=256, NH=8, DQK=256, DV=512) in the launch
    configuration the benchmark times; ``MLSTM_DECODE_STEPS`` steps (default 1024).  Every head
    runs on the GPU; 64 heads spread over the batch (plus three fixed ones) are checked against
    the oracle at every step, each h row and each d-row of the final state."""
    w = configs.DECODE_B256
    steps = int(os.environ.get("MLSTM_DECODE_STEPS", w.steps))
    S = w.heads
    mb = _mlstm()
    C, n, m = decode_initial_state(None)
    dec = w.decode_inputs(steps=steps)
    sample = np.unique(np.concatenate([np.linspace(0, S - 1, 64).round().astype(np.int64), [1, 777, 1024]]))
    Cd, nd, md = dev(C).reshape(w.B, w.NH, 256, 512), dev(n).reshape(w.B, w.NH, 256), dev(m).reshape(w.B, w.NH)
    q, k, v = dev(dec.q), dev(dec.k), dev(dec.v)
    ip, fp = dev(dec.ipre), dev(dec.fpre)
    hs = torch.empty(steps, len(sample), 512, dtype=torch.float64)
    h = torch.empty(w.B, w.NH, 512, dtype=torch.bfloat16, device="cuda")
    sel = torch.from_numpy(sample).cuda()
    for t in range(steps):
        mb.mlstm_step(q[:, :, t].contiguous(), k[:, :, t].contiguous(), v[:, :, t].contiguous(),
                      ip[:, :, t].contiguous(), fp[:, :, t].contiguous(), Cd, nd, md, h, Cd, nd, md)
        hs[t] = h.reshape(S, 512).index_select(0, sel).double().cpu()
    torch.cuda.synchronize()
    sub = w.decode_inputs(steps=steps, heads=sample)
    hr, Cr, nr, mr = coracle.recurrent(sub.as_f64("q")[0], sub.as_f64("k")[0], sub.as_f64("v")[0],
                                       sub.as_f64("ipre")[0], sub.as_f64("fpre")[0], C[sample].astype(np.float64),
                                       n[sample].astype(np.float64), m[sample].astype(np.float64))
    eh = row_err(hs.numpy().transpose(1, 0, 2), hr, 512, f"{len(sample)} heads x {steps} steps: h")
    Cg = host_f64(Cd.reshape(S, 256, 512)[sel])
    ng = host_f64(nd.reshape(S, 256)[sel])
    mg = host_f64(md.reshape(S)[sel])
    eC, en, em = state_errs(Cg, ng, mg, Cr, nr, mr, "final state")
    print(f"steps {steps}: max row errors h {eh:.3e} C {eC:.3e} n {en:.3e} m {em:.3e}")
    assert eh <= TOL_BF16 and eC <= TOL_BF16 and en <= TOL_BF16 and em <= TOL_BF16
    assert torch.isfinite(Cd).all()
