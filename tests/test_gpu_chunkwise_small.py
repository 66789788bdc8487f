"""mlstm_chunkwise_fwd on small heads (the fp32 VALU kernel) against the fp64 oracle.

Covers the tiny fp32 workload (B=1, NH=1, T=64, d=16, L=16) at the fp32 bar of
1e-5, chunk-size independence, an initial state, T = 0, document resets (f~ = -inf),
bf16 inputs through the same kernel, and T decode steps == one prefill of T tokens.
"""
import numpy as np
import pytest
import torch

from oracle import coracle
from paper_2503_13427_amd import configs
from paper_2503_13427_amd.inputs import GateDist, StateDist, make_prefill
from tests.helpers import (TOL_BF16, TOL_F32, alloc_prefill_outputs, host_f64, row_err, state_errs,
                           upload_prefill)

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def run_chunk(inp, L, workspace=None):
    d = upload_prefill(inp)
    o = alloc_prefill_outputs(inp)
    _mb().mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], L,
                              o["h"], o["CT"], o["nT"], o["mT"], workspace=workspace)
    torch.cuda.synchronize()
    return {k: host_f64(t) for k, t in o.items()}


def compare(inp, out, tol, label=""):
    S = inp.B * inp.NH
    hr, Cr, nr, mr = coracle.recurrent_inputs(inp)
    eh = row_err(out["h"].reshape(S, inp.T, inp.DV), hr, inp.DV, f"{label} h")
    eC, en, em = state_errs(out["CT"].reshape(S, inp.DQK, inp.DV), out["nT"].reshape(S, inp.DQK),
                            out["mT"].reshape(S), Cr, nr, mr)
    print(f"{label} h {eh:.3e} C {eC:.3e} n {en:.3e} m {em:.3e}")
    assert eh <= tol and eC <= tol and en <= tol and em <= tol, (eh, eC, en, em)
    return eh


def test_tiny_fp32_workload():
    w = configs.TINY_F32
    inp = w.prefill_inputs()
    out = run_chunk(inp, w.L)
    compare(inp, out, TOL_F32, w.name)


SMALL = [
    # (B, NH, T, DQK, DV, L, dtype, state, gates)
    (2, 3, 96, 16, 16, 16, "f32", True, GateDist()),
    (1, 2, 128, 32, 64, 32, "f32", True, GateDist(f_mu=5, f_sd=2, cap=15.0)),
    (2, 2, 64, 64, 32, 64, "f32", False, GateDist(i_mu=-10)),
    (1, 4, 192, 16, 128, 64, "f32", True, GateDist(f_mu=-1, f_sd=2)),
    (1, 2, 64, 128, 16, 16, "f32", False, GateDist()),
    (3, 2, 128, 32, 32, 32, "bf16", True, GateDist()),
    # partial last chunk
    (1, 2, 50, 16, 16, 16, "f32", True, GateDist()),
    (2, 1, 70, 32, 64, 32, "f32", False, GateDist(f_mu=5, f_sd=2, cap=15.0)),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "B{}NH{}T{}d{}x{}L{}{}".format(*c[:7]))
def test_small_heads_match_oracle(case):
    B, NH, T, DQK, DV, L, dt, st, g = case
    inp = make_prefill(workload=90, B=B, NH=NH, T=T, DQK=DQK, DV=DV, dtype=dt, gates=g,
                       state=StateDist() if st else None, k_scale=1 / np.sqrt(DQK))
    out = run_chunk(inp, L)
    compare(inp, out, TOL_F32 if dt == "f32" else TOL_BF16)


@pytest.mark.parametrize("borders", ["edges", "every", 20.0])
@pytest.mark.parametrize("L", [16, 32])
def test_document_resets_fp32(borders, L):
    """f~ = -inf (a document border, App. B) restarts the state; fp32 bar."""
    from paper_2503_13427_amd.inputs import pack_documents
    T = 150
    inp = make_prefill(workload=93, B=1, NH=3, T=T, DQK=16, DV=32, dtype="f32", gates=GateDist(),
                       state=StateDist(), k_scale=0.25)
    if borders == "edges":
        inp.fpre[..., [0, L - 1, L, L + 1, 2 * L + 5, 2 * L + 6, T - 1]] = -np.inf
    elif borders == "every":
        inp.fpre[...] = -np.inf
    else:
        pack_documents(inp, borders, workload=93)
    out = run_chunk(inp, L)
    compare(inp, out, TOL_F32, f"resets L{L} {borders}")


def test_chunk_size_independence_fp32():
    inp = make_prefill(workload=91, B=1, NH=3, T=64, DQK=16, DV=32, dtype="f32", gates=GateDist(),
                       state=StateDist(), k_scale=0.25)
    outs = [run_chunk(inp, L) for L in (16, 32, 64)]
    for o in outs[1:]:
        assert row_err(o["h"], outs[0]["h"], 32, "L vs L16") < 2e-6
        np.testing.assert_allclose(o["mT"], outs[0]["mT"], rtol=1e-6, atol=1e-6)


def test_empty_sequence_copies_initial_state():
    inp = make_prefill(workload=92, B=1, NH=2, T=0, DQK=16, DV=16, dtype="f32", gates=GateDist(),
                       state=StateDist())
    out = run_chunk(inp, 16)
    np.testing.assert_array_equal(out["CT"], inp.C0)
    np.testing.assert_array_equal(out["nT"], inp.n0)
    np.testing.assert_array_equal(out["mT"], inp.m0)


def test_decode_steps_equal_prefill_fp32():
    """T steps of mlstm_step == one mlstm_chunkwise_fwd over the same T tokens."""
    inp = make_prefill(workload=93, B=1, NH=2, T=32, DQK=16, DV=16, dtype="f32", gates=GateDist(),
                       state=StateDist(), k_scale=0.25)
    out = run_chunk(inp, 16)
    d = upload_prefill(inp)
    C, n, m = d["C0"].clone(), d["n0"].clone(), d["m0"].clone()
    hs = []
    for t in range(inp.T):
        h = torch.empty(1, 2, 16, device="cuda")
        _mb().mlstm_step(d["q"][:, :, t].contiguous(), d["k"][:, :, t].contiguous(), d["v"][:, :, t].contiguous(),
                         d["ipre"][:, :, t].contiguous(), d["fpre"][:, :, t].contiguous(), C, n, m, h, C, n, m)
        hs.append(h)
    torch.cuda.synchronize()
    hstep = host_f64(torch.stack(hs, dim=2))
    assert row_err(hstep, out["h"].reshape(hstep.shape), 16, "steps vs prefill") < 2e-6
    eC, en, em = state_errs(host_f64(C).reshape(2, 16, 16), host_f64(n).reshape(2, 16), host_f64(m).reshape(2),
                            out["CT"].reshape(2, 16, 16), out["nT"].reshape(2, 16), out["mT"].reshape(2))
    assert max(eC, en, em) < 2e-6
