"""mlstm_chunkwise_fwd_noalloc: the prefill with its segment slots in the library's fixed device
scratch instead of a caller workspace, for callers that cannot allocate.

Checked through the C ABI against mlstm_chunkwise_fwd given a workspace (the same kernels and
schedule: the results must be bit-identical), on two calls in a row, the second with a smaller
input (the scratch keeps the first call's slots), plus the smaller call against the fp64 oracle at
the bf16 bar.
"""
import numpy as np
import pytest
import torch

from oracle import coracle
from paper_2503_13427_amd import configs
from paper_2503_13427_amd.inputs import GateDist, StateDist, make_prefill
from tests.helpers import TOL_BF16, alloc_prefill_outputs, host_f64, row_err, state_errs, upload_prefill

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def _with_workspace(inp, L):
    mb = _mb()
    d = upload_prefill(inp)
    o = alloc_prefill_outputs(inp)
    nb = mb.mlstm_chunkwise_workspace_bytes(inp.B, inp.NH, inp.T, inp.DQK, inp.DV, L)
    assert 0 < nb <= mb.mlstm_chunkwise_scratch_bytes()
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    mb.mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], L,
                           o["h"], o["CT"], o["nT"], o["mT"], workspace=ws)
    return d, o


def _no_alloc(inp, d, L):
    o = alloc_prefill_outputs(inp)
    _mb().mlstm_chunkwise_fwd_noalloc(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], L,
                                      o["h"], o["CT"], o["nT"], o["mT"])
    return o


def test_no_alloc_matches_the_workspace_entry_point_on_two_calls():
    big = configs.PREFILL_T2048.prefill_inputs()       # 8 sequences x 7 segment slots (29.4 MB)
    small = make_prefill(workload=120, B=1, NH=3, T=1000, DQK=256, DV=512, dtype="bf16",
                         gates=GateDist(f_mu=5, f_sd=2, cap=15.0), state=StateDist())   # ragged, L = 128
    cases = [(big, 64), (small, 128)]
    refs = [_with_workspace(inp, L) for inp, L in cases]
    torch.cuda.synchronize()
    for (inp, L), (d, ref) in zip(cases, refs):
        got = _no_alloc(inp, d, L)
        torch.cuda.synchronize()
        for key in ("h", "CT", "nT", "mT"):
            assert torch.equal(got[key], ref[key]), (inp.T, key)
        print(f"T={inp.T} L={L}: bit-identical to the workspace entry point")
    # the smaller call against the oracle
    inp, L = cases[1]
    got = _no_alloc(inp, refs[1][0], L)
    torch.cuda.synchronize()
    hr, Cr, nr, mr = coracle.recurrent_inputs(inp)
    S = inp.B * inp.NH
    eh = row_err(host_f64(got["h"]).reshape(S, inp.T, -1), hr, 512, "no-alloc h")
    eC, en, em = state_errs(host_f64(got["CT"]).reshape(S, 256, 512), host_f64(got["nT"]).reshape(S, 256),
                            host_f64(got["mT"]).reshape(S), Cr, nr, mr, "no-alloc")
    assert max(eh, eC, en, em) <= TOL_BF16


def test_no_alloc_without_a_segment_schedule():
    """A shape the fused pass serves alone (enough sequences to fill the chip) uses no scratch."""
    inp = make_prefill(workload=121, B=1, NH=2, T=64, DQK=256, DV=512, dtype="bf16", gates=GateDist())
    mb = _mb()
    assert mb.mlstm_chunkwise_workspace_bytes(1, 2, 64, 256, 512, 64) == 0
    d = upload_prefill(inp)
    ref = alloc_prefill_outputs(inp)
    mb.mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], None, None, None, 64,
                           ref["h"], ref["CT"], ref["nT"], ref["mT"])
    got = _no_alloc(inp, d, 64)
    torch.cuda.synchronize()
    for key in ("h", "CT", "nT", "mT"):
        assert torch.equal(got[key], ref[key]), key
