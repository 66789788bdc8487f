"""mlstm_chunkwise_fwd_strided: q, k, v as strided views (per-head views of one projection output
[B, T, NH * (2 DQK + 2 DV)], padded rows, a mix of strided and contiguous operands) give results
bit-identical to mlstm_chunkwise_fwd on contiguous head-major copies of the same values (h, C, n, m),
which the MFMA parity tests hold to the fp64 oracle; one case is also checked against the oracle
directly.  Rows past the end of a sequence in the strided layout (the next sequence's rows, or NaN
padding) are never read into the result: a partial last chunk reads zeros there as it does for
contiguous rows.
"""
import numpy as np
import pytest
import torch

from paper_2503_13427_amd.inputs import GateDist, StateDist, make_prefill
from tests.helpers import alloc_prefill_outputs, upload_prefill

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def _ws(inp, L):
    nb = _mb().mlstm_chunkwise_workspace_bytes(inp.B, inp.NH, inp.T, inp.DQK, inp.DV, L)
    return torch.empty(nb, dtype=torch.uint8, device="cuda") if nb else None


def projection_views(d, B, NH, T, pad_rows=0, pad_cols=0, fill=float("nan")):
    """One buffer [B, T + pad_rows, NH (2 DQK + 2 DV) + pad_cols] laid out as the layer's projection
    output (q | k | v | o~ per token), filled with ``fill``, the q, k, v values copied in; returns the
    head-major [B, NH, T, D] views of q, k and v."""
    DQK, DV = d["q"].shape[-1], d["v"].shape[-1]
    W = NH * (2 * DQK + 2 * DV) + pad_cols
    P = torch.full((B, T + pad_rows, W), fill, dtype=torch.bfloat16, device="cuda")
    c = [0, NH * DQK, 2 * NH * DQK, NH * (2 * DQK + DV)]
    views = []
    for j, (name, D) in enumerate((("q", DQK), ("k", DQK), ("v", DV))):
        view = P[:, :T, c[j]:c[j + 1]].view(B, T, NH, D).transpose(1, 2)
        view.copy_(d[name])
        views.append(view)
    return P, views


def run_pair(inp, L, workspace, views):
    d = upload_prefill(inp)
    ref = alloc_prefill_outputs(inp)
    out = alloc_prefill_outputs(inp)
    ws = _ws(inp, L) if workspace else None
    _mb().mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], L,
                              ref["h"], ref["CT"], ref["nT"], ref["mT"], workspace=ws)
    q, k, v = views(d)
    assert not (q.is_contiguous() and k.is_contiguous() and v.is_contiguous())
    _mb().mlstm_chunkwise_fwd_strided(q, k, v, d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], L,
                                      out["h"], out["CT"], out["nT"], out["mT"], workspace=ws)
    torch.cuda.synchronize()
    return ref, out


def assert_identical(ref, out):
    for key in ("h", "CT", "nT", "mT"):
        assert torch.isfinite(out[key].float()).all(), key
        assert torch.equal(ref[key].view(torch.int16) if ref[key].dtype == torch.bfloat16 else ref[key].view(torch.int32),
                           out[key].view(torch.int16) if out[key].dtype == torch.bfloat16 else out[key].view(torch.int32)), key


CASES = [
    # (B, NH, T, L, workspace, gates, state)
    (1, 2, 256, 64, False, GateDist(), None),
    (2, 2, 100, 64, True, GateDist(), StateDist()),                 # partial last chunk, next batch's rows follow
    (1, 2, 1000, 64, True, GateDist(), StateDist()),               # 8 segments, the last ragged
    (2, 1, 300, 128, False, GateDist(f_mu=5, f_sd=2, cap=15.0), StateDist()),
    (1, 2, 700, 128, True, GateDist(), None),
    (1, 1, 17, 64, False, GateDist(), StateDist()),                 # one partial chunk
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c[0]}NH{c[1]}T{c[2]}L{c[3]}-{'seg' if c[4] else 'fused'}")
def test_projection_views_equal_contiguous(case):
    B, NH, T, L, workspace, gd, sd = case
    inp = make_prefill(workload=120, B=B, NH=NH, T=T, DQK=256, DV=512, dtype="bf16", gates=gd, state=sd, seed=T + L)
    keep = []
    ref, out = run_pair(inp, L, workspace, lambda d: keep.append(projection_views(d, B, NH, T)) or keep[0][1])
    assert_identical(ref, out)


@pytest.mark.parametrize("T,L,workspace", [(100, 64, True), (300, 128, False), (1000, 64, True)])
def test_padding_rows_past_T_are_not_read(T, L, workspace):
    """NaN rows right after each sequence's last token and NaN columns after each row: a read of any
    of them into the result would turn it NaN."""
    inp = make_prefill(workload=121, B=2, NH=2, T=T, DQK=256, DV=512, dtype="bf16", gates=GateDist(),
                       state=StateDist(), seed=T)
    keep = []
    ref, out = run_pair(inp, L, workspace,
                        lambda d: keep.append(projection_views(d, 2, 2, T, pad_rows=130, pad_cols=64)) or keep[0][1])
    assert_identical(ref, out)


def test_mixed_strided_and_contiguous_operands():
    """k contiguous head-major, q and v strided with different row strides."""
    B, NH, T, L = 1, 2, 520, 64
    inp = make_prefill(workload=122, B=B, NH=NH, T=T, DQK=256, DV=512, dtype="bf16", gates=GateDist(),
                       state=StateDist())

    def views(d):
        qb = torch.full((B, T, NH, 256 + 8), float("nan"), dtype=torch.bfloat16, device="cuda")
        vb = torch.full((B, T, NH + 1, 512), float("nan"), dtype=torch.bfloat16, device="cuda")
        q = qb[..., :256].transpose(1, 2)
        v = vb[:, :, :NH].transpose(1, 2)
        q.copy_(d["q"])
        v.copy_(d["v"])
        views.keep = (qb, vb)
        return q, d["k"], v

    ref, out = run_pair(inp, L, True, views)
    assert_identical(ref, out)


def test_strided_matches_oracle():
    from oracle import coracle
    from tests.helpers import TOL_BF16, host_f64, row_err, state_errs
    B, NH, T, L = 1, 2, 384, 128
    inp = make_prefill(workload=123, B=B, NH=NH, T=T, DQK=256, DV=512, dtype="bf16",
                       gates=GateDist(f_mu=5, f_sd=2, cap=15.0), state=StateDist())
    keep = []
    _, out = run_pair(inp, L, True, lambda d: keep.append(projection_views(d, B, NH, T)) or keep[0][1])
    hr, Cr, nr, mr = coracle.recurrent_inputs(inp)
    S = B * NH
    eh = row_err(host_f64(out["h"].reshape(S, T, -1)), hr, 512, "strided h")
    eC, en, em = state_errs(host_f64(out["CT"].reshape(S, 256, 512)), host_f64(out["nT"].reshape(S, 256)),
                            host_f64(out["mT"].reshape(S)), Cr, nr, mr, "strided")
    assert max(eh, eC, en, em) <= TOL_BF16, (eh, eC, en, em)


def test_layer_prefill_passes_views_without_copies():
    """The layer's prefill hands the cell per-head views of its projection output: its state equals,
    bit for bit, the cell's on head-major copies of the same projections."""
    from paper_2503_13427_amd.layer import LayerWeights, MLSTMLayer
    from paper_2503_13427_amd.inputs import make_layer
    li = make_layer(workload=124, B=2, T=200, NH=2, DQK=256, DV=512)
    layer = MLSTMLayer(LayerWeights.from_inputs(li), L=64, eps=1e-6, cap=15.0)
    x = torch.from_numpy(li.x).view(torch.bfloat16).cuda()
    y, (C, n, m) = layer.prefill(x)
    q, k, v, o, ig, fg = layer.project_heads(x)
    h = torch.empty(2, 2, 200, 512, dtype=torch.bfloat16, device="cuda")
    C2, n2, m2 = torch.empty_like(C), torch.empty_like(n), torch.empty_like(m)
    nb = _mb().mlstm_chunkwise_workspace_bytes(2, 2, 200, 256, 512, 64)   # the schedule the prefill takes
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda") if nb else None
    _mb().mlstm_chunkwise_fwd(q, k, v, ig, fg, None, None, None, 64, h, C2, n2, m2, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(C, C2) and torch.equal(n, n2) and torch.equal(m, m2)
    assert np.isfinite(y.float().cpu().numpy()).all()
