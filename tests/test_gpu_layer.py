"""The mLSTM layer (Eq. 11) around libmlstm against the fp64 oracle.

bf16 weights and input.  The layer stores q, k, v and o~ in bf16 after its projections, as a bf16
model does, and keeps the gates in fp32; the oracle takes the same storage step
(``proj_dtype="bf16"``: its own fp64 projections rounded to bf16), so the comparison holds y to
the cell's bar, max relative error <= 2e-2 per batch slice.  The projections are checked
against the oracle's rounded ones to one bf16 rounding step, and the capped gate pre-activations
(fp32 throughout) against the oracle's to fp32 accumulation error.  Decode steps after a prefill are
checked against the whole sequence."""
import numpy as np
import pytest
import torch

from oracle import mlstm_ref as R
from paper_2503_13427_amd.inputs import bf16_bits_to_f32, make_layer
from tests.helpers import TOL_BF16, host_f64, row_err, state_errs

pytestmark = pytest.mark.gpu


def _layer(li, L=64):
    from paper_2503_13427_amd.layer import LayerWeights, MLSTMLayer
    return MLSTMLayer(LayerWeights.from_inputs(li), L=L, eps=1e-6, cap=15.0)


def _oracle(li, proj_dtype="bf16"):
    return R.mlstm_layer(bf16_bits_to_f32(li.x), bf16_bits_to_f32(li.W_in), bf16_bits_to_f32(li.W_proj),
                         li.gate_bias, li.norm_weight, li.NH, li.DQK, li.DV, eps=1e-6, cap=15.0,
                         proj_dtype=proj_dtype)


@pytest.mark.parametrize("B,T,NH,L", [(1, 192, 2, 64), (2, 160, 1, 128)])
def test_layer_prefill_matches_oracle(B, T, NH, L):
    li = make_layer(workload=70, B=B, T=T, NH=NH, DQK=256, DV=512)
    layer = _layer(li, L)
    x = torch.from_numpy(li.x).view(torch.bfloat16).cuda()
    heads = layer.project_heads(x)
    q, ig, fg = host_f64(heads[0]), host_f64(heads[4]), host_f64(heads[5])
    y, (C, n, m) = layer.prefill(x)
    torch.cuda.synchronize()
    yr, (Cr, nr, mr) = _oracle(li)
    err = row_err(host_f64(y), yr, yr.shape[-1], "y")
    xw = bf16_bits_to_f32(li.x).astype(np.float64) @ bf16_bits_to_f32(li.W_in).astype(np.float64)
    q_ref = R.round_bf16(np.moveaxis(xw[..., :NH * 256].reshape(B, T, NH, 256), 2, 1))
    e_q = row_err(q, q_ref, 256)
    a = NH * (2 * 256 + 512)
    gates = [np.moveaxis(R.soft_cap(xw[..., a + j * NH:a + (j + 1) * NH] + li.gate_bias[j], 15.0), 2, 1) for j in (0, 1)]
    e_g = max(float(np.abs(got - ref).max()) for got, ref in zip((ig, fg), gates))
    e_C, e_n, e_m = state_errs(host_f64(C).reshape(B * NH, 256, 512), host_f64(n).reshape(B * NH, 256),
                               host_f64(m).reshape(B * NH), Cr, nr, mr)
    print(f"layer B{B} T{T} NH{NH} L{L}: y {err:.3e}, state C {e_C:.3e} n {e_n:.3e} m {e_m:.3e}, q {e_q:.3e}, "
          f"gates {e_g:.3e}")
    assert np.isfinite(host_f64(y)).all() and err <= TOL_BF16
    assert max(e_C, e_n) <= TOL_BF16 and e_m <= TOL_BF16
    assert e_q <= 2 ** -8
    assert e_g <= 1e-4     # fp32 accumulation of bf16 products; a bf16 round trip would show ~1e-2


def test_layer_prefill_with_document_borders():
    """A packed sequence: borders (f~ = -inf from the gate kernel) restart the state per document
    (App. B); against the oracle layer with the same border mask."""
    from paper_2503_13427_amd.layer import MLSTMLayer  # noqa: F401  (import check)
    B, T, NH = 2, 300, 2
    li = make_layer(workload=73, B=B, T=T, NH=NH, DQK=256, DV=512)
    border = np.zeros((B, T), bool)
    border[0, [40, 64, 65, 200]] = True
    border[1, [0, 128, 299]] = True
    layer = _layer(li)
    x = torch.from_numpy(li.x).view(torch.bfloat16).cuda()
    y, _ = layer.prefill(x, border=torch.from_numpy(border).cuda())
    torch.cuda.synchronize()
    yr, _ = R.mlstm_layer(bf16_bits_to_f32(li.x), bf16_bits_to_f32(li.W_in), bf16_bits_to_f32(li.W_proj),
                          li.gate_bias, li.norm_weight, NH, 256, 512, eps=1e-6, cap=15.0, proj_dtype="bf16",
                          border=border)
    err = row_err(host_f64(y), yr, yr.shape[-1], "y")
    print(f"layer with borders: y {err:.3e}")
    assert np.isfinite(host_f64(y)).all() and err <= TOL_BF16


def test_layer_decode_continues_the_prefill():
    li = make_layer(workload=71, B=2, T=132, NH=2, DQK=256, DV=512)
    layer = _layer(li)
    x = torch.from_numpy(li.x).view(torch.bfloat16).cuda()
    _, state = layer.prefill(x[:, :128].contiguous())
    ys = [layer.step(x[:, t].contiguous(), state) for t in range(128, 132)]
    torch.cuda.synchronize()
    yr, _ = _oracle(li)
    got = np.stack([host_f64(y) for y in ys], axis=1)      # [B, 4, d]
    err = row_err(got, yr[:, 128:], yr.shape[-1], "y")
    print(f"layer decode: y {err:.3e}")
    assert err <= TOL_BF16


def test_graphed_decode_replays_match_eager():
    """Four replays of the captured decode step, with eager work and synchronisations between them,
    each against the eager step from the same state (same kernels on the same data)."""
    from paper_2503_13427_amd.layer import GraphedDecode
    li = make_layer(workload=72, B=2, T=68, NH=2, DQK=256, DV=512)
    layer = _layer(li)
    x = torch.from_numpy(li.x).view(torch.bfloat16).cuda()
    _, st_e = layer.prefill(x[:, :64].contiguous())
    st_g = tuple(t.clone() for t in st_e)
    gd = GraphedDecode(layer, st_g, B=2)
    for t in range(64, 68):
        ye = layer.step(x[:, t].contiguous(), st_e)
        junk = torch.randn(1 << 20, device="cuda").sum()          # eager work between replays
        yg = gd(x[:, t].contiguous()).clone()
        torch.cuda.synchronize()
        e_y = row_err(host_f64(yg), host_f64(ye), ye.shape[-1])
        e_C = row_err(host_f64(st_g[0]), host_f64(st_e[0]), 512)
        print(f"graphed decode t={t}: y {e_y:.3e}, C {e_C:.3e}, junk {float(junk):.1f}")
        assert e_y <= 1e-3 and e_C <= 1e-5
        np.testing.assert_allclose(host_f64(st_g[2]), host_f64(st_e[2]), rtol=1e-6, atol=1e-6)
