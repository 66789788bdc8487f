"""mlstm_output_norm (h = sigmoid(o~) * (Norm(h~) * weight + bias), Eq. 6 with Eq. 9) on the GPU
against the fp64 oracle, per (batch, head) slice: <= 2e-2 for bf16 rows, <= 1e-5 for fp32 rows.
Covers LayerNorm and RMSNorm, with and without weight / bias, several row widths, the decode
shape, in-place use, no write past the last row, and the whole cell output: chunkwise h~ from
the MFMA kernel followed by the norm, against the recurrent oracle followed by the oracle norm."""
import numpy as np
import pytest
import torch

from oracle import coracle
from oracle import mlstm_ref as R
from paper_2503_13427_amd.inputs import GateDist, make_prefill
from tests.helpers import TOL_BF16, TOL_F32, alloc_prefill_outputs, host_f64, row_err, upload_prefill

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def _inputs(seed, B, NH, T, DV, dtype, affine):
    rng = np.random.default_rng(seed)
    # rows with their own offset and scale, as h~ rows have
    x = rng.normal(0, 1, (B, NH, T, DV)) * rng.uniform(0.05, 3.0, (B, NH, T, 1)) + rng.normal(0, 0.5, (B, NH, T, 1))
    o = rng.normal(0, 2.0, (B, NH, T, DV))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    xt = torch.from_numpy(x).to(tdt).cuda()
    ot = torch.from_numpy(o).to(tdt).cuda()
    w = torch.from_numpy(rng.normal(1, 0.2, (NH, DV))).float().cuda() if affine else None
    b = torch.from_numpy(rng.normal(0, 0.2, (NH, DV))).float().cuda() if affine else None
    return xt, ot, w, b


def _oracle(xt, ot, w, b, eps, norm):
    return R.output_gate_norm(host_f64(xt), host_f64(ot), None if w is None else host_f64(w),
                              None if b is None else host_f64(b), eps=eps, norm=norm)


CASES = [
    # (B, NH, T, DV, dtype, norm, affine)
    (1, 8, 64, 512, "bf16", "layer", True),
    (1, 8, 64, 512, "bf16", "rms", True),
    (2, 2, 33, 512, "bf16", "layer", False),
    (1, 3, 17, 2048, "f32", "layer", True),
    (2, 2, 5, 4, "f32", "layer", True),
    (1, 4, 9, 64, "f32", "rms", False),
    (3, 1, 7, 1000, "bf16", "rms", True),
    (1, 2, 11, 16, "f32", "rms", True),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}NH{}T{}DV{}-{}-{}-{}".format(*c))
def test_output_norm_matches_oracle(case):
    B, NH, T, DV, dt, norm, affine = case
    xt, ot, w, b = _inputs(100 + CASES.index(case), B, NH, T, DV, dt, affine)
    h = torch.empty_like(xt)
    eps = 1e-6 if dt == "f32" else 1e-5
    _mb().mlstm_output_norm(xt, ot, w, b, eps, norm, h)
    torch.cuda.synchronize()
    ref = _oracle(xt, ot, w, b, eps, norm)
    err = row_err(host_f64(h), ref, ref.shape[-1], "h")
    print(case, f"{err:.3e}")
    assert np.isfinite(host_f64(h)).all()
    assert err <= (TOL_F32 if dt == "f32" else TOL_BF16), err


TOKEN_CASES = [
    # (B, NH, T, DV, dtype, norm, affine, extra columns per projection row)
    (2, 8, 64, 512, "bf16", "layer", True, 8 * (2 * 256 + 512)),
    (3, 2, 33, 512, "bf16", "rms", False, 8),   # base 16-byte aligned, rows 8-byte aligned
    (1, 3, 17, 2048, "f32", "layer", True, 0),
    (2, 4, 9, 64, "f32", "rms", True, 12),
]


@pytest.mark.parametrize("case", TOKEN_CASES, ids=lambda c: "B{}NH{}T{}DV{}-{}-{}-{}-pad{}".format(*c))
def test_output_norm_tokens_matches_oracle(case):
    """o~ as columns of a wider token-major projection output, y token-major: element by element
    the same result as the head-major oracle, transposed."""
    B, NH, T, DV, dt, norm, affine, pad = case
    xt, ot, w, b = _inputs(300 + TOKEN_CASES.index(case), B, NH, T, DV, dt, affine)
    P = torch.full((B * T, pad + NH * DV + 4), 7.0, dtype=xt.dtype, device="cuda")
    o_view = P[:, pad:pad + NH * DV].view(B, T, NH, DV)
    o_view.copy_(ot.transpose(1, 2))
    y = torch.full((B, T, NH, DV + 0), -5.0, dtype=xt.dtype, device="cuda")
    eps = 1e-6 if dt == "f32" else 1e-5
    _mb().mlstm_output_norm_tokens(xt, o_view, w, b, eps, norm, y)
    torch.cuda.synchronize()
    ref = _oracle(xt, ot, w, b, eps, norm).transpose(0, 2, 1, 3)
    err = row_err(host_f64(y), ref, ref.shape[-1], "y")
    print(case, f"{err:.3e}")
    assert err <= (TOL_F32 if dt == "f32" else TOL_BF16), err
    # the head-major call on the same rows gives the same bits
    h = torch.empty_like(xt)
    _mb().mlstm_output_norm(xt, ot, w, b, eps, norm, h)
    torch.cuda.synchronize()
    assert torch.equal(h.transpose(1, 2), y)


def test_decode_shape_and_in_place():
    xt, ot, w, b = _inputs(7, 256, 8, 1, 512, "bf16", True)
    x3, o3 = xt[:, :, 0].contiguous(), ot[:, :, 0].contiguous()
    h = torch.empty_like(x3)
    _mb().mlstm_output_norm(x3, o3, w, b, 1e-6, "layer", h)
    ref = _oracle(xt, ot, w, b, 1e-6, "layer")[:, :, 0]
    torch.cuda.synchronize()
    assert row_err(host_f64(h), ref, ref.shape[-1], "h") <= TOL_BF16
    y = x3.clone()
    _mb().mlstm_output_norm(y, o3, w, b, 1e-6, "layer", y)   # in place
    torch.cuda.synchronize()
    assert torch.equal(y, h)


def test_no_write_past_the_last_row():
    T, DV = 13, 512   # 13 rows: the last workgroup has three idle waves
    xt, ot, w, b = _inputs(8, 1, 1, T, DV, "bf16", True)
    big = torch.full((T + 8, DV), 3.0, dtype=torch.bfloat16, device="cuda")
    h = big[:T].view(1, 1, T, DV)
    _mb().mlstm_output_norm(xt, ot, w, b, 1e-6, "rms", h)
    torch.cuda.synchronize()
    assert bool((big[T:] == 3.0).all())
    assert row_err(host_f64(h), _oracle(xt, ot, w, b, 1e-6, "rms"), DV, "h") <= TOL_BF16


def test_cell_output_end_to_end():
    """h = sigmoid(o~) * LayerNorm(h~) with h~ from the chunkwise MFMA kernel, against the fp64
    recurrent h~ followed by the oracle norm."""
    inp = make_prefill(workload=96, B=1, NH=2, T=320, DQK=256, DV=512, dtype="bf16", gates=GateDist(), state=None)
    d = upload_prefill(inp)
    o = alloc_prefill_outputs(inp)
    _mb().mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], None, None, None, 64,
                              o["h"], o["CT"], o["nT"], o["mT"])
    rng = np.random.default_rng(11)
    ot = torch.from_numpy(rng.normal(0, 2, (1, 2, 320, 512))).to(torch.bfloat16).cuda()
    w = torch.from_numpy(rng.normal(1, 0.2, (2, 512))).float().cuda()
    b = torch.from_numpy(rng.normal(0, 0.2, (2, 512))).float().cuda()
    h = torch.empty_like(o["h"])
    _mb().mlstm_output_norm(o["h"], ot, w, b, 1e-6, "layer", h)
    torch.cuda.synchronize()
    hr, _, _, _ = coracle.recurrent_inputs(inp)
    ref = R.output_gate_norm(hr.reshape(1, 2, 320, 512), host_f64(ot), host_f64(w), host_f64(b), eps=1e-6,
                             norm="layer")
    err = row_err(host_f64(h), ref, ref.shape[-1], "h")
    print(f"cell output {err:.3e}")
    assert err <= TOL_BF16
