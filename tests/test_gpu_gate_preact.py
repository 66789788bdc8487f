"""mlstm_gate_preact (gate projection, bias, soft-cap, document borders; Eq. 11, Eq. 13, App. B)
against the fp64 oracle ``gate_preact``.

bf16 x and weights (the oracle upcasts the same bf16 values exactly), fp32 accumulation and
fp32 gates: the bar is the fp32 one, max relative error <= 1e-5 per (batch, head) slice, and
border tokens must hold exactly -inf in f~ while keeping their i~.  Covers the three launch shapes
(at most 16 tokens, fewer and more than 4096 tokens), ragged token tiles, a partial gate-column tile (2 NH = 6),
several column tiles (NH = 16, 32), a decode step ([B, d] input), no cap, no bias, and the
65 536-token layer shape on sampled tokens.
"""
import numpy as np
import pytest
import torch

from oracle import mlstm_ref as R
from paper_2503_13427_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits
from tests.helpers import TOL_F32, rel_err

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def draw(seed, B, T, d, NH, border_rate=0.01):
    rng = np.random.default_rng(seed)
    x = f32_to_bf16_bits(rng.standard_normal((B, T, d), dtype=np.float32))
    w_t = f32_to_bf16_bits((rng.standard_normal((2 * NH, d)) * d ** -0.5).astype(np.float32))
    bias = np.stack([rng.normal(-2, 1, NH), rng.normal(3, 1, NH)]).astype(np.float32)
    border = rng.random((B, T)) < border_rate
    return x, w_t, bias, border


def run(x, w_t, bias, cap, border, decode=False):
    B, T, d = x.shape
    NH = w_t.shape[0] // 2
    xd = torch.from_numpy(x).view(torch.bfloat16).cuda()
    if decode:
        xd = xd.reshape(B, d)
    wd = torch.from_numpy(w_t).view(torch.bfloat16).cuda()
    bd = None if bias is None else torch.from_numpy(bias).cuda()
    brd = None if border is None else torch.from_numpy(border.astype(np.uint8)).cuda()
    ip = torch.full((B, NH, T), 7.0, device="cuda")
    fp = torch.full((B, NH, T), 7.0, device="cuda")
    _mb().mlstm_gate_preact(xd, wd, bd, cap, brd, ip.reshape(B, NH, T) if not decode else ip.reshape(B, NH),
                            fp.reshape(B, NH, T) if not decode else fp.reshape(B, NH))
    torch.cuda.synchronize()
    return ip.cpu().numpy().astype(np.float64), fp.cpu().numpy().astype(np.float64)


def compare(got, want, label, per_head=True):
    """Relative error per (batch, head) slice of T gates, or (per_head=False, a decode step whose
    slices would hold one gate each) over the whole tensor."""
    ig, fg = got
    ir, fr = want
    S = ir.shape[0] * ir.shape[1] if per_head else 1
    inf = np.isneginf(fr)
    assert np.array_equal(np.isneginf(fg), inf), label
    ei = rel_err(ig.reshape(S, -1), ir.reshape(S, -1), 1)
    ef = rel_err(np.where(inf, 0, fg).reshape(S, -1), np.where(inf, 0, fr).reshape(S, -1), 1)
    print(f"{label}: i~ {ei:.3e} f~ {ef:.3e} borders {int(inf.sum())}")
    assert np.isfinite(ig).all() and ei <= TOL_F32 and ef <= TOL_F32


CASES = [
    # (B, T, d, NH, cap, bias, border)
    (2, 100, 512, 8, 15.0, True, True),      # 200 tokens: single-tile path, ragged last tile
    (1, 5000, 256, 8, 15.0, True, True),     # four-tile path, ragged last workgroup
    (1, 70, 256, 3, 15.0, True, False),      # 2 NH = 6: a partial column tile
    (1, 300, 384, 16, 0.0, False, True),     # two column tiles, no cap, no bias
    (1, 64, 128, 32, 15.0, True, True),      # four column tiles
    (3, 4100, 128, 8, 0.0, True, False),     # tiles crossing batch boundaries
    (1, 1, 4096, 8, 15.0, True, True),       # one token: sixteen-wave path
    (3, 5, 512, 16, 15.0, True, True),       # 15 tokens, two column tiles: sixteen-wave path
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c[0]}T{c[1]}d{c[2]}NH{c[3]}cap{c[4]:g}")
def test_gate_preact_matches_oracle(case):
    B, T, d, NH, cap, has_bias, has_border = case
    x, w_t, bias, border = draw(200 + CASES.index(case), B, T, d, NH)
    bias = bias if has_bias else None
    border = border if has_border else None
    got = run(x, w_t, bias, cap, border)
    want = R.gate_preact(bf16_bits_to_f32(x), bf16_bits_to_f32(w_t).T, np.zeros((2, NH)) if bias is None else bias,
                         cap=cap if cap > 0 else None, border=border)
    compare(got, want, str(case), per_head=T >= 16)


def test_gate_preact_decode_step():
    """A decode step passes x [B, d] and receives [B, NH] gates (T = 1)."""
    x, w_t, bias, _ = draw(210, 256, 1, 4096, 8)
    got = run(x, w_t, bias, 15.0, None, decode=True)
    want = R.gate_preact(bf16_bits_to_f32(x), bf16_bits_to_f32(w_t).T, bias, cap=15.0)
    compare(got, want, "decode B256", per_head=False)


def test_gate_preact_layer_shape_sampled():
    """65 536 tokens at d = 4096, NH = 8 (the layer benchmark's prefill), checked on 2048 sampled tokens."""
    B, T, d, NH = 8, 8192, 4096, 8
    rng = np.random.default_rng(211)
    x = f32_to_bf16_bits(rng.standard_normal((B, T, d), dtype=np.float32))
    w_t = f32_to_bf16_bits((rng.standard_normal((2 * NH, d)) * d ** -0.5).astype(np.float32))
    bias = np.stack([rng.normal(-2, 1, NH), rng.normal(3, 1, NH)]).astype(np.float32)
    border = rng.random((B, T)) < 1 / 300
    ig, fg = run(x, w_t, bias, 15.0, border)
    ts = np.sort(rng.choice(T, 256, replace=False))
    want = R.gate_preact(bf16_bits_to_f32(x[:, ts]), bf16_bits_to_f32(w_t).T, bias, cap=15.0, border=border[:, ts])
    compare((ig[:, :, ts], fg[:, :, ts]), want, "layer shape, 2048 sampled tokens")
