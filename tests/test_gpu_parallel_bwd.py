"""mlstm_parallel_bwd (the training-mode backward pass over the parallel form) against the fp64
gradient oracle: ``recurrent_grad`` (autograd over the step-by-step cell) for small shapes and
``parallel_grad`` (its closed form, pinned to it) for the xLSTM-7B head shape.

Bars: dq, dk, dv per token row at the spec bars, 1e-5 for fp32 q/k/v and 2e-2 for bf16 (the
oracle upcasts the same bf16 values), a row that is zero in exact arithmetic held to 1e-3 of its
tensor's largest row.  A row whose value is far below its terms (dq_t sums W_ts k_s over s with
W_ts = dh_t . (v_s - sign(D_t) h_t) F~_ts / den_t, which nearly vanishes when h_t is close to v_s, as
with a short memory) may instead meet the bar elementwise against the magnitudes of all the terms an
evaluation sums, inner dot products included (``parallel_grad_scales``); a row passes if either
error is within the bar.  The gate gradients are sums of terms of both signs that cancel:
di~_t = k_t . dk_t and dlogsig(f~_t) = sum_{t' >= t} (q_t' . dq_t' - k_t' . dk_t'), so an error
relative to their cancelled value says nothing about the arithmetic.  Their bar is the same
relative bar applied to the magnitude of the summands, from the oracle's own gradients:
|di~_t - ref| <= tol sum_d |k_td dk_td| and
|df~_t - ref| <= tol sigmoid(-f~_t) sum_{t' >= t} sum_d (|q_t'd dq_t'd| + |k_t'd dk_t'd|),
which is what a relative error of tol in every summand produces.  Covers ragged T (not a multiple
of the 16-token tile), one token, the floor branch and short memory, on both the VALU passes (DQK or
DV not a multiple of 64) and the MFMA passes, and the benchmarked shape (8 heads, T = 2048) with
sampled heads."""
import numpy as np
import pytest
import torch

from oracle import mlstm_grad as G
from paper_2503_13427_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits
from tests.helpers import TOL_BF16, TOL_F32, gate_scales, row_errs

TOL_BWD_F32 = TOL_F32

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def draw(seed, B, NH, T, DQK, DV, dtype, i_mu=0.0, f_mu=3.0, f_sd=1.0):
    rng = np.random.default_rng(seed)
    S = B * NH
    q = rng.standard_normal((S, T, DQK)).astype(np.float32)
    k = (rng.standard_normal((S, T, DQK)) / np.sqrt(DQK) * 4).astype(np.float32)
    v = rng.standard_normal((S, T, DV)).astype(np.float32)
    if dtype == "bf16":
        q, k, v = (bf16_bits_to_f32(f32_to_bf16_bits(x)) for x in (q, k, v))
    ip = rng.normal(i_mu, 1.0, (S, T)).astype(np.float32)
    fp = rng.normal(f_mu, f_sd, (S, T)).astype(np.float32)
    dh = rng.standard_normal((S, T, DV)).astype(np.float32)
    return q, k, v, ip, fp, dh


def run(B, NH, q, k, v, ip, fp, dh, dtype):
    S, T, DQK = q.shape
    DV = v.shape[2]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = lambda x, *shape: torch.from_numpy(np.ascontiguousarray(x)).reshape(*shape).cuda()
    qd, kd = dev(q, B, NH, T, DQK).to(tdt), dev(k, B, NH, T, DQK).to(tdt)
    vd = dev(v, B, NH, T, DV).to(tdt)
    ipd, fpd, dhd = dev(ip, B, NH, T), dev(fp, B, NH, T), dev(dh, B, NH, T, DV)
    outs = [torch.full_like(qd, 9.0, dtype=torch.float32), torch.full_like(kd, 9.0, dtype=torch.float32),
            torch.full_like(vd, 9.0, dtype=torch.float32), torch.full_like(ipd, 9.0), torch.full_like(fpd, 9.0)]
    ws = torch.empty(_mb().mlstm_parallel_bwd_workspace_bytes(B, NH, T, DV), dtype=torch.uint8, device="cuda")
    _mb().mlstm_parallel_bwd(qd, kd, vd, ipd, fpd, dhd, *outs, ws)
    torch.cuda.synchronize()
    return [o.cpu().numpy().astype(np.float64).reshape(S, T, -1) for o in outs]


def compare(got, ref, tol, label, q, k, fp, term_scales=None):
    names = ["dq", "dk", "dv", "di", "df"]
    errs = []
    sc = gate_scales(q, k, fp, ref)
    for n, g, r in zip(names, got, ref):
        assert np.isfinite(g).all(), n
        if n in ("dq", "dk", "dv"):
            # per token row; a row that is zero in exact arithmetic (such as dq of a first token whose
            # denominator is above the floor) is held to 1e-3 of the tensor's largest row
            er = row_errs(g, r, r.shape[2], floor=1e-3)
            if term_scales is not None:
                ts = np.asarray(term_scales[names.index(n)]).reshape(g.shape)
                et = (np.abs(g - r) / np.where(ts > 0, ts, 1.0)).reshape(er.size, -1).max(axis=1)
                er = np.minimum(er, et)
            e = float(er.max()) if er.size else 0.0
            print(f"{label} {n}: {er.size} rows, median {np.median(er):.2e}, max {e:.2e}")
        else:
            S, T = r.shape[0], r.shape[1]
            scale = sc[0] if n == "di" else sc[1]
            d = np.abs(g.reshape(S, T) - r.reshape(S, T))
            e = float((d / np.where(scale > 0, scale, 1.0)).max()) if d.size else 0.0
        errs.append(e)
    print(label + " " + " ".join(f"{n} {e:.2e}" for n, e in zip(names, errs)))
    assert max(errs) <= tol, dict(zip(names, errs))


SMALL = [
    # (B, NH, T, DQK, DV, dist)
    (1, 2, 40, 16, 16, "standard"),       # ragged: 40 = 2 x 16 + 8
    (2, 1, 64, 32, 48, "short_memory"),
    (1, 1, 17, 16, 32, "floor_active"),
    (1, 1, 1, 16, 16, "standard"),        # one token
    (1, 2, 100, 64, 128, "standard"),     # DQK, DV multiples of 64: the MFMA passes
    (2, 1, 77, 64, 64, "short_memory"),   # MFMA passes, ragged T
    (1, 1, 50, 128, 192, "floor_active"), # MFMA passes, three 16-column tiles per wave
    (1, 1, 40, 256, 512, "standard"),     # the xLSTM-7B head in fp32: MFMA passes
]
DIST = {"standard": {}, "short_memory": dict(f_mu=-1.0, f_sd=2.0), "floor_active": dict(i_mu=-6.0)}


@pytest.mark.parametrize("case", SMALL, ids=lambda c: f"B{c[0]}NH{c[1]}T{c[2]}d{c[3]}x{c[4]}-{c[5]}")
def test_parallel_bwd_fp32_matches_oracle(case):
    B, NH, T, DQK, DV, dist = case
    q, k, v, ip, fp, dh = draw(300 + SMALL.index(case), B, NH, T, DQK, DV, "f32", **DIST[dist])
    got = run(B, NH, q, k, v, ip, fp, dh, "f32")
    ref = G.recurrent_grad(q, k, v, ip, fp, dh)
    ref = [r.reshape(r.shape[0], r.shape[1], -1) for r in ref]
    compare(got, ref, TOL_BWD_F32, str(case), q, k, fp, G.parallel_grad_scales(q, k, v, ip, fp, dh))


@pytest.mark.parametrize("T", [128, 300])
def test_parallel_bwd_bf16_xlstm_head(T):
    B, NH, DQK, DV = 1, 2, 256, 512
    q, k, v, ip, fp, dh = draw(310 + T, B, NH, T, DQK, DV, "bf16")
    got = run(B, NH, q, k, v, ip, fp, dh, "bf16")
    ref = G.parallel_grad(q, k, v, ip, fp, dh)
    ref = [r.reshape(r.shape[0], r.shape[1], -1) for r in ref]
    compare(got, ref, TOL_BF16, f"7B head T{T}", q, k, fp)


@pytest.mark.parametrize("dtype,DQK,DV", [("f32", 64, 128), ("bf16", 256, 512)])
def test_autograd_cell_gradients(dtype, DQK, DV):
    """Gradients through ``mlstm_cell`` (forward on the chunkwise kernels; backward on the parallel-form
    kernels for fp32 64 x 128 heads, on the chunkwise backward for the bf16 xLSTM-7B head) for a loss
    sum(h * w), against the fp64 gradient oracle with dh = w (for bf16 the forward output h, and so
    dh = w, enter in bf16, and the gradients return in bf16: the bf16 bar)."""
    from paper_2503_13427_amd.cell import mlstm_cell
    B, NH, T = 1, 2, 90
    q, k, v, ip, fp, w = draw(330, B, NH, T, DQK, DV, dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = lambda x, dt, *shape: torch.from_numpy(np.ascontiguousarray(x)).reshape(*shape).cuda().to(dt).requires_grad_(True)
    tq, tk, tv = dev(q, tdt, B, NH, T, DQK), dev(k, tdt, B, NH, T, DQK), dev(v, tdt, B, NH, T, DV)
    tip, tfp = dev(ip, torch.float32, B, NH, T), dev(fp, torch.float32, B, NH, T)
    h = mlstm_cell(tq, tk, tv, tip, tfp, L=64)
    assert h.dtype == tdt
    (h * torch.from_numpy(w).reshape(B, NH, T, DV).cuda().to(tdt)).sum().backward()
    torch.cuda.synchronize()
    got = [t.grad.float().cpu().numpy().astype(np.float64).reshape(B * NH, T, -1) for t in (tq, tk, tv, tip, tfp)]
    wr = w if dtype == "f32" else bf16_bits_to_f32(f32_to_bf16_bits(w))
    ref = G.recurrent_grad(q, k, v, ip, fp, wr)
    ref = [r.reshape(r.shape[0], r.shape[1], -1) for r in ref]
    compare(got, ref, TOL_BWD_F32 if dtype == "f32" else TOL_BF16, f"autograd cell {dtype}", q, k, fp,
            G.parallel_grad_scales(q, k, v, ip, fp, wr))


def test_parallel_bwd_full_size_sampled_heads():
    """The benchmarked backward shape (8 heads of 256 x 512, T = 2048, bf16) in one call; two
    heads are checked against the closed-form oracle run on those heads alone."""
    B, NH, T, DQK, DV = 1, 8, 2048, 256, 512
    q, k, v, ip, fp, dh = draw(330, B, NH, T, DQK, DV, "bf16")
    got = run(B, NH, q, k, v, ip, fp, dh, "bf16")
    for h in (0, 5):
        sl = slice(h, h + 1)
        ref = G.parallel_grad(q[sl], k[sl], v[sl], ip[sl], fp[sl], dh[sl])
        ref = [r.reshape(1, T, -1) for r in ref]
        compare([g[sl] for g in got], ref, TOL_BF16, f"T{T} head {h}", q[sl], k[sl], fp[sl])
    assert all(np.isfinite(g).all() for g in got)
