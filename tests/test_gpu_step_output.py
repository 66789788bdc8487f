"""mlstm_step_output: a decode step that returns the cell's hidden-state output
h = sigmoid(o~) * (Norm(h~) w + b) (Eq. 6 with Eq. 9) against the fp64 oracle: the recurrent step
(Eqs. 2-5) followed by ``output_gate_norm``.

Many sequences take the fused launch (the norm in the step kernel's epilogue, from the unrounded h~);
few sequences take the column-split step and the output pass in place.  Per-row bar: 2e-2 for bf16,
1e-5 for fp32.  The state the call leaves is bit-identical to mlstm_step's.
"""
import numpy as np
import pytest
import torch

from oracle import coracle, mlstm_ref
from tests.helpers import TOL_BF16, TOL_F32, dev, host_f64, row_err, state_errs

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def _bf16(x):
    from paper_2503_13427_amd.inputs import f32_to_bf16_bits
    return f32_to_bf16_bits(x.astype(np.float32))


def _widen(x):
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


CASES = [
    # (B, NH, DQK, DV, dtype, norm, affine, steps)
    (64, 8, 256, 512, "bf16", "layer", True, 3),    # 512 sequences: fused epilogue
    (40, 8, 256, 512, "bf16", "rms", False, 2),     # 320 sequences: fused, RMSNorm, no affine
    (1, 8, 256, 512, "bf16", "layer", True, 3),     # 8 sequences: column split + output pass
    (300, 1, 64, 128, "f32", "layer", True, 3),     # fp32, fused
    (2, 2, 16, 32, "f32", "rms", True, 2),          # fp32, few sequences
    (1, 4, 32, 2048, "f32", "layer", False, 2),     # the widest row the output takes
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}NH{}d{}x{}-{}-{}-{}".format(*c[:7]))
def test_step_output_matches_oracle(case):
    B, NH, DQK, DV, dt, norm, affine, steps = case
    S = B * NH
    rng = np.random.default_rng(400 + CASES.index(case))
    mk = (lambda x: _bf16(x)) if dt == "bf16" else (lambda x: x.astype(np.float32))
    q = mk(rng.standard_normal((S, steps, DQK)))
    k = mk(rng.standard_normal((S, steps, DQK)) / (1.0 if dt == "bf16" else np.sqrt(DQK)))
    v = mk(rng.standard_normal((S, steps, DV)))
    o = mk(rng.normal(0, 2, (S, steps, DV)))
    ip = rng.standard_normal((S, steps)).astype(np.float32)
    fp = rng.normal(3, 1, (S, steps)).astype(np.float32)
    fp[0, 1] = -np.inf                                        # a document border on one sequence
    C0 = rng.normal(0, 0.1, (S, DQK, DV)).astype(np.float32)
    n0 = np.abs(rng.standard_normal((S, DQK))).astype(np.float32)
    m0 = rng.standard_normal(S).astype(np.float32)
    w = rng.normal(1, 0.2, (NH, DV)).astype(np.float32) if affine else None
    b = rng.normal(0, 0.2, (NH, DV)).astype(np.float32) if affine else None
    eps = 1e-6 if dt == "bf16" else 1e-5

    mb = _mb()
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    C, n, m = dev(C0).reshape(B, NH, DQK, DV), dev(n0).reshape(B, NH, DQK), dev(m0).reshape(B, NH)
    C2, n2, m2 = C.clone(), n.clone(), m.clone()                # mlstm_step on a copy: same state
    wt, bt = (dev(w) if affine else None), (dev(b) if affine else None)
    hs = []
    for t in range(steps):
        cp = lambda a: dev(np.ascontiguousarray(a[:, t])).reshape(B, NH, -1)
        qt, kt, vt, ot = cp(q), cp(k), cp(v), cp(o)
        it = dev(np.ascontiguousarray(ip[:, t])).reshape(B, NH)
        ft = dev(np.ascontiguousarray(fp[:, t])).reshape(B, NH)
        h = torch.empty(B, NH, DV, dtype=tdt, device="cuda")
        mb.mlstm_step_output(qt, kt, vt, it, ft, C, n, m, ot, wt, bt, eps, norm, h, C, n, m)
        h2 = torch.empty_like(h)
        mb.mlstm_step(qt, kt, vt, it, ft, C2, n2, m2, h2, C2, n2, m2)
        hs.append(h)
    torch.cuda.synchronize()
    for a, c in ((C, C2), (n, n2), (m, m2)):
        assert torch.equal(a, c), "the state differs from mlstm_step's"
    got = np.stack([host_f64(x).reshape(S, DV) for x in hs], axis=1)           # [S, steps, DV]

    hr, Cr, nr, mr = coracle.recurrent(_widen(q), _widen(k), _widen(v), ip.astype(np.float64), fp.astype(np.float64),
                                       C0.astype(np.float64), n0.astype(np.float64), m0.astype(np.float64))
    ref = mlstm_ref.output_gate_norm(hr.reshape(B, NH, steps, DV), _widen(o).reshape(B, NH, steps, DV),
                                     None if w is None else w.astype(np.float64),
                                     None if b is None else b.astype(np.float64), eps=eps, norm=norm)
    tol = TOL_BF16 if dt == "bf16" else TOL_F32
    e = row_err(got, ref.reshape(S, steps, DV), DV, f"{case} h")
    eC, en, em = state_errs(host_f64(C).reshape(S, DQK, DV), host_f64(n).reshape(S, DQK), host_f64(m).reshape(S),
                            Cr, nr, mr)
    assert np.isfinite(got).all()
    assert e <= tol and max(eC, en, em) <= tol, (e, eC, en, em)


def test_fused_and_split_paths_are_both_exercised():
    from paper_2503_13427_amd import binding as mb  # noqa: F401  (library loaded)
    import ctypes
    lib = ctypes.CDLL(mb.LIB_PATH)
    f = lib._ZN5mlstm17step_output_fusedEiiii
    f.restype = ctypes.c_bool
    assert f(64, 8, 256, 512) and f(300, 1, 64, 128)
    assert not f(1, 8, 256, 512) and not f(1, 4, 32, 2048)
