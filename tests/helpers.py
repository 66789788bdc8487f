"""Shared test helpers: device upload, the error metric, oracle runs on workloads.

Error metric (the reading adopted for "max relative error"), per row: an
output row is the vector one (batch, head, step) produces (an h row of DV
values), or one d-row of the matrix state C (DV values).  Each row's error is
max|x - x_ref| / max|x_ref| over that row, and the bar applies to the largest
row error, so every row is held to its own magnitude (a row of small values
cannot hide under a large one elsewhere in its sequence).  A row whose
reference is exactly zero is held to max|x|.  The max state m is compared
absolutely, |dm| <= tol * max(1, |m_ref|), and the matrix state is compared
scale-free, C * exp(m - m_ref) against C_ref.  The normaliser n of a sequence
is one row.
"""
from __future__ import annotations

import numpy as np
import torch

from paper_2503_13427_amd.inputs import Inputs, bf16_bits_to_f32

TOL_BF16 = 2e-2
TOL_F32 = 1e-5


def dev(x: np.ndarray, device="cuda") -> torch.Tensor:
    """Host array -> device tensor; uint16 arrays are bf16 bit patterns."""
    if x is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(x))
    if x.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.to(device)


def host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_err(x: np.ndarray, ref: np.ndarray, slice_dims: int) -> float:
    """max over the leading ``slice_dims`` axes of max|x-ref| / max|ref| within each slice."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    lead = int(np.prod(ref.shape[:slice_dims]))
    xs = x.reshape(lead, -1)
    rs = ref.reshape(lead, -1)
    num = np.abs(xs - rs).max(axis=1)
    den = np.abs(rs).max(axis=1)
    den = np.where(den == 0, 1.0, den)
    return float((num / den).max()) if lead else 0.0


def row_errs(x: np.ndarray, ref: np.ndarray, row_len: int, floor: float = 0.0) -> np.ndarray:
    """Per-row errors over rows of ``row_len`` consecutive values: max|x-ref| / max|ref| per row,
    max|x| for a row whose reference is all zero.  ``floor`` > 0 (gradient checks only) holds a
    row to at least that fraction of the largest row of its tensor: a gradient row that is zero
    in exact arithmetic has no relative error to speak of."""
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    if ref.size == 0:
        return np.zeros(0)
    xs = x.reshape(-1, row_len)
    rs = ref.reshape(-1, row_len)
    num = np.abs(xs - rs).max(axis=1)
    den = np.maximum(np.abs(rs).max(axis=1), floor * np.abs(rs).max())
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), num)


def row_err(x: np.ndarray, ref: np.ndarray, row_len: int, label: str = None, floor: float = 0.0) -> float:
    """Largest per-row error (see ``row_errs``); with a label, prints the row count, median,
    99.9th percentile and maximum."""
    e = row_errs(x, ref, row_len, floor)
    if not e.size:
        return 0.0
    if label is not None:
        print(f"{label}: {e.size} rows of {row_len}, median {np.median(e):.2e}, "
              f"p99.9 {np.quantile(e, 0.999):.2e}, max {e.max():.2e}")
    return float(e.max())


def m_err(m: np.ndarray, m_ref: np.ndarray) -> float:
    m = np.asarray(m, np.float64).ravel()
    r = np.asarray(m_ref, np.float64).ravel()
    return float((np.abs(m - r) / np.maximum(1.0, np.abs(r))).max()) if r.size else 0.0


def state_errs(C, n, m, C_ref, n_ref, m_ref, label=None):
    """Errors of (C, n, m) against the oracle, C and n compared scale-free: C per d-row (DV
    values), n per sequence."""
    S = C_ref.shape[0]
    DV = C_ref.shape[-1]
    sc = np.exp(np.asarray(m, np.float64).reshape(S) - np.asarray(m_ref, np.float64).reshape(S))
    eC = row_err(np.asarray(C, np.float64).reshape(S, -1) * sc[:, None], C_ref.reshape(S, -1), DV,
                 None if label is None else f"{label} C")
    en = row_err(np.asarray(n, np.float64).reshape(S, -1) * sc[:, None], n_ref.reshape(S, -1), n_ref.reshape(S, -1).shape[1])
    return eC, en, m_err(m, m_ref)


def subset(inp: Inputs, heads) -> Inputs:
    """The inputs of the given global heads (b * NH + h), shaped [1, len(heads), ...]."""
    sel = np.asarray(heads, dtype=np.int64)
    S = inp.B * inp.NH
    pick = lambda a: None if a is None else a.reshape(S, *a.shape[2:])[sel][None]
    return Inputs(dtype=inp.dtype, q=pick(inp.q), k=pick(inp.k), v=pick(inp.v), ipre=pick(inp.ipre),
                  fpre=pick(inp.fpre), C0=pick(inp.C0), n0=pick(inp.n0), m0=pick(inp.m0), heads=sel)


def upload_prefill(inp: Inputs, device="cuda"):
    return dict(q=dev(inp.q, device), k=dev(inp.k, device), v=dev(inp.v, device), ipre=dev(inp.ipre, device),
                fpre=dev(inp.fpre, device), C0=dev(inp.C0, device), n0=dev(inp.n0, device),
                m0=dev(inp.m0, device))


def alloc_prefill_outputs(inp: Inputs, device="cuda"):
    B, NH, T, DQK, DV = inp.B, inp.NH, inp.T, inp.DQK, inp.DV
    dt = torch.bfloat16 if inp.dtype == "bf16" else torch.float32
    return dict(h=torch.empty(B, NH, T, DV, dtype=dt, device=device),
                CT=torch.empty(B, NH, DQK, DV, dtype=torch.float32, device=device),
                nT=torch.empty(B, NH, DQK, dtype=torch.float32, device=device),
                mT=torch.empty(B, NH, dtype=torch.float32, device=device))


def gate_scales(q, k, fp, ref):
    """Magnitudes of the summands of the gate gradients, [S, T] each, from the reference gradients
    ref = (dq, dk, ...): di~_t = k_t . dk_t sums k_td dk_td; dlogsig(f~_t) sums q_t'd dq_t'd - k_t'd dk_t'd
    over t' >= t, times sigmoid(-f~_t) for df~.  A gate gradient's error is measured against these."""
    S, T = ref[0].shape[0], ref[0].shape[1]
    q = np.asarray(q, np.float64).reshape(S, T, -1)
    k = np.asarray(k, np.float64).reshape(S, T, -1)
    aq = np.abs(q * ref[0].reshape(S, T, -1)).sum(axis=2)
    ak = np.abs(k * ref[1].reshape(S, T, -1)).sum(axis=2)
    tail = np.cumsum((aq + ak)[:, ::-1], axis=1)[:, ::-1]
    sig = 1.0 / (1.0 + np.exp(np.asarray(fp, np.float64).reshape(S, T)))
    return ak, sig * tail
