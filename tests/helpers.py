"""Shared test helpers: device upload, the error metric, oracle runs on workloads.

Error metric (the reading adopted for "max relative error"): for an output
tensor, take each (batch, head) slice, compute max|x - x_ref| / max|x_ref|
over the slice, and report the maximum over slices.  The max state m is
compared absolutely, |dm| <= tol * max(1, |m_ref|), and the matrix state is
compared scale-free, C * exp(m - m_ref) against C_ref.
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


def m_err(m: np.ndarray, m_ref: np.ndarray) -> float:
    m = np.asarray(m, np.float64).ravel()
    r = np.asarray(m_ref, np.float64).ravel()
    return float((np.abs(m - r) / np.maximum(1.0, np.abs(r))).max()) if r.size else 0.0


def state_errs(C, n, m, C_ref, n_ref, m_ref):
    """Errors of (C, n, m) against the oracle, C and n compared scale-free."""
    S = C_ref.shape[0]
    sc = np.exp(np.asarray(m, np.float64).reshape(S) - np.asarray(m_ref, np.float64).reshape(S))
    eC = rel_err(np.asarray(C, np.float64).reshape(S, -1) * sc[:, None], C_ref.reshape(S, -1), 1)
    en = rel_err(np.asarray(n, np.float64).reshape(S, -1) * sc[:, None], n_ref.reshape(S, -1), 1)
    return eC, en, m_err(m, m_ref)


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
