"""Gradients of the mLSTM cell for the training-mode backward pass, fp64 on the CPU.

TEST INFRASTRUCTURE ONLY: the oracle side of the backward parity tests.  Only ``tests/``, the
smoke check and the benchmark's CPU-baseline leg may import this module; it shares no code with
the HIP library.

Two forms, for q, k [S, T, DQK], v [S, T, DV], ipre, fpre [S, T] and an upstream gradient
dh [S, T, DV] of the outputs h~ (Eq. 5), from the zero initial state (m_0 = 0):

* ``recurrent_grad``  the definition: the cell of Sec. 2 (Eqs. 2-5 with Eqs. 7-8) written step
                      by step in torch fp64, differentiated by autograd.  A library primitive
                      (reverse-mode differentiation) supplies the derivative of that code.
                      ``recurrent_grad_state`` is the same from a given initial state
                      (C0, n0, m0), and also returns the gradients of C0, n0 and m0.
* ``parallel_grad``   the same gradients in closed form over the parallel form (Eq. 10), written
                      out from the chain rule (below), with every exponential taken relative to
                      the row's max state so that each weight is <= 1.

Closed form.  In unscaled units the cell output is h_t = N_t / max(|D_t|, 1) with
N_t = sum_{s<=t} A_ts v_s, D_t = sum_{s<=t} A_ts, A_ts = exp(b_t - b_s + i~_s) (k_s . q^_t),
b the prefix sums of logsig(f~), q^ = q / sqrt(DQK) (the floor exp(-m_t) of Eq. 5 is 1 in these
units).  With the stabiliser m_t of Eq. 2 every quantity is carried scaled by exp(-m_t)
(A~ = A e^{-m_t}, N~, D~, den_t = max(|D~_t|, e^{-m_t})), and the chain rule gives

    dN~_t = dh_t / den_t
    dD~_t = -(dh_t . h_t) / den_t * sign(D~_t)   where |D~_t| > e^{-m_t}, else 0
    G_ts  = (dN~_t . v_s + dD~_t) A~_ts          (the gradient flowing through A_ts times A_ts)
    dq_t  = sum_s (dN~_t . v_s + dD~_t) F~_ts k_s / sqrt(DQK),   F~_ts = exp(b_t - b_s + i~_s - m_t)
    dk_s  = sum_t (dN~_t . v_s + dD~_t) F~_ts q^_t
    dv_s  = sum_t A~_ts dN~_t
    di~_s = sum_t G_ts
    P_t   = sum_s G_ts = dN~_t . N~_t + dD~_t D~_t
    da_j  = sum_{s < j <= t} G_ts = sum_{t >= j} (P_t - di~_t)     (a = logsig f~)
    df~_j = da_j * sigmoid(-f~_j)

The pins in ``tests/test_grad_oracle.py`` tie ``recurrent_grad`` to central finite differences
of the NumPy recurrent form, and ``parallel_grad`` to ``recurrent_grad``.

``parallel_grad_scales`` gives, for the same closed form, the componentwise magnitude of every term
an evaluation of dq, dk, dv sums, the inner dot products included:
    |W|_ts   = (sum_v |dN~_tv v_sv| + sum_v |dh_tv h_tv| / den_t) F~_ts   (second term where |D~_t| > e^{-m_t})
    |A~|_ts  = sum_d |q^_td k_sd| F~_ts
    dq: sum_s |W|_ts |k_sd| / sqrt(DQK),  dk: sum_t |W|_ts |q^_td|,  dv: sum_t |A~|_ts |dN~_tv|.
A gradient element whose terms cancel (W_ts nearly vanishes when h_t is close to v_s) is measured
against these: a relative error of tol in every term is an error of at most tol times the scale.
"""
from __future__ import annotations

import numpy as np
import torch


def _recurrent_torch(q, k, v, ip, fp, C=None, n=None, m=None):
    """Eqs. 2-5, 7-8 step by step from (C, n, m), the zero state (m_0 = 0) when not given,
    differentiable."""
    S, T, DQK = q.shape
    DV = v.shape[2]
    if C is None:
        C = torch.zeros(S, DQK, DV, dtype=torch.float64)
        n = torch.zeros(S, DQK, dtype=torch.float64)
        m = torch.zeros(S, dtype=torch.float64)
    hs = []
    for t in range(T):
        a = torch.nn.functional.logsigmoid(fp[:, t])
        m_new = torch.maximum(a + m, ip[:, t])                         # Eq. 2
        f = torch.exp(a + m - m_new)                                   # Eq. 7
        i = torch.exp(ip[:, t] - m_new)                                # Eq. 8
        C = f[:, None, None] * C + i[:, None, None] * k[:, t, :, None] * v[:, t, None, :]   # Eq. 3
        n = f[:, None] * n + i[:, None] * k[:, t]                      # Eq. 4
        qh = q[:, t] / np.sqrt(DQK)
        num = torch.einsum("sdv,sd->sv", C, qh)
        den = torch.maximum(torch.abs(torch.einsum("sd,sd->s", n, qh)), torch.exp(-m_new))   # Eq. 5
        hs.append(num / den[:, None])
        m = m_new
    return torch.stack(hs, dim=1)


def recurrent_grad(q, k, v, ip, fp, dh):
    """Gradients of sum(h * dh) with respect to q, k, v, ipre, fpre (fp64 numpy arrays)."""
    ts = [torch.tensor(np.asarray(x, dtype=np.float64), requires_grad=True) for x in (q, k, v, ip, fp)]
    h = _recurrent_torch(*ts)
    (h * torch.tensor(np.asarray(dh, dtype=np.float64))).sum().backward()
    return tuple(t.grad.numpy() for t in ts)


def recurrent_grad_state(q, k, v, ip, fp, C0, n0, m0, dh):
    """Gradients of sum(h * dh) with respect to q, k, v, ipre, fpre and the initial state C0 [S, DQK, DV],
    n0 [S, DQK], m0 [S] (fp64 numpy arrays).  A forget gate of zero (f~ = -inf) restarts the state; its
    own f~ gradient is zero (sigmoid has zero slope there)."""
    xs = (q, k, v, ip, fp, C0, n0, m0)
    ts = [torch.tensor(np.asarray(x, dtype=np.float64), requires_grad=True) for x in xs]
    h = _recurrent_torch(*ts)
    (h * torch.tensor(np.asarray(dh, dtype=np.float64))).sum().backward()
    out = [t.grad.numpy() for t in ts]
    out[4] = np.where(np.isneginf(np.asarray(fp)), 0.0, out[4])
    return tuple(out)


def _logsigmoid(x):
    return np.minimum(x, 0.0) - np.log1p(np.exp(-np.abs(x)))


def parallel_grad(q, k, v, ip, fp, dh):
    """The closed form of the module docstring over the parallel form, per sequence."""
    q, k, v, ip, fp, dh = (np.asarray(x, dtype=np.float64) for x in (q, k, v, ip, fp, dh))
    S, T, DQK = q.shape
    out = [np.zeros_like(x) for x in (q, k, v, ip, fp)]
    tri = np.tril(np.ones((T, T), dtype=bool))
    for s in range(S):
        b = np.cumsum(_logsigmoid(fp[s]))
        logF = np.where(tri, b[:, None] - b[None, :] + ip[s][None, :], -np.inf)   # log of F_ts e^{m_t}
        m = np.maximum(np.maximum.accumulate(ip[s] - b) + b, b)                   # Eq. 2 from m_0 = 0
        Ft = np.exp(logF - m[:, None])                                            # F~_ts <= 1
        qh = q[s] / np.sqrt(DQK)
        Sqk = qh @ k[s].T                                                         # k_s . q^_t
        At = Ft * Sqk                                                             # A~_ts
        Nt = At @ v[s]
        Dt = At.sum(axis=1)
        den = np.maximum(np.abs(Dt), np.exp(-m))
        h = Nt / den[:, None]
        dN = dh[s] / den[:, None]
        dD = np.where(np.abs(Dt) > np.exp(-m), -(dh[s] * h).sum(axis=1) / den * np.sign(Dt), 0.0)
        W = (dN @ v[s].T + dD[:, None]) * Ft                                      # (dN~_t . v_s + dD~_t) F~_ts
        out[0][s] = (W @ k[s]) / np.sqrt(DQK)
        out[1][s] = W.T @ qh
        out[2][s] = At.T @ dN
        G = W * Sqk
        di = G.sum(axis=0)
        P = (dN * Nt).sum(axis=1) + dD * Dt
        da = np.cumsum((P - di)[::-1])[::-1]
        out[3][s] = di
        out[4][s] = da / (1.0 + np.exp(fp[s]))                                    # sigmoid(-f~)
    return tuple(out)


def parallel_grad_scales(q, k, v, ip, fp, dh):
    """Componentwise term magnitudes of dq, dk, dv in the closed form of ``parallel_grad`` (zero
    initial state; see the module docstring): arrays of the shapes of q, k, v."""
    q, k, v, ip, fp, dh = (np.asarray(x, dtype=np.float64) for x in (q, k, v, ip, fp, dh))
    S, T, DQK = q.shape
    out = [np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)]
    tri = np.tril(np.ones((T, T), dtype=bool))
    for s in range(S):
        b = np.cumsum(_logsigmoid(fp[s]))
        logF = np.where(tri, b[:, None] - b[None, :] + ip[s][None, :], -np.inf)
        m = np.maximum(np.maximum.accumulate(ip[s] - b) + b, b)
        Ft = np.exp(logF - m[:, None])
        qh = q[s] / np.sqrt(DQK)
        At = Ft * (qh @ k[s].T)
        Nt = At @ v[s]
        Dt = At.sum(axis=1)
        den = np.maximum(np.abs(Dt), np.exp(-m))
        h = Nt / den[:, None]
        dN = dh[s] / den[:, None]
        act = np.abs(Dt) > np.exp(-m)
        dDa = np.where(act, (np.abs(dh[s]) * np.abs(h)).sum(axis=1) / den, 0.0)
        Wa = (np.abs(dN) @ np.abs(v[s]).T + dDa[:, None]) * Ft
        Aa = Ft * (np.abs(qh) @ np.abs(k[s]).T)
        out[0][s] = (Wa @ np.abs(k[s])) / np.sqrt(DQK)
        out[1][s] = Wa.T @ np.abs(qh)
        out[2][s] = Aa.T @ np.abs(dN)
    return tuple(out)
