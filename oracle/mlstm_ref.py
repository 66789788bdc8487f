"""NumPy fp64 forms of the mLSTM cell.

TEST INFRASTRUCTURE ONLY: the oracle side of the parity tests.  Only
``tests/``, the smoke check and the benchmark's CPU-baseline leg may import
this module; it shares no code with the HIP library and imports nothing from
it.

All functions take fp64 arrays with a leading sequence axis S (= B * NH,
every (batch, head) pair is an independent cell):

    q, k   [S, T, DQK]      v [S, T, DV]      ipre, fpre [S, T]
    C0     [S, DQK, DV]     n0 [S, DQK]       m0 [S]     (all None: zero state, m0 = 0)

and return ``h [S, T, DV]`` (the h~ of Eq. 5) and the final state
``(C [S, DQK, DV], n [S, DQK], m [S])``.

Forms, each written from the paper's statement of the cell (Sec. 2):

* ``recurrent``              Eqs. 2-5, 7-8, step by step (the definition).
* ``recurrent_unstabilized`` the same recurrence without the max state:
                             C~_t = e^{logsig f~_t} C~_{t-1} + e^{i~_t} k v^T, and the
                             floor exp(-m_t) becomes 1 in these unscaled units.
* ``parallel_quadratic``     the fully parallel form H = mLSTMCell(X) (Eq. 10):
                             a causal, gate-weighted T x T matrix.
* ``chunkwise``              the chunkwise-parallel form, following the sub-steps
                             of the FLOP count in App. D.1 (chunkwise gates, gates and
                             max state, inter-chunk numerator and denominator, gate
                             matrix, gated logits, intra-chunk numerator and
                             denominator, output combination), for any chunk size;
                             the last chunk may be shorter.
* ``output_gate_norm``       the hidden-state output h = o * Norm(h~) with o = sigmoid(o~)
                             (Eq. 6 with Eq. 9), Norm the headwise LayerNorm or RMSNorm that
                             Sec. 2 allows; it takes [B, NH, T, DV] rows, not the S axis.
* ``mlstm_layer``            the multi-head mLSTM layer (Eq. 11): dense projections of x to
                             q, k, v, the gate pre-activations (soft-capped, Eq. 13) and o~,
                             one cell per head, the output gate and norm, concatenation and
                             the output projection; it takes x [B, T, d].  With
                             proj_dtype="bf16" the projections q, k, v and o~ are stored in
                             bf16 (``round_bf16``) before the cell, as a bf16 model holds them.
* ``round_bf16``             fp64 -> nearest bf16 value (ties to even), returned as fp64.
* ``gate_preact``            the gate pre-activations of the layer: i~, f~ = softcap(x W + b)
                             per head (Eq. 11 with the soft-cap of Eq. 13), f~ = -inf on
                             document-border tokens (the reset of App. B), head-major [B, NH, T].
"""
from __future__ import annotations

import numpy as np


def logsigmoid(x):
    """log(sigmoid(x)) = min(x, 0) - log1p(exp(-|x|)), exact in value, no overflow."""
    x = np.asarray(x, dtype=np.float64)
    return np.minimum(x, 0.0) - np.log1p(np.exp(-np.abs(x)))


def _init_state(S, DQK, DV, C0, n0, m0):
    if C0 is None:
        assert n0 is None and m0 is None
        return np.zeros((S, DQK, DV)), np.zeros((S, DQK)), np.zeros((S,))
    return (np.array(C0, dtype=np.float64, copy=True), np.array(n0, dtype=np.float64, copy=True),
            np.array(m0, dtype=np.float64, copy=True))


def recurrent(q, k, v, ipre, fpre, C0=None, n0=None, m0=None):
    """Recurrent form, Eqs. 2-5 with Eqs. 7-8 (Sec. 2, generation mode)."""
    S, T, DQK = q.shape
    DV = v.shape[2]
    C, n, m = _init_state(S, DQK, DV, C0, n0, m0)
    h = np.empty((S, T, DV))
    scale = 1.0 / np.sqrt(DQK)
    for t in range(T):
        a = logsigmoid(fpre[:, t])
        it = ipre[:, t]
        m_new = np.maximum(a + m, it)                      # Eq. 2
        f = np.exp(a + m - m_new)                          # Eq. 7
        i = np.exp(it - m_new)                             # Eq. 8
        kt, vt = k[:, t, :], v[:, t, :]
        C = f[:, None, None] * C + i[:, None, None] * kt[:, :, None] * vt[:, None, :]   # Eq. 3
        n = f[:, None] * n + i[:, None] * kt               # Eq. 4
        m = m_new
        qh = q[:, t, :] * scale
        num = np.einsum("sdv,sd->sv", C, qh)               # C_t^T q^_t
        den = np.maximum(np.abs(np.einsum("sd,sd->s", n, qh)), np.exp(-m))
        h[:, t, :] = num / den[:, None]                    # Eq. 5
    return h, C, n, m


def recurrent_unstabilized(q, k, v, ipre, fpre, C0=None, n0=None, m0=None):
    """The recurrence in unscaled units (no max state).

    With C~ = e^{m} C and n~ = e^{m} n, Eqs. 3-5 become
    C~_t = e^{logsig f~_t} C~_{t-1} + e^{i~_t} k_t v_t^T (same for n~), and the
    floor max(|n^T q^|, e^{-m}) turns into max(|n~^T q^|, 1).  Returns h and the
    unscaled final (C~, n~).  Only for small inputs: e^{i~} is not bounded.
    """
    S, T, DQK = q.shape
    DV = v.shape[2]
    C, n, m = _init_state(S, DQK, DV, C0, n0, m0)
    Cb = np.exp(m)[:, None, None] * C
    nb = np.exp(m)[:, None] * n
    h = np.empty((S, T, DV))
    scale = 1.0 / np.sqrt(DQK)
    for t in range(T):
        fa = np.exp(logsigmoid(fpre[:, t]))
        ia = np.exp(ipre[:, t])
        kt, vt = k[:, t, :], v[:, t, :]
        Cb = fa[:, None, None] * Cb + ia[:, None, None] * kt[:, :, None] * vt[:, None, :]
        nb = fa[:, None] * nb + ia[:, None] * kt
        qh = q[:, t, :] * scale
        num = np.einsum("sdv,sd->sv", Cb, qh)
        den = np.maximum(np.abs(np.einsum("sd,sd->s", nb, qh)), 1.0)
        h[:, t, :] = num / den[:, None]
    return h, Cb, nb


def parallel_quadratic(q, k, v, ipre, fpre, C0=None, n0=None, m0=None):
    """Fully parallel form (Eq. 10): every output row is a gate-weighted sum over all
    earlier tokens plus the decayed initial state.

    Token j reaches step t >= j with log weight i~_j + sum_{j<s<=t} logsig(f~_s) and the
    initial state with log weight m_0 + sum_{s<=t} logsig(f~_s).  The row maximum
    of these log weights is the max state m_t, which stabilises the row and sets the
    floor exp(-m_t).
    """
    S, T, DQK = q.shape
    DV = v.shape[2]
    C, n, m = _init_state(S, DQK, DV, C0, n0, m0)
    h = np.empty((S, T, DV))
    CT = np.empty((S, DQK, DV))
    nT = np.empty((S, DQK))
    mT = np.empty((S,))
    scale = 1.0 / np.sqrt(DQK)
    for s in range(S):
        a = logsigmoid(fpre[s])
        # seg[t, j] = sum_{j < s' <= t} logsig(f~_s'), summed directly (not as a difference of
        # prefix sums) so that a forget gate of exactly zero (logsig = -inf) stays exact.
        seg = np.full((T, T), -np.inf)
        for j in range(T):
            seg[j, j] = 0.0
            if j + 1 < T:
                seg[j + 1:, j] = np.cumsum(a[j + 1:])
        logD = ipre[s][None, :] + seg
        log0 = m[s] + np.cumsum(a)                         # initial-state weight per row
        mrow = np.maximum(log0, logD.max(axis=1)) if T else log0
        D = np.exp(logD - mrow[:, None])
        w0 = np.exp(log0 - mrow)
        Qh = q[s] * scale
        Sm = (Qh @ k[s].T) * D
        num = Sm @ v[s] + w0[:, None] * (Qh @ C[s])
        den = Sm.sum(axis=1) + w0 * (Qh @ n[s])
        h[s] = num / np.maximum(np.abs(den), np.exp(-mrow))[:, None]
        if T:
            mT[s] = mrow[-1]
            wl = D[-1]                                     # last row: weights of every token at T
            CT[s] = w0[-1] * C[s] + (k[s] * wl[:, None]).T @ v[s]
            nT[s] = w0[-1] * n[s] + k[s].T @ wl
        else:
            mT[s], CT[s], nT[s] = m[s], C[s], n[s]
    return h, CT, nT, mT


def chunkwise(q, k, v, ipre, fpre, C0=None, n0=None, m0=None, L=64):
    """Chunkwise-parallel form with chunk size L, in the sub-steps of App. D.1.

    Within chunk k (positions tau = 1..Lc) with previous state (C, n, m_prev):
      chunkwise gates   b_tau = sum_{s<=tau} logsig(f~_s),  g = b_Lc
      max state         m_tau = max(b_tau + m_prev, max_{sig<=tau}(i~_sig + b_tau - b_sig))
                        m_k   = max(g + m_prev, max_tau(i~_tau + g - b_tau))
      gate matrix       D[tau, sig] = exp(i~_sig + b_tau - b_sig - m_tau),  sig <= tau
      gated logits      S = (Q^ K^T) * D
      numerator         e^{b_tau + m_prev - m_tau} Q^ C  +  S V
      denominator       e^{b_tau + m_prev - m_tau} Q^ n  +  rowsum(S)
      output            h_tau = numerator / max(|denominator|, e^{-m_tau})
      state update      C <- e^{g + m_prev - m_k} C + (w * K)^T V,  w_tau = e^{i~_tau + g - b_tau - m_k}
                        n <- e^{g + m_prev - m_k} n + K^T w,        m_prev <- m_k
    """
    S, T, DQK = q.shape
    DV = v.shape[2]
    C, n, m = _init_state(S, DQK, DV, C0, n0, m0)
    h = np.empty((S, T, DV))
    scale = 1.0 / np.sqrt(DQK)
    for s in range(S):
        Cs, ns, mp = C[s].copy(), n[s].copy(), m[s]
        for t0 in range(0, T, L):
            t1 = min(T, t0 + L)
            a = logsigmoid(fpre[s, t0:t1])
            it = ipre[s, t0:t1]
            b = np.cumsum(a)
            g = b[-1]
            Lc = t1 - t0
            tri = np.tril(np.ones((Lc, Lc), dtype=bool))
            logD = np.where(tri, it[None, :] + b[:, None] - b[None, :], -np.inf)
            m_tau = np.maximum(b + mp, logD.max(axis=1))
            D = np.exp(logD - m_tau[:, None])
            Qh = q[s, t0:t1] * scale
            K, V = k[s, t0:t1], v[s, t0:t1]
            Sm = (Qh @ K.T) * D
            inter = np.exp(b + mp - m_tau)
            num = inter[:, None] * (Qh @ Cs) + Sm @ V
            den = inter * (Qh @ ns) + Sm.sum(axis=1)
            h[s, t0:t1] = num / np.maximum(np.abs(den), np.exp(-m_tau))[:, None]
            m_k = max(g + mp, np.max(it + g - b))
            w = np.exp(it + g - b - m_k)
            decay = np.exp(g + mp - m_k)
            Cs = decay * Cs + (K * w[:, None]).T @ V
            ns = decay * ns + K.T @ w
            mp = m_k
        C[s], n[s], m[s] = Cs, ns, mp
    return h, C, n, m


def sigmoid(x):
    """1 / (1 + exp(-x)), written so that neither branch overflows."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def output_gate_norm(h_tilde, o_pre, weight=None, bias=None, eps=1e-6, norm="layer"):
    """Hidden-state output h = o * Norm(h~), o = sigmoid(o~) (Eq. 6 with Eq. 9).

    Norm acts on each row of DV values, one head at one step (the headwise norm of Sec. 2 and
    of the 7B model's cell), then scales by ``weight`` and shifts by ``bias`` (both [NH, DV],
    None meaning 1 and 0):
      layer: (x - mean(x)) / sqrt(var(x) + eps), var the mean squared deviation;
      rms:   x / sqrt(mean(x^2) + eps).
    h_tilde, o_pre: [B, NH, T, DV].  Returns h [B, NH, T, DV] in fp64.
    """
    x = np.asarray(h_tilde, dtype=np.float64)
    o = np.asarray(o_pre, dtype=np.float64)
    assert x.ndim == 4 and o.shape == x.shape
    if norm == "layer":
        mu = x.mean(axis=-1, keepdims=True)
        y = (x - mu) / np.sqrt(((x - mu) ** 2).mean(axis=-1, keepdims=True) + eps)
    elif norm == "rms":
        y = x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)
    else:
        raise ValueError(norm)
    if weight is not None:
        y = y * np.asarray(weight, dtype=np.float64)[None, :, None, :]
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)[None, :, None, :]
    return sigmoid(o) * y


def soft_cap(x, cap):
    """cap * tanh(x / cap) (Eq. 13); cap = None leaves x unchanged."""
    x = np.asarray(x, dtype=np.float64)
    return x if cap is None else cap * np.tanh(x / cap)


def round_bf16(x):
    """Nearest bf16 value of each element (ties to even), as fp64.  bf16 keeps 8 significant bits
    and fp32's exponent range: a normal |x| in [2^E, 2^(E+1)) has the quantum 2^(E-7), and below
    the smallest normal 2^-126 the quantum stays 2^-133 (subnormals).  Dividing by a power of two
    and multiplying back are exact in fp64, and np.round rounds halves to even.  Overflow past the
    largest bf16 value is not handled (no caller comes near it)."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                       # x = f 2^e, f in [0.5, 1): leading bit 2^(e-1)
    quantum = np.ldexp(1.0, np.maximum(e - 1, -126) - 7)
    return np.round(x / quantum) * quantum


def gate_preact(x, W_gates, gate_bias, cap=15.0, border=None):
    """Gate pre-activations of one layer, head-major.

    x [B, T, d]; W_gates [d, 2 NH]: the input gate column of each head, then the forget gate
    column of each head; gate_bias [2, NH].  i~ = softcap(x w_i + b_i), f~ = softcap(x w_f + b_f)
    (cap None: no cap).  ``border`` [B, T] (bool, optional) marks the first token of a new
    document, whose forget gate is exactly zero: f~ = -inf there.  Returns ipre, fpre [B, NH, T]
    in fp64."""
    x = np.asarray(x, dtype=np.float64)
    W = np.asarray(W_gates, dtype=np.float64)
    NH = W.shape[1] // 2
    b = np.asarray(gate_bias, dtype=np.float64)
    z = x @ W                                                        # [B, T, 2 NH]
    ig = soft_cap(z[..., :NH] + b[0], cap)
    fg = soft_cap(z[..., NH:] + b[1], cap)
    if border is not None:
        fg = np.where(np.asarray(border, dtype=bool)[..., None], -np.inf, fg)
    return np.ascontiguousarray(np.moveaxis(ig, 2, 1)), np.ascontiguousarray(np.moveaxis(fg, 2, 1))


def mlstm_layer(x, W_in, W_proj, gate_bias, norm_weight, NH, DQK, DV, eps=1e-6, cap=15.0,
                C0=None, n0=None, m0=None, proj_dtype=None, border=None):
    """Multi-head mLSTM layer (Eq. 11), x [B, T, d] -> y [B, T, d] and the final cell state.

    W_in [d, NH * (2 DQK + 2 DV + 2)] holds, in column order, the q, k, v projections (head-major:
    the DQK or DV columns of head 0, then head 1, ...), the input and forget gate projections
    (one column per head) and the output gate projection (head-major); gate_bias [2, NH] is added
    to the two gate pre-activations before the soft-cap.  Each head runs the cell of Sec. 2 from
    (C0, n0, m0) ([B * NH, ...], None: zero state), its h~ goes through the output gate and the
    headwise LayerNorm (weight norm_weight [NH, DV]), the heads are concatenated and projected by
    W_proj [NH * DV, d].  proj_dtype="bf16" rounds q, k, v and o~ to bf16 after the projection
    (the gates stay in full precision); None keeps every projection in fp64.  ``border`` [B, T]
    (optional) marks document borders of a packed sequence: the forget gate is zero there
    (``gate_preact``), so each document runs as if from the zero state.
    """
    x = np.asarray(x, dtype=np.float64)
    B, T, d = x.shape
    P = x @ np.asarray(W_in, dtype=np.float64)                      # [B, T, N_in]
    o0 = 0
    def take(width):
        nonlocal o0
        part = P[..., o0:o0 + width]
        o0 += width
        return part
    q = take(NH * DQK).reshape(B, T, NH, DQK)
    k = take(NH * DQK).reshape(B, T, NH, DQK)
    v = take(NH * DV).reshape(B, T, NH, DV)
    o_gates = o0
    take(2 * NH)
    ig, fg = gate_preact(x, np.asarray(W_in, dtype=np.float64)[:, o_gates:o_gates + 2 * NH], gate_bias, cap,
                         border)                                    # [B, NH, T] each
    og = take(NH * DV).reshape(B, T, NH, DV)
    assert o0 == P.shape[-1]
    if proj_dtype == "bf16":
        q, k, v, og = round_bf16(q), round_bf16(k), round_bf16(v), round_bf16(og)
    elif proj_dtype is not None:
        raise ValueError(proj_dtype)
    heads = lambda a: np.ascontiguousarray(np.moveaxis(a, 2, 1))    # [B, T, NH, D] -> [B, NH, T, D]
    S = B * NH
    h, C, n, m = recurrent(heads(q).reshape(S, T, DQK), heads(k).reshape(S, T, DQK), heads(v).reshape(S, T, DV),
                           ig.reshape(S, T), fg.reshape(S, T), C0, n0, m0)
    hy = output_gate_norm(h.reshape(B, NH, T, DV), heads(og), norm_weight, None, eps=eps, norm="layer")
    y = np.moveaxis(hy, 1, 2).reshape(B, T, NH * DV) @ np.asarray(W_proj, dtype=np.float64)
    return y, (C, n, m)
