"""Seeded synthetic inputs for the mLSTM cell.

This module only draws random numbers and rounds them to the storage dtypes.
It holds none of the cell's arithmetic, so both the HIP path and the CPU
oracle can consume the same arrays.

Stream layout.  Every tensor of every (batch, head) sequence comes from its
own PCG64 stream, keyed by ``SeedSequence([seed, workload_id, head, tensor])``
where ``head = b * NH + h``.  Consequences:

* any subset of heads can be regenerated without drawing the others (the
  full-size parity tests check sampled heads against the oracle);
* a shorter sequence is a prefix of a longer one (stream prefixes);
* generation parallelises over heads with a thread pool (NumPy releases the
  GIL while filling large arrays).

Distributions.  ``N(mu, s)`` means mean ``mu`` and standard deviation ``s``.
q, k, v are drawn in fp32 and, for bf16 workloads, rounded to bf16 with
round-to-nearest-even; the rounded values are the inputs (the oracle upcasts
them exactly).  Gate pre-activations are drawn in fp64, optionally passed
through the soft-cap ``a * tanh(x / a)`` of the paper's gate stabilisation
(Sec. 3.2, Eq. 13, a = 15), and rounded once to fp32.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

# tensor ids inside a head's key
_Q, _K, _V, _I, _F, _C0, _N0, _M0 = 0, 1, 2, 3, 4, 5, 6, 7
_DEC_OFFSET = 10  # decode-step tensors use ids 10..14
_DOC = 20         # document lengths of a packed sequence


def _rng(seed: int, workload: int, head: int, tensor: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, workload, head, tensor])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); returns uint16 bit patterns.

    Inputs here are finite, so NaN handling is not needed.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def softcap(x: np.ndarray, cap: float) -> np.ndarray:
    """Soft-cap of the gate pre-activations, a * tanh(x / a) (Sec. 3.2, Eq. 13), in fp64."""
    return cap * np.tanh(x / cap)


def _workers() -> int:
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(16, n))


def _parallel(fn, items):
    items = list(items)
    if len(items) <= 1:
        for it in items:
            fn(it)
        return
    with _cf.ThreadPoolExecutor(_workers()) as ex:
        for _ in ex.map(fn, items):
            pass


@dataclass
class GateDist:
    """Gate pre-activation distribution: ipre ~ N(i_mu, i_sd), fpre ~ N(f_mu, f_sd), optional soft-cap."""
    i_mu: float = 0.0
    i_sd: float = 1.0
    f_mu: float = 3.0
    f_sd: float = 1.0
    cap: Optional[float] = None


@dataclass
class StateDist:
    """Initial state distribution: C0 ~ N(0, c_sd), n0 ~ |N(0, 1)|, m0 ~ N(0, 1)."""
    c_sd: float = 0.1


@dataclass
class Inputs:
    """One batch of cell inputs, host side.

    ``q, k, v`` are uint16 bf16 bit patterns when ``dtype == 'bf16'`` and
    float32 when ``dtype == 'f32'``; layouts are [B, NH, T, D] row-major.
    Gates are float32 [B, NH, T].  The initial state is either all None
    (zero state, m0 = 0) or float32 C0 [B, NH, DQK, DV], n0 [B, NH, DQK],
    m0 [B, NH].
    """
    dtype: str
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    ipre: np.ndarray
    fpre: np.ndarray
    C0: Optional[np.ndarray] = None
    n0: Optional[np.ndarray] = None
    m0: Optional[np.ndarray] = None
    heads: Optional[np.ndarray] = field(default=None)  # global head indices held, if a subset

    @property
    def B(self) -> int:
        return self.q.shape[0]

    @property
    def NH(self) -> int:
        return self.q.shape[1]

    @property
    def T(self) -> int:
        return self.q.shape[2]

    @property
    def DQK(self) -> int:
        return self.q.shape[3]

    @property
    def DV(self) -> int:
        return self.v.shape[3]

    def as_f64(self, name: str) -> np.ndarray:
        """Exact fp64 copy of an input tensor (bf16 and fp32 both widen exactly)."""
        x = getattr(self, name)
        if x is None:
            return None
        if x.dtype == np.uint16:
            x = bf16_bits_to_f32(x)
        return x.astype(np.float64)


def _draw_qkv(rng: np.random.Generator, n: int, bf16: bool, scale: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(n, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return f32_to_bf16_bits(x) if bf16 else x


def _draw_gate(rng: np.random.Generator, n: int, mu: float, sd: float, cap: Optional[float]) -> np.ndarray:
    x = rng.normal(mu, sd, n)
    if cap is not None:
        x = softcap(x, cap)
    return x.astype(np.float32)


def make_prefill(*, workload: int, B: int, NH: int, T: int, DQK: int, DV: int, dtype: str,
                 gates: GateDist, state: Optional[StateDist] = None, k_scale: float = 1.0,
                 seed: int = 0, heads: Optional[np.ndarray] = None,
                 tensor_base: int = 0) -> Inputs:
    """Draw a prefill batch.  ``heads`` (global indices b*NH+h) selects a subset; the result
    then has shape [1, len(heads), ...] and holds exactly the values those heads have in the
    full batch."""
    bf16 = dtype == "bf16"
    all_heads = np.arange(B * NH) if heads is None else np.asarray(heads, dtype=np.int64)
    nsel = len(all_heads)
    qkv_dt = np.uint16 if bf16 else np.float32
    q = np.empty((nsel, T * DQK), qkv_dt)
    k = np.empty((nsel, T * DQK), qkv_dt)
    v = np.empty((nsel, T * DV), qkv_dt)
    ipre = np.empty((nsel, T), np.float32)
    fpre = np.empty((nsel, T), np.float32)
    if state is not None:
        C0 = np.empty((nsel, DQK * DV), np.float32)
        n0 = np.empty((nsel, DQK), np.float32)
        m0 = np.empty((nsel,), np.float32)
    tb = tensor_base

    def one(j):
        hg = int(all_heads[j])
        q[j] = _draw_qkv(_rng(seed, workload, hg, tb + _Q), T * DQK, bf16)
        k[j] = _draw_qkv(_rng(seed, workload, hg, tb + _K), T * DQK, bf16, k_scale)
        v[j] = _draw_qkv(_rng(seed, workload, hg, tb + _V), T * DV, bf16)
        ipre[j] = _draw_gate(_rng(seed, workload, hg, tb + _I), T, gates.i_mu, gates.i_sd, gates.cap)
        fpre[j] = _draw_gate(_rng(seed, workload, hg, tb + _F), T, gates.f_mu, gates.f_sd, gates.cap)
        if state is not None:
            C0[j] = (_rng(seed, workload, hg, _C0).normal(0.0, state.c_sd, DQK * DV)).astype(np.float32)
            n0[j] = np.abs(_rng(seed, workload, hg, _N0).standard_normal(DQK)).astype(np.float32)
            m0[j] = np.float32(_rng(seed, workload, hg, _M0).standard_normal())

    _parallel(one, range(nsel))
    shp = (B, NH) if heads is None else (1, nsel)
    out = Inputs(dtype=dtype,
                 q=q.reshape(*shp, T, DQK), k=k.reshape(*shp, T, DQK), v=v.reshape(*shp, T, DV),
                 ipre=ipre.reshape(*shp, T), fpre=fpre.reshape(*shp, T),
                 heads=None if heads is None else all_heads)
    if state is not None:
        out.C0 = C0.reshape(*shp, DQK, DV)
        out.n0 = n0.reshape(*shp, DQK)
        out.m0 = m0.reshape(*shp)
    return out


def pack_documents(inp: Inputs, mean_len: float, *, workload: int, seed: int = 0,
                   first: bool = False) -> list:
    """Mark document borders in ``inp.fpre`` in place: each sequence is a run of packed documents
    with i.i.d. geometric lengths of mean ``mean_len`` (at least one token), and the first token
    of every document after the first gets f~ = -inf, a forget gate of exactly zero (the reset at
    document borders of sequence packing, App. B).  ``first`` also marks token 0, which drops an
    initial state.  Returns the marked positions per sequence (global head order)."""
    fp = inp.fpre.reshape(-1, inp.T)
    heads = np.arange(fp.shape[0]) if inp.heads is None else inp.heads
    out = []
    for j, hg in enumerate(heads):
        rng = _rng(seed, workload, int(hg), _DOC)
        pos, t = [0] if first else [], 0
        while True:
            t += int(rng.geometric(1.0 / mean_len))
            if t >= inp.T:
                break
            pos.append(t)
        fp[j, pos] = -np.inf
        out.append(np.asarray(pos, dtype=np.int64))
    return out


def make_decode_steps(*, workload: int, B: int, NH: int, steps: int, DQK: int, DV: int,
                      gates: GateDist, dtype: str = "bf16", seed: int = 0,
                      heads: Optional[np.ndarray] = None) -> Inputs:
    """Per-step decode inputs for ``steps`` consecutive tokens, returned with a time axis
    ([B, NH, steps, D]); step s reads index s of that axis.  Drawn from the decode tensor
    ids, so the first s steps of a longer run are identical."""
    return make_prefill(workload=workload, B=B, NH=NH, T=steps, DQK=DQK, DV=DV, dtype=dtype,
                        gates=gates, state=None, seed=seed, heads=heads, tensor_base=_DEC_OFFSET)


@dataclass
class LayerInputs:
    """Synthetic weights and input of one mLSTM layer (bf16 arrays as uint16 bit patterns).

    W_in [d, NH (2 DQK + 2 DV + 2)]: q, k, v projections (head-major), the input and forget
    gate projections (one column per head), the output gate projection (head-major);
    W_proj [NH DV, d]; gate_bias [2, NH] fp32 (input gate around -2, forget gate around +3);
    norm_weight [NH, DV] fp32; x [B, T, d] bf16.
    """
    d: int
    NH: int
    DQK: int
    DV: int
    W_in: np.ndarray
    W_proj: np.ndarray
    gate_bias: np.ndarray
    norm_weight: np.ndarray
    x: np.ndarray


def make_layer(*, workload: int, B: int, T: int, NH: int, DQK: int, DV: int, seed: int = 0) -> LayerInputs:
    """Weights drawn N(0, 1/sqrt(fan_in)), norm weights N(1, 0.1), x N(0, 1)."""
    d = NH * DV
    n_in = NH * (2 * DQK + 2 * DV + 2)
    r = lambda t: _rng(seed, workload, 1 << 20, t)
    W_in = r(0).standard_normal((d, n_in), dtype=np.float32) * np.float32(d ** -0.5)
    W_proj = r(1).standard_normal((NH * DV, d), dtype=np.float32) * np.float32((NH * DV) ** -0.5)
    gb = np.stack([r(2).normal(-2.0, 1.0, NH), r(3).normal(3.0, 1.0, NH)]).astype(np.float32)
    nw = r(4).normal(1.0, 0.1, (NH, DV)).astype(np.float32)
    x = r(5).standard_normal((B, T, d), dtype=np.float32)
    return LayerInputs(d, NH, DQK, DV, f32_to_bf16_bits(W_in), f32_to_bf16_bits(W_proj), gb, nw, f32_to_bf16_bits(x))
