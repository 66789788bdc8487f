"""Work and traffic accounting for the mLSTM cell: the roofline denominators.

* ``flops_chunkwise``: the FLOP count of the chunkwise forward pass, App. D.1
  ("FLOPs for the mLSTM Operation"), a factor 2 per multiply-accumulate and
  every F_X factor (exp, max, mask, abs) = 1.
* ``state_bytes``: the fp32 memory-state size formula of Sec. 3.1
  (#blocks x #heads x d_qk x d_hv x 4 bytes).
* ``prefill_bytes`` / ``step_bytes``: algorithmic HBM bytes of one call, i.e.
  every input read once and every output written once, at the call's dtypes.
* ``flops_layer_projections``: the dense projections of one mLSTM layer, App. D.2
  ("FLOPs for the mLSTM in a Transformer Backbone"), per token count.
* ``layer_step_bytes``: algorithmic HBM bytes of one layer decode step (weights,
  state, token in and out).
* ``flops_parallel_bwd``: the FLOP count of the backward pass over the parallel
  form, per causal (t, s) pair.
"""
from __future__ import annotations

from dataclasses import dataclass

# MI355X published peaks
PEAK_BF16_MFMA_TFLOPS = 2500.0      # dense bf16 MFMA, TFLOP/s
PEAK_HBM_GBS = 8000.0               # HBM3E, GB/s
PEAK_FP32_VALU_TFLOPS = 157.3


@dataclass(frozen=True)
class FlopSplit:
    chunk_gates: float
    gates_max_state: float
    inter_numerator: float
    inter_denominator: float
    gate_matrix: float
    gated_logits: float
    intra_numerator: float
    intra_denominator: float
    output_combination: float

    @property
    def total(self) -> float:
        return (self.chunk_gates + self.gates_max_state + self.inter_numerator + self.inter_denominator
                + self.gate_matrix + self.gated_logits + self.intra_numerator + self.intra_denominator
                + self.output_combination)

    @property
    def contractions(self) -> float:
        """The matrix products: K~^T V and Q^ C (inside the inter numerator), Q^ K^T and S~ V."""
        return self.inter_numerator + self.gated_logits + self.intra_numerator


def flops_chunkwise(heads: int, T: int, L: int, dqk: int, dv: int,
                    F_exp: float = 1, F_max: float = 1, F_mask: float = 1, F_abs: float = 1) -> FlopSplit:
    """App. D.1 FLOP count of the chunkwise mLSTM forward over ``heads`` sequences of T tokens.

    ``heads`` is the number of independent (batch, head) sequences; num_chunks = T / L.
    """
    nc = T / L
    hc = heads * nc
    return FlopSplit(
        chunk_gates=hc * (0.5 * L * (L + 1) + 2 * L),
        gates_max_state=hc * (3 + F_max + F_exp + L * (3 + 2 * F_exp)),
        inter_numerator=hc * (2 * dqk * dv + 4 * L * dqk * dv + 3 * L * dqk),
        inter_denominator=hc * (dqk + 4 * L * dqk),
        gate_matrix=hc * (0.5 * L * (L + 1) + L * L * (3 + F_mask + F_max + F_exp) + L * (1 + F_max)),
        gated_logits=hc * 2 * L * L * (1 + dqk),
        intra_numerator=hc * 2 * L * L * dv,
        intra_denominator=hc * 2 * L * L,
        output_combination=hc * (L * (1 + F_max) + L * (2 + F_abs + F_exp + F_max + 2 * dv)),
    )


def state_bytes(blocks: int, heads: int, dqk: int, dhv: int, elem_bytes: int = 4) -> int:
    """Total memory-state size, #blocks x #heads x d_qk x d_hv x 4 bytes (Sec. 3.1)."""
    return blocks * heads * dqk * dhv * elem_bytes


def prefill_bytes(B: int, NH: int, T: int, dqk: int, dv: int, qkv_bytes: int = 2,
                  with_initial_state: bool = False) -> int:
    """Algorithmic HBM bytes of one chunkwise prefill call: q, k, v, both gate arrays and
    (optionally) C0, n0, m0 read once; h (same dtype as q, k, v) and C_T, n_T, m_T written once."""
    S = B * NH
    tok = S * T * (2 * dqk * qkv_bytes + dv * qkv_bytes + 2 * 4 + dv * qkv_bytes)
    state = S * (dqk * dv + dqk + 1) * 4
    return tok + state * (2 if with_initial_state else 1)


def step_bytes(B: int, NH: int, dqk: int, dv: int, qkv_bytes: int = 2) -> int:
    """Algorithmic HBM bytes of one decode step: C, n, m read and written once (fp32),
    q, k, v and the two gates read, h written."""
    S = B * NH
    return S * (2 * (dqk * dv + dqk + 1) * 4 + (2 * dqk + dv) * qkv_bytes + 2 * 4 + dv * qkv_bytes)


def step_flops(B: int, NH: int, dqk: int, dv: int) -> int:
    """Arithmetic of one decode step: the C update f*C + (i*k)*v is 3 FLOPs per element, the
    read-out C'^T q^ one multiply-add (2 FLOPs) per element; n and its dot product add 6 per row."""
    S = B * NH
    return S * (5 * dqk * dv + 6 * dqk)


def output_norm_bytes(B: int, NH: int, T: int, dv: int, elem_bytes: int = 2, affine: bool = True) -> int:
    """Algorithmic HBM bytes of the hidden-state output h = sigmoid(o~) * (Norm(h~) w + b): every
    row of h~ and o~ read once and of h written once, plus the per-head weight and bias once."""
    return 3 * B * NH * T * dv * elem_bytes + (2 * NH * dv * 4 if affine else 0)


def flops_layer_projections(tokens: int, d: int, NH: int, dqk: int, dv: int, F_sig: int = 1) -> int:
    """App. D.2, one mLSTM layer without the cell: the q, k, v, input and forget gate projections,
    2 tokens d NH (2 dqk + dv + 2), and the output gate with the output projection,
    4 tokens d NH dv + tokens NH dv F_sig."""
    return 2 * tokens * d * NH * (2 * dqk + dv + 2) + 4 * tokens * d * NH * dv + tokens * NH * dv * F_sig


def layer_weight_bytes(d: int, NH: int, dqk: int, dv: int) -> int:
    """The layer's weights as stored: q, k, v, o~ projection and output projection in bf16, the gate
    projection (2 NH columns), the gate biases and the norm weight in fp32."""
    return 2 * d * NH * (2 * dqk + 2 * dv) + 2 * NH * dv * d + 4 * (2 * d * NH + 2 * NH + NH * dv)


def layer_step_bytes(B: int, d: int, NH: int, dqk: int, dv: int) -> int:
    """Algorithmic HBM bytes of one layer decode step of B tokens: every weight read once, the fp32
    state (C, n, m) read and written once, x read and y written once (bf16)."""
    state = 4 * B * NH * (dqk * dv + dqk + 1)
    return layer_weight_bytes(d, NH, dqk, dv) + 2 * state + 2 * 2 * B * d


def flops_parallel_bwd(heads: int, T: int, dqk: int, dv: int) -> int:
    """FLOPs of the backward pass over the parallel form (Eq. 10) as the library computes it: per
    causal pair (t, s <= t) the dot products q^_t . k_s (twice), dN~_t . v_s (twice) and the
    accumulations into N~_t, dq_t, dk_s and dv_s, each 2 FLOP per element: 8 (dqk + dv)."""
    return heads * (T * (T + 1) // 2) * 8 * (dqk + dv)
