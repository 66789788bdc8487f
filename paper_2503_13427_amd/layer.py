"""Multi-head mLSTM layer of xLSTM 7B (Eq. 11) around libmlstm, with synthetic weights.

x [B, T, d] -> y [B, T, d], d = NH * DV:

1. input projection: one bf16 GEMM for q, k, v and o~ (head-major columns, bf16 output;
   hipBLASLt on ROCm);
2. ``mlstm_gate_preact``: the two gate pre-activations per head (bf16 products, fp32), their
   biases, the soft-cap a * tanh(x / a) of Eq. 13 (a = 15) and the document borders of a packed
   sequence (f~ = -inf, App. B), written head-major;
3. the cell: ``mlstm_chunkwise_fwd_strided`` for a prefill, which reads q, k and v as per-head
   views of the projection output (no head-major copies), ``mlstm_step_output`` for one decode
   step (the step with the output norm of step 4 in its epilogue; q, k, v, o~ contiguous);
4. the output norm h = sigmoid(o~) * LayerNorm(h~) * weight, per head: for a prefill
   ``mlstm_output_norm_tokens`` reads o~ in place in the projection output and writes h
   token-major [B, T, NH, DV], which is already the concatenation of the heads;
5. the output projection (bf16 GEMM).

The q, k, v, o~ and output projections are plain library GEMMs around the cell; the gates, the
cell and the output norm run in libmlstm.  The layer's pre-norm (Norm(x) in the block, Eq. 12) belongs to
the block, not to the layer, and is not applied.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Tuple

import torch

from . import binding as mb

State = Tuple[torch.Tensor, torch.Tensor, torch.Tensor]   # C [B, NH, DQK, DV], n [B, NH, DQK], m [B, NH]


@dataclass
class LayerWeights:
    W_qkvo: torch.Tensor      # [d, NH (2 DQK + 2 DV)] bf16: q, k, v, o~ columns, head-major
    W_gates_t: torch.Tensor   # [2 NH, d] bf16: input gate rows, then forget gate rows
    W_proj: torch.Tensor      # [NH DV, d] bf16
    gate_bias: torch.Tensor   # [2, NH] fp32
    norm_weight: torch.Tensor # [NH, DV] fp32
    NH: int
    DQK: int
    DV: int

    @staticmethod
    def from_inputs(li, device="cuda") -> "LayerWeights":
        """From ``inputs.LayerInputs`` (bf16 bit patterns): W_in split into the q, k, v, o~ columns
        and the gate columns."""
        import numpy as np
        NH, DQK, DV = li.NH, li.DQK, li.DV
        W = torch.from_numpy(np.ascontiguousarray(li.W_in)).view(torch.bfloat16)
        a = NH * (2 * DQK + DV)
        W_qkvo = torch.cat([W[:, :a], W[:, a + 2 * NH:]], dim=1).contiguous()
        W_gates_t = W[:, a:a + 2 * NH].t().contiguous()
        Wp = torch.from_numpy(np.ascontiguousarray(li.W_proj)).view(torch.bfloat16)
        return LayerWeights(W_qkvo.to(device), W_gates_t.to(device), Wp.to(device),
                            torch.from_numpy(li.gate_bias).to(device), torch.from_numpy(li.norm_weight).to(device),
                            NH, DQK, DV)


class MLSTMLayer:
    def __init__(self, w: LayerWeights, L: int = 64, eps: float = 1e-6, cap: Optional[float] = 15.0):
        self.w, self.L, self.eps, self.cap = w, L, eps, cap

    def _project(self, x2: torch.Tensor):
        """x2 [R, d] bf16 -> q, k [R, NH, DQK], v, o [R, NH, DV] bf16 (views of one GEMM output)."""
        w = self.w
        NH, DQK, DV = w.NH, w.DQK, w.DV
        P = torch.matmul(x2, w.W_qkvo)
        R = x2.shape[0]
        c = [0, NH * DQK, 2 * NH * DQK, NH * (2 * DQK + DV), NH * (2 * DQK + 2 * DV)]
        q = P[:, c[0]:c[1]].view(R, NH, DQK)
        k = P[:, c[1]:c[2]].view(R, NH, DQK)
        v = P[:, c[2]:c[3]].view(R, NH, DV)
        o = P[:, c[3]:c[4]].view(R, NH, DV)
        return q, k, v, o

    def gates(self, x: torch.Tensor, border: Optional[torch.Tensor] = None):
        """i~, f~ head-major, fp32: [B, NH, T] for x [B, T, d], [B, NH] for a decode step x [B, d];
        ``border`` [B, T] (bool or uint8) marks the first token of each new document."""
        w = self.w
        shape = (x.shape[0], w.NH) if x.dim() == 2 else (x.shape[0], w.NH, x.shape[1])
        ig = torch.empty(shape, dtype=torch.float32, device=x.device)
        fg = torch.empty(shape, dtype=torch.float32, device=x.device)
        mb.mlstm_gate_preact(x, w.W_gates_t, w.gate_bias, self.cap or 0.0, border, ig, fg)
        return ig, fg

    def project_heads(self, x: torch.Tensor, border: Optional[torch.Tensor] = None):
        """Steps 1-3 for a prefill: x [B, T, d] -> head-major q, k [B, NH, T, DQK], v, o~
        [B, NH, T, DV] (bf16) and the capped gate pre-activations i~, f~ [B, NH, T] (fp32)."""
        w = self.w
        B, T, d = x.shape
        NH, DQK, DV = w.NH, w.DQK, w.DV
        q, k, v, o = self._project(x.reshape(B * T, d))
        hm = lambda a, D: a.view(B, T, NH, D).transpose(1, 2).contiguous()   # head-major [B, NH, T, D]
        ig, fg = self.gates(x, border)
        return hm(q, DQK), hm(k, DQK), hm(v, DV), hm(o, DV), ig, fg

    def prefill(self, x: torch.Tensor, state: Optional[State] = None,
                workspace: Optional[torch.Tensor] = None,
                border: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, State]:
        """x [B, T, d] bf16 -> (y [B, T, d] bf16, the cell state after the T tokens).  ``workspace``
        (uint8, ``mlstm_chunkwise_workspace_bytes``) is allocated per call when not given;
        ``border`` [B, T] marks document borders of packed sequences (the state restarts there)."""
        w = self.w
        B, T, d = x.shape
        NH, DQK, DV = w.NH, w.DQK, w.DV
        q, k, v, o = self._project(x.reshape(B * T, d))
        # head-major views of the projection output, no copy: the cell takes strided q, k, v rows
        hv = lambda a, D: a.view(B, T, NH, D).transpose(1, 2)
        q, k, v = hv(q, DQK), hv(k, DQK), hv(v, DV)
        ig, fg = self.gates(x, border)
        h = torch.empty(B, NH, T, DV, dtype=torch.bfloat16, device=x.device)
        C = torch.empty(B, NH, DQK, DV, device=x.device)
        n = torch.empty(B, NH, DQK, device=x.device)
        m = torch.empty(B, NH, device=x.device)
        C0, n0, m0 = state if state is not None else (None, None, None)
        if workspace is None:   # the segment schedule needs one; without it the call runs one block per sequence
            nb = mb.mlstm_chunkwise_workspace_bytes(B, NH, T, DQK, DV, self.L)
            workspace = torch.empty(nb, dtype=torch.uint8, device=x.device) if nb else None
        mb.mlstm_chunkwise_fwd_strided(q, k, v, ig, fg, C0, n0, m0, self.L, h, C, n, m, workspace=workspace)
        # o~ stays in the projection output and the result comes out token-major for W_proj
        yh = torch.empty(B, T, NH, DV, dtype=torch.bfloat16, device=x.device)
        mb.mlstm_output_norm_tokens(h, o.view(B, T, NH, DV), w.norm_weight, None, self.eps, "layer", yh)
        y = torch.matmul(yh.view(B * T, NH * DV), w.W_proj)
        return y.view(B, T, d), (C, n, m)

    def step(self, x: torch.Tensor, state: State) -> torch.Tensor:
        """One decode step: x [B, d] bf16 -> y [B, d]; the state is updated in place."""
        w = self.w
        B, d = x.shape
        q, k, v, o = self._project(x)
        q, k, v, o = q.contiguous(), k.contiguous(), v.contiguous(), o.contiguous()
        ig, fg = self.gates(x)
        C, n, m = state
        h = torch.empty(B, w.NH, w.DV, dtype=torch.bfloat16, device=x.device)
        mb.mlstm_step_output(q, k, v, ig, fg, C, n, m, o, w.norm_weight, None, self.eps, "layer", h, C, n, m)
        return torch.matmul(h.reshape(B, w.NH * w.DV), w.W_proj)


class GraphedDecode:
    """One decode step of ``layer`` captured as a HIP graph, for batch B and the given state.

    A single-token step is a dozen small launches (projections, gate cap, the cell, the norm, the
    output projection); replaying them as one graph removes the per-launch host cost.  The graph
    reads ``self.x`` and the state tensors it was captured with, updates that state in place and
    writes ``self.y``: call it with the next token's x [B, d]; the returned y is overwritten by the
    next call.  Nothing in the captured work clears memory with a memset node."""

    def __init__(self, layer: MLSTMLayer, state: State, B: int):
        w = layer.w
        d = w.W_proj.shape[1]
        dev = w.W_proj.device
        self.x = torch.zeros(B, d, dtype=torch.bfloat16, device=dev)
        self.state = state
        # library set-up (GEMM handles, workspaces) happens on warm-up calls before capture; they run
        # on a copy of the state so the caller's state is untouched
        scratch = tuple(t.clone() for t in state)
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(torch.cuda.current_stream(dev))
        with torch.cuda.stream(side):
            for _ in range(2):
                layer.step(self.x, scratch)
        torch.cuda.current_stream(dev).wait_stream(side)
        torch.cuda.synchronize(dev)
        del scratch
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.y = layer.step(self.x, state)

    def __call__(self, x: torch.Tensor) -> torch.Tensor:
        self.x.copy_(x)
        self.graph.replay()
        return self.y
