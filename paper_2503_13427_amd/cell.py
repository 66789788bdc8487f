"""The mLSTM cell as a differentiable torch operation for training (Sec. 2, "Training Mode").

``mlstm_cell(q, k, v, ipre, fpre, L, state)`` runs the chunkwise forward (``mlstm_chunkwise_fwd``,
from the zero state or a given one) and, on backward, the chunkwise backward
(``mlstm_chunkwise_bwd``: bf16 q, k, v with the xLSTM-7B head shape DQK = 256, DV = 512; document
borders f~ = -inf and the initial state's gradients included) or, for other shapes and dtypes, the
parallel-form backward (``mlstm_parallel_bwd``: zero initial state, no borders).  Both run in
libmlstm.  This module only marshals tensors: it allocates the outputs, the workspaces and the
gradient buffers and casts the incoming gradient to the dtype the backward takes.
"""
from __future__ import annotations

from typing import Optional, Tuple

import torch

from . import binding as mb

BWD_L = 64   # the chunkwise backward's chunk length (independent of the forward's)


def chunkwise_bwd_supported(q: torch.Tensor, v: torch.Tensor) -> bool:
    return q.dtype == torch.bfloat16 and q.shape[3] == 256 and v.shape[3] == 512


class _MLSTMCell(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, ipre, fpre, C0, n0, m0, L):
        B, NH, T, DQK = q.shape
        DV = v.shape[3]
        dev = q.device
        h = torch.empty(B, NH, T, DV, dtype=q.dtype, device=dev)
        CT = torch.empty(B, NH, DQK, DV, device=dev)
        nT = torch.empty(B, NH, DQK, device=dev)
        mT = torch.empty(B, NH, device=dev)
        nb = mb.mlstm_chunkwise_workspace_bytes(B, NH, T, DQK, DV, L, q.dtype)
        ws = torch.empty(nb, dtype=torch.uint8, device=dev) if nb else None
        mb.mlstm_chunkwise_fwd(q, k, v, ipre, fpre, C0, n0, m0, L, h, CT, nT, mT, workspace=ws)
        ctx.chunkwise = chunkwise_bwd_supported(q, v)
        ctx.has_state = C0 is not None
        if not ctx.chunkwise:
            if ctx.has_state:
                raise ValueError("the parallel-form backward (shapes other than bf16 DQK=256, DV=512) starts "
                                 "from the zero state; an initial state is not supported there")
            if bool(torch.isneginf(fpre).any()):
                raise ValueError("the parallel-form backward (shapes other than bf16 DQK=256, DV=512) does not "
                                 "take document borders (f~ = -inf): its gradients would be NaN")
        ctx.save_for_backward(q, k, v, ipre, fpre, C0, n0, m0)
        ctx.mark_non_differentiable(CT, nT, mT)
        return h, CT, nT, mT

    @staticmethod
    def backward(ctx, dh, _dCT, _dnT, _dmT):
        q, k, v, ipre, fpre, C0, n0, m0 = ctx.saved_tensors
        B, NH, T, DQK = q.shape
        DV = v.shape[3]
        dev = q.device
        dq = torch.empty(B, NH, T, DQK, device=dev)
        dk = torch.empty(B, NH, T, DQK, device=dev)
        dv = torch.empty(B, NH, T, DV, device=dev)
        di = torch.empty(B, NH, T, device=dev)
        df = torch.empty(B, NH, T, device=dev)
        dC0 = dn0 = dm0 = None
        if ctx.chunkwise:
            if ctx.has_state:
                dC0 = torch.empty(B, NH, DQK, DV, device=dev)
                dn0 = torch.empty(B, NH, DQK, device=dev)
                dm0 = torch.empty(B, NH, device=dev)
            nb = mb.mlstm_chunkwise_bwd_workspace_bytes(B, NH, T, DQK, DV, BWD_L)
            ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
            mb.mlstm_chunkwise_bwd(q, k, v, ipre, fpre, C0, n0, m0, BWD_L, dh.to(torch.bfloat16).contiguous(),
                                   dq, dk, dv, di, df, dC0, dn0, dm0, ws)
        else:
            ws = torch.empty(mb.mlstm_parallel_bwd_workspace_bytes(B, NH, T, DV), dtype=torch.uint8, device=dev)
            mb.mlstm_parallel_bwd(q, k, v, ipre, fpre, dh.float().contiguous(), dq, dk, dv, di, df, ws)
        return dq.to(q.dtype), dk.to(k.dtype), dv.to(v.dtype), di, df, dC0, dn0, dm0, None


State = Tuple[torch.Tensor, torch.Tensor, torch.Tensor]


def mlstm_cell(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, ipre: torch.Tensor, fpre: torch.Tensor,
               L: int = 64, state: Optional[State] = None, return_state: bool = False):
    """h~ [B, NH, T, DV] (the dtype of q, k, v) from the zero state or ``state`` = (C0 [B, NH, DQK, DV],
    n0 [B, NH, DQK], m0 [B, NH], fp32); differentiable with respect to q, k, v [B, NH, T, D], the fp32
    gate pre-activations ipre, fpre [B, NH, T] and the initial state.  ``return_state`` also returns
    the final state (CT, nT, mT), which carries no gradient (the loss is taken not to depend on it)."""
    C0, n0, m0 = (None, None, None) if state is None else tuple(s.contiguous() for s in state)
    h, CT, nT, mT = _MLSTMCell.apply(q.contiguous(), k.contiguous(), v.contiguous(), ipre.contiguous(),
                                     fpre.contiguous(), C0, n0, m0, L)
    return (h, (CT, nT, mT)) if return_state else h
