"""The mLSTM cell as a differentiable torch operation for training (Sec. 2, "Training Mode").

``mlstm_cell(q, k, v, ipre, fpre, L)`` runs the chunkwise forward (``mlstm_chunkwise_fwd``, zero
initial state) and, on backward, the gradients of ``mlstm_parallel_bwd``; both run in libmlstm.
This module only marshals tensors: it allocates the outputs, the workspaces and the gradient
buffers and casts the incoming gradient to the fp32 the backward takes.
"""
from __future__ import annotations

import torch

from . import binding as mb


class _MLSTMCell(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, ipre, fpre, L):
        B, NH, T, DQK = q.shape
        DV = v.shape[3]
        dev = q.device
        h = torch.empty(B, NH, T, DV, dtype=q.dtype, device=dev)
        CT = torch.empty(B, NH, DQK, DV, device=dev)
        nT = torch.empty(B, NH, DQK, device=dev)
        mT = torch.empty(B, NH, device=dev)
        nb = mb.mlstm_chunkwise_workspace_bytes(B, NH, T, DQK, DV, L, q.dtype)
        ws = torch.empty(nb, dtype=torch.uint8, device=dev) if nb else None
        mb.mlstm_chunkwise_fwd(q, k, v, ipre, fpre, None, None, None, L, h, CT, nT, mT, workspace=ws)
        ctx.save_for_backward(q, k, v, ipre, fpre)
        ctx.has_borders = bool(torch.isneginf(fpre).any())
        return h

    @staticmethod
    def backward(ctx, dh):
        q, k, v, ipre, fpre = ctx.saved_tensors
        if ctx.has_borders:
            raise ValueError("mlstm_parallel_bwd does not take document borders (f~ = -inf); "
                             "its gradients would be NaN")
        B, NH, T, DQK = q.shape
        DV = v.shape[3]
        dev = q.device
        dq = torch.empty(B, NH, T, DQK, device=dev)
        dk = torch.empty(B, NH, T, DQK, device=dev)
        dv = torch.empty(B, NH, T, DV, device=dev)
        di = torch.empty(B, NH, T, device=dev)
        df = torch.empty(B, NH, T, device=dev)
        ws = torch.empty(mb.mlstm_parallel_bwd_workspace_bytes(B, NH, T, DV), dtype=torch.uint8, device=dev)
        mb.mlstm_parallel_bwd(q, k, v, ipre, fpre, dh.float().contiguous(), dq, dk, dv, di, df, ws)
        return dq.to(q.dtype), dk.to(k.dtype), dv.to(v.dtype), di, df, None


def mlstm_cell(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, ipre: torch.Tensor, fpre: torch.Tensor,
               L: int = 64) -> torch.Tensor:
    """h~ [B, NH, T, DV] (the dtype of q, k, v) from the zero state; differentiable with respect to
    q, k, v [B, NH, T, D] and the fp32 gate pre-activations ipre, fpre [B, NH, T]."""
    return _MLSTMCell.apply(q.contiguous(), k.contiguous(), v.contiguous(), ipre.contiguous(), fpre.contiguous(), L)
