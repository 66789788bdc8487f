"""ctypes binding of libmlstm (``include/mlstm.h``): argument marshalling only.

Every step of the cell runs in the HIP library; this module turns torch
tensors into device pointers and sizes, picks the current HIP stream, and
raises ``MlstmError`` on a non-OK status.  torch supplies device memory and
streams only.  If ``libmlstm.so`` is not built, importing this module fails
loudly: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# MLSTM_LIBRARY selects another build of the same library (the host-sanitized libmlstm_san.so of
# build_sanitize.py, for CPU-side checking); the default is the in-tree libmlstm.so
LIB_PATH = os.environ.get("MLSTM_LIBRARY") or os.path.join(_HERE, "libmlstm.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libmlstm is not built at {LIB_PATH}; run __graft_entry__.build() "
                      "or python -m paper_2503_13427_amd.build")

lib = ctypes.CDLL(LIB_PATH)

MLSTM_OK = 0
MLSTM_F32 = 0
MLSTM_BF16 = 1
MLSTM_NORM_LAYER = 0
MLSTM_NORM_RMS = 1
STATUS_NAMES = {0: "MLSTM_OK", 1: "MLSTM_ERR_NULL_PTR", 2: "MLSTM_ERR_BAD_SHAPE", 3: "MLSTM_ERR_UNSUPPORTED",
                4: "MLSTM_ERR_MISALIGNED", 5: "MLSTM_ERR_ALIAS", 6: "MLSTM_ERR_WORKSPACE", 7: "MLSTM_ERR_HIP"}

_vp = ctypes.c_void_p
_i = ctypes.c_int
lib.mlstm_chunkwise_fwd.argtypes = [_vp, _vp, _vp, _i, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                    _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
lib.mlstm_chunkwise_fwd.restype = _i
lib.mlstm_chunkwise_fwd_strided.argtypes = [_vp, _vp, _vp, ctypes.POINTER(ctypes.c_int64), _i, _vp, _vp, _vp, _vp, _vp,
                                            _i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
lib.mlstm_chunkwise_fwd_strided.restype = _i
lib.mlstm_chunkwise_fwd_noalloc.argtypes = [_vp, _vp, _vp, _i, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                            _vp, _vp, _vp, _vp, _vp]
lib.mlstm_chunkwise_fwd_noalloc.restype = _i
lib.mlstm_chunkwise_scratch_bytes.argtypes = []
lib.mlstm_chunkwise_scratch_bytes.restype = ctypes.c_size_t
lib.mlstm_chunkwise_workspace_bytes.argtypes = [_i, _i, _i, _i, _i, _i, _i]
lib.mlstm_chunkwise_workspace_bytes.restype = ctypes.c_size_t
lib.mlstm_step.argtypes = [_vp, _vp, _vp, _i, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp]
lib.mlstm_step.restype = _i
lib.mlstm_step_output.argtypes = [_vp, _vp, _vp, _i, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_float, _i, _i, _i,
                                  _i, _i, _vp, _vp, _vp, _vp, _vp]
lib.mlstm_step_output.restype = _i
lib.mlstm_output_norm.argtypes = [_vp, _vp, _i, _vp, _vp, ctypes.c_float, _i, _i, _i, _i, _i, _vp, _vp]
lib.mlstm_output_norm.restype = _i
lib.mlstm_output_norm_tokens.argtypes = [_vp, _vp, ctypes.c_int64, _i, _vp, _vp, ctypes.c_float, _i, _i, _i, _i,
                                         _i, _vp, _vp]
lib.mlstm_output_norm_tokens.restype = _i
lib.mlstm_gate_preact.argtypes = [_vp, _i, _vp, _vp, ctypes.c_float, _vp, _i, _i, _i, _i, _vp, _vp, _vp]
lib.mlstm_gate_preact.restype = _i
lib.mlstm_parallel_bwd_workspace_bytes.argtypes = [_i, _i, _i, _i]
lib.mlstm_parallel_bwd_workspace_bytes.restype = ctypes.c_size_t
lib.mlstm_parallel_bwd.argtypes = [_vp, _vp, _vp, _i, _vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp,
                                   ctypes.c_size_t, _vp]
lib.mlstm_parallel_bwd.restype = _i
lib.mlstm_chunkwise_bwd_workspace_bytes.argtypes = [_i, _i, _i, _i, _i, _i, _i]
lib.mlstm_chunkwise_bwd_workspace_bytes.restype = ctypes.c_size_t
lib.mlstm_chunkwise_bwd.argtypes = [_vp, _vp, _vp, _i, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp,
                                    _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
lib.mlstm_chunkwise_bwd.restype = _i
lib.mlstm_status_string.argtypes = [_i]
lib.mlstm_status_string.restype = ctypes.c_char_p
lib.mlstm_version.argtypes = []
lib.mlstm_version.restype = _i
lib.mlstm_debug_flags.argtypes = []
lib.mlstm_debug_flags.restype = ctypes.c_uint


class MlstmError(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(mlstm_status_string(status))


def mlstm_status_string(status: int) -> str:
    return lib.mlstm_status_string(int(status)).decode()


def mlstm_version() -> int:
    return lib.mlstm_version()


MLSTM_DEBUG_NOT_BUILT = 0x80000000


def mlstm_debug_flags() -> int:
    """Debug builds: the bounds-check bits set since the last call (0: none failed); other builds
    return MLSTM_DEBUG_NOT_BUILT.  Synchronise the device first."""
    return int(lib.mlstm_debug_flags())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return MLSTM_BF16
    if t.dtype == torch.float32:
        return MLSTM_F32
    raise TypeError(f"q/k/v must be bfloat16 or float32, got {t.dtype}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("libmlstm needs contiguous tensors")
    return t.data_ptr()


def _view_ptr(t: torch.Tensor) -> int:
    """Data pointer of a strided view (its strides travel separately)."""
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(status: int) -> None:
    if status != MLSTM_OK:
        raise MlstmError(status)


def mlstm_chunkwise_workspace_bytes(B: int, NH: int, T: int, DQK: int, DV: int, L: int,
                                    dtype: torch.dtype = torch.bfloat16) -> int:
    code = MLSTM_BF16 if dtype == torch.bfloat16 else MLSTM_F32
    return int(lib.mlstm_chunkwise_workspace_bytes(B, NH, T, DQK, DV, L, code))


def mlstm_chunkwise_fwd(q, k, v, ipre, fpre, C0, n0, m0, L, h, CT, nT, mT,
                        workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """Chunkwise prefill.  Tensors as in ``include/mlstm.h``; shapes are read from q and v.
    ``C0, n0, m0`` all None means the zero state.  ``workspace`` is an optional uint8 device
    tensor of at least ``mlstm_chunkwise_workspace_bytes`` bytes."""
    B, NH, T, DQK = q.shape
    DV = v.shape[3]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.mlstm_chunkwise_fwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(ipre), _ptr(fpre),
                                   _ptr(C0), _ptr(n0), _ptr(m0), B, NH, T, DQK, DV, int(L),
                                   _ptr(h), _ptr(CT), _ptr(nT), _ptr(mT), _ptr(workspace), ws_bytes,
                                   _stream(stream)))


def mlstm_chunkwise_fwd_strided(q, k, v, ipre, fpre, C0, n0, m0, L, h, CT, nT, mT,
                                workspace=None, stream=None) -> None:
    """mlstm_chunkwise_fwd on strided views q, k [B, NH, T, DQK], v [B, NH, T, DV] (bf16, rows of D
    contiguous), for instance ``x.view(B, T, NH, D).transpose(1, 2)`` of a projection output."""
    B, NH, T, DQK = q.shape
    DV = v.shape[3]
    for t in (q, k, v):
        if t.stride(3) != 1:
            raise ValueError("the rows (last axis) of q, k, v must be contiguous")
    st = (ctypes.c_int64 * 9)(*(q.stride()[:3] + k.stride()[:3] + v.stride()[:3]))
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib.mlstm_chunkwise_fwd_strided(_view_ptr(q), _view_ptr(k), _view_ptr(v), st, _dtype_code(q), _ptr(ipre),
                                           _ptr(fpre),
                                           _ptr(C0), _ptr(n0), _ptr(m0), B, NH, T, DQK, DV, L, _ptr(h), _ptr(CT),
                                           _ptr(nT), _ptr(mT), _ptr(workspace), ws_bytes, _stream(stream)))


def mlstm_chunkwise_scratch_bytes() -> int:
    return int(lib.mlstm_chunkwise_scratch_bytes())


def mlstm_chunkwise_fwd_noalloc(q, k, v, ipre, fpre, C0, n0, m0, L, h, CT, nT, mT, stream=None) -> None:
    """Chunkwise prefill without a workspace and without allocating: the segment slots live in the
    library's fixed device scratch (``mlstm_chunkwise_scratch_bytes``)."""
    B, NH, T, DQK = q.shape
    DV = v.shape[3]
    _check(lib.mlstm_chunkwise_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(ipre), _ptr(fpre),
                                           _ptr(C0), _ptr(n0), _ptr(m0), B, NH, T, DQK, DV, int(L),
                                           _ptr(h), _ptr(CT), _ptr(nT), _ptr(mT), _stream(stream)))


def mlstm_step(q, k, v, ipre, fpre, C, n, m, h, C_out, n_out, m_out, stream=None) -> None:
    """One decode step.  q, k [B, NH, DQK]; v, h [B, NH, DV]; state outputs may be the inputs."""
    B, NH, DQK = q.shape
    DV = v.shape[2]
    _check(lib.mlstm_step(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(ipre), _ptr(fpre), _ptr(C),
                          _ptr(n), _ptr(m), B, NH, DQK, DV, _ptr(h), _ptr(C_out), _ptr(n_out), _ptr(m_out),
                          _stream(stream)))


def mlstm_step_output(q, k, v, ipre, fpre, C, n, m, o_pre, weight, bias, eps: float, norm: str, h, C_out, n_out,
                      m_out, stream=None) -> None:
    """One decode step returning h = sigmoid(o~) * (Norm(h~) * weight + bias); o_pre and h [B, NH, DV];
    weight, bias [NH, DV] fp32 or None; norm "layer" or "rms"; state outputs may be the inputs."""
    B, NH, DQK = q.shape
    DV = v.shape[2]
    code = {"layer": MLSTM_NORM_LAYER, "rms": MLSTM_NORM_RMS}[norm]
    _check(lib.mlstm_step_output(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(ipre), _ptr(fpre), _ptr(C), _ptr(n),
                                 _ptr(m), _ptr(o_pre), _ptr(weight), _ptr(bias), float(eps), code, B, NH, DQK, DV,
                                 _ptr(h), _ptr(C_out), _ptr(n_out), _ptr(m_out), _stream(stream)))


def mlstm_output_norm(h_tilde, o_pre, weight, bias, eps: float, norm: str, h, stream=None) -> None:
    """Hidden-state output h = sigmoid(o~) * (Norm(h~) * weight + bias) over the rows of
    h_tilde / o_pre / h [B, NH, T, DV] (a decode step: [B, NH, DV], taken as T = 1); weight and
    bias [NH, DV] fp32 or None; norm "layer" or "rms".  h may be h_tilde (in place)."""
    shape = h_tilde.shape
    if len(shape) == 3:
        B, NH, DV = shape
        T = 1
    else:
        B, NH, T, DV = shape
    code = {"layer": MLSTM_NORM_LAYER, "rms": MLSTM_NORM_RMS}[norm]
    _check(lib.mlstm_output_norm(_ptr(h_tilde), _ptr(o_pre), _dtype_code(h_tilde), _ptr(weight), _ptr(bias),
                                 float(eps), code, B, NH, T, DV, _ptr(h), _stream(stream)))


def mlstm_output_norm_tokens(h_tilde, o_pre, weight, bias, eps: float, norm: str, y, stream=None) -> None:
    """The output norm in token-major layouts: h_tilde [B, NH, T, DV] head-major, o_pre a
    [B, T, NH, DV] view whose tokens are ``o_pre.stride(1)`` elements apart (columns of a
    projection output), y [B, T, NH, DV] contiguous."""
    B, NH, T, DV = h_tilde.shape
    if tuple(o_pre.shape) != (B, T, NH, DV) or o_pre.stride(3) != 1 or o_pre.stride(2) != DV or \
            (B > 1 and o_pre.stride(0) != T * o_pre.stride(1)):
        raise ValueError("o_pre must be a [B, T, NH, DV] view with contiguous heads and evenly spaced tokens")
    if tuple(y.shape) != (B, T, NH, DV) or not y.is_contiguous():
        raise ValueError("y must be a contiguous [B, T, NH, DV] tensor")
    code = {"layer": MLSTM_NORM_LAYER, "rms": MLSTM_NORM_RMS}[norm]
    # o_pre is a strided view by design: its layout was checked above, so its pointer is taken as is
    _check(lib.mlstm_output_norm_tokens(_ptr(h_tilde), o_pre.data_ptr(), o_pre.stride(1), _dtype_code(h_tilde),
                                        _ptr(weight), _ptr(bias), float(eps), code, B, NH, T, DV, _ptr(y),
                                        _stream(stream)))


def mlstm_gate_preact(x, w_t, bias, cap: float, border, ipre, fpre, stream=None) -> None:
    """Gate pre-activations of a layer: x [B, T, d] bf16 (a decode step: [B, d], taken as T = 1),
    w_t [2 NH, d] bf16 (input gate rows, then forget gate rows), bias [2, NH] fp32 or None,
    cap (0: none), border [B, T] uint8/bool or None -> ipre, fpre [B, NH, T] fp32 (decode:
    [B, NH])."""
    if x.dim() == 2:
        B, d = x.shape
        T = 1
    else:
        B, T, d = x.shape
    NH = w_t.shape[0] // 2
    if border is not None and border.dtype == torch.bool:
        border = border.view(torch.uint8)
    _check(lib.mlstm_gate_preact(_ptr(x), _dtype_code(x), _ptr(w_t), _ptr(bias), float(cap), _ptr(border), B, T, d,
                                 NH, _ptr(ipre), _ptr(fpre), _stream(stream)))


def mlstm_parallel_bwd_workspace_bytes(B: int, NH: int, T: int, DV: int) -> int:
    return int(lib.mlstm_parallel_bwd_workspace_bytes(B, NH, T, DV))


def mlstm_parallel_bwd(q, k, v, ipre, fpre, dh, dq, dk, dv, dipre, dfpre, workspace, stream=None) -> None:
    """Gradients of a loss with respect to q, k, v [B, NH, T, D] (bf16 or fp32) and ipre, fpre
    [B, NH, T] given dh [B, NH, T, DV] fp32, from the zero initial state; outputs fp32 of the
    input shapes; workspace: uint8 tensor of mlstm_parallel_bwd_workspace_bytes bytes."""
    B, NH, T, DQK = q.shape
    DV = v.shape[3]
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib.mlstm_parallel_bwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(ipre), _ptr(fpre), _ptr(dh), B, NH, T,
                                  DQK, DV, _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dipre), _ptr(dfpre), _ptr(workspace),
                                  ws_bytes, _stream(stream)))


def mlstm_chunkwise_bwd_workspace_bytes(B: int, NH: int, T: int, DQK: int, DV: int, L: int,
                                        dtype: torch.dtype = torch.bfloat16) -> int:
    code = MLSTM_BF16 if dtype == torch.bfloat16 else MLSTM_F32
    return int(lib.mlstm_chunkwise_bwd_workspace_bytes(B, NH, T, DQK, DV, L, code))


def mlstm_chunkwise_bwd(q, k, v, ipre, fpre, C0, n0, m0, L, dh, dq, dk, dv, dipre, dfpre, dC0, dn0, dm0,
                        workspace, stream=None) -> None:
    """Gradients of a loss with respect to q, k, v [B, NH, T, D] (bf16), ipre, fpre [B, NH, T] and the
    initial state (C0, n0, m0, or all None), given dh [B, NH, T, DV] (bf16), the loss's gradient with
    respect to the forward's output h~;
    outputs fp32 of the input shapes, dC0/dn0/dm0 all None when not wanted; workspace: uint8 tensor
    of mlstm_chunkwise_bwd_workspace_bytes bytes."""
    B, NH, T, DQK = q.shape
    DV = v.shape[3]
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib.mlstm_chunkwise_bwd(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(ipre), _ptr(fpre), _ptr(C0),
                                   _ptr(n0), _ptr(m0), B, NH, T, DQK, DV, L, _ptr(dh), _ptr(dq), _ptr(dk),
                                   _ptr(dv), _ptr(dipre), _ptr(dfpre), _ptr(dC0), _ptr(dn0), _ptr(dm0),
                                   _ptr(workspace), ws_bytes, _stream(stream)))
