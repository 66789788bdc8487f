"""libmlstm: the mLSTM matrix-memory cell of xLSTM 7B (arXiv 2503.13427) on MI355X (gfx950).

The compute path is the C-ABI library ``libmlstm.so`` (hand-written HIP
kernels); ``binding`` is a thin ctypes layer over it that only marshals
arguments.  Submodules:

* ``binding``     ``mlstm_chunkwise_fwd``, ``mlstm_step`` and friends (loads the library)
* ``inputs``      seeded synthetic input generator
* ``configs``     the five synthetic workloads
* ``accounting``  FLOP / byte counts for the roofline
* ``build``       compiles the HIP library for gfx950
"""
__version__ = "0.1.0"

_BINDING_NAMES = ("mlstm_chunkwise_fwd", "mlstm_chunkwise_workspace_bytes", "mlstm_step",
                  "mlstm_status_string", "mlstm_version", "MlstmError")


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
