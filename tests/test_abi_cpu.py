"""The C ABI on the host (no GPU): symbols, status strings, and argument validation.

Every call here is rejected by validation before anything is launched, so the
fake (aligned, never dereferenced) addresses are never touched.
"""
import ctypes
import os
import re

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mlstm.h")

from paper_2503_13427_amd import binding as Bd  # noqa: E402

lib = Bd.lib


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mlstm_[a-z_]+)\s*\(", src)))


def test_header_declares_expected_entry_points():
    assert declared_functions() == sorted(["mlstm_chunkwise_fwd", "mlstm_chunkwise_workspace_bytes", "mlstm_step",
                                           "mlstm_chunkwise_fwd_noalloc", "mlstm_chunkwise_scratch_bytes",
                                           "mlstm_chunkwise_fwd_strided",
                                           "mlstm_step_output", "mlstm_chunkwise_bwd",
                                           "mlstm_chunkwise_bwd_workspace_bytes",
                                           "mlstm_output_norm", "mlstm_output_norm_tokens", "mlstm_gate_preact", "mlstm_parallel_bwd",
                                           "mlstm_parallel_bwd_workspace_bytes", "mlstm_status_string",
                                           "mlstm_version", "mlstm_debug_flags"])


@pytest.mark.parametrize("name", declared_functions())
def test_library_exports_every_declared_symbol(name):
    assert hasattr(lib, name)


def test_default_build_reports_no_debug_checks():
    """The default library carries no device bounds checks and says so without touching a device."""
    if os.path.basename(Bd.LIB_PATH) != "libmlstm.so":
        pytest.skip("another build of the library is loaded")
    assert Bd.mlstm_debug_flags() == Bd.MLSTM_DEBUG_NOT_BUILT


@pytest.mark.skipif(not os.path.exists(os.path.join(ROOT, "paper_2503_13427_amd", "libmlstm_debug.so")),
                    reason="libmlstm_debug.so is not built")
def test_debug_build_exports_every_declared_symbol():
    path = os.path.join(ROOT, "paper_2503_13427_amd", "libmlstm_debug.so")
    dbg = ctypes.CDLL(path)
    out = os.popen(f"nm -D --defined-only {path}").read()
    for name in declared_functions():
        assert hasattr(dbg, name), name
        assert re.search(rf"\bT {name}$", out, flags=re.M), name


def test_status_strings_and_version():
    for code, name in Bd.STATUS_NAMES.items():
        assert Bd.mlstm_status_string(code).startswith(name)
    assert Bd.mlstm_status_string(99) == "MLSTM_UNKNOWN_STATUS"
    assert Bd.mlstm_version() == 100


# ---- prefill validation --------------------------------------------------------------------------

BASE = 1 << 40           # fake, 16-byte aligned addresses, far apart
GAP = 1 << 34


def fake(i, off=0):
    return BASE + i * GAP + off


def chunk_args(**over):
    a = dict(q=fake(0), k=fake(1), v=fake(2), dt=Bd.MLSTM_BF16, ipre=fake(3), fpre=fake(4), C0=None, n0=None,
             m0=None, B=1, NH=8, T=256, DQK=256, DV=512, L=64, h=fake(5), CT=fake(6), nT=fake(7), mT=fake(8),
             ws=None, ws_bytes=0, stream=None)
    a.update(over)
    return a


def call_chunk(a):
    return lib.mlstm_chunkwise_fwd(a["q"], a["k"], a["v"], a["dt"], a["ipre"], a["fpre"], a["C0"], a["n0"],
                                   a["m0"], a["B"], a["NH"], a["T"], a["DQK"], a["DV"], a["L"], a["h"], a["CT"],
                                   a["nT"], a["mT"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("field", ["q", "k", "v", "ipre", "fpre", "h", "CT", "nT", "mT"])
def test_chunk_null_pointer(field):
    assert call_chunk(chunk_args(**{field: None})) == 1


def test_chunk_empty_sequence_needs_only_state_pointers():
    # T == 0 with a NULL q is not a NULL-pointer error; a NULL CT still is
    assert call_chunk(chunk_args(T=0, q=None, CT=None)) == 1
    a = chunk_args(T=0, q=None, k=None, v=None, ipre=None, fpre=None, h=None)
    a["mT"] = a["nT"] + 16     # overlapping outputs: rejected by validation, nothing launched
    assert call_chunk(a) == 5


@pytest.mark.parametrize("given", [("C0",), ("n0",), ("m0",), ("C0", "n0")])
def test_chunk_partial_initial_state(given):
    over = {g: fake(10 + i) for i, g in enumerate(given)}
    assert call_chunk(chunk_args(**over)) == 1


@pytest.mark.parametrize("over", [dict(B=0), dict(NH=-1), dict(T=-64), dict(DQK=0), dict(DV=0), dict(L=0)])
def test_chunk_bad_shape(over):
    assert call_chunk(chunk_args(**over)) == 2


@pytest.mark.parametrize("over", [dict(dt=7), dict(dt=Bd.MLSTM_BF16, DQK=96, DV=100, L=64, T=128),
                                  dict(dt=Bd.MLSTM_F32, DQK=4096, DV=4096, L=64, T=128)])
def test_chunk_unsupported(over):
    assert call_chunk(chunk_args(**over)) == 3


@pytest.mark.parametrize("field", ["q", "v", "ipre", "h", "CT", "mT"])
def test_chunk_misaligned(field):
    a = chunk_args()
    a[field] = a[field] + 2
    assert call_chunk(a) == 4


@pytest.mark.parametrize("out,inp", [("h", "q"), ("CT", "v"), ("nT", "fpre"), ("h", "CT"), ("mT", "nT")])
def test_chunk_alias(out, inp):
    a = chunk_args()
    a[out] = a[inp] + 16
    assert call_chunk(a) == 5


def test_chunk_alias_with_initial_state():
    a = chunk_args(C0=fake(10), n0=fake(11), m0=fake(12))
    a["CT"] = a["C0"]
    assert call_chunk(a) == 5


def test_chunk_workspace_without_pointer():
    assert call_chunk(chunk_args(ws=None, ws_bytes=1024)) == 1


def test_workspace_query_is_pure_host():
    assert lib.mlstm_chunkwise_workspace_bytes(1, 8, 100, 256, 512, 64, Bd.MLSTM_BF16) == 0   # 2 chunks: 1 segment
    # a partial last chunk counts as a chunk: 16 chunks of 64 for T = 1000, 8 segments
    assert lib.mlstm_chunkwise_workspace_bytes(1, 8, 1000, 256, 512, 64, Bd.MLSTM_BF16) > 0
    assert lib.mlstm_chunkwise_workspace_bytes(1, 1, 64, 16, 16, 16, Bd.MLSTM_F32) == 0       # fp32 kernel


# ---- step validation -----------------------------------------------------------------------------

def step_args(**over):
    a = dict(q=fake(0), k=fake(1), v=fake(2), dt=Bd.MLSTM_BF16, ipre=fake(3), fpre=fake(4), C=fake(5), n=fake(6),
             m=fake(7), B=256, NH=8, DQK=256, DV=512, h=fake(8), Co=fake(9), no=fake(10), mo=fake(11), stream=None)
    a.update(over)
    return a


def call_step(a):
    return lib.mlstm_step(a["q"], a["k"], a["v"], a["dt"], a["ipre"], a["fpre"], a["C"], a["n"], a["m"], a["B"],
                          a["NH"], a["DQK"], a["DV"], a["h"], a["Co"], a["no"], a["mo"], a["stream"])


@pytest.mark.parametrize("field", ["q", "k", "v", "ipre", "fpre", "C", "n", "m", "h", "Co", "no", "mo"])
def test_step_null_pointer(field):
    assert call_step(step_args(**{field: None})) == 1


@pytest.mark.parametrize("over", [dict(B=0), dict(NH=0), dict(DQK=0), dict(DV=6), dict(DV=0)])
def test_step_bad_shape(over):
    assert call_step(step_args(**over)) == 2


@pytest.mark.parametrize("over", [dict(dt=3), dict(DQK=8192, DV=4), dict(DQK=2048, DV=1024)])
def test_step_unsupported(over):
    assert call_step(step_args(**over)) == 3


def test_step_misaligned():
    a = step_args()
    a["C"] += 4
    assert call_step(a) == 4


@pytest.mark.parametrize("out,inp,off", [("Co", "C", 16), ("no", "n", 64), ("mo", "m", 4 * 16), ("h", "v", 0),
                                         ("Co", "q", 0), ("no", "C", 0), ("h", "Co", 0)])
def test_step_alias(out, inp, off):
    a = step_args()
    a[out] = a[inp] + off
    assert call_step(a) == 5


# ---- output gate + norm validation ---------------------------------------------------------------

def norm_args(**over):
    a = dict(x=fake(0), o=fake(1), dt=Bd.MLSTM_BF16, w=fake(2), b=fake(3), eps=1e-6, norm=Bd.MLSTM_NORM_LAYER,
             B=1, NH=8, T=2048, DV=512, h=fake(4), stream=None)
    a.update(over)
    return a


def call_norm(a):
    return lib.mlstm_output_norm(a["x"], a["o"], a["dt"], a["w"], a["b"], a["eps"], a["norm"], a["B"], a["NH"],
                                 a["T"], a["DV"], a["h"], a["stream"])


@pytest.mark.parametrize("field", ["x", "o", "h"])
def test_norm_null_pointer(field):
    assert call_norm(norm_args(**{field: None})) == 1


def test_norm_empty_rows_is_ok_without_pointers():
    # T == 0: nothing to do, no row pointer needed, nothing launched
    assert call_norm(norm_args(T=0, x=None, o=None, h=None)) == 0


@pytest.mark.parametrize("over", [dict(B=0), dict(NH=-1), dict(T=-1), dict(DV=0), dict(eps=0.0), dict(eps=-1e-6),
                                  dict(eps=float("nan")), dict(eps=float("inf")), dict(norm=2)])
def test_norm_bad_shape(over):
    assert call_norm(norm_args(**over)) == 2


@pytest.mark.parametrize("over", [dict(dt=3), dict(DV=6), dict(DV=4096)])
def test_norm_unsupported(over):
    assert call_norm(norm_args(**over)) == 3


@pytest.mark.parametrize("field", ["x", "o", "w", "b", "h"])
def test_norm_misaligned(field):
    a = norm_args()
    a[field] += 8
    assert call_norm(a) == 4


# ---- the token-major output norm: the same checks plus the o~ token stride -----------------------

def call_norm_tokens(a, stride=None):
    ostride = 4 * a["NH"] * a["DV"] if stride is None else stride
    return lib.mlstm_output_norm_tokens(a["x"], a["o"], ostride, a["dt"], a["w"], a["b"], a["eps"], a["norm"],
                                        a["B"], a["NH"], a["T"], a["DV"], a["h"], a["stream"])


@pytest.mark.parametrize("field", ["x", "o", "h"])
def test_norm_tokens_null_pointer(field):
    assert call_norm_tokens(norm_args(**{field: None})) == 1


def test_norm_tokens_empty_rows_is_ok_without_pointers():
    assert call_norm_tokens(norm_args(T=0, x=None, o=None, h=None)) == 0


@pytest.mark.parametrize("over", [dict(B=0), dict(NH=-1), dict(DV=0), dict(eps=0.0), dict(norm=2)])
def test_norm_tokens_bad_shape(over):
    assert call_norm_tokens(norm_args(**over)) == 2


@pytest.mark.parametrize("stride", [8 * 512 - 4, 8 * 512 + 2, -4, 0])
def test_norm_tokens_bad_stride(stride):
    # the o~ rows of one token would overlap, or rows would lose their 4-element alignment
    assert call_norm_tokens(norm_args(), stride) == 2


@pytest.mark.parametrize("over", [dict(dt=3), dict(DV=6), dict(DV=4096)])
def test_norm_tokens_unsupported(over):
    assert call_norm_tokens(norm_args(**over)) == 3


@pytest.mark.parametrize("field", ["x", "o", "w", "b", "h"])
def test_norm_tokens_misaligned(field):
    a = norm_args()
    a[field] += 8
    assert call_norm_tokens(a) == 4


def test_norm_tokens_output_may_not_overlap_inputs():
    # unlike the head-major call, y may not be h~ itself: the two layouts differ
    a = norm_args()
    a["h"] = a["x"]
    assert call_norm_tokens(a) == 5


@pytest.mark.parametrize("inp,off", [("x", 16), ("o", 0), ("o", 4096), ("w", 0), ("b", 16)])
def test_norm_alias(inp, off):
    a = norm_args()
    a["h"] = a[inp] + off
    assert call_norm(a) == 5


# ---- gate pre-activation validation ------------------------------------------------------------

def gate_args(**over):
    a = dict(x=fake(0), dt=Bd.MLSTM_BF16, w=fake(1), b=fake(2), cap=15.0, border=fake(3), B=2, T=2048, d=4096,
             NH=8, ip=fake(4), fp=fake(5), stream=None)
    a.update(over)
    return a


def call_gate(a):
    return lib.mlstm_gate_preact(a["x"], a["dt"], a["w"], a["b"], a["cap"], a["border"], a["B"], a["T"], a["d"],
                                 a["NH"], a["ip"], a["fp"], a["stream"])


@pytest.mark.parametrize("field", ["x", "w", "ip", "fp"])
def test_gate_null_pointer(field):
    assert call_gate(gate_args(**{field: None})) == 1


def test_gate_optional_pointers_and_empty_batch():
    # bias and border are optional; B T == 0 needs no pointer and launches nothing
    assert call_gate(gate_args(B=0, x=None, w=None, ip=None, fp=None)) == 0
    assert call_gate(gate_args(T=0, x=None, w=None, ip=None, fp=None, b=None, border=None)) == 0


@pytest.mark.parametrize("over", [dict(B=-1), dict(T=-1), dict(d=0), dict(NH=0), dict(cap=-1.0),
                                  dict(cap=float("nan")), dict(cap=float("inf"))])
def test_gate_bad_shape(over):
    assert call_gate(gate_args(**over)) == 2


@pytest.mark.parametrize("over", [dict(dt=Bd.MLSTM_F32), dict(d=4000), dict(d=64), dict(NH=33)])
def test_gate_unsupported(over):
    assert call_gate(gate_args(**over)) == 3


@pytest.mark.parametrize("field", ["x", "w", "b", "border", "ip", "fp"])
def test_gate_misaligned(field):
    a = gate_args()
    a[field] += 4
    assert call_gate(a) == 4


@pytest.mark.parametrize("out,inp,off", [("fp", "ip", 16), ("ip", "x", 4096), ("fp", "w", 0), ("ip", "b", 0),
                                         ("fp", "border", 16)])
def test_gate_alias(out, inp, off):
    a = gate_args()
    a[out] = a[inp] + off
    assert call_gate(a) == 5


# ---- backward validation -------------------------------------------------------------------------

def bwd_args(**over):
    a = dict(q=fake(0), k=fake(1), v=fake(2), dt=Bd.MLSTM_BF16, ip=fake(3), fp=fake(4), dh=fake(5), B=1, NH=8,
             T=2048, DQK=256, DV=512, dq=fake(6), dk=fake(7), dv=fake(8), di=fake(9), df=fake(10), ws=fake(11),
             ws_bytes=1 << 30, stream=None)
    a.update(over)
    return a


def call_bwd(a):
    return lib.mlstm_parallel_bwd(a["q"], a["k"], a["v"], a["dt"], a["ip"], a["fp"], a["dh"], a["B"], a["NH"], a["T"],
                                  a["DQK"], a["DV"], a["dq"], a["dk"], a["dv"], a["di"], a["df"], a["ws"],
                                  a["ws_bytes"], a["stream"])


def test_bwd_workspace_size():
    # per sequence: five fp32 vectors of T (rounded up to four floats) and dN~ [T][DV]
    assert lib.mlstm_parallel_bwd_workspace_bytes(2, 8, 100, 512) == 2 * 8 * (500 + 100 * 512) * 4
    assert lib.mlstm_parallel_bwd_workspace_bytes(1, 1, 3, 16) == (16 + 3 * 16) * 4
    assert lib.mlstm_parallel_bwd_workspace_bytes(0, 8, 100, 512) == 0


@pytest.mark.parametrize("field", ["q", "k", "v", "ip", "fp", "dh", "dq", "dk", "dv", "di", "df", "ws"])
def test_bwd_null_pointer(field):
    assert call_bwd(bwd_args(**{field: None})) == 1


def test_bwd_empty_sequence_is_ok_without_pointers():
    assert call_bwd(bwd_args(T=0, q=None, k=None, v=None, dh=None, dq=None, ws=None, ws_bytes=0)) == 0


@pytest.mark.parametrize("over", [dict(B=0), dict(NH=-1), dict(T=-1), dict(DQK=0), dict(DV=0)])
def test_bwd_bad_shape(over):
    assert call_bwd(bwd_args(**over)) == 2


@pytest.mark.parametrize("over", [dict(dt=3), dict(DQK=24), dict(DV=520), dict(DQK=272), dict(DV=1024)])
def test_bwd_unsupported(over):
    assert call_bwd(bwd_args(**over)) == 3


def test_bwd_workspace_too_small():
    need = lib.mlstm_parallel_bwd_workspace_bytes(1, 8, 2048, 512)
    assert call_bwd(bwd_args(ws_bytes=need - 1)) == 6
    # enough workspace passes that check and stops at the next one (no call here may launch)
    assert call_bwd(bwd_args(ws_bytes=need, q=fake(0, 4))) == 4


@pytest.mark.parametrize("field", ["q", "dh", "dq", "df", "ws"])
def test_bwd_misaligned(field):
    a = bwd_args()
    a[field] += 4
    assert call_bwd(a) == 4


@pytest.mark.parametrize("out,other,off", [("dq", "q", 0), ("dv", "dh", 4096), ("dk", "dq", 16), ("df", "di", 0),
                                           ("ws", "dv", 64), ("di", "ip", 0)])
def test_bwd_alias(out, other, off):
    a = bwd_args()
    a[out] = a[other] + off
    assert call_bwd(a) == 5


# ---- the no-allocation prefill (fixed device scratch) ---------------------------------------------

def call_chunk_noalloc(a):
    return lib.mlstm_chunkwise_fwd_noalloc(a["q"], a["k"], a["v"], a["dt"], a["ipre"], a["fpre"], a["C0"], a["n0"],
                                           a["m0"], a["B"], a["NH"], a["T"], a["DQK"], a["DV"], a["L"], a["h"],
                                           a["CT"], a["nT"], a["mT"], a["stream"])


def test_noalloc_scratch_size():
    assert Bd.mlstm_chunkwise_scratch_bytes() == 64 << 20


def test_noalloc_rejects_a_schedule_larger_than_the_scratch():
    """The B=4 x T=32768 prefill's segment schedule needs 67.2 MB of slots, more than the 64 MiB
    scratch: rejected on the host, nothing launched."""
    a = chunk_args(B=4, NH=8, T=32768, L=128)
    assert Bd.mlstm_chunkwise_workspace_bytes(4, 8, 32768, 256, 512, 128) > Bd.mlstm_chunkwise_scratch_bytes()
    assert call_chunk_noalloc(a) == 6
    assert "scratch" in Bd.mlstm_status_string(6)


@pytest.mark.parametrize("field", ["q", "fpre", "h", "mT"])
def test_noalloc_validates_like_the_workspace_entry_point(field):
    assert call_chunk_noalloc(chunk_args(**{field: None})) == 1
    a = chunk_args()
    a[field] = a[field] + 2
    assert call_chunk_noalloc(a) == 4
    assert call_chunk_noalloc(chunk_args(B=0)) == 2
    assert call_chunk_noalloc(chunk_args(h=fake(1, 64))) == 5


# ---- strided q, k, v ------------------------------------------------------------------------------

def proj_strides(B=1, NH=8, T=256, DQK=256, DV=512):
    """q, k, v as per-head views of one projection output [B, T, NH * (2 DQK + DV)] (element strides)."""
    row = NH * (2 * DQK + DV)
    return [T * row, DQK, row, T * row, DQK, row, T * row, DV, row]


def call_strided(a, st):
    arr = None if st is None else (ctypes.c_int64 * 9)(*st)
    return lib.mlstm_chunkwise_fwd_strided(a["q"], a["k"], a["v"], arr, a["dt"], a["ipre"], a["fpre"], a["C0"],
                                           a["n0"], a["m0"], a["B"], a["NH"], a["T"], a["DQK"], a["DV"], a["L"],
                                           a["h"], a["CT"], a["nT"], a["mT"], a["ws"], a["ws_bytes"], a["stream"])


def test_strided_null_strides_and_pointers():
    assert call_strided(chunk_args(), None) == 1
    assert call_strided(chunk_args(k=None), proj_strides()) == 1


@pytest.mark.parametrize("i,val,status", [(2, 4100, 4), (0, 8 * 3 + 4, 4), (4, -256, 2), (5, 248, 2), (8, 504, 2),
                                          (2, 1 << 24, 3)])
def test_strided_stride_checks(i, val, status):
    """A stride that is not a multiple of 8 elements is misaligned; a negative one, or a token stride
    under D (rows that overlap), is a bad shape; a sequence whose rows (plus the rows a partial last
    chunk reads past its end) span 2^31 bytes or more is unsupported."""
    st = proj_strides()
    st[i] = val
    assert call_strided(chunk_args(), st) == status


def test_strided_span_bound_counts_the_padding_rows():
    # T = 1 with a token stride of 2^23 elements: the row itself fits, the 127 padding rows do not
    st = proj_strides(T=1)
    st[2] = 1 << 23
    assert call_strided(chunk_args(T=1), st) == 3
    st[2] = (1 << 23) - 8
    a = chunk_args(T=1)
    a["h"] = a["CT"]                   # within the bound: validation goes on to the alias checks
    assert call_strided(a, st) == 5


@pytest.mark.parametrize("over", [dict(dt=Bd.MLSTM_F32), dict(DQK=128, DV=128, L=64), dict(L=32),
                                  dict(B=1 << 20, NH=64, T=64)])
def test_strided_unsupported_shapes(over):
    st = proj_strides(DQK=over.get("DQK", 256), DV=over.get("DV", 512))
    assert call_strided(chunk_args(**over), st) == 3


def test_strided_alias_covers_the_view_extent():
    """h placed past q's contiguous size but inside the range its strided view spans is an alias."""
    a = chunk_args()
    nq = 1 * 8 * 256 * 256
    a["h"] = a["q"] + 2 * nq * 2      # 2 nq elements in: beyond [B, NH, T, DQK], inside the strided view
    assert call_strided(a, proj_strides()) == 5


# ---- the decode step with the output epilogue ----------------------------------------------------

def step_out_args(**over):
    a = dict(q=fake(0), k=fake(1), v=fake(2), dt=Bd.MLSTM_BF16, ipre=fake(3), fpre=fake(4), C=fake(5), n=fake(6),
             m=fake(7), o=fake(8), w=fake(9), b=fake(10), eps=1e-6, norm=0, B=2, NH=8, DQK=256, DV=512, h=fake(11),
             Co=fake(5), no=fake(6), mo=fake(7), stream=None)
    a.update(over)
    return a


def call_step_out(a):
    return lib.mlstm_step_output(a["q"], a["k"], a["v"], a["dt"], a["ipre"], a["fpre"], a["C"], a["n"], a["m"], a["o"],
                                 a["w"], a["b"], ctypes.c_float(a["eps"]), a["norm"], a["B"], a["NH"], a["DQK"],
                                 a["DV"], a["h"], a["Co"], a["no"], a["mo"], a["stream"])


@pytest.mark.parametrize("over,status", [
    (dict(o=None), 1), (dict(q=None), 1), (dict(eps=0.0), 2), (dict(eps=float("nan")), 2), (dict(norm=5), 2),
    (dict(DV=4096, DQK=64), 3), (dict(DV=6), 2), (dict(o=fake(8, 2)), 4), (dict(w=fake(9, 4)), 4),
    (dict(h=fake(8, 16)), 5), (dict(h=fake(9, 64)), 5), (dict(Co=fake(8)), 5)])
def test_step_output_validation(over, status):
    assert call_step_out(step_out_args(**over)) == status


# ---- the chunkwise backward ----------------------------------------------------------------------

def cbwd_args(**over):
    a = dict(q=fake(0), k=fake(1), v=fake(2), dt=Bd.MLSTM_BF16, ip=fake(3), fp=fake(4), C0=None, n0=None, m0=None,
             B=1, NH=8, T=2048, DQK=256, DV=512, L=64, dh=fake(6), dq=fake(7), dk=fake(8), dv=fake(9),
             di=fake(10), df=fake(11), dC0=None, dn0=None, dm0=None, ws=fake(12), ws_bytes=1 << 40, stream=None)
    a.update(over)
    return a


def call_cbwd(a):
    return lib.mlstm_chunkwise_bwd(a["q"], a["k"], a["v"], a["dt"], a["ip"], a["fp"], a["C0"], a["n0"], a["m0"],
                                   a["B"], a["NH"], a["T"], a["DQK"], a["DV"], a["L"], a["dh"], a["dq"],
                                   a["dk"], a["dv"], a["di"], a["df"], a["dC0"], a["dn0"], a["dm0"], a["ws"],
                                   a["ws_bytes"], a["stream"])


def test_chunk_bwd_workspace_size():
    """Slots of every chunk but the first (n, m, then L_c, z_c); the segment slots of the walk (32
    sequence-tile workgroups per segment, so eight segments of four chunks: seven segment slots per
    sequence); the four dv tiles' partial sums of X; Gam_c in bf16; L_0, gam per chunk,
    per-token key weights and partial sums, per-chunk decays, dm0 partial sums; each region 256-byte
    aligned."""
    al = lambda b: (b + 255) // 256 * 256
    S, T, NC = 8, 2048, 32
    slot = 256 * 512 + 256 + 4
    want = (al(S * (NC - 1) * slot * 4) + al(S * 7 * slot * 4) + al(4 * S * T * 256 * 4)
            + al(S * (NC - 1) * 256 * 512 * 2)
            + al(S * (256 * 512 + 256) * 4)
            + al(S * NC * 256 * 4) + al(S * T * 4) + al(S * T * 32) + al(S * NC * 4) + al(S * 129 * 4))
    assert Bd.mlstm_chunkwise_bwd_workspace_bytes(1, 8, T, 256, 512, 64) == want
    assert Bd.mlstm_chunkwise_bwd_workspace_bytes(1, 8, T, 256, 512, 128) == 0
    assert Bd.mlstm_chunkwise_bwd_workspace_bytes(1, 8, T, 256, 512, 64, torch.float32) == 0


@pytest.mark.parametrize("field", ["q", "k", "v", "ip", "fp", "dh", "dq", "dk", "dv", "di", "df", "ws"])
def test_chunk_bwd_null_pointer(field):
    assert call_cbwd(cbwd_args(**{field: None})) == 1


@pytest.mark.parametrize("over", [dict(C0=fake(13)), dict(C0=fake(13), n0=fake(14)), dict(dC0=fake(13)),
                                  dict(dn0=fake(13), dm0=fake(14))])
def test_chunk_bwd_partial_state_triples(over):
    assert call_cbwd(cbwd_args(**over)) == 1


def test_chunk_bwd_empty_sequence_is_ok_without_pointers():
    assert call_cbwd(cbwd_args(T=0, q=None, k=None, v=None, dh=None, dq=None, ws=None, ws_bytes=0)) == 0


@pytest.mark.parametrize("over", [dict(B=0), dict(NH=-1), dict(T=-1), dict(DQK=0), dict(DV=0), dict(L=0)])
def test_chunk_bwd_bad_shape(over):
    assert call_cbwd(cbwd_args(**over)) == 2


@pytest.mark.parametrize("over", [dict(dt=3), dict(dt=Bd.MLSTM_F32), dict(DQK=128), dict(DV=256), dict(L=128),
                                  dict(B=65536, NH=1), dict(T=1 << 21)])
def test_chunk_bwd_unsupported(over):
    assert call_cbwd(cbwd_args(**over)) == 3


def test_chunk_bwd_workspace_too_small():
    need = Bd.mlstm_chunkwise_bwd_workspace_bytes(1, 8, 2048, 256, 512, 64)
    assert call_cbwd(cbwd_args(ws_bytes=need - 1)) == 6
    assert call_cbwd(cbwd_args(ws_bytes=need, q=fake(0, 4))) == 4


@pytest.mark.parametrize("field", ["q", "dh", "dq", "df", "ws"])
def test_chunk_bwd_misaligned(field):
    a = cbwd_args()
    a[field] += 4
    assert call_cbwd(a) == 4


@pytest.mark.parametrize("out,other,off", [("dq", "q", 0), ("dv", "dh", 4096), ("dk", "dq", 16), ("df", "di", 0),
                                           ("ws", "dv", 64), ("di", "ip", 0), ("dq", "k", 1024)])
def test_chunk_bwd_alias(out, other, off):
    a = cbwd_args()
    a[out] = a[other] + off
    assert call_cbwd(a) == 5


def test_chunk_bwd_state_gradient_alias():
    a = cbwd_args(C0=fake(13), n0=fake(14), m0=fake(15), dC0=fake(13, 64), dn0=fake(16), dm0=fake(17))
    assert call_cbwd(a) == 5
