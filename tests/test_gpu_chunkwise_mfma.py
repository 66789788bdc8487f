"""mlstm_chunkwise_fwd on the bf16 MFMA kernel (DQK=256, DV=512, L in {64, 128}) against the
fp64 recurrent oracle.

Parity bar: max relative error <= 2e-2 per row (each h row of one (batch, head, step), each
d-row of the final C; bf16 q/k/v/h, fp32 state).  Covers several chunks and segments, an initial state, the
floor branch, short and long memory, the soft-capped gates, T = 0, a partial last chunk
(T not a multiple of L: no h row beyond T is written), the segment-parallel schedule
(workspace), document resets (f~ = -inf) at chunk edges, consecutive tokens, segment starts
and packed-document borders, chunk-size independence, state carry, decode steps == prefill,
run-to-run determinism, and the three prefill workloads at full size, every head checked.
"""
import numpy as np
import pytest
import torch

from oracle import coracle
from paper_2503_13427_amd import configs
from paper_2503_13427_amd.inputs import GateDist, StateDist, make_prefill
from tests.helpers import (TOL_BF16, alloc_prefill_outputs, host_f64, row_err, state_errs, subset, upload_prefill)

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def run(inp, L, workspace=True, dev_inputs=None):
    d = dev_inputs or upload_prefill(inp)
    o = alloc_prefill_outputs(inp)
    ws = None
    if workspace:
        nb = _mb().mlstm_chunkwise_workspace_bytes(inp.B, inp.NH, inp.T, inp.DQK, inp.DV, L)
        if nb:
            ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    _mb().mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], L,
                              o["h"], o["CT"], o["nT"], o["mT"], workspace=ws)
    torch.cuda.synchronize()
    return o


def check(inp, o, heads=None, label=""):
    """Compare device outputs with the oracle; ``heads`` selects global head indices (then
    ``inp`` must be the matching subset drawn with the same heads)."""
    S_all = o["h"].shape[0] * o["h"].shape[1]
    hr, Cr, nr, mr = coracle.recurrent_inputs(inp)
    sel = np.arange(S_all) if heads is None else np.asarray(heads)
    idx = torch.from_numpy(sel).cuda()
    T = o["h"].shape[2]
    h = host_f64(o["h"].reshape(S_all, T, -1).index_select(0, idx))
    C = host_f64(o["CT"].reshape(S_all, 256, 512).index_select(0, idx))
    n = host_f64(o["nT"].reshape(S_all, 256).index_select(0, idx))
    m = host_f64(o["mT"].reshape(S_all).index_select(0, idx))
    eh = row_err(h, hr, 512, f"{label} h")
    eC, en, em = state_errs(C, n, m, Cr, nr, mr, label)
    print(f"{label} max row errors: h {eh:.3e} C {eC:.3e} n {en:.3e} m {em:.3e}")
    assert np.isfinite(h).all()
    assert eh <= TOL_BF16 and eC <= TOL_BF16 and en <= TOL_BF16 and em <= TOL_BF16, (eh, eC, en, em)
    return eh, eC, en, em


CASES = [
    # (B, NH, T, L, gates, state)
    (1, 2, 256, 64, GateDist(), None),
    (1, 2, 256, 128, GateDist(), None),
    (2, 1, 384, 64, GateDist(f_mu=5, f_sd=2, cap=15.0), StateDist()),
    (1, 2, 512, 128, GateDist(f_mu=5, f_sd=2, cap=15.0), StateDist()),
    (1, 2, 192, 64, GateDist(i_mu=-10.0), None),                 # floor branch active
    (1, 2, 256, 64, GateDist(f_mu=-1.0, f_sd=2.0), StateDist()),  # short memory
    (1, 1, 64, 64, GateDist(), StateDist()),                     # a single chunk
    (1, 1, 128, 128, GateDist(i_mu=2.0, i_sd=3.0), None),        # large input gates
    # partial last chunk
    (1, 2, 100, 64, GateDist(), None),
    (1, 1, 17, 64, GateDist(), StateDist()),                     # one partial chunk
    (1, 2, 300, 128, GateDist(f_mu=5, f_sd=2, cap=15.0), StateDist()),
    (1, 2, 1000, 64, GateDist(), StateDist()),                   # 8 segments, the last one ragged
    (1, 1, 700, 128, GateDist(), None),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c[0]}NH{c[1]}T{c[2]}L{c[3]}-{c[4]}-{c[5] is not None}")
@pytest.mark.parametrize("workspace", [False, True], ids=["fused", "segments"])
def test_mfma_matches_oracle(case, workspace):
    B, NH, T, L, g, st = case
    inp = make_prefill(workload=95, B=B, NH=NH, T=T, DQK=256, DV=512, dtype="bf16", gates=g, state=st)
    o = run(inp, L, workspace=workspace)
    check(inp, o, label=str(case))


def _edge_borders(T, L):
    """Restarts at the first token (drops an initial state), at the last and first rows of a
    chunk, on consecutive tokens, at a segment's start and at the last token."""
    pos = [0, L - 1, L, L + 1, 2 * L + 2, 2 * L + 3, T // 2, T - 1]
    return sorted({p for p in pos if 0 <= p < T})


RESET_CASES = [
    # (B, NH, T, L, gates, state, borders: "edges", "every" or a mean document length)
    (1, 2, 1000, 64, GateDist(), StateDist(), "edges"),
    (1, 2, 700, 128, GateDist(f_mu=5, f_sd=2, cap=15.0), StateDist(), "edges"),
    (1, 2, 2048, 64, GateDist(), None, 150.0),
    (2, 1, 3000, 128, GateDist(f_mu=5, f_sd=2, cap=15.0), StateDist(), 400.0),
    (1, 2, 4096, 64, GateDist(f_mu=5, f_sd=2, cap=15.0), None, 1500.0),   # few borders, long memory
    (1, 1, 256, 64, GateDist(), StateDist(), "every"),
]


@pytest.mark.parametrize("case", RESET_CASES, ids=lambda c: f"B{c[0]}NH{c[1]}T{c[2]}L{c[3]}-{c[6]}")
@pytest.mark.parametrize("workspace", [False, True], ids=["fused", "segments"])
def test_document_resets_match_oracle(case, workspace):
    """f~ = -inf at document borders (sequence packing, App. B): the state restarts there, in the
    chunk loop, in the local segment states and in their combination."""
    from paper_2503_13427_amd.inputs import pack_documents
    B, NH, T, L, g, st, borders = case
    inp = make_prefill(workload=98, B=B, NH=NH, T=T, DQK=256, DV=512, dtype="bf16", gates=g, state=st)
    if borders == "edges":
        inp.fpre[..., _edge_borders(T, L)] = -np.inf
    elif borders == "every":
        inp.fpre[...] = -np.inf
    else:
        pack_documents(inp, borders, workload=98)
    o = run(inp, L, workspace=workspace)
    check(inp, o, label=f"resets {case[:4]} {borders}")


@pytest.mark.parametrize("T,L", [(100, 64), (300, 128), (1000, 64)])
def test_partial_chunk_writes_no_row_beyond_T(T, L):
    """h is a view of the first T rows of a larger buffer: the rows after it keep their
    sentinel, and the chunk-size-independent result matches the oracle."""
    inp = make_prefill(workload=97, B=1, NH=1, T=T, DQK=256, DV=512, dtype="bf16", gates=GateDist(),
                       state=StateDist())
    d = upload_prefill(inp)
    o = alloc_prefill_outputs(inp)
    big = torch.full((T + 128, 512), -7.0, dtype=torch.bfloat16, device="cuda")
    h = big[:T].view(1, 1, T, 512)
    for workspace in (False, True):
        ws = None
        nb = _mb().mlstm_chunkwise_workspace_bytes(1, 1, T, 256, 512, L)
        if workspace and nb:
            ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        _mb().mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], L,
                                  h, o["CT"], o["nT"], o["mT"], workspace=ws)
        torch.cuda.synchronize()
        assert bool((big[T:] == -7.0).all()), "a row beyond T was written"
        check(inp, dict(h=h, CT=o["CT"], nT=o["nT"], mT=o["mT"]), label=f"T{T}L{L}ws{workspace}")


def test_segment_schedule_is_used_and_agrees():
    """The workload shape of the T=2048 prefill asks for a workspace; both schedules agree."""
    w = configs.PREFILL_T2048
    assert _mb().mlstm_chunkwise_workspace_bytes(w.B, w.NH, w.T, 256, 512, w.L) > 0
    inp = w.prefill_inputs(T=1024)
    a = run(inp, 64, workspace=False)
    b = run(inp, 64, workspace=True)
    assert row_err(host_f64(a["h"]), host_f64(b["h"]), 512, "fused vs segments") < TOL_BF16
    np.testing.assert_allclose(host_f64(a["mT"]), host_f64(b["mT"]), rtol=1e-5, atol=1e-5)


def test_workspace_too_small_is_rejected():
    w = configs.PREFILL_T2048
    inp = w.prefill_inputs(T=512)
    nb = _mb().mlstm_chunkwise_workspace_bytes(1, 8, 512, 256, 512, 64)
    assert nb > 0
    d = upload_prefill(inp)
    o = alloc_prefill_outputs(inp)
    ws = torch.empty(nb - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(_mb().MlstmError) as e:
        _mb().mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], None, None, None, 64,
                                  o["h"], o["CT"], o["nT"], o["mT"], workspace=ws)
    assert e.value.status == 6


def test_empty_sequence_mfma():
    inp = make_prefill(workload=96, B=1, NH=2, T=0, DQK=256, DV=512, dtype="bf16", gates=GateDist(),
                       state=StateDist())
    o = run(inp, 64)
    np.testing.assert_array_equal(host_f64(o["CT"]), inp.C0.astype(np.float64))
    np.testing.assert_array_equal(host_f64(o["nT"]), inp.n0.astype(np.float64))
    np.testing.assert_array_equal(host_f64(o["mT"]), inp.m0.astype(np.float64))


def test_chunk_size_independence_and_determinism():
    inp = make_prefill(workload=97, B=1, NH=2, T=512, DQK=256, DV=512, dtype="bf16", gates=GateDist(),
                       state=StateDist())
    a = run(inp, 64)
    b = run(inp, 128)
    c = run(inp, 64)
    assert row_err(host_f64(a["h"]), host_f64(b["h"]), 512, "L64 vs L128") < TOL_BF16
    np.testing.assert_allclose(host_f64(a["mT"]), host_f64(b["mT"]), rtol=1e-5, atol=1e-5)
    for k in a:
        assert torch.equal(a[k], c[k]), k


def test_state_carry():
    """prefill(T1) -> (C, n, m) -> prefill(T2) == prefill(T1 + T2), within the bf16 bar."""
    inp = make_prefill(workload=98, B=1, NH=2, T=512, DQK=256, DV=512, dtype="bf16", gates=GateDist(),
                       state=StateDist())
    d = upload_prefill(inp)
    full = run(inp, 64, dev_inputs=d)
    first = {k: (v[:, :, :256].contiguous() if k in ("q", "k", "v", "ipre", "fpre") else v) for k, v in d.items()}
    second = {k: (v[:, :, 256:].contiguous() if k in ("q", "k", "v", "ipre", "fpre") else v) for k, v in d.items()}
    o1 = alloc_prefill_outputs(make_prefill(workload=98, B=1, NH=2, T=256, DQK=256, DV=512, dtype="bf16",
                                            gates=GateDist()))
    mb = _mb()
    mb.mlstm_chunkwise_fwd(first["q"], first["k"], first["v"], first["ipre"], first["fpre"], d["C0"], d["n0"],
                           d["m0"], 64, o1["h"], o1["CT"], o1["nT"], o1["mT"])
    o2 = alloc_prefill_outputs(make_prefill(workload=98, B=1, NH=2, T=256, DQK=256, DV=512, dtype="bf16",
                                            gates=GateDist()))
    mb.mlstm_chunkwise_fwd(second["q"], second["k"], second["v"], second["ipre"], second["fpre"], o1["CT"],
                           o1["nT"], o1["mT"], 64, o2["h"], o2["CT"], o2["nT"], o2["mT"])
    torch.cuda.synchronize()
    h12 = torch.cat([o1["h"], o2["h"]], dim=2)
    assert row_err(host_f64(h12), host_f64(full["h"]), 512, "carried vs one call") < TOL_BF16
    eC, en, em = state_errs(host_f64(o2["CT"]).reshape(2, 256, 512), host_f64(o2["nT"]).reshape(2, 256),
                            host_f64(o2["mT"]).reshape(2), host_f64(full["CT"]).reshape(2, 256, 512),
                            host_f64(full["nT"]).reshape(2, 256), host_f64(full["mT"]).reshape(2))
    assert max(eC, en) < 1e-2 and em < 1e-5


def test_decode_steps_equal_prefill_bf16():
    """T steps of mlstm_step == mlstm_chunkwise_fwd over the same T tokens (both on the GPU)."""
    inp = make_prefill(workload=99, B=1, NH=2, T=128, DQK=256, DV=512, dtype="bf16", gates=GateDist(),
                       state=StateDist())
    d = upload_prefill(inp)
    pre = run(inp, 64, dev_inputs=d)
    C, n, m = d["C0"].clone(), d["n0"].clone(), d["m0"].clone()
    hs = []
    for t in range(inp.T):
        h = torch.empty(1, 2, 512, dtype=torch.bfloat16, device="cuda")
        _mb().mlstm_step(d["q"][:, :, t].contiguous(), d["k"][:, :, t].contiguous(), d["v"][:, :, t].contiguous(),
                         d["ipre"][:, :, t].contiguous(), d["fpre"][:, :, t].contiguous(), C, n, m, h, C, n, m)
        hs.append(h)
    torch.cuda.synchronize()
    hstep = host_f64(torch.stack(hs, dim=2))
    assert row_err(hstep, host_f64(pre["h"]), 512, "steps vs prefill") < TOL_BF16
    eC, en, em = state_errs(host_f64(C).reshape(2, 256, 512), host_f64(n).reshape(2, 256), host_f64(m).reshape(2),
                            host_f64(pre["CT"]).reshape(2, 256, 512), host_f64(pre["nT"]).reshape(2, 256),
                            host_f64(pre["mT"]).reshape(2))
    assert max(eC, en) < 1e-2 and em < 1e-5


# ---- the prefill workloads at full size -----------------------------------------------------------

def test_prefill_T2048_full():
    """B=1, NH=8, T=2048, L=64, zero state: every head against the oracle."""
    w = configs.PREFILL_T2048
    inp = w.prefill_inputs()
    o = run(inp, w.L)
    check(inp, o, label=w.name)


@pytest.mark.slow
@pytest.mark.parametrize("wl", [configs.PREFILL_T8192, configs.CONT_PREFILL_T32768], ids=lambda w: w.name)
def test_prefill_full_size_every_head(wl):
    """Full-size launch (every head on the GPU, the benchmark's launch configuration, workspace
    included); every head is checked against the oracle, eight at a time."""
    inp = wl.prefill_inputs()
    o = run(inp, wl.L)
    worst = [0.0] * 4
    for h0 in range(0, wl.heads, 8):
        heads = list(range(h0, min(wl.heads, h0 + 8)))
        errs = check(subset(inp, heads), o, heads=heads, label=f"{wl.name} heads {heads[0]}-{heads[-1]}")
        worst = [max(a, b) for a, b in zip(worst, errs)]
    print(f"{wl.name}: all {wl.heads} heads, max row errors h {worst[0]:.3e} C {worst[1]:.3e} "
          f"n {worst[2]:.3e} m {worst[3]:.3e}")


def test_maximum_sequence_length():
    """The longest sequence the MFMA prefill takes: T = 2^21 - 64, whose h spans just under the 2^31
    bytes a buffer resource addresses.  A document border every 4096 tokens makes every document a
    fresh run (App. B; pinned on the oracle), so sampled documents, including the ragged last one
    that ends at the last token, and the final state are checked against the oracle run on that
    document alone."""
    T = (1 << 21) - 64
    L, doc = 64, 4096
    assert T * 512 * 2 < (1 << 31) and (T + 64) * 512 * 2 >= (1 << 31)
    g = torch.Generator(device="cuda").manual_seed(90)
    q = torch.randn(1, 1, T, 256, generator=g, device="cuda").bfloat16()
    k = (torch.randn(1, 1, T, 256, generator=g, device="cuda") / 16).bfloat16()
    v = torch.randn(1, 1, T, 512, generator=g, device="cuda").bfloat16()
    ip = torch.randn(1, 1, T, generator=g, device="cuda")
    fp = torch.randn(1, 1, T, generator=g, device="cuda") + 3
    fp[..., ::doc] = float("-inf")
    h = torch.empty(1, 1, T, 512, dtype=torch.bfloat16, device="cuda")
    CT = torch.empty(1, 1, 256, 512, device="cuda")
    nT = torch.empty(1, 1, 256, device="cuda")
    mT = torch.empty(1, 1, device="cuda")
    nb = _mb().mlstm_chunkwise_workspace_bytes(1, 1, T, 256, 512, L)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    _mb().mlstm_chunkwise_fwd(q, k, v, ip, fp, None, None, None, L, h, CT, nT, mT, workspace=ws)
    torch.cuda.synchronize()
    starts = [0, doc * 257, (T - 1) // doc * doc]
    for s0 in starts:
        e0 = min(T, s0 + doc)
        sl = lambda x: host_f64(x[0, 0, s0:e0]).reshape(1, e0 - s0, -1)
        qd, kd, vd = sl(q), sl(k), sl(v)
        ipd, fpd = host_f64(ip[0, 0, s0:e0]).reshape(1, -1), host_f64(fp[0, 0, s0:e0]).reshape(1, -1)
        hr, Cr, nr, mr = coracle.recurrent(qd, kd, vd, ipd, fpd, None, None, None)
        eh = row_err(sl(h), hr, 512, f"T = {T}: document at {s0} ({e0 - s0} tokens): h")
        assert np.isfinite(sl(h)).all() and eh <= TOL_BF16
    eC, en, em = state_errs(host_f64(CT).reshape(1, 256, 512), host_f64(nT).reshape(1, 256), host_f64(mT).reshape(1),
                            Cr, nr, mr)
    print(f"final state: C {eC:.3e} n {en:.3e} m {em:.3e}")
    assert max(eC, en, em) <= TOL_BF16
