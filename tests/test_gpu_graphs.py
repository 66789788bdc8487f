"""The cell entry points captured in HIP graphs: mlstm_chunkwise_fwd on the segment schedule
(local-state, combine and chunkwise kernels with a workspace) and mlstm_step in place.

Each graph is replayed several times with new inputs copied into its static buffers and eager
work and synchronisations between replays; every replay must equal the eager call on the same
inputs bit for bit (same kernels, same data, no atomics).  No kernel of these calls clears
memory with a memset node: the workspace is written in full before it is read."""
import numpy as np
import pytest
import torch

from paper_2503_13427_amd import configs
from tests.helpers import host_f64

pytestmark = pytest.mark.gpu


def _mb():
    from paper_2503_13427_amd import binding
    return binding


def _prefill_buffers(B, NH, T, g):
    q = torch.randn(B, NH, T, 256, generator=g, device="cuda").bfloat16()
    k = torch.randn(B, NH, T, 256, generator=g, device="cuda").bfloat16()
    v = torch.randn(B, NH, T, 512, generator=g, device="cuda").bfloat16()
    ip = torch.randn(B, NH, T, generator=g, device="cuda")
    fp = torch.randn(B, NH, T, generator=g, device="cuda") + 3
    return q, k, v, ip, fp


def test_prefill_graph_replays_match_eager():
    mb = _mb()
    w = configs.PREFILL_T2048
    B, NH, T, L = w.B, w.NH, w.T, w.L
    g = torch.Generator(device="cuda").manual_seed(31)
    ins = _prefill_buffers(B, NH, T, g)
    outs = (torch.empty(B, NH, T, 512, dtype=torch.bfloat16, device="cuda"), torch.empty(B, NH, 256, 512, device="cuda"),
            torch.empty(B, NH, 256, device="cuda"), torch.empty(B, NH, device="cuda"))
    ws = torch.empty(mb.mlstm_chunkwise_workspace_bytes(B, NH, T, 256, 512, L), dtype=torch.uint8, device="cuda")
    assert ws.numel() > 0   # the segment schedule: three kernels per call
    call = lambda i, o: mb.mlstm_chunkwise_fwd(*i, None, None, None, L, *o, workspace=ws)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(ins, outs)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(ins, outs)
    for r in range(3):
        new = _prefill_buffers(B, NH, T, g)
        for dst, src in zip(ins, new):
            dst.copy_(src)
        graph.replay()
        got = [o.clone() for o in outs]
        torch.randn(1 << 20, device="cuda").sum()                     # eager work between replays
        torch.cuda.synchronize()
        call(ins, outs)                                               # the eager call on the same inputs
        torch.cuda.synchronize()
        for a, b in zip(got, outs):
            assert torch.equal(a, b), f"replay {r}"
        print(f"prefill graph replay {r}: equal, h max {host_f64(got[0]).max():.3f}")


def test_step_graph_replays_match_eager():
    mb = _mb()
    B, NH = 1, 8
    g = torch.Generator(device="cuda").manual_seed(32)
    mk = lambda: (torch.randn(B, NH, 256, generator=g, device="cuda").bfloat16(),
                  torch.randn(B, NH, 256, generator=g, device="cuda").bfloat16(),
                  torch.randn(B, NH, 512, generator=g, device="cuda").bfloat16(),
                  torch.randn(B, NH, generator=g, device="cuda"), torch.randn(B, NH, generator=g, device="cuda") + 3)
    ins = mk()
    st = (torch.randn(B, NH, 256, 512, generator=g, device="cuda") * 0.1,
          torch.randn(B, NH, 256, generator=g, device="cuda").abs(), torch.zeros(B, NH, device="cuda"))
    st_e = tuple(t.clone() for t in st)
    h = torch.empty(B, NH, 512, dtype=torch.bfloat16, device="cuda")
    h_e = torch.empty_like(h)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        mb.mlstm_step(*ins, *st, h, *st)                              # in place, column-split launch
    for r in range(4):
        new = mk()
        for dst, src in zip(ins, new):
            dst.copy_(src)
        graph.replay()
        mb.mlstm_step(*ins, *st_e, h_e, *st_e)
        torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        assert torch.equal(h, h_e) and all(torch.equal(a, b) for a, b in zip(st, st_e)), f"replay {r}"
    print("step graph: 4 replays equal to eager")
