#!/usr/bin/env python3
"""Benchmark of libmlstm on one MI355X: prefill tokens/s (%MFMA) and decode step us (%HBM).

One JSON line on stdout.  The headline ``value`` is the chunkwise prefill of the
largest xLSTM-7B-shaped workload, the continued prefill B=4, NH=8, T=32768,
DQK=256, DV=512, L=128 from a nonzero fp32 initial state (bf16 q/k/v, fp32 gates
soft-capped at 15, fp32 state): one "step" is one mlstm_chunkwise_fwd call over
that batch, all of its kernels included.  Inputs are seeded synthetic data
already resident in HBM (the working set, 3.3 GB, is far beyond the 256 MB
Infinity Cache).  Every timed call is bracketed by HIP events on the launch
stream: ``ms_per_step`` is the mean over the K timed calls, and the median,
p10 and p90 of the per-call times are reported beside it.

Extra objects on the same line:
  roofline      achieved bf16 TFLOP/s (App. D.1 FLOP count per call / mean call
                duration) vs 2.5 PFLOP/s, and the HBM bytes per call from the
                committed rocprofv3 FETCH_SIZE/WRITE_SIZE summary;
  cpu_baseline  the fp64 CPU oracle on a sample of the same workload (host
                cores), plus every other workload and a 1-thread run;
  prefill_other the two other prefill workloads (B=1 x T=2048, L=64, with rotated
                input copies and warm-cache figure; B=8 x T=8192 soft-capped, L=64),
                each >= 20 calls with median, p10, p90;
  decode        1024 consecutive mlstm_step calls at B=256, NH=8: us per step,
                us per sequence-token, achieved GB/s vs 8 TB/s;
  decode_b1     mlstm_step at B=1, NH=8 (single-sequence generation), in place;
  decode_output the step returning h = sigmoid(o~) * LayerNorm(h~) w: mlstm_step_output
                (fused epilogue at B=256; column split + output pass at B=1) against
                mlstm_step followed by mlstm_output_norm;
  output_norm   the hidden-state output h = sigmoid(o~) * LayerNorm(h~) w + b
                (mlstm_output_norm) on the T=2048 prefill's h shape and the
                decode step's h shape: us per call and achieved GB/s vs 8 TB/s;
  layer         one xLSTM-7B-shaped mLSTM layer (d = 4096, random weights): prefill
                of 65536 tokens as batch x context (1 x 65536, 8 x 8192, 64 x 1024)
                with the time of each stage, and decode steps at B = 1 and 256,
                eager and as a captured HIP graph;
  backward      the training-mode backward pass on the T=2048 prefill shape;
  env           GPU, ROCm and torch versions, git commit when available, and a
                hash of the kernel sources.
Every timed section is preceded by 0.25 s of untimed calls (clock settle).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2503_13427_amd import accounting as acc  # noqa: E402
from paper_2503_13427_amd import configs  # noqa: E402

METRIC = "mLSTM prefill tokens/s (%MFMA peak); decode step µs/token (%HBM BW)"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def dev(x, device="cuda"):
    if x is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(x))
    if x.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.to(device)


class Prefill:
    """Device buffers for one prefill workload, NINPUT rotated input copies."""

    def __init__(self, w, ninput=1, device="cuda"):
        from paper_2503_13427_amd import binding
        self.mb = binding
        self.w = w
        inp = w.prefill_inputs()
        self.sets = []
        for i in range(ninput):
            self.sets.append(dict(q=dev(inp.q), k=dev(inp.k), v=dev(inp.v), ipre=dev(inp.ipre), fpre=dev(inp.fpre),
                                  C0=dev(inp.C0), n0=dev(inp.n0), m0=dev(inp.m0)))
        B, NH, T = w.B, w.NH, w.T
        self.h = torch.empty(B, NH, T, w.DV, dtype=torch.bfloat16, device=device)
        self.CT = torch.empty(B, NH, w.DQK, w.DV, device=device)
        self.nT = torch.empty(B, NH, w.DQK, device=device)
        self.mT = torch.empty(B, NH, device=device)
        nb = binding.mlstm_chunkwise_workspace_bytes(B, NH, T, w.DQK, w.DV, w.L)
        self.ws = torch.empty(nb, dtype=torch.uint8, device=device) if nb else None
        self.i = 0

    def step(self, stream=None):
        d = self.sets[self.i % len(self.sets)]
        self.i += 1
        self.mb.mlstm_chunkwise_fwd(d["q"], d["k"], d["v"], d["ipre"], d["fpre"], d["C0"], d["n0"], d["m0"], self.w.L,
                                    self.h, self.CT, self.nT, self.mT, workspace=self.ws, stream=stream)

    def flops(self):
        w = self.w
        return acc.flops_chunkwise(w.B * w.NH, w.T, w.L, w.DQK, w.DV).total

    def bytes(self):
        w = self.w
        return acc.prefill_bytes(w.B, w.NH, w.T, w.DQK, w.DV, with_initial_state=w.state is not None)


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "chunkwise_traffic_B4_NH8_T32768_L128.md")
CSRC = os.path.join(ROOT, "paper_2503_13427_amd", "csrc")
# the chunkwise prefill's source and the device headers it includes, hashed in this order
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in
                  ("mlstm_chunkwise_mfma.hip", "chunk_common.h", "mfma_common.h", "device_common.h")]


def kernel_source_sha16():
    """First 16 hex digits of the SHA-256 over the prefill kernel's source files, concatenated."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per headline call from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE summary, or None
    when that summary is missing or was taken on a different chunkwise kernel source."""
    try:
        text = open(TRAFFIC_PROFILE).read()
        src_sha = kernel_source_sha16()
    except OSError:
        return None
    nbytes = sha = None
    for line in text.splitlines():
        if line.startswith("traffic_bytes_per_call:"):
            nbytes = float(line.split(":")[1])
        elif line.startswith("kernel_source_sha256_16:"):
            sha = line.split(":")[1].split()[0]
    if nbytes is None or sha != src_sha:
        return None
    return nbytes


SETTLE_S = 0.25


def settle(fn, seconds=SETTLE_S):
    """Untimed calls of fn until ``seconds`` of wall time have passed: the GPU raises its clocks over
    the first milliseconds under load, so short warm-ups alone time a partly idle-clocked chip."""
    t0 = time.perf_counter()
    n = 1
    while time.perf_counter() - t0 < seconds:
        for _ in range(n):
            fn()
        torch.cuda.synchronize()
        n = min(2 * n, 64)


def time_steps(fn, steps, warmup, stream):
    """Wall time and HIP-event time (on the launch stream) of ``steps`` calls of fn, after the clock
    settle phase and ``warmup`` untimed calls."""
    settle(fn)
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, e0.elapsed_time(e1) / 1e3


def bench_prefill(w, steps, warmup, ninput, stream):
    """``steps`` calls, each bracketed by HIP events on the launch stream: mean, median, p10 and
    p90 of the per-call times; the throughput and roofline figures use the mean."""
    p = Prefill(w, ninput)
    fn = lambda: p.step(stream)
    settle(fn)
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i].record(stream)
        fn()
    ev[steps].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]) / 1e3
    t = ev[0].elapsed_time(ev[steps]) / 1e3 / steps
    fl = p.flops()
    tok = w.B * w.T
    out = dict(workload=w.name, tokens_per_s=tok / t, us_per_call=t * 1e6,
               us_per_call_median=float(np.median(per)) * 1e6, us_per_call_p10=float(np.quantile(per, 0.1)) * 1e6,
               us_per_call_p90=float(np.quantile(per, 0.9)) * 1e6, tflops=fl / t / 1e12,
               mfma_frac=fl / t / 1e12 / acc.PEAK_BF16_MFMA_TFLOPS,
               mfma_frac_median=fl / float(np.median(per)) / 1e12 / acc.PEAK_BF16_MFMA_TFLOPS,
               gbs=p.bytes() / t / 1e9, hbm_frac=p.bytes() / t / 1e9 / acc.PEAK_HBM_GBS, wall_s=wall, steps=steps,
               flops_per_call=fl, bytes_per_call=p.bytes(), input_sets=ninput,
               workspace_bytes=0 if p.ws is None else p.ws.numel())
    return out, p


def bench_decode(w, steps, stream, warm=16):
    """``steps`` consecutive decode steps on device-resident per-step inputs; the initial state
    comes from the library's own prefill of the workload's 128-token prompt."""
    from paper_2503_13427_amd import binding as mb
    log(f"decode: drawing {steps} steps of inputs for {w.heads} heads")
    dec = w.decode_inputs(steps=steps)
    q, k, v = dev(dec.q), dev(dec.k), dev(dec.v)
    ip, fp = dev(dec.ipre), dev(dec.fpre)
    del dec
    # per-step contiguous slices, resident before timing
    qs = [q[:, :, t].contiguous() for t in range(steps)]
    ks = [k[:, :, t].contiguous() for t in range(steps)]
    vs = [v[:, :, t].contiguous() for t in range(steps)]
    ips = [ip[:, :, t].contiguous() for t in range(steps)]
    fps = [fp[:, :, t].contiguous() for t in range(steps)]
    del q, k, v, ip, fp
    pre = w.prefill_inputs()
    C = torch.empty(w.B, w.NH, w.DQK, w.DV, device="cuda")
    n = torch.empty(w.B, w.NH, w.DQK, device="cuda")
    m = torch.empty(w.B, w.NH, device="cuda")
    hpre = torch.empty(w.B, w.NH, w.T, w.DV, dtype=torch.bfloat16, device="cuda")
    mb.mlstm_chunkwise_fwd(dev(pre.q), dev(pre.k), dev(pre.v), dev(pre.ipre), dev(pre.fpre), None, None, None, w.L,
                           hpre, C, n, m, stream=stream)
    h = torch.empty(w.B, w.NH, w.DV, dtype=torch.bfloat16, device="cuda")
    C0, n0, m0 = C.clone(), n.clone(), m.clone()
    settle(lambda: mb.mlstm_step(qs[0], ks[0], vs[0], ips[0], fps[0], C0, n0, m0, h, C0, n0, m0, stream=stream))
    for t in range(warm):   # warm-up on a copy of the state
        mb.mlstm_step(qs[t], ks[t], vs[t], ips[t], fps[t], C0, n0, m0, h, C0, n0, m0, stream=stream)
    del C0, n0, m0
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for t in range(steps):
        mb.mlstm_step(qs[t], ks[t], vs[t], ips[t], fps[t], C, n, m, h, C, n, m, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    t_step = e0.elapsed_time(e1) / 1e3 / steps
    by = acc.step_bytes(w.B, w.NH, w.DQK, w.DV)
    finite = bool(torch.isfinite(C).all().item())
    return dict(workload=w.name, steps=steps, us_per_step=t_step * 1e6, us_per_token=t_step * 1e6 / w.B,
                gbs=by / t_step / 1e9, hbm_frac=by / t_step / 1e9 / acc.PEAK_HBM_GBS, bytes_per_step=by,
                wall_s=wall, state_finite=finite)


def bench_step_small(B, NH, steps, stream):
    """mlstm_step for a small batch (B = 1: the single-sequence generation of the paper's speed
    benchmarks), the state updated in place; the C stream is split over many workgroups per
    sequence.  us per step and the step's algorithmic bytes against HBM bandwidth."""
    from paper_2503_13427_amd import binding as mb
    DQK, DV = 256, 512
    g = torch.Generator(device="cuda").manual_seed(7)
    q = torch.randn(B, NH, DQK, generator=g, device="cuda").bfloat16()
    k = torch.randn(B, NH, DQK, generator=g, device="cuda").bfloat16()
    v = torch.randn(B, NH, DV, generator=g, device="cuda").bfloat16()
    ip = torch.randn(B, NH, generator=g, device="cuda")
    fp = torch.randn(B, NH, generator=g, device="cuda") + 3
    C = torch.randn(B, NH, DQK, DV, generator=g, device="cuda") * 0.1
    n = torch.randn(B, NH, DQK, generator=g, device="cuda").abs()
    m = torch.zeros(B, NH, device="cuda")
    h = torch.empty(B, NH, DV, dtype=torch.bfloat16, device="cuda")
    fn = lambda: mb.mlstm_step(q, k, v, ip, fp, C, n, m, h, C, n, m, stream=stream)
    _, ev = time_steps(fn, steps, 10, stream)
    t = ev / steps
    by = acc.step_bytes(B, NH, DQK, DV)
    return dict(workload=f"decode_B{B}_NH{NH}", us_per_step=t * 1e6, bytes_per_step=by, gbs=by / t / 1e9,
                hbm_frac=by / t / 1e9 / acc.PEAK_HBM_GBS)


def bench_step_output(B, NH, steps, stream):
    """The decode step returning the hidden-state output h = sigmoid(o~) * LayerNorm(h~) w (Eq. 6, 9):
    mlstm_step_output (the norm in the step's epilogue at this batch) against mlstm_step followed by
    mlstm_output_norm, both in place on the same state; us per step."""
    from paper_2503_13427_amd import binding as mb
    DQK, DV = 256, 512
    g = torch.Generator(device="cuda").manual_seed(9)
    rn = lambda *shape: torch.randn(*shape, generator=g, device="cuda")
    q, k, v = rn(B, NH, DQK).bfloat16(), rn(B, NH, DQK).bfloat16(), rn(B, NH, DV).bfloat16()
    o = rn(B, NH, DV).bfloat16()
    ip, fp = rn(B, NH), rn(B, NH) + 3
    C, n, m = rn(B, NH, DQK, DV) * 0.1, rn(B, NH, DQK).abs(), torch.zeros(B, NH, device="cuda")
    w = 1 + 0.1 * rn(NH, DV)
    h = torch.empty(B, NH, DV, dtype=torch.bfloat16, device="cuda")
    fused = lambda: mb.mlstm_step_output(q, k, v, ip, fp, C, n, m, o, w, None, 1e-6, "layer", h, C, n, m, stream=stream)

    def pair():
        mb.mlstm_step(q, k, v, ip, fp, C, n, m, h, C, n, m, stream=stream)
        mb.mlstm_output_norm(h, o, w, None, 1e-6, "layer", h, stream=stream)
    t_f = time_steps(fused, steps, 10, stream)[1] / steps
    t_p = time_steps(pair, steps, 10, stream)[1] / steps
    by = acc.step_bytes(B, NH, DQK, DV) + B * NH * DV * 2   # plus o~ read once
    return dict(workload=f"decode_output_B{B}_NH{NH}", us_per_step_fused=t_f * 1e6, us_per_step_step_then_norm=t_p * 1e6,
                saved_us=(t_p - t_f) * 1e6, bytes_per_step=by, gbs_fused=by / t_f / 1e9,
                hbm_frac_fused=by / t_f / 1e9 / acc.PEAK_HBM_GBS)


def bench_output_norm(B, NH, T, DV, steps, stream, label):
    """h = sigmoid(o~) * LayerNorm(h~) * w + b on bf16 rows already in HBM (HBM-bound)."""
    from paper_2503_13427_amd import binding as mb
    g = torch.Generator(device="cuda").manual_seed(5)
    shape = (B, NH, T, DV)
    x = torch.randn(shape, generator=g, device="cuda").bfloat16()
    o = torch.randn(shape, generator=g, device="cuda").bfloat16()
    w = torch.randn(NH, DV, generator=g, device="cuda") * 0.2 + 1
    b = torch.randn(NH, DV, generator=g, device="cuda") * 0.2
    h = torch.empty_like(x)
    fn = lambda: mb.mlstm_output_norm(x, o, w, b, 1e-6, "layer", h, stream=stream)
    _, ev = time_steps(fn, steps, 10, stream)
    t = ev / steps
    by = acc.output_norm_bytes(B, NH, T, DV)
    return dict(workload=label, rows=B * NH * T, dv=DV, us_per_call=t * 1e6, bytes_per_call=by,
                gbs=by / t / 1e9, hbm_frac=by / t / 1e9 / acc.PEAK_HBM_GBS)


LAYER_D, LAYER_NH, LAYER_DQK, LAYER_DV = 4096, 8, 256, 512
LAYER_PREFILL_SPLITS = ((1, 65536), (8, 8192), (64, 1024))   # 65536 tokens as batch x context


def synthetic_layer(seed=11, L=64):
    """An xLSTM-7B-shaped mLSTM layer (d = 4096, 8 heads, dqk = 256, dv = 512) with random weights:
    projections N(0, 1/fan_in) in bf16, input/forget gate biases around
    -2 and +3, norm weight around 1."""
    from paper_2503_13427_amd.layer import LayerWeights, MLSTMLayer
    d, NH, DQK, DV = LAYER_D, LAYER_NH, LAYER_DQK, LAYER_DV
    g = torch.Generator(device="cuda").manual_seed(seed)
    rn = lambda *shape: torch.randn(*shape, generator=g, device="cuda")
    w = LayerWeights(W_qkvo=(rn(d, NH * (2 * DQK + 2 * DV)) * d ** -0.5).bfloat16(),
                     W_gates_t=(rn(2 * NH, d) * d ** -0.5).bfloat16(),
                     W_proj=(rn(NH * DV, d) * (NH * DV) ** -0.5).bfloat16(),
                     gate_bias=rn(2, NH) + torch.tensor([[-2.0], [3.0]], device="cuda"),
                     norm_weight=1 + 0.1 * rn(NH, DV), NH=NH, DQK=DQK, DV=DV)
    return MLSTMLayer(w, L=L, eps=1e-6, cap=15.0)


def bench_layer_prefill(layer, B, T, steps, stream):
    """One layer forward over B x T tokens (x resident in HBM), and the same work stage by stage."""
    from paper_2503_13427_amd import binding as mb
    w = layer.w
    NH, DQK, DV, d = w.NH, w.DQK, w.DV, LAYER_D
    g = torch.Generator(device="cuda").manual_seed(12)
    x = torch.randn(B, T, d, generator=g, device="cuda").bfloat16()
    nb = mb.mlstm_chunkwise_workspace_bytes(B, NH, T, DQK, DV, layer.L)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda") if nb else None
    run = lambda fn: time_steps(fn, steps, 1, stream)[1] / steps
    t_total = run(lambda: layer.prefill(x, workspace=ws))
    x2 = x.reshape(B * T, d)
    t_proj = run(lambda: layer._project(x2))
    t_gates = run(lambda: layer.gates(x))
    # the stages as the prefill runs them: the cell reads q, k, v as per-head views of the projection
    # output and the norm reads o~ in place (no head-major copies)
    q4, k4, v4, o4 = layer._project(x2)
    hv = lambda a, D: a.view(B, T, NH, D).transpose(1, 2)
    q, k, v = hv(q4, DQK), hv(k4, DQK), hv(v4, DV)
    ig, fg = layer.gates(x)
    h = torch.empty(B, NH, T, DV, dtype=torch.bfloat16, device="cuda")
    C = torch.empty(B, NH, DQK, DV, device="cuda")
    n = torch.empty(B, NH, DQK, device="cuda")
    m = torch.empty(B, NH, device="cuda")
    t_cell = run(lambda: mb.mlstm_chunkwise_fwd_strided(q, k, v, ig, fg, None, None, None, layer.L, h, C, n, m,
                                                         workspace=ws, stream=stream))
    # for comparison: the cell on head-major copies (what the copies would cost is not in the total)
    qc, kc, vc = q.contiguous(), k.contiguous(), v.contiguous()
    t_cell_contig = run(lambda: mb.mlstm_chunkwise_fwd(qc, kc, vc, ig, fg, None, None, None, layer.L, h, C, n, m,
                                                        workspace=ws, stream=stream))
    del qc, kc, vc
    yh = torch.empty(B, T, NH, DV, dtype=torch.bfloat16, device="cuda")
    o_view = o4.view(B, T, NH, DV)
    t_norm = run(lambda: mb.mlstm_output_norm_tokens(h, o_view, w.norm_weight, None, layer.eps, "layer", yh,
                                                     stream=stream))
    t_out = run(lambda: torch.matmul(yh.view(B * T, NH * DV), w.W_proj))
    tok = B * T
    fl_proj = acc.flops_layer_projections(tok, d, NH, DQK, DV)
    fl_cell = acc.flops_chunkwise(B * NH, T, layer.L, DQK, DV).total
    stages = dict(projections=t_proj, gates=t_gates, cell=t_cell, output_norm=t_norm, output_projection=t_out)
    return dict(workload=f"layer_prefill_B{B}_T{T}_d{d}_NH{NH}", B=B, T=T, tokens_per_s=tok / t_total,
                ms_per_call=t_total * 1e3, tflops=(fl_proj + fl_cell) / t_total / 1e12,
                flops_projections=fl_proj, flops_cell=fl_cell,
                stages_ms={k: v * 1e3 for k, v in stages.items()}, cell_on_contiguous_copies_ms=t_cell_contig * 1e3,
                stages_share={k: v / t_total for k, v in stages.items()})


def bench_layer_decode(layer, B, steps, stream):
    """Consecutive decode steps of B tokens through one layer: eager launches, then the same step
    replayed as a captured HIP graph; algorithmic bytes per step against HBM bandwidth."""
    from paper_2503_13427_amd.layer import GraphedDecode
    w = layer.w
    NH, DQK, DV, d = w.NH, w.DQK, w.DV, LAYER_D
    g = torch.Generator(device="cuda").manual_seed(13)
    x = torch.randn(B, d, generator=g, device="cuda").bfloat16()
    state = (torch.zeros(B, NH, DQK, DV, device="cuda"), torch.zeros(B, NH, DQK, device="cuda"),
             torch.zeros(B, NH, device="cuda"))
    t_eager = time_steps(lambda: layer.step(x, state), steps, 10, stream)[1] / steps
    gd = GraphedDecode(layer, tuple(t.clone() for t in state), B)
    gd.x.copy_(x)
    t_graph = time_steps(gd.graph.replay, steps, 10, stream)[1] / steps
    by = acc.layer_step_bytes(B, d, NH, DQK, DV)
    return dict(workload=f"layer_decode_B{B}_d{d}_NH{NH}", B=B, us_per_step_eager=t_eager * 1e6,
                us_per_step_graph=t_graph * 1e6, tokens_per_s_graph=B / t_graph, bytes_per_step=by,
                gbs_graph=by / t_graph / 1e9, hbm_frac_graph=by / t_graph / 1e9 / acc.PEAK_HBM_GBS)


def bench_layer(steps, decode_steps, stream):
    layer = synthetic_layer()
    out = {"prefill": [], "decode": []}
    for B, T in LAYER_PREFILL_SPLITS:
        log(f"layer prefill B={B} T={T}")
        out["prefill"].append(bench_layer_prefill(layer, B, T, steps, stream))
        torch.cuda.empty_cache()
    for B in (1, 256):
        log(f"layer decode B={B}")
        out["decode"].append(bench_layer_decode(layer, B, decode_steps, stream))
    return out


def backward_inputs(w):
    """Seeded inputs of the training-mode backward on a prefill shape (bf16 q/k/v and dh, fp32 gates,
    zero initial state), its fp32 outputs and its workspace."""
    from paper_2503_13427_amd import binding as mb
    g = torch.Generator(device="cuda").manual_seed(17)
    B, NH, T, DQK, DV = w.B, w.NH, w.T, w.DQK, w.DV
    q = torch.randn(B, NH, T, DQK, generator=g, device="cuda").bfloat16()
    k = (torch.randn(B, NH, T, DQK, generator=g, device="cuda") / 16).bfloat16()
    v = torch.randn(B, NH, T, DV, generator=g, device="cuda").bfloat16()
    ip = torch.randn(B, NH, T, generator=g, device="cuda")
    fp = torch.randn(B, NH, T, generator=g, device="cuda") + 3
    dh = torch.randn(B, NH, T, DV, generator=g, device="cuda").bfloat16()
    outs = [torch.empty(B, NH, T, DQK, device="cuda"), torch.empty(B, NH, T, DQK, device="cuda"),
            torch.empty(B, NH, T, DV, device="cuda"), torch.empty(B, NH, T, device="cuda"),
            torch.empty(B, NH, T, device="cuda")]
    wsb = torch.empty(mb.mlstm_chunkwise_bwd_workspace_bytes(B, NH, T, DQK, DV, 64), dtype=torch.uint8, device="cuda")
    return q, k, v, ip, fp, dh, outs, wsb


def bench_backward(w, steps, stream, parallel=True):
    """The training-mode backward on a prefill shape (inputs of ``backward_inputs``):
    mlstm_chunkwise_bwd (per-call median of ``steps`` calls), the forward on the same inputs
    for the ratio, and (``parallel``) mlstm_parallel_bwd for comparison.  FLOP figures use App. D.2's
    count, twice the App. D.1 forward, against the bf16 MFMA peak."""
    from paper_2503_13427_amd import binding as mb
    B, NH, T, DQK, DV = w.B, w.NH, w.T, w.DQK, w.DV
    q, k, v, ip, fp, dh, outs, wsb = backward_inputs(w)

    def per_call(fn, n):
        settle(fn)
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        for i in range(n):
            ev[i].record(stream)
            fn()
        ev[n].record(stream)
        torch.cuda.synchronize()
        return np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(n)]) / 1e3

    bwd = per_call(lambda: mb.mlstm_chunkwise_bwd(q, k, v, ip, fp, None, None, None, 64, dh, *outs, None, None, None,
                                                  wsb, stream=stream), steps)
    del wsb
    h = torch.empty(B, NH, T, DV, dtype=torch.bfloat16, device="cuda")
    CT, nT, mT = (torch.empty(B, NH, DQK, DV, device="cuda"), torch.empty(B, NH, DQK, device="cuda"),
                  torch.empty(B, NH, device="cuda"))
    nb = mb.mlstm_chunkwise_workspace_bytes(B, NH, T, DQK, DV, w.L)
    wsf = torch.empty(nb, dtype=torch.uint8, device="cuda") if nb else None
    fwd = per_call(lambda: mb.mlstm_chunkwise_fwd(q, k, v, ip, fp, None, None, None, w.L, h, CT, nT, mT, workspace=wsf,
                                                  stream=stream), steps)
    tb, tf = float(np.median(bwd)), float(np.median(fwd))
    fl_d2 = 2 * acc.flops_chunkwise(B * NH, T, 64, DQK, DV).total
    out = dict(workload=f"backward_{w.name}", kernel="mlstm_chunkwise_bwd", calls=steps, ms_per_call=tb * 1e3,
               ms_per_call_p10=float(np.quantile(bwd, 0.1)) * 1e3, ms_per_call_p90=float(np.quantile(bwd, 0.9)) * 1e3,
               tokens_per_s=B * T / tb, forward_ms_per_call=tf * 1e3, backward_over_forward=tb / tf,
               app_d2_flops=fl_d2, app_d2_tflops=fl_d2 / tb / 1e12,
               mfma_frac=fl_d2 / tb / 1e12 / acc.PEAK_BF16_MFMA_TFLOPS)
    if parallel:
        dh32 = dh.float()
        ws = torch.empty(mb.mlstm_parallel_bwd_workspace_bytes(B, NH, T, DV), dtype=torch.uint8, device="cuda")
        par = per_call(lambda: mb.mlstm_parallel_bwd(q, k, v, ip, fp, dh32, *outs, ws, stream=stream), max(3, steps // 4))
        tp = float(np.median(par))
        fl = acc.flops_parallel_bwd(B * NH, T, DQK, DV)
        out["parallel_form"] = dict(kernel="mlstm_parallel_bwd", ms_per_call=tp * 1e3, flops_per_call=fl,
                                    tflops=fl / tp / 1e12, valu_frac=fl / tp / 1e12 / acc.PEAK_FP32_VALU_TFLOPS)
    return out


def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_prefill(w, heads, threads, T=None):
    """Seconds the fp64 oracle takes on ``heads`` of workload w (full sequence, or its first T tokens)."""
    from oracle import coracle
    inp = w.prefill_inputs(heads=heads, T=T)
    t0 = time.perf_counter()
    coracle.recurrent_inputs(inp, nthreads=threads)
    return time.perf_counter() - t0


def _oracle_decode(w, heads, steps, threads):
    """Seconds the fp64 oracle takes for ``steps`` decode steps of ``heads`` sequences from a state."""
    from oracle import coracle
    rng = np.random.default_rng(3)
    S = len(heads)
    C = rng.normal(0, 0.1, (S, w.DQK, w.DV))
    n = np.abs(rng.standard_normal((S, w.DQK)))
    m = rng.standard_normal(S)
    dec = w.decode_inputs(steps=steps, heads=heads)
    args = [dec.as_f64(x)[0] for x in ("q", "k", "v", "ipre", "fpre")]
    t0 = time.perf_counter()
    coracle.recurrent(*args, C, n, m, nthreads=threads)
    return time.perf_counter() - t0


def cpu_baseline(w):
    """The fp64 recurrent oracle (the CPU baseline, never tuned) timed on the host.  Heads are
    independent sequences, so each workload's sample is a subset of its heads over the full
    sequence; token rates are scaled to whole-workload tokens (B T per call) by the sampled share
    of the heads.  The headline entry is workload w; ``per_workload`` holds every workload, and the
    T=2048 prefill is also timed on one thread."""
    aff = len(os.sched_getaffinity(0))
    threads = max(1, min(aff, 16))

    def prefill_entry(wl, nheads, nthreads=threads):
        heads = list(range(min(nheads, wl.heads)))
        dt = _oracle_prefill(wl, heads, nthreads)
        share = len(heads) / wl.heads
        return dict(workload=wl.name, tokens_per_s=wl.B * wl.T * share / dt, seconds=dt, threads=nthreads,
                    sample=f"{len(heads)} of {wl.heads} heads x {wl.T} tokens")

    log(f"cpu baseline: fp64 oracle on {threads} threads")
    w2 = configs.PREFILL_T2048
    first = prefill_entry(w2, 8)
    # heads for a budget of about ``seconds`` of oracle time, from the T=2048 rate (threads work on
    # one head each)
    per_head_token = first["seconds"] / min(8, threads) / w2.T / math.ceil(8 / threads)

    def budget_heads(wl, seconds):
        rounds = max(1, int(seconds / (per_head_token * wl.T)))
        return max(1, min(wl.heads, rounds * threads))

    head = prefill_entry(w, budget_heads(w, 12.0))
    per = [prefill_entry(configs.TINY_F32, 1, 1), first, prefill_entry(w2, 8, 1),
           prefill_entry(configs.PREFILL_T8192, budget_heads(configs.PREFILL_T8192, 4.0))]
    dw = configs.DECODE_B256
    dheads = list(range(2 * threads))
    dt = _oracle_decode(dw, dheads, dw.steps, threads)
    us_step = dt / dw.steps * dw.heads / len(dheads) * 1e6
    per.append(dict(workload=dw.name, us_per_step=us_step, us_per_token=us_step / dw.B, seconds=dt, threads=threads,
                    sample=f"{len(dheads)} of {dw.heads} heads x {dw.steps} steps, scaled to all heads"))
    per.append(head)
    return dict(value=head["tokens_per_s"], unit="tokens/s", cores=threads, kind="oracle",
                sample=f"{head['sample']} of {w.name} (fp64 recurrent form, {head['seconds']:.2f} s wall); "
                       "tokens/s scaled to the whole workload by the sampled share of heads",
                seconds=head["seconds"], cpu_model=cpu_model(), affinity_cpus=aff, per_workload=per)


def env_info():
    """What produced the numbers: GPU, ROCm, torch, git commit (when the tree has one) and a hash of
    the HIP sources and the built library."""
    import hashlib
    import subprocess
    info = dict(torch=torch.__version__, hip=getattr(torch.version, "hip", None))
    try:
        props = torch.cuda.get_device_properties(0)
        info.update(gpu=props.name, arch=getattr(props, "gcnArchName", None), cus=props.multi_processor_count)
    except RuntimeError:
        pass
    for path in ("/opt/rocm/.info/version", "/opt/rocm/.info/version-dev"):
        try:
            info["rocm"] = open(path).read().strip()
            break
        except OSError:
            pass
    try:
        r = subprocess.run(["git", "-C", ROOT, "rev-parse", "HEAD"], capture_output=True, text=True, timeout=10)
        info["git_commit"] = r.stdout.strip() if r.returncode == 0 else None
    except (OSError, subprocess.SubprocessError):
        info["git_commit"] = None
    # a copy of the tree without .git: the commit the library was built from (build.py records it)
    try:
        b = json.load(open(os.path.join(ROOT, "paper_2503_13427_amd", "build_info.json")))
        info["built_from_commit"] = b.get("git_commit")
        info["built_from_dirty_tree"] = b.get("git_dirty")
    except (OSError, ValueError):
        pass
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        h.update(name.encode())
        h.update(open(os.path.join(CSRC, name), "rb").read())
    info["csrc_sha256_16"] = h.hexdigest()[:16]
    lib = os.path.join(ROOT, "paper_2503_13427_amd", "libmlstm.so")
    if os.path.exists(lib):
        info["libmlstm_sha256_16"] = hashlib.sha256(open(lib, "rb").read()).hexdigest()[:16]
    return info


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--ninput", type=int, default=8, help="rotated input copies of the T=2048 prefill (defeats a "
                                                            "warm Infinity Cache)")
    ap.add_argument("--other-steps", type=int, default=50, help="timed calls of each other prefill workload")
    ap.add_argument("--decode-steps", type=int, default=1024)
    ap.add_argument("--skip-decode", action="store_true")
    ap.add_argument("--skip-other", action="store_true")
    ap.add_argument("--skip-output-norm", action="store_true")
    ap.add_argument("--skip-cpu-baseline", action="store_true")
    ap.add_argument("--skip-layer", action="store_true")
    ap.add_argument("--skip-backward", action="store_true")
    ap.add_argument("--only", choices=["prefill", "other", "decode", "decode_b1", "decode_output", "output_norm", "layer",
                                       "backward",
                                       "calls", "cpu"],
                    default=None,
                    help="run one part only (profiling runs); 'calls' makes --calls untimed prefill calls of "
                         "--workload and then one --copy-mib MiB device copy, for counter runs")
    ap.add_argument("--workload", default=configs.CONT_PREFILL_T32768.name,
                    help="workload name for --only calls")
    ap.add_argument("--calls", type=int, default=3)
    ap.add_argument("--backward", action="store_true",
                    help="with --only calls on a prefill workload: chunkwise backward calls instead of the forward")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="size of the calibration copy after the calls (0: none)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU; --gpus {args.gpus} is not supported (every (batch, head) "
              "sequence is independent, so more GPUs would shard B*NH with no exchange)", file=sys.stderr)
        sys.exit(2)
    if args.only == "cpu":
        print(json.dumps(cpu_baseline(configs.CONT_PREFILL_T32768)), flush=True)
        return
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    w = configs.CONT_PREFILL_T32768

    if args.only == "calls":
        wl = {x.name: x for x in configs.ALL}[args.workload]
        if wl.kind == "decode":
            # in-place steps of the full decode batch from a random state (counter runs of the step)
            from paper_2503_13427_amd import binding as mb
            g = torch.Generator(device="cuda").manual_seed(7)
            rn = lambda *shape: torch.randn(*shape, generator=g, device="cuda")
            q, k, v = rn(wl.B, wl.NH, wl.DQK).bfloat16(), rn(wl.B, wl.NH, wl.DQK).bfloat16(), rn(wl.B, wl.NH, wl.DV).bfloat16()
            ip, fp = rn(wl.B, wl.NH), rn(wl.B, wl.NH) + 3
            C, n, m = rn(wl.B, wl.NH, wl.DQK, wl.DV) * 0.1, rn(wl.B, wl.NH, wl.DQK).abs(), torch.zeros(wl.B, wl.NH, device="cuda")
            h = torch.empty(wl.B, wl.NH, wl.DV, dtype=torch.bfloat16, device="cuda")
            torch.cuda.synchronize()
            for _ in range(args.calls):
                mb.mlstm_step(q, k, v, ip, fp, C, n, m, h, C, n, m, stream=stream)
        elif args.backward:
            # the chunkwise backward on the prefill shape (counter runs of the training-mode passes)
            from paper_2503_13427_amd import binding as mb
            q, k, v, ip, fp, dh, outs, wsb = backward_inputs(wl)
            torch.cuda.synchronize()
            for _ in range(args.calls):
                mb.mlstm_chunkwise_bwd(q, k, v, ip, fp, None, None, None, 64, dh, *outs, None, None, None, wsb,
                                       stream=stream)
        else:
            p = Prefill(wl, 1)
            for _ in range(args.calls):
                p.step(stream)
        torch.cuda.synchronize()
        if args.copy_mib:
            src = torch.ones(args.copy_mib * (1 << 18), dtype=torch.float32, device="cuda")
            dst = torch.empty_like(src)
            dst.copy_(src)
            torch.cuda.synchronize()
        log(f"calls: {args.calls} x {wl.name}, copy {args.copy_mib} MiB")
        return

    res = {}
    if args.only in (None, "prefill"):
        log(f"prefill {w.name}: {args.warmup} warm-up + {args.steps} timed calls")
        res["prefill"], p = bench_prefill(w, args.steps, args.warmup, 1, stream)
        del p
        torch.cuda.empty_cache()
    if args.only in (None, "other") and not args.skip_other:
        res["prefill_other"] = []
        w2 = configs.PREFILL_T2048
        log(f"prefill {w2.name}: {args.other_steps} timed calls, {args.ninput} rotated inputs")
        r, p = bench_prefill(w2, args.other_steps, 5, args.ninput, stream)
        del p
        warm, p = bench_prefill(w2, args.other_steps, 5, 1, stream)   # warm-cache figure: one input set
        del p
        r["warm_mall_us_per_call_median"] = warm["us_per_call_median"]
        res["prefill_other"].append(r)
        w3 = configs.PREFILL_T8192
        log(f"prefill {w3.name}: {args.other_steps} timed calls")
        r, p = bench_prefill(w3, args.other_steps, 3, 1, stream)
        res["prefill_other"].append(r)
        del p
        torch.cuda.empty_cache()
    if args.only in (None, "output_norm") and not args.skip_output_norm:
        log("output gate + headwise LayerNorm on the prefill and decode h shapes")
        w2 = configs.PREFILL_T2048
        res["output_norm"] = [bench_output_norm(w2.B, w2.NH, w2.T, w2.DV, 200, stream, "prefill_B1_NH8_T2048_DV512"),
                              bench_output_norm(256, 8, 1, 512, 200, stream, "decode_B256_NH8_DV512")]
        torch.cuda.empty_cache()
    if args.only in (None, "layer") and not args.skip_layer:
        log("mLSTM layer (projections + cell + output norm + output projection)")
        res["layer"] = bench_layer(10, max(50, args.decode_steps // 4), stream)
        torch.cuda.empty_cache()
    if args.only in (None, "backward") and not args.skip_backward:
        log(f"backward, {configs.PREFILL_T2048.name} and {configs.PREFILL_T8192.name}")
        res["backward"] = [bench_backward(configs.PREFILL_T2048, 20, stream),
                           bench_backward(configs.PREFILL_T8192, 10, stream, parallel=False)]
        torch.cuda.empty_cache()
    if args.only in (None, "decode") and not args.skip_decode:
        log(f"decode {configs.DECODE_B256.name}: {args.decode_steps} steps")
        res["decode"] = bench_decode(configs.DECODE_B256, args.decode_steps, stream)
        torch.cuda.empty_cache()
    if args.only in (None, "decode_b1") and not args.skip_decode:
        res["decode_b1"] = bench_step_small(1, 8, args.decode_steps, stream)
    if args.only in (None, "decode_output") and not args.skip_decode:
        log("decode step with the output gate and norm: fused vs step + output pass")
        res["decode_output"] = [bench_step_output(256, 8, 256, stream), bench_step_output(1, 8, 256, stream)]
        torch.cuda.empty_cache()

    line = {"metric": METRIC, "value": None, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": None, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": w.name, "B": w.B, "NH": w.NH, "T": w.T, "dqk": w.DQK, "dv": w.DV, "L": w.L,
                       "qkv": "bf16", "gates_state": "fp32", "initial_state": "C0~N(0,0.1), n0~|N(0,1)|, m0~N(0,1)",
                       "gates": "ipre~N(0,1), fpre~N(5,2), both soft-capped at 15"}}
    if "prefill" in res:
        hp = res["prefill"]
        line["value"] = hp["tokens_per_s"]
        line["ms_per_step"] = hp["us_per_call"] / 1e3
        line["roofline"] = {"bound": "mfma", "achieved": hp["tflops"], "peak": acc.PEAK_BF16_MFMA_TFLOPS,
                            "unit": "TFLOP/s", "frac": hp["mfma_frac"], "traffic": measured_traffic(),
                            "kernel": "mlstm_chunkwise_fwd call (every kernel of the call: the segment schedule's "
                                      "local-state and combine passes and the chunkwise pass); achieved and traffic "
                                      "are per call, over the call's mean duration",
                            "flops_per_call": hp["flops_per_call"], "hbm_frac": hp["hbm_frac"]}
        line["prefill"] = hp
    for key in ("prefill_other", "decode", "decode_b1", "decode_output", "output_norm", "layer", "backward"):
        if key in res:
            line[key] = res[key]
    if not args.skip_cpu_baseline and args.only in (None, "prefill"):
        line["cpu_baseline"] = cpu_baseline(w)
    line["env"] = env_info()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
