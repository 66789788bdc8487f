"""The five synthetic workloads of the mLSTM cell.

Shapes follow the xLSTM 7B cell: 8 heads, d_hv = 512 and d_qk = d_hv / 2 = 256
(Sec. 3.1, "Optimizing the Memory Capacity"; Tab. 3).  The long prefill uses
the 65 536-token budget of the prefill-throughput experiment (Sec. 4.3, Fig. 7)
as 8 x 8192.  The gate soft-cap a = 15 is Eq. 13 (Sec. 3.2).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

from .inputs import GateDist, Inputs, StateDist, make_decode_steps, make_prefill


@dataclass(frozen=True)
class Workload:
    wid: int                 # workload id, keys the input streams
    name: str
    kind: str                # "prefill" or "decode"
    B: int
    NH: int
    T: int                   # prefill tokens (decode: the state-building prefill length)
    DQK: int
    DV: int
    L: int                   # chunk size of the prefill call
    dtype: str               # "bf16" or "f32" for q, k, v, h
    gates: GateDist
    state: Optional[StateDist] = None
    k_scale: float = 1.0
    steps: int = 0           # decode: consecutive mlstm_step calls

    @property
    def heads(self) -> int:
        return self.B * self.NH

    def prefill_inputs(self, seed: int = 0, heads=None, T: Optional[int] = None) -> Inputs:
        return make_prefill(workload=self.wid, B=self.B, NH=self.NH, T=self.T if T is None else T,
                            DQK=self.DQK, DV=self.DV, dtype=self.dtype, gates=self.gates,
                            state=self.state, k_scale=self.k_scale, seed=seed, heads=heads)

    def decode_inputs(self, seed: int = 0, heads=None, steps: Optional[int] = None) -> Inputs:
        assert self.kind == "decode"
        return make_decode_steps(workload=self.wid, B=self.B, NH=self.NH,
                                 steps=self.steps if steps is None else steps,
                                 DQK=self.DQK, DV=self.DV, gates=self.gates, dtype=self.dtype,
                                 seed=seed, heads=heads)


_G2 = GateDist(i_mu=0.0, i_sd=1.0, f_mu=3.0, f_sd=1.0, cap=None)

TINY_F32 = Workload(1, "tiny_f32_B1_NH1_T64_d16_L16", "prefill", B=1, NH=1, T=64, DQK=16, DV=16, L=16,
                    dtype="f32", gates=_G2, k_scale=1.0 / np.sqrt(16.0))
PREFILL_T2048 = Workload(2, "prefill_B1_NH8_T2048_L64", "prefill", B=1, NH=8, T=2048, DQK=256, DV=512,
                         L=64, dtype="bf16", gates=_G2)
PREFILL_T8192 = Workload(3, "prefill_B8_NH8_T8192_L64_softcap15", "prefill", B=8, NH=8, T=8192, DQK=256,
                         DV=512, L=64, dtype="bf16",
                         gates=GateDist(i_mu=0.0, i_sd=1.0, f_mu=3.0, f_sd=1.0, cap=15.0))
DECODE_B256 = Workload(4, "decode_B256_NH8_1024steps", "decode", B=256, NH=8, T=128, DQK=256, DV=512,
                       L=64, dtype="bf16", gates=_G2, steps=1024)
CONT_PREFILL_T32768 = Workload(5, "continued_prefill_B4_NH8_T32768_L128", "prefill", B=4, NH=8, T=32768,
                               DQK=256, DV=512, L=128, dtype="bf16",
                               gates=GateDist(i_mu=0.0, i_sd=1.0, f_mu=5.0, f_sd=2.0, cap=15.0),
                               state=StateDist(c_sd=0.1))

ALL = [TINY_F32, PREFILL_T2048, PREFILL_T8192, DECODE_B256, CONT_PREFILL_T32768]
BY_ID = {w.wid: w for w in ALL}
