"""The roofline denominators reproduce the paper's closed-form columns (CPU only).

Tab. 3's "FLOPs forward" column is the App. D.1 count at context 8192; its
"Total Memory State in MB" column is the Sec. 3.1 state-size formula.  Both
are stored in tests/golden/tab3_head_ablation.json with their citation.
"""
import json
import os

import pytest

from paper_2503_13427_amd import accounting as A

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "tab3_head_ablation.json")))


@pytest.mark.parametrize("row", GOLDEN["rows"], ids=lambda r: f"NH{r['heads']}")
def test_state_size_matches_tab3(row):
    mb = A.state_bytes(GOLDEN["blocks"], row["heads"], row["d_hv"] // 2, row["d_hv"]) / 1e6
    assert round(mb, 1) == row["state_MB"]


@pytest.mark.parametrize("row", GOLDEN["rows"], ids=lambda r: f"NH{r['heads']}")
def test_flops_forward_matches_tab3(row):
    f = A.flops_chunkwise(row["heads"], GOLDEN["context"], GOLDEN["chunk_size_reading"], row["d_hv"] // 2,
                          row["d_hv"]).total
    # printed to two significant digits
    assert float(f"{f:.1e}") == pytest.approx(row["flops_fwd_read"], rel=1e-12)


def test_flops_split_dominated_by_inter_chunk():
    f = A.flops_chunkwise(8, 2048, 64, 256, 512)
    assert f.inter_numerator / f.total == pytest.approx(0.84, abs=0.01)
    assert f.total == pytest.approx(1.033e10, rel=1e-3)


def test_bytes():
    assert A.prefill_bytes(1, 8, 2048, 256, 512) == 8 * 2048 * (2 * 256 * 2 + 512 * 2 + 8 + 512 * 2) + 8 * (256 * 512 + 257) * 4
    assert A.step_bytes(256, 8, 256, 512) == pytest.approx(2.158e9, rel=1e-3)


def test_layer_projection_flops_are_the_layer_gemms():
    """App. D.2's projection count, sigmoid left out, equals 2 m n k summed over the GEMMs the layer
    runs: x [T, d] by the q, k, v, o~ columns NH (2 dqk + 2 dv), by the 2 NH gate columns, and the
    concatenated heads [T, NH dv] by the output projection [NH dv, d]."""
    T, d, NH, dqk, dv = 2048, 4096, 8, 256, 512
    gemms = [(T, NH * (2 * dqk + 2 * dv), d), (T, 2 * NH, d), (T, d, NH * dv)]
    assert A.flops_layer_projections(T, d, NH, dqk, dv, F_sig=0) == sum(2 * m * n * k for m, n, k in gemms)
    assert A.flops_layer_projections(T, d, NH, dqk, dv) - A.flops_layer_projections(T, d, NH, dqk, dv, 0) == T * d


def test_layer_step_bytes():
    """One 7B-shaped decode step at B=1: 2 bytes per bf16 weight of the App. E count with d_model =
    NH dv (qkv, output gate, output projection), fp32 gates and norm, and the 4 MiB-scale state twice."""
    d, NH, dqk, dv = 4096, 8, 256, 512
    bf16_params = d * NH * (2 * dqk + dv) + d * d + d * d
    f32_params = 2 * d * NH + 2 * NH + d
    assert A.layer_weight_bytes(d, NH, dqk, dv) == 2 * bf16_params + 4 * f32_params
    state = A.state_bytes(1, NH, dqk, dv) + 4 * NH * (dqk + 1)
    assert A.layer_step_bytes(1, d, NH, dqk, dv) == 2 * bf16_params + 4 * f32_params + 2 * state + 4 * d
