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
