"""The seeded input generator (CPU only): determinism, head subsets, prefixes, bf16 rounding."""
import numpy as np
import pytest
import torch

from paper_2503_13427_amd import configs
from paper_2503_13427_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits


def test_bf16_round_to_nearest_even_matches_torch():
    x = np.random.default_rng(0).standard_normal(200_000).astype(np.float32) * 7
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 0.0]       # ties: round to even
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(bf16_bits_to_f32(ours), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_deterministic_and_head_subsets():
    w = configs.PREFILL_T2048
    a = w.prefill_inputs(T=128)
    b = w.prefill_inputs(T=128)
    np.testing.assert_array_equal(a.q, b.q)
    sub = w.prefill_inputs(T=128, heads=[6, 1])
    np.testing.assert_array_equal(sub.q[0, 0], a.q[0, 6])
    np.testing.assert_array_equal(sub.v[0, 1], a.v[0, 1])
    np.testing.assert_array_equal(sub.fpre[0, 0], a.fpre[0, 6])


def test_shorter_sequence_is_prefix():
    w = configs.PREFILL_T2048
    a = w.prefill_inputs(T=64, heads=[3])
    b = w.prefill_inputs(T=128, heads=[3])
    np.testing.assert_array_equal(a.k[0, 0], b.k[0, 0, :64])
    np.testing.assert_array_equal(a.ipre[0, 0], b.ipre[0, 0, :64])


def test_distributions():
    w = configs.CONT_PREFILL_T32768
    x = w.prefill_inputs(T=4096, heads=[0, 1, 2, 3])
    f = x.fpre.astype(np.float64)
    assert np.all(np.abs(f) < 15.0)                      # soft-capped at 15
    assert 4.5 < f.mean() < 5.3 and 1.7 < f.std() < 2.2  # N(5, 2) before the cap
    assert x.C0.std() == pytest.approx(0.1, rel=0.02)
    assert np.all(x.n0 >= 0)
    q = bf16_bits_to_f32(x.q)
    assert abs(q.mean()) < 0.01 and q.std() == pytest.approx(1.0, rel=0.01)
    t = configs.TINY_F32.prefill_inputs()
    assert t.q.dtype == np.float32 and t.k.std() == pytest.approx(0.25, rel=0.15)


def test_decode_steps_prefix():
    w = configs.DECODE_B256
    a = w.decode_inputs(steps=4, heads=[100])
    b = w.decode_inputs(steps=8, heads=[100])
    np.testing.assert_array_equal(a.q[0, 0], b.q[0, 0, :4])
    assert a.q.shape == (1, 1, 4, 256) and a.v.shape == (1, 1, 4, 512)


def test_pack_documents_marks_borders():
    """Borders are f~ = -inf exactly at the returned positions, reproducible per head, with the
    requested mean document length on a long sequence."""
    from paper_2503_13427_amd.inputs import GateDist, make_prefill, pack_documents
    a = make_prefill(workload=5, B=1, NH=2, T=20000, DQK=4, DV=4, dtype="f32", gates=GateDist())
    pos = pack_documents(a, 100.0, workload=5)
    for j in range(2):
        fp = a.fpre.reshape(2, -1)[j]
        assert np.array_equal(np.flatnonzero(np.isneginf(fp)), pos[j])
        assert pos[j][0] > 0 and 80 < 20000 / (len(pos[j]) + 1) < 125
    b = make_prefill(workload=5, B=1, NH=2, T=20000, DQK=4, DV=4, dtype="f32", gates=GateDist())
    pos_b = pack_documents(b, 100.0, workload=5, first=True)
    assert pos_b[1][0] == 0 and np.array_equal(pos_b[1][1:], pos[1])
