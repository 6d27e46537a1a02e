"""The seeded generator: shapes, offsets, determinism, planted structure."""
import numpy as np
import pytest
import torch

from paper_2607_25422_amd import workloads as wls


def test_named_workload_shapes():
    b = wls.make_batch("tiny_fp32", 2026)
    assert b.V.shape == (1, 576, 256) and b.V.dtype == torch.float32
    assert b.Qtok.shape == (16, 256)
    assert b.k.tolist() == [96] and b.P.tolist() == [4]
    assert b.Kh.shape == (256, 4, 64) and b.Vh.shape == (256, 4, 64)
    assert b.passage_offsets.tolist() == [0, 64, 128, 192, 256]
    assert b.planted[0].size == 24
    b2 = wls.make_batch("llava_bf16", 42, B=2)
    assert b2.V.dtype == torch.bfloat16 and b2.V.shape == (2, 576, 1024)
    assert b2.Kh.shape == (2 * 5 * 128, 16, 64)


def test_determinism_and_seed_sensitivity():
    a = wls.make_batch("llava_bf16", 137, B=2, N=100, k=(10,))
    b = wls.make_batch("llava_bf16", 137, B=2, N=100, k=(10,))
    c = wls.make_batch("llava_bf16", 42, B=2, N=100, k=(10,))
    assert torch.equal(a.V, b.V) and torch.equal(a.Kh, b.Kh) and torch.equal(a.Qtok, b.Qtok)
    assert not torch.equal(a.V, c.V)
    # per-question streams: question 0 does not depend on the batch size
    d = wls.make_batch("llava_bf16", 137, B=3, N=100, k=(10,))
    assert torch.equal(a.V[0], d.V[0])


def test_ragged_offsets_consistent():
    b = wls.make_batch("mixed_bf16", 2026, B=6, N=64, H=2, d_h=16, T=(1, 4),
                       k=(0, 5, 64), P=(0, 2, 3), L_p=(1, 7))
    assert b.q_offsets[0] == 0 and np.all(np.diff(b.q_offsets) >= 1)
    assert b.q_offsets[-1] == b.Qtok.shape[0]
    assert np.all(np.isin(b.k, [0, 5, 64]))
    assert b.query_passages[-1] == b.passage_offsets.size - 1
    assert b.passage_offsets[-1] == b.Kh.shape[0]
    assert np.all(np.diff(b.passage_offsets) >= 1)


def test_tile_planting_forms_two_8x8_blocks():
    b = wls.make_batch("highres_bf16", 2026, B=2, N=2304, d=256, H=2,
                       P=(1,), L_p=2)
    for pl in b.planted:
        assert pl.size == 128
        tiles = np.unique(pl // 576)
        assert tiles.size == 2
        for t in tiles:
            cell = pl[pl // 576 == t] % 576
            r, c = cell // 24, cell % 24
            assert r.max() - r.min() == 7 and c.max() - c.min() == 7


def test_mixed_budgets_cover_choices():
    b = wls.make_batch("mixed_bf16", 2026, N=400, d=64, H=2, L_p=1, k=(48, 96, 192, 384))
    assert set(b.k.tolist()) == {48, 96, 192, 384}
    assert set(b.P.tolist()) == {2, 5, 10, 20}


def test_keep_budget_rejects_nothing_silently():
    with pytest.raises(ValueError):
        wls.make_batch("tiny_fp32", 1, N=50)      # k = 96 > N
