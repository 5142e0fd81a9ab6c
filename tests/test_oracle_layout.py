"""Pins of the oracle's layout metadata against what the paper fixes."""
import json
import os

import numpy as np
import pytest

from oracle import layout
from paper_2609_30379_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_worked_example_offsets_and_splits():
    g = _gold("worked_example_2_3.json")
    L = g["lengths"]
    assert layout.single_offsets(L).tolist() == g["single_offsets"]
    assert layout.pair_offsets(L).tolist() == g["pair_offsets"]
    lvl1, lvl2 = layout.pair_row_splits(L)
    assert lvl1.tolist() == g["pair_row_splits_level1"]
    assert lvl2.tolist() == g["pair_row_splits_level2"]
    assert len(lvl2) == 1 + sum(L)
    # first-level splits equal the single offsets but not the pair offsets
    assert lvl1.tolist() == layout.single_offsets(L).tolist()
    assert lvl1.tolist() != layout.pair_offsets(L).tolist()


def test_worked_example_gather_lists():
    g = _gold("worked_example_2_3.json")
    rows, cols = layout.pair_gather_indices(g["lengths"])
    assert rows.tolist() == g["rows"]
    assert cols.tolist() == g["columns"]
    assert len(rows) == 13


@pytest.mark.parametrize("seed", range(6))
def test_offset_invariants(seed):
    rng = np.random.default_rng(seed)
    L = rng.integers(0, 9, size=rng.integers(1, 12))
    for o, p in ((layout.single_offsets(L), L), (layout.pair_offsets(L), L * L)):
        assert o[0] == 0
        assert np.array_equal(np.diff(o), p)
        assert o[-1] == p.sum()
    _, lvl2 = layout.pair_row_splits(L)
    assert len(lvl2) == 1 + L.sum()
    assert lvl2[-1] == (L * L).sum()
    assert np.all(np.diff(lvl2) >= 0)


def test_position_count_is_sum_of_squares():
    # pair states occupy sum_i N_i^2 positions rather than B N_max^2 (abstract)
    L = [5, 1, 3]
    assert layout.pair_offsets(L)[-1] == 25 + 1 + 9
    assert layout.pair_offsets(L)[-1] < len(L) * max(L) ** 2


def test_zero_volume_shapes_are_distinct():
    # (0,3) and (0,7) have coincident offsets but different sizes (Sec. 3.1)
    a, b = [(0, 3)], [(0, 7)]
    assert layout.rect_pair_offsets([0], [3]).tolist() == layout.rect_pair_offsets([0], [7]).tolist()
    assert not layout.compatible(a, b)


def test_equal_volume_shapes_are_incompatible():
    # (2,6,C) and (3,4,C) both hold twelve rows but cannot be added (Sec. 3.2)
    assert layout.rect_pair_offsets([2], [6])[-1] == layout.rect_pair_offsets([3], [4])[-1] == 12
    assert not layout.compatible([(2, 6)], [(3, 4)])
    assert layout.compatible([(2, 6)], [(2, 6)])


def test_coordinate_map_matches_packing_order():
    L = [3, 0, 4, 1]
    o = layout.pair_offsets(L)
    rows = 0
    for i, n in enumerate(L):
        for a in range(n):
            for b in range(n):
                assert layout.coordinate(o[i], (n, n), (a, b)) == o[i] + a * n + b == rows
                rows += 1
    assert rows == o[-1]
    with pytest.raises(IndexError):
        layout.coordinate(0, (2, 2), (2, 0))


def test_pack_unpack_roundtrip():
    rng = np.random.default_rng(3)
    L = [2, 0, 3]
    elems = [rng.standard_normal((n, n, 4)) for n in L]
    V = layout.pack(elems, (4,))
    assert V.shape == (13, 4)
    back = layout.unpack(V, layout.pair_offsets(L), [(n, n) for n in L])
    for e, b in zip(elems, back):
        assert np.array_equal(e, b)


def test_occupancy():
    assert layout.pair_occupancy([2, 4]) == pytest.approx((4 + 16) / (2 * 16))
    assert layout.seq_occupancy([2, 4]) == pytest.approx(6 / 8)
    assert layout.pair_occupancy([3, 2], [1, 5]) == pytest.approx((3 + 10) / (2 * 3 * 5))


def test_generator_lengths_fixture():
    g = _gold("workload_lengths.json")
    for name, w in synth.WORKLOADS.items():
        assert synth.lengths_for(w).tolist() == g[name], name
        if w.col_dist:
            assert synth.cols_for(w).tolist() == g[name + ".cols"], name
