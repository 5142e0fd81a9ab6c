"""Packed-layout metadata, written out from the definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Notation (Sec. 3.1 "Numerical storage"): for sample i with ragged extents
n_{i,r_1..r_q}, p_i is its packed row count, T = sum_i p_i, and the sample
offsets are o_i = sum_{k<i} p_k, so o_0 = 0, o_{i+1} - o_i = p_i, o_B = T
(Appendix A, "Structural invariants").  For singles p_i = N_i; for square
pairs p_i = N_i^2.
"""
from __future__ import annotations

import numpy as np


def offsets(p) -> np.ndarray:
    """Sample offsets o (length B+1) of packed row counts p (Sec. 3.1, Eq. packing)."""
    p = [int(v) for v in p]
    o = [0]
    for v in p:
        if v < 0:
            raise ValueError("negative extent")
        o.append(o[-1] + v)
    return np.asarray(o, dtype=np.int64)


def single_offsets(lengths) -> np.ndarray:
    """eta / cu_seqlens: offsets of a single-axis element of N_i rows."""
    return offsets(lengths)


def pair_offsets(lengths) -> np.ndarray:
    """Offsets of square pair elements (N_i, N_i, C): p_i = N_i * N_i."""
    return offsets([int(n) * int(n) for n in lengths])


def rect_pair_offsets(rows, cols) -> np.ndarray:
    """Offsets of rectangular pair elements (N_i, M_i, C): p_i = N_i * M_i."""
    return offsets([int(n) * int(m) for n, m in zip(rows, cols)])


def pair_row_splits(lengths):
    """Hierarchical row splits of a square pair tensor (Fig. "representation",
    Appendix A "Structural invariants").

    Level 1 counts pair rows per sample, so it equals the single offsets.
    Level 2 delimits the cells of every pair row; it has 1 + sum_i N_i entries.
    """
    level1 = single_offsets(lengths)
    o = pair_offsets(lengths)
    level2 = [0]
    for i, n in enumerate(lengths):
        for a in range(int(n)):
            level2.append(int(o[i]) + (a + 1) * int(n))
    return level1, np.asarray(level2, dtype=np.int64)


def coordinate(o_i: int, extents, coords) -> int:
    """Packed row of ragged coordinates (a_1..a_q) in sample i (Sec. 3.2, Eq. coordinate):
    l_i(a) = o_i + sum_j a_j * prod_{k>j} n_{i,r_k}."""
    row = int(o_i)
    for j, a in enumerate(coords):
        if not 0 <= a < extents[j]:
            raise IndexError("coordinate outside the element")
        stride = 1
        for n in extents[j + 1:]:
            stride *= int(n)
        row += int(a) * stride
    return row


def pair_gather_indices(lengths):
    """The explicit-packing gathers of Fig. "program": for every pair cell, in
    packed order, the single row of its row coordinate and of its column
    coordinate (`rows` and `columns`)."""
    eta = single_offsets(lengths)
    rows, cols = [], []
    for i, n in enumerate(lengths):
        for a in range(int(n)):
            for b in range(int(n)):
                rows.append(int(eta[i]) + a)
                cols.append(int(eta[i]) + b)
    return np.asarray(rows, dtype=np.int64), np.asarray(cols, dtype=np.int64)


def compatible(sizes_a, sizes_b) -> bool:
    """Elementwise alignment check (Sec. 3.2 "Compatibility and semantics"):
    two packed operands align only if every sample has the same logical
    extents, not merely the same packed row count."""
    if len(sizes_a) != len(sizes_b):
        return False
    return all(tuple(x) == tuple(y) for x, y in zip(sizes_a, sizes_b))


def pair_occupancy(rows, cols=None) -> float:
    """rho_pair = sum_i N_i M_i / (B N_max M_max) (Appendix C)."""
    cols = rows if cols is None else cols
    rows = [int(v) for v in rows]
    cols = [int(v) for v in cols]
    return sum(n * m for n, m in zip(rows, cols)) / (len(rows) * max(rows) * max(cols))


def seq_occupancy(lengths) -> float:
    """rho_seq = sum_i N_i / (B N_max) (Sec. 4.4 "Batching policy")."""
    lengths = [int(v) for v in lengths]
    return sum(lengths) / (len(lengths) * max(lengths))


def unpack(values: np.ndarray, o: np.ndarray, shapes) -> list:
    """Logical view D of a packed tensor: sample i's rows o_i..o_{i+1} reshaped
    back to its element shape (inverse of Eq. packing with the ragged-first order)."""
    out = []
    for i, shp in enumerate(shapes):
        blk = values[int(o[i]):int(o[i + 1])]
        out.append(blk.reshape(tuple(shp) + values.shape[1:]))
    return out


def pack(elements, static_shape) -> np.ndarray:
    """Eq. packing: collapse each element's ragged prefix and concatenate."""
    rows = [np.asarray(e).reshape((-1,) + tuple(static_shape)) for e in elements]
    if not rows:
        return np.zeros((0,) + tuple(static_shape))
    return np.concatenate(rows, axis=0)
