"""Pins of the oracle's surface-code geometry (App. A.1.2) against code-theoretic facts."""
import itertools
import os

import numpy as np
import pytest

from oracle import decoder as O

DISTANCES = [3, 5, 7, 9, 11, 13, 17, 25]


def gf2_rank(rows):
    m = np.array(rows, dtype=np.uint8) % 2
    rank = 0
    ncols = m.shape[1]
    for col in range(ncols):
        piv = None
        for r in range(rank, m.shape[0]):
            if m[r, col]:
                piv = r
                break
        if piv is None:
            continue
        m[[rank, piv]] = m[[piv, rank]]
        for r in range(m.shape[0]):
            if r != rank and m[r, col]:
                m[r] ^= m[rank]
        rank += 1
    return rank


def check_matrix(d, kind):
    cells = [c for c in O.stabilizer_cells(d) if O.stabilizer_kind(c) == kind]
    H = np.zeros((len(cells), d * d), dtype=np.uint8)
    for k, cell in enumerate(cells):
        for i, j in O.stabilizer_support(d, cell):
            H[k, i * d + j] = 1
    return H


@pytest.mark.parametrize("d", DISTANCES)
def test_counts(d):
    cells = O.stabilizer_cells(d)
    assert len(cells) == d * d - 1
    weights = [len(O.stabilizer_support(d, c)) for c in cells]
    assert weights.count(4) == (d - 1) ** 2
    assert weights.count(2) == 2 * (d - 1)
    kinds = [O.stabilizer_kind(c) for c in cells]
    assert kinds.count("X") == kinds.count("Z") == (d * d - 1) // 2
    assert cells == sorted(cells)                       # row-major token order
    pos = O.grid_positions(d)
    assert len(set(pos.tolist())) == len(pos) and pos.max() < (d + 1) ** 2


@pytest.mark.parametrize("d", DISTANCES)
def test_commuting_independent_one_logical(d):
    HX, HZ = check_matrix(d, "X"), check_matrix(d, "Z")
    # every X check overlaps every Z check on an even number of data qubits
    assert not ((HX.astype(int) @ HZ.T.astype(int)) % 2).any()
    # independent checks, n - rank(HX) - rank(HZ) = 1 encoded qubit
    assert gf2_rank(HX) == HX.shape[0] and gf2_rank(HZ) == HZ.shape[0]
    assert d * d - gf2_rank(HX) - gf2_rank(HZ) == 1
    # each data qubit is checked by one or two stabilizers of each kind
    for H in (HX, HZ):
        col = H.sum(axis=0)
        assert col.min() >= 1 and col.max() <= 2


def test_distance_three():
    """The smallest undetectable logical error of the d=3 layout has weight 3."""
    d = 3
    HX, HZ = check_matrix(d, "X"), check_matrix(d, "Z")
    rowspace_x = {tuple((np.array(c) @ HX) % 2) for c in itertools.product([0, 1], repeat=HX.shape[0])}
    best = d * d
    for v in itertools.product([0, 1], repeat=d * d):
        v = np.array(v, dtype=np.uint8)
        if v.any() and not ((HZ @ v) % 2).any() and tuple(v) not in rowspace_x:
            best = min(best, int(v.sum()))
    assert best == 3


def test_d3_layout_golden():
    path = os.path.join(os.path.dirname(__file__), "golden", "d3_layout.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    cells = O.stabilizer_cells(3)
    assert len(rows) == len(cells)
    for tok, row in enumerate(rows):
        assert int(row[0]) == tok
        cell = (int(row[1]), int(row[2]))
        assert cells[tok] == cell
        assert O.stabilizer_kind(cell) == row[3]
        support = sorted(tuple(int(x) for x in s.strip("()").split(",")) for s in row[4:])
        assert sorted(O.stabilizer_support(3, cell)) == support
