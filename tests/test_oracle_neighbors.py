"""Pins for the oracle's neighbour sets: brute force vs cell list, vs SciPy's
periodic k-d tree (an independent library routine), exact boundary cases."""
import numpy as np
import pytest
from scipy.spatial import cKDTree

import oracle.neighbors as nb


def _sets(offsets, idx):
    return [set(idx[offsets[i]:offsets[i + 1]].tolist()) for i in range(len(offsets) - 1)]


@pytest.mark.parametrize("shape,n,rl", [
    ((13.0, 13.0, 13.0), 150, 6.5),      # one cell per axis
    ((14.0, 19.5, 27.0), 300, 6.5),      # 2, 3 and 4 cells per axis
    ((30.0, 30.0, 13.1), 500, 6.0),      # non-cubic
])
def test_cell_list_equals_brute_force(shape, n, rl):
    rng = np.random.default_rng(n)
    box = np.array(shape)
    pos = rng.uniform(0, 1, (n, 3)) * box
    pos[:10] += box * rng.integers(-2, 3, (10, 3))   # some atoms outside [0, L)
    a = nb.brute_force_neighbors(pos, box, rl)
    b = nb.cell_list_neighbors(pos, box, rl)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_matches_periodic_kdtree():
    rng = np.random.default_rng(11)
    box = np.array([20.0, 22.0, 25.0])
    pos = rng.uniform(0, 1, (700, 3)) * box
    rl = 6.5
    off, idx = nb.brute_force_neighbors(pos, box, rl)
    tree = cKDTree(pos, boxsize=box)
    pairs = tree.query_pairs(rl)
    ref = [set() for _ in range(len(pos))]
    for i, j in pairs:
        ref[i].add(j)
        ref[j].add(i)
    assert _sets(off, idx) == ref


def test_symmetric_and_no_self():
    rng = np.random.default_rng(5)
    box = np.array([15.0, 15.0, 15.0])
    pos = rng.uniform(0, 15, (200, 3))
    off, idx = nb.brute_force_neighbors(pos, box, 6.5)
    S = _sets(off, idx)
    for i, s in enumerate(S):
        assert i not in s
        for j in s:
            assert i in S[j]


def test_exact_boundary_is_excluded():
    box = np.array([20.0, 20.0, 20.0])
    rl = 6.5
    below = np.nextafter(6.5, 0.0)
    pos = np.array([[1.0, 1.0, 1.0],
                    [7.5, 1.0, 1.0],            # dx = 6.5 exactly: d2 == rl^2 -> excluded
                    [1.0, 1.0 + below, 1.0],    # just inside
                    [1.0, 1.0, 1.0 - 6.5 + 20.0]])  # 6.5 through the periodic face -> excluded
    off, idx = nb.brute_force_neighbors(pos, box, rl)
    S = _sets(off, idx)
    assert 1 not in S[0]
    assert 2 in S[0]
    assert 3 not in S[0]


def test_wrap_definition():
    box = np.array([10.0, 10.0, 10.0])
    x = np.array([[-1e-20, 10.0, 25.0], [-10.0, 9.999999999999998, -0.5]])
    w = nb.wrap_positions(x, box)
    assert np.all(w >= 0) and np.all(w < box)
    np.testing.assert_array_equal(w[0], [0.0, 0.0, 5.0])   # -1e-20 + 10 rounds to 10 -> 0
    np.testing.assert_array_equal(w[1], [0.0, 9.999999999999998, 9.5])


def test_fcc_shell_counts():
    """Perfect FCC a = 3.6: 78 neighbours within 6.0 (shells 12+6+24+12+24)
    and 86 within 6.5 (adds the 8 at a*sqrt(3))."""
    import synth
    pos, box = synth.lattice("fcc", 4, 3.6)
    off, idx = nb.brute_force_neighbors(pos, box, 6.0)
    assert set(np.diff(off)) == {78}
    off, idx = nb.brute_force_neighbors(pos, box, 6.5)
    assert set(np.diff(off)) == {86}
    pos, box = synth.lattice("bcc", 5, 3.2)
    off, idx = nb.brute_force_neighbors(pos, box, 6.0)
    assert set(np.diff(off)) == {58}
