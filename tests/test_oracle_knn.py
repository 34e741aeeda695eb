"""Pins of the oracle's 3D neighbour tables (Eq. 13) on the CPU."""
import numpy as np
import pytest
from scipy.spatial import cKDTree

from oracle import knn
from scenes import make_scene, subscene


def _pos(n, seed):
    s = make_scene("n4096_d1152", seed)
    return subscene(s, np.arange(n)).pos


@pytest.mark.parametrize("g", [1, 5, 32])
def test_distances_match_kdtree(g):
    # A KD-tree (an independent algorithm) returns the same neighbour
    # distances; where no two distances tie, the same neighbours.
    pos = _pos(700, 0)
    nb = knn.knn_ref(pos, g)
    tree = cKDTree(pos.astype(np.float64))
    dist, idx = tree.query(pos.astype(np.float64), k=g)
    dist = dist.reshape(len(pos), g)
    idx = idx.reshape(len(pos), g)
    p = pos.astype(np.float64)
    ours = np.sqrt(((p[:, None, :] - p[nb]) ** 2).sum(axis=2))
    assert np.allclose(ours, dist, rtol=1e-12, atol=1e-12)
    d_sorted = np.sort(knn.sq_dist_rows(pos), axis=1)
    untied = np.all(np.diff(d_sorted[:, : g + 1], axis=1) > 0, axis=1)
    assert untied.sum() > 600
    assert np.array_equal(nb[untied], idx[untied])


def test_self_is_nearest_without_duplicates():
    pos = _pos(300, 1)
    nb = knn.knn_ref(pos, 4)
    assert np.array_equal(nb[:, 0], np.arange(300))


def test_ties_go_to_smaller_index():
    # Duplicated positions are at distance 0 from each other: the neighbour
    # list starts with all copies in index order, whichever copy asks.
    pos = _pos(50, 2).copy()
    pos[[7, 20, 33]] = pos[20]
    nb = knn.knn_ref(pos, 3)
    for t in (7, 20, 33):
        assert nb[t].tolist() == [7, 20, 33]
    # Four tokens on a cross around a centre: equal distances, index order.
    cross = np.array([[0, 0, 0], [1, 0, 0], [-1, 0, 0], [0, 1, 0], [0, -1, 0], [5, 5, 5]], np.float32)
    assert knn.knn_ref(cross, 5, rows=[0]).tolist() == [[0, 1, 2, 3, 4]]


def test_full_neighbourhood_is_everyone_by_distance():
    pos = _pos(40, 3)
    nb = knn.knn_ref(pos, 40)
    assert all(sorted(r.tolist()) == list(range(40)) for r in nb)
    d = knn.sq_dist_rows(pos)
    for t in range(40):
        assert np.all(np.diff(d[t, nb[t]]) >= 0)


def test_rows_subset_matches_full_table():
    pos = _pos(200, 4)
    full = knn.knn_ref(pos, 9)
    rows = np.array([0, 17, 199, 100])
    assert np.array_equal(knn.knn_ref(pos, 9, rows=rows), full[rows])
