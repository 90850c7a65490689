"""Pins for the oracle's radius-graph builder (CPU only)."""

import itertools

import numpy as np
import pytest
from scipy import stats

from oracle import radius_graph as rg
from oracle import rng


def _edges(row_ptr, col):
    dst = rg.dst_of_edges(row_ptr)
    return set(zip(dst.tolist(), np.asarray(col).tolist()))


def _scalar_d2(pi, pj):
    # one pair at a time with numpy float32 scalars: the canonical order
    acc = np.float32(0)
    for a in range(len(pi)):
        dx = np.float32(np.float32(pj[a]) - np.float32(pi[a]))
        sq = np.float32(dx * dx)
        acc = sq if a == 0 else np.float32(acc + sq)
    return acc


def _pairs_bruteforce(pos, n_dst, r, cap=0, mode=rg.CAP_KNN, seed=0):
    """Pure-Python all-pairs reference on tiny inputs."""
    r32 = np.float32(r)
    r2 = np.float32(r32 * r32)
    n_src = pos.shape[0]
    rows = []
    for i in range(n_dst):
        cand = []
        for j in range(n_src):
            if j == i:
                continue
            d2 = _scalar_d2(pos[i], pos[j])
            if d2 <= r2:
                key = float(d2) if mode == rg.CAP_KNN else rng.splitmix64_scalar(seed, i * n_src + j)
                cand.append((key, j))
        if cap and len(cand) > cap:
            cand = sorted(cand)[:cap]
        rows.append(sorted(j for _, j in cand))
    return rows


def _rows(row_ptr, col):
    return [col[row_ptr[i]:row_ptr[i + 1]].tolist() for i in range(len(row_ptr) - 1)]


@pytest.mark.parametrize("D", [2, 3])
@pytest.mark.parametrize("cap,mode", [(0, rg.CAP_KNN), (5, rg.CAP_KNN), (4, rg.CAP_RANDOM)])
def test_matches_pure_python_bruteforce(D, cap, mode):
    g = np.random.default_rng(10 + D)
    pos = g.uniform(0, 1, (120, D)).astype(np.float32)
    r = 0.25 if D == 2 else 0.35
    rp, col = rg.radius_graph(pos, 100, r, cap, mode, seed=77, method="brute")
    assert _rows(rp, col) == _pairs_bruteforce(pos, 100, r, cap, mode, seed=77)


@pytest.mark.parametrize("D", [2, 3])
@pytest.mark.parametrize("cap,mode", [(0, rg.CAP_KNN), (7, rg.CAP_KNN), (7, rg.CAP_RANDOM)])
def test_tree_candidates_equal_all_pairs(D, cap, mode):
    g = np.random.default_rng(20 + D)
    pos = g.uniform(0, 1, (1500, D)).astype(np.float32)
    r = 0.06 if D == 2 else 0.12
    a = rg.radius_graph(pos, 1400, r, cap, mode, seed=3, method="brute")
    b = rg.radius_graph(pos, 1400, r, cap, mode, seed=3, method="tree")
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    rows = [3, 999, 0, 1399]
    sub = rg.rows_subset(pos, rows, 1400, r, cap, mode, seed=3)
    for i, lst in zip(rows, sub):
        assert lst.tolist() == a[1][a[0][i]:a[0][i + 1]].tolist()


def _lattice_points_in_ball(R2, D):
    """Closed form: integer points with |v|^2 <= R2, excluding the origin;
    also the smallest gap between R2 and any lattice |v|^2 (to check that
    float32 rounding cannot change the answer)."""
    R = int(np.floor(np.sqrt(R2))) + 1
    cnt, gap = 0, np.inf
    for v in itertools.product(range(-R, R + 1), repeat=D):
        s = sum(t * t for t in v)
        gap = min(gap, abs(s - R2))
        if s <= R2 and s > 0:
            cnt += 1
    return cnt, gap


@pytest.mark.parametrize("n,D,r,want", [(64, 2, 0.08, 80), (256, 2, 0.04, None),
                                         (21, 3, 0.12, 56), (11, 3, 0.25, 80)])
def test_interior_lattice_degree_closed_form(n, D, r, want):
    R2 = (r * (n - 1)) ** 2
    closed, gap = _lattice_points_in_ball(R2, D)
    assert gap / R2 > 1e-4        # no lattice point near the sphere
    if want is not None:
        assert closed == want
    t = np.linspace(0, 1, n)
    grids = np.meshgrid(*([t] * D), indexing="ij")
    pos = np.stack([g.ravel() for g in grids], 1).astype(np.float32)
    rp, col = rg.radius_graph(pos, pos.shape[0], r, method="tree")
    deg = np.diff(rp)
    R = int(np.ceil(np.sqrt(R2)))
    idx = np.stack(np.unravel_index(np.arange(pos.shape[0]), [n] * D), 1)
    interior = np.all((idx >= R) & (idx <= n - 1 - R), axis=1)
    assert interior.any()
    assert np.all(deg[interior] == closed)
    assert np.all(deg[~interior] <= closed)


def test_uncapped_graph_is_symmetric():
    g = np.random.default_rng(3)
    pos = g.uniform(0, 1, (2000, 2)).astype(np.float32)
    rp, col = rg.radius_graph(pos, 2000, 0.05)
    E = _edges(rp, col)
    assert all((j, i) in E for (i, j) in E)
    assert all(i != j for (i, j) in E)


def test_complete_and_empty_graphs():
    g = np.random.default_rng(4)
    pos = g.uniform(0, 1, (300, 3)).astype(np.float32)
    rp, col = rg.radius_graph(pos, 300, 10.0)
    assert np.all(np.diff(rp) == 299)
    rp, col = rg.radius_graph(pos, 300, 1e-6)
    assert rp[-1] == 0 and col.size == 0


def test_coincident_points_and_no_self_loops():
    pos = np.array([[0.5, 0.5], [0.5, 0.5], [0.5, 0.5], [0.9, 0.9]], np.float32)
    rp, col = rg.radius_graph(pos, 4, 0.0)      # r = 0 keeps exact coincidences only
    assert _rows(rp, col) == [[1, 2], [0, 2], [0, 1], []]


def test_knn_tie_break_by_index():
    # 1-D-like line: node 0 at centre, 4 neighbours at equal distance
    pos = np.array([[0, 0], [1, 0], [-1, 0], [0, 1], [0, -1], [2, 0]], np.float32)
    rp, col = rg.radius_graph(pos, 1, 1.0, cap=2, cap_mode=rg.CAP_KNN)
    assert _rows(rp, col) == [[1, 2]]
    rp, col = rg.radius_graph(pos, 1, 2.0, cap=5, cap_mode=rg.CAP_KNN)
    assert _rows(rp, col) == [[1, 2, 3, 4, 5]]
    rp, col = rg.radius_graph(pos, 1, 2.0, cap=4, cap_mode=rg.CAP_KNN)
    assert _rows(rp, col) == [[1, 2, 3, 4]]


def test_halo_sources_are_not_destinations():
    g = np.random.default_rng(8)
    pos = g.uniform(0, 1, (500, 2)).astype(np.float32)
    rp, col = rg.radius_graph(pos, 400, 0.1)
    assert rp.size == 401
    assert col.max() >= 400          # halo nodes do feed owned ones
    full_rp, full_col = rg.radius_graph(pos, 500, 0.1)
    assert np.array_equal(rp, full_rp[:401]) and np.array_equal(col, full_col[:rp[-1]])


def test_random_cap_is_uniform_subset():
    # centre 0 with 10 equidistant-enough candidates; keep 3 of them
    ang = np.linspace(0, 2 * np.pi, 10, endpoint=False)
    pos = np.concatenate([[[0, 0]], np.stack([np.cos(ang), np.sin(ang)], 1) * 0.5]).astype(np.float32)
    counts = np.zeros(11)
    trials = 3000
    for seed in range(trials):
        rp, col = rg.radius_graph(pos, 1, 1.0, cap=3, cap_mode=rg.CAP_RANDOM, seed=seed)
        assert col.size == 3 and np.all(np.diff(col) > 0)
        counts[col] += 1
    expected = trials * 3 / 10
    chi2 = ((counts[1:] - expected) ** 2 / expected).sum()
    assert stats.chi2.sf(chi2, 9) > 1e-4


def test_transpose_groups_by_source_in_edge_order():
    g = np.random.default_rng(9)
    pos = g.uniform(0, 1, (300, 2)).astype(np.float32)
    rp, col = rg.radius_graph(pos, 250, 0.1, cap=6)
    cp, ceid = rg.transpose(rp, col, 300)
    assert cp[-1] == col.size
    for j in range(300):
        eids = ceid[cp[j]:cp[j + 1]]
        assert np.all(col[eids] == j)
        assert np.all(np.diff(eids) > 0)
