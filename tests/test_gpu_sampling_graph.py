"""GPU parity: node sampling and radius graph against the oracle, bit for bit."""

import numpy as np
import pytest

import oracle
from oracle import radius_graph as org
from tests.helpers import announce, gpu_lib
from workloads import make_config

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    return gpu_lib()


@pytest.mark.parametrize("M,s,seed", [(1, 1, 0), (10, 0, 3), (10, 10, 3), (37, 9, 2024), (4096, 1024, 4001),
                                      (65536, 8192, 4002), (1000003, 12345, 2 ** 64 - 5), (300000, 299999, 9)])
def test_sampling_bit_exact(env, M, s, seed):
    dm, lib, torch = env
    announce("sample", M, s, seed)
    got = lib.dsmp_sample_nodes(M, s, seed).cpu().numpy()
    assert np.array_equal(got, oracle.sampling.sample_nodes(M, s, seed))


def test_sampling_rejects_bad_sizes(env):
    dm, lib, torch = env
    with pytest.raises(dm.DsmpError) as ei:
        lib.dsmp_sample_nodes(5, 6, 0)
    assert ei.value.status == dm.INVALID_ARG


def _check_graph(lib, torch, pos, n_dst, r, cap=0, mode=0, seed=0, rows=None):
    dev = torch.device("cuda", 0)
    tpos = torch.from_numpy(np.ascontiguousarray(pos, np.float32)).to(dev)
    E = lib.dsmp_radius_graph_count(tpos, n_dst, r, cap, mode, seed)
    g = lib.dsmp_radius_graph_build(tpos, n_dst, r, cap, mode, seed, capacity=E)
    assert g.n_edges == E
    rp = g.row_ptr.cpu().numpy().astype(np.int64)
    col = g.col[:E].cpu().numpy()
    dst = g.dst[:E].cpu().numpy()
    if rows is None:
        rp_ref, col_ref = org.radius_graph(pos, n_dst, r, cap, mode, seed)
        assert np.array_equal(rp, rp_ref)
        assert np.array_equal(col, col_ref)
        assert np.array_equal(dst, org.dst_of_edges(rp_ref))
        cp_ref, ceid_ref = org.transpose(rp_ref, col_ref, pos.shape[0])
        assert np.array_equal(g.csc_ptr.cpu().numpy(), cp_ref)
        assert np.array_equal(g.csc_eid[:E].cpu().numpy(), ceid_ref)
    else:
        ref = org.rows_subset(pos, rows, n_dst, r, cap, mode, seed)
        for i, lst in zip(rows, ref):
            assert col[rp[i]:rp[i + 1]].tolist() == lst.tolist(), i
        assert np.all(np.diff(rp) >= 0) and rp[-1] == E
        assert np.array_equal(dst, np.repeat(np.arange(n_dst), np.diff(rp)))
        cp = g.csc_ptr.cpu().numpy().astype(np.int64)
        ceid = g.csc_eid[:E].cpu().numpy()
        assert cp[-1] == E and np.array_equal(np.bincount(col, minlength=pos.shape[0]), np.diff(cp))
        assert np.array_equal(col[ceid], np.repeat(np.arange(pos.shape[0]), np.diff(cp)))
        assert np.array_equal(np.sort(ceid), np.arange(E))
        for j in range(0, pos.shape[0], max(1, pos.shape[0] // 50)):
            assert np.all(np.diff(ceid[cp[j]:cp[j + 1]]) > 0)
    return g


def _rand(n, D, seed):
    return np.random.default_rng(seed).uniform(0, 1, (n, D)).astype(np.float32)


def _two_clusters(seed):
    """513 points within 0.002 of each other, and 514 more far away."""
    return np.concatenate([_rand(513, 3, seed) * 1e-3, _rand(514, 3, seed + 1) * 1e-3 + 10.0])


def _long_line(r=0.02, length=300.0, pairs=4000, seed=17):
    """Points along a line 15,000 cells long (one cell across) with pairs at
    the largest float32 distance that passes the radius test, the first point
    just past a cell bound, far from the origin, where the rounding of a cell
    coordinate is largest against the cell margin of 2^-10."""
    g = np.random.default_rng(seed)
    f32 = np.float32
    r2 = f32(r) * f32(r)
    c = r * (1.0 + 2.0 ** -10)
    k = g.integers(int(0.6 * length / c), int(length / c) - 2, pairs)
    x1 = ((k + g.uniform(0.9e-3, 1.5e-3, pairs)) * c).astype(f32)
    x2 = (x1 + f32(r)).astype(f32)
    for _ in range(8):   # the largest x2 with fl(fl(x2 - x1)^2) <= fl(r^2)
        d = (x2 - x1).astype(f32)
        over = (d * d).astype(f32) > r2
        x2 = np.where(over, np.nextafter(x2, f32(-np.inf)), x2)
    up = np.nextafter(x2, f32(np.inf))
    du = (up - x1).astype(f32)
    x2 = np.where((du * du).astype(f32) <= r2, up, x2)
    y = np.full(pairs, 5e-4, f32)
    pts = [np.array([[0.0, 0.0], [length, 1e-3]], f32),
           np.stack([x1, y], 1), np.stack([x2, y], 1),
           np.stack([g.uniform(0, length, 2000), g.uniform(0, 1e-3, 2000)], 1).astype(f32)]
    return np.concatenate(pts)


CASES = {
    "2d_uncapped": (lambda: _rand(3000, 2, 1), 2500, 0.03, 0, 0),
    "2d_knn5": (lambda: _rand(3000, 2, 2), 3000, 0.05, 5, 0),
    "2d_random5": (lambda: _rand(3000, 2, 3), 2800, 0.05, 5, 1),
    "3d_uncapped": (lambda: _rand(3000, 3, 4), 3000, 0.08, 0, 0),
    "3d_knn7": (lambda: _rand(3000, 3, 5), 2000, 0.12, 7, 0),
    "3d_random7": (lambda: _rand(3000, 3, 6), 3000, 0.12, 7, 1),
    "lattice64_ties_knn": (lambda: np.stack(np.meshgrid(np.linspace(0, 1, 64), np.linspace(0, 1, 64),
                                                        indexing="ij"), -1).reshape(-1, 2).astype(np.float32),
                           4096, 0.08, 12, 0),
    "lattice_uncapped": (lambda: np.stack(np.meshgrid(np.linspace(0, 1, 64), np.linspace(0, 1, 64),
                                                      indexing="ij"), -1).reshape(-1, 2).astype(np.float32),
                         4096, 0.08, 0, 0),
    "coincident_r0": (lambda: np.repeat(_rand(200, 2, 7), 3, axis=0), 600, 0.0, 0, 0),
    "empty_tiny_r": (lambda: _rand(2000, 3, 8), 2000, 1e-6, 0, 0),
    "complete_graph": (lambda: _rand(1500, 2, 9), 1500, 5.0, 0, 0),
    "complete_capped": (lambda: _rand(1500, 3, 10), 1500, 5.0, 100, 0),
    "clustered": (lambda: np.concatenate([_rand(1000, 2, 11) * 1e-3, _rand(1000, 2, 12)]), 2000, 0.01, 16, 0),
    "no_destinations": (lambda: _rand(100, 2, 13), 0, 0.1, 0, 0),
    "single_point": (lambda: _rand(1, 3, 14), 1, 0.1, 0, 0),
    "halo_far": (lambda: np.concatenate([_rand(500, 2, 15), _rand(500, 2, 16) + 5.0]), 500, 0.08, 0, 0),
    "long_line_15k_cells": (lambda: _long_line(), 10002, 0.02, 0, 0),
    # rows of 65..168 candidates capped at 40: the cap is selected in registers
    "dense_knn40": (lambda: _rand(4000, 3, 20), 4000, 0.2, 40, 0),
    # rows of 130..555 candidates, a cap above 64: both the register select
    # (up to 512 candidates) and the sort in shared memory (beyond)
    "dense_random80": (lambda: _rand(4000, 2, 21), 4000, 0.2, 80, 1),
    # two tight clusters: rows of exactly 512 and of 513 candidates
    "clusters_512_513_knn": (lambda: _two_clusters(22), 1027, 0.01, 30, 0),
    "clusters_512_513_random": (lambda: _two_clusters(24), 1027, 0.01, 30, 1),
    # capped graphs select each row in one pass: rows of 58..264 candidates
    # (the last few beyond what that pass holds), and a cap of exactly 64
    "dense_random48": (lambda: _rand(4000, 2, 25), 4000, 0.132, 48, 1),
    "dense_knn64": (lambda: _rand(4000, 3, 26), 4000, 0.2, 64, 0),
    # a cap of one (the select keeps the single smallest key), and a cap above
    # every row's size (no select; the fill pass, caps above 64)
    "3d_knn1": (lambda: _rand(3000, 3, 27), 3000, 0.12, 1, 0),
    "2d_random1": (lambda: _rand(3000, 2, 28), 3000, 0.05, 1, 1),
    "3d_cap200": (lambda: _rand(3000, 3, 29), 3000, 0.12, 200, 0),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_graph_bit_exact(env, name):
    dm, lib, torch = env
    mk, n_dst, r, cap, mode = CASES[name]
    announce("graph", name)
    _check_graph(lib, torch, mk(), n_dst, r, cap, mode, seed=123)


@pytest.mark.parametrize("cap", [0, 10])
def test_graph_capacity_error_reports_E(env, cap):
    dm, lib, torch = env
    pos = torch.from_numpy(_rand(1000, 2, 20)).cuda()
    E = lib.dsmp_radius_graph_count(pos, 1000, 0.05, cap)
    with pytest.raises(dm.DsmpError) as ei:
        lib.dsmp_radius_graph_build(pos, 1000, 0.05, cap, capacity=E - 1)
    assert ei.value.status == dm.CAPACITY


def test_graph_row_limit_is_unsupported(env):
    dm, lib, torch = env
    pos = torch.from_numpy(_rand(5000, 2, 21)).cuda()
    with pytest.raises(dm.DsmpError) as ei:
        lib.dsmp_radius_graph_count(pos, 5000, 10.0)
    assert ei.value.status == dm.UNSUPPORTED


def _sampled(k):
    w = make_config(k)
    pos, n_dst = [], w.n_dst
    for p in w.parts:
        idx = oracle.sampling.sample_nodes(p.pos.shape[0], p.s, p.seed)
        pos.append(p.pos[idx])
    return w, np.concatenate(pos)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_graph_workload_full(env, k):
    dm, lib, torch = env
    announce("graph workload", k)
    w, pos = _sampled(k)
    _check_graph(lib, torch, pos, w.n_dst, w.r, w.cap, w.cap_mode)


@pytest.mark.parametrize("k", [4, 5])
def test_graph_workload_rows(env, k):
    dm, lib, torch = env
    announce("graph workload rows", k)
    w, pos = _sampled(k)
    rows = np.random.default_rng(k).choice(w.n_dst, 400, replace=False)
    rows = np.concatenate([rows, [0, w.n_dst - 1]])
    _check_graph(lib, torch, pos, w.n_dst, w.r, w.cap, w.cap_mode, rows=rows)


def test_graph_is_deterministic(env):
    dm, lib, torch = env
    pos = torch.from_numpy(_rand(20000, 3, 30)).cuda()
    a = lib.dsmp_radius_graph_build(pos, 20000, 0.05, 10)
    b = lib.dsmp_radius_graph_build(pos, 20000, 0.05, 10)
    for x, y in ((a.row_ptr, b.row_ptr), (a.col, b.col), (a.csc_eid, b.csc_eid)):
        assert torch.equal(x, y)
