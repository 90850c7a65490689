"""Radius-graph kernel construction with edge cap (oracle side; test infrastructure only).

Sec. 2.1 builds, around every sampled centre node i, a graph kernel whose edges
join i to the nodes j within radius r; when a centre has more than n_e such
edges, n_e of them are kept.  Algorithm 1 does this with its edge-index
creation step followed by its edge-sampling step.

Readings (the paper is silent on each):

* no self loops (j != i); the root term of the layer carries i itself;
* the radius test is inclusive and evaluated in float32 without fused
  multiply-add, in this order:
      dx_a = fl(p_j[a] - p_i[a])            for each axis a
      d2   = fl(fl(dx_0*dx_0) + fl(dx_1*dx_1))                 (D = 2)
      d2   = fl(fl(fl(dx_0*dx_0) + fl(dx_1*dx_1)) + fl(dx_2*dx_2))   (D = 3)
      keep iff d2 <= fl(r*r)
* the cap has two modes:
    - "knn"    keep the n_e smallest (d2, j) pairs (the workloads' cap);
    - "random" keep the n_e smallest (splitmix64(seed, i*N_src + j), j) pairs,
               i.e. a uniform random subset without replacement (the
               paper's own edge sampling);
* destinations are the first n_dst nodes; sources are all n_src nodes (owned
  nodes first, then halo nodes of a sub-domain);
* every row is returned with its sources in ascending order (CSR).

Candidates are found with a KD-tree at a padded radius (or by brute force);
the final decision always uses the float32 formula above.

Pinned by: brute-force all-pairs search, closed-form lattice degrees (integer
lattice-point counts in a disc or ball), symmetry of uncapped graphs, the
complete and the empty graph, coincident points, and brute-force selection
for both cap modes.
"""

import numpy as np

from .rng import splitmix64

CAP_KNN = 0
CAP_RANDOM = 1


def _d2_f32(pi: np.ndarray, pj: np.ndarray) -> np.ndarray:
    """Canonical float32 squared distance, rows of pj against rows of pi."""
    pi = np.asarray(pi, dtype=np.float32)
    pj = np.asarray(pj, dtype=np.float32)
    D = pi.shape[-1]
    acc = None
    for a in range(D):
        dx = np.subtract(pj[..., a], pi[..., a], dtype=np.float32)
        sq = np.multiply(dx, dx, dtype=np.float32)
        acc = sq if acc is None else np.add(acc, sq, dtype=np.float32)
    return acc


def _row_select(i, cand, d2, r2, cap, cap_mode, seed, n_src):
    keep = (d2 <= r2) & (cand != i)
    cj = cand[keep]
    cd = d2[keep]
    if cap > 0 and cj.size > cap:
        if cap_mode == CAP_KNN:
            order = np.lexsort((cj, cd))              # primary d2, then j
        elif cap_mode == CAP_RANDOM:
            keys = splitmix64(seed, np.uint64(i) * np.uint64(n_src) + cj.astype(np.uint64))
            order = np.lexsort((cj, keys))
        else:
            raise ValueError("unknown cap mode")
        cj = cj[order[:cap]]
    return np.sort(cj)


def radius_graph(pos, n_dst: int, r: float, cap: int = 0, cap_mode: int = CAP_KNN,
                 seed: int = 0, method: str = "auto"):
    """CSR radius graph.

    pos   : float32 [n_src, D] positions (D = 2 or 3)
    n_dst : destinations are rows [0, n_dst)
    r     : radius (converted to float32; the test uses fl32(r*r))
    cap   : 0 for no cap, else n_e
    method: "brute" (all pairs), "tree" (KD-tree candidates) or "auto"

    Returns (row_ptr int64 [n_dst+1], col int32 [E]).
    """
    pos = np.ascontiguousarray(pos, dtype=np.float32)
    n_src, D = pos.shape
    if not (0 <= n_dst <= n_src):
        raise ValueError("need 0 <= n_dst <= n_src")
    r32 = np.float32(r)
    r2 = np.multiply(r32, r32, dtype=np.float32)
    if method == "auto":
        method = "brute" if n_src <= 3000 else "tree"
    rows = []
    if method == "brute":
        allj = np.arange(n_src)
        for i in range(n_dst):
            d2 = _d2_f32(pos[i][None, :], pos)
            rows.append(_row_select(i, allj, d2, r2, cap, cap_mode, seed, n_src))
    elif method == "tree":
        from scipy.spatial import cKDTree
        tree = cKDTree(pos.astype(np.float64))
        # padded radius: float32 rounding moves d2 by a few ulp at most
        pad = float(r32) * (1.0 + 1e-4) + 1e-6 * float(np.abs(pos).max(initial=0.0))
        lists = tree.query_ball_point(pos[:n_dst].astype(np.float64), pad)
        for i in range(n_dst):
            cand = np.asarray(lists[i], dtype=np.int64)
            d2 = _d2_f32(pos[i][None, :], pos[cand]) if cand.size else np.zeros(0, np.float32)
            rows.append(_row_select(i, cand, d2, r2, cap, cap_mode, seed, n_src))
    else:
        raise ValueError(method)
    counts = np.array([x.size for x in rows], dtype=np.int64)
    row_ptr = np.zeros(n_dst + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col = np.concatenate(rows).astype(np.int32) if rows else np.zeros(0, np.int32)
    return row_ptr, col


def rows_subset(pos, rows, n_dst: int, r: float, cap: int = 0, cap_mode: int = CAP_KNN,
                seed: int = 0):
    """Sorted source lists for the destination rows listed in ``rows`` only.

    Same rule as ``radius_graph``; used to check sampled rows of graphs too
    large to build whole on the host.
    """
    pos = np.ascontiguousarray(pos, dtype=np.float32)
    n_src = pos.shape[0]
    r32 = np.float32(r)
    r2 = np.multiply(r32, r32, dtype=np.float32)
    from scipy.spatial import cKDTree
    tree = cKDTree(pos.astype(np.float64))
    pad = float(r32) * (1.0 + 1e-4) + 1e-6 * float(np.abs(pos).max(initial=0.0))
    out = []
    for i in rows:
        i = int(i)
        if not (0 <= i < n_dst):
            raise ValueError("row out of range")
        cand = np.asarray(tree.query_ball_point(pos[i].astype(np.float64), pad), dtype=np.int64)
        d2 = _d2_f32(pos[i][None, :], pos[cand]) if cand.size else np.zeros(0, np.float32)
        out.append(_row_select(i, cand, d2, r2, cap, cap_mode, seed, n_src).astype(np.int32))
    return out


def dst_of_edges(row_ptr) -> np.ndarray:
    """Destination (row) of every CSR edge."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    return np.repeat(np.arange(row_ptr.size - 1), np.diff(row_ptr)).astype(np.int32)


def transpose(row_ptr, col, n_src: int):
    """Edges grouped by source: csc_ptr [n_src+1], csc_eid [E] (ascending edge id per source)."""
    col = np.asarray(col, dtype=np.int64)
    order = np.argsort(col, kind="stable")
    counts = np.bincount(col, minlength=n_src)
    csc_ptr = np.zeros(n_src + 1, dtype=np.int64)
    np.cumsum(counts, out=csc_ptr[1:])
    return csc_ptr, order.astype(np.int32)
