"""Pins for the oracle's sub-domain inference with reassembly (CPU only)."""

import numpy as np
import pytest

from oracle import infer, nnconv as nn
from oracle import radius_graph as rg
from workloads import layer_params


def _case(seed, n=260, D=2, d=8, H=16, layers=2, r=0.11, dtype="f32"):
    g = np.random.default_rng(seed)
    pos = g.uniform(0, 1, (n, D)).astype(np.float32)
    attr = np.concatenate([pos, g.uniform(0, 1, (n, 1)).astype(np.float32)], 1)
    h0 = g.normal(size=(n, d)).astype(np.float32)
    if dtype == "bf16":
        h0 = nn.bf16(h0).astype(np.float32)
    params = [layer_params(g, d, 2 * D + 2, H, H, dtype) for _ in range(layers)]
    return pos, attr, h0, params, r


def _grid_boxes(cx, cy):
    e = lambda c: [-np.inf] + list(c) + [np.inf]
    ex, ey = e(cx), e(cy)
    return [([ex[i], ey[j]], [ex[i + 1], ey[j + 1]]) for i in range(len(ex) - 1) for j in range(len(ey) - 1)]


def _whole(pos, attr, h0, params, r, dtype="f32"):
    n = pos.shape[0]
    rp, col = rg.radius_graph(pos, n, r)
    return infer.forward_stack(params, attr, h0, rp, col, n, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_overlap_of_the_receptive_field_reproduces_the_whole_domain(dtype):
    """With an overlap of layers * r every owned node sees the same
    neighbourhood at every layer as in the whole domain."""
    pos, attr, h0, params, r = _case(1, dtype=dtype)
    boxes = _grid_boxes([0.37, 0.61], [0.52])
    got, stats = infer.infer(params, pos, attr, h0, boxes, len(params) * r, r, dtype=dtype)
    want = _whole(pos, attr, h0, params, r, dtype)
    assert np.allclose(got, want, rtol=0, atol=1e-12)
    assert sum(s[0] for s in stats) == pos.shape[0]
    assert all(s[1] > s[0] for s in stats)           # every box has overlap nodes


def test_short_overlap_changes_owned_nodes_near_the_cuts():
    pos, attr, h0, params, r = _case(2)
    boxes = _grid_boxes([0.5], [])
    want = _whole(pos, attr, h0, params, r)
    for l in (0.0, r):                                 # l = r is complete for the first layer only
        got, _ = infer.infer(params, pos, attr, h0, boxes, l, r)
        bad = np.abs(got - want).max(1) > 1e-9
        assert bad.any()
        # only nodes within layers * r of the cut can differ
        assert np.all(np.abs(pos[bad, 0] - 0.5) <= len(params) * r + 1e-6)


def test_one_box_is_the_whole_domain():
    pos, attr, h0, params, r = _case(3)
    got, stats = infer.infer(params, pos, attr, h0, [([-np.inf] * 2, [np.inf] * 2)], 0.0, r)
    assert stats[0][:2] == (pos.shape[0], pos.shape[0])
    assert np.array_equal(got, _whole(pos, attr, h0, params, r))


def test_membership_brute_force():
    g = np.random.default_rng(4)
    pos = g.uniform(-1, 2, (500, 3)).astype(np.float32)
    pos[:20] = np.float32(0.25)                      # nodes exactly on a bound
    lo, hi, l = [0.25, -0.5, 0.0], [1.0, 0.75, 1.5], 0.2
    own, ovl = infer.subdomain_nodes(pos, lo, hi, l)
    f = np.float32
    for i in range(500):
        p = pos[i]
        o = all(f(lo[a]) <= p[a] < f(hi[a]) for a in range(3))
        e = all(f(f(lo[a]) - f(l)) <= p[a] < f(f(hi[a]) + f(l)) for a in range(3))
        assert (i in own) == o and (i in ovl) == (e and not o), i
    assert np.all(np.diff(own) > 0) and np.all(np.diff(ovl) > 0)
    assert 0 in own                                  # the lower bound is inclusive


def test_boxes_that_tile_own_every_node_once():
    pos, attr, h0, params, r = _case(5)
    boxes = _grid_boxes([0.2, 0.3, 0.9], [0.1, 0.5])
    count = np.zeros(pos.shape[0], int)
    for lo, hi in boxes:
        own, _ = infer.subdomain_nodes(pos, lo, hi, 0.1)
        count[own] += 1
    assert np.all(count == 1)
