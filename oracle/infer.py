"""Sub-domain inference with reassembly (oracle; test infrastructure only).

At test time the paper cuts the domain into smaller, randomly chosen
sub-domains, each with its overlap region, runs them through the trained
model one after another, and puts the outputs back together into the output
over the whole domain (Sec. 3, Methodology, testing procedure).

Readings where the paper is silent:
* a sub-domain is an axis-aligned box [lo, hi) (half-open in every axis, so
  boxes that tile the domain give every node exactly one owner); its nodes
  are the owned nodes (lo <= p < hi in every axis) and the overlap nodes
  (not owned, lo - l <= p < hi + l in every axis), with the bounds lo - l and
  hi + l rounded to float32 and the tests in float32;
* the nodes of a sub-domain are ordered owned first, then overlap, each in
  ascending index order; the sub-domain is a graph of its own: every one of
  its nodes is a destination, joined to its nodes within r (the same cap);
* the model is the stack of layers of ``oracle.nnconv`` (each layer's
  output, rounded to the layer's operand type, is the next layer's input
  features); overlap nodes are recomputed at every layer like the owned
  ones, since no neighbour updates them;
* reassembly keeps each sub-domain's final outputs on its owned nodes only.

With an overlap of at least layers * r every owned node sees, at every layer,
the same neighbours with the same input features as in the whole domain, so
the reassembled output equals the output over the whole domain: this is the
pin.  Smaller overlaps (the paper's l = r) change the owned outputs near the
cuts.

Pinned by: equality with the whole-domain forward at overlap layers * r (and
inequality at overlap 0 with more than one sub-domain), a single box holding
everything, every node owned exactly once, and brute-force membership.
"""

import numpy as np

from . import nnconv
from .radius_graph import radius_graph


def subdomain_nodes(pos, lo, hi, overlap):
    """(owned, overlap) node indices of the box [lo, hi) with overlap l, both
    ascending.  pos [n, D] float32; lo, hi [D]."""
    p = np.asarray(pos, dtype=np.float32)
    lo32 = np.asarray(lo, dtype=np.float32)
    hi32 = np.asarray(hi, dtype=np.float32)
    l32 = np.float32(overlap)
    elo = np.subtract(lo32, l32, dtype=np.float32)
    ehi = np.add(hi32, l32, dtype=np.float32)
    own = np.all((p >= lo32) & (p < hi32), axis=1)
    ext = np.all((p >= elo) & (p < ehi), axis=1)
    return np.nonzero(own)[0].astype(np.int32), np.nonzero(ext & ~own)[0].astype(np.int32)


def forward_stack(params, node_attr, h0, row_ptr, col, n, dtype, mode="concat"):
    """Outputs of the layer stack on one graph whose n nodes are all
    destinations; float64 [n, d]."""
    x = nnconv.edge_attr(node_attr, row_ptr, col, mode)
    h = np.asarray(h0, dtype=np.float64)
    out = None
    for P in params:
        out, _ = nnconv.forward(P, x, h, row_ptr, col, n)
        h = nnconv.bf16(out) if dtype == "bf16" else out
    return out


def infer(params, pos, node_attr, h0, boxes, overlap, r, cap=0, cap_mode=0, dtype="f32", seed=0, only=None):
    """Reassembled output [n, d] (float64) of sub-domain inference.

    params: list of layer parameter dicts; pos [n, D] float32; node_attr
    [n, D+1]; h0 [n, d] input features (values of the layer type); boxes: a
    list of (lo, hi) pairs; overlap: l.  ``only`` (optional) lists the boxes
    to run (the others leave zero rows).  Also returns the per-box node
    counts (owned, total) and edge counts.
    """
    pos = np.asarray(pos, dtype=np.float32)
    n = pos.shape[0]
    d = np.asarray(h0).shape[1]
    out = np.zeros((n, d))
    stats = []
    for b, (lo, hi) in enumerate(boxes):
        own, ovl = subdomain_nodes(pos, lo, hi, overlap)
        if only is not None and b not in only:
            stats.append((own.size, own.size + ovl.size, None))
            continue
        nodes = np.concatenate([own, ovl])
        m = nodes.size
        rp, col = radius_graph(pos[nodes], m, r, cap, cap_mode, seed)
        if m:
            res = forward_stack(params, np.asarray(node_attr)[nodes], np.asarray(h0)[nodes], rp, col, m, dtype)
            out[own] = res[:own.size]
        stats.append((own.size, m, int(rp[-1])))
    return out, stats
