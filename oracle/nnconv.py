"""Edge-conditioned convolution layer, forward and backward (oracle; test infrastructure only).

The layer is the graph convolution of eq. (1) (Sec. 2.1) and eq. (ii)
(Sec. 2.2), applied once per radius hop in Algorithm 1 (graph-convolution
step followed by the residual addition):

    x_e      edge attributes of edge e = (i <- j), i the centre (destination),
             j the neighbour (source)
    z1       = ReLU(W1 x_e + b1)                  kernel MLP, layer 1
    z        = ReLU(W2 z1  + b2)                  kernel MLP, layer 2
    w_e      = W3 z + b3                          kernel MLP, last layer (d*d)
    Theta_e  = w_e viewed as a d x d matrix, Theta_e[p, q] = w_e[p*d + q]
    m_e      = Theta_e^T h_j                      message, m_e[q] = sum_p Theta_e[p,q] h_j[p]
    agg_i    = (1/|E_i|) sum_{e in E_i} m_e      mean over the retained edges
    y_i      = agg_i + Wr h_i + br                root linear term and bias
    out_i    = h_i + act(y_i)   (residual)   or   act(y_i)

Parameters use the torch ``Linear`` layout [out, in]:
W1 [H1, de], b1 [H1], W2 [H2, H1], b2 [H2], W3 [d*d, H2], b3 [d*d],
Wr [d, d], br [d].

Readings where the paper is silent:
* the kernel MLP output is reshaped input-channel-major (Theta[p, q] with p
  the input channel), and the message is Theta^T h_j;
* the mean runs over the retained (capped) edges; a centre with no edges
  gets agg = 0;
* a root term Wr h_i joins the paper's bias b; act is the identity unless
  ReLU is asked for; ReLU'(0) = 0;
* edge attributes are, in "concat" mode, [p_i, p_j, s_i, s_j] (positions and
  the node scalar of both ends); in "diff" mode they are v_i - v_j, the
  relative difference the paper describes (Sec. 2.1; Algorithm 1, edge
  attribute step).

Everything is float64; Theta is materialised per chunk of edges, which the
GPU path never does.  The backward pass is written out by hand from the
chain rule.

ReLU decisions.  The sign of a pre-activation (a1, a2, and y when act is
ReLU) is a discrete decision taken by floating point, and the paper fixes no
precision.  With ``decide=None`` the oracle decides on its float64 values.
With ``decide="f32"`` or ``decide="bf16"`` it decides on the values a kernel
of that precision produces: a1 as a float32 chain of fused multiply-adds over
the attributes in order starting from b1; for "bf16" also z1 and z rounded to
bfloat16 (nearest-even) before they enter the layer-2 and last-layer
products, the products accumulated exactly.  Values themselves stay float64.
Decisions that a float32 accumulation could still take either way
(|a2| or |y| within 2^-16 resp. 2^-14 of the sum of absolute terms, |a1|
within 2^-20) are reported: forward returns them, and backward returns, for
each gradient an ambiguous a1/a2 decision can reach (dW1, db1, dW2, db2), an
elementwise bound on how much the choice can move it.

Pinned by: hand-computed messages on a 3-node graph, the constant kernel
(reduces to a neighbour mean), a constant matrix kernel (reduces to a mean of
A^T h_j, checked against a library matmul), linearity in h, node-permutation
equivariance, isolated nodes, central finite differences and the adjoint
(dot-product) identity for the backward pass; the decision path against
plain float32 arithmetic and against the float64 decisions away from zero.
"""

import numpy as np

ACT_IDENTITY = 0
ACT_RELU = 1

_EPS_A1 = 2.0 ** -20
_EPS_A2 = 2.0 ** -16
_EPS_Y = 2.0 ** -14


def edge_attr(node_attr, row_ptr, col, mode: str = "concat") -> np.ndarray:
    """Edge attributes in CSR edge order.

    node_attr: [n_src, D+1] = (position, scalar) per node.
    concat: x_e = [p_i (D), p_j (D), s_i, s_j]   (de = 2D + 2)
    diff  : x_e = v_i - v_j                       (de = D + 1)
    """
    na = np.asarray(node_attr, dtype=np.float64)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    dst = np.repeat(np.arange(row_ptr.size - 1), np.diff(row_ptr))
    src = np.asarray(col, dtype=np.int64)
    D = na.shape[1] - 1
    if mode == "concat":
        return np.concatenate([na[dst, :D], na[src, :D], na[dst, D:D + 1], na[src, D:D + 1]], axis=1)
    if mode == "diff":
        return na[dst] - na[src]
    raise ValueError(mode)


def _relu(a):
    return np.maximum(a, 0.0)


def _chunk_size(d: int) -> int:
    return max(1, (1 << 24) // (d * d))


def bf16(x) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even) via float32; returned as float64."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
    return u.astype(np.uint32).view(np.float32).astype(np.float64).reshape(np.shape(x))


def a1_float32(P, x) -> np.ndarray:
    """W1 x + b1 as a float32 kernel evaluates it: start from b1, then one fused
    multiply-add per attribute in order (exact product, one rounding)."""
    W1 = np.asarray(P["W1"], dtype=np.float32).astype(np.float64)
    b1 = np.asarray(P["b1"], dtype=np.float32).astype(np.float64)
    x32 = np.asarray(x, dtype=np.float32).astype(np.float64)
    v = np.broadcast_to(b1, (x32.shape[0], b1.size)).copy()
    for c in range(x32.shape[1]):
        v = (x32[:, c:c + 1] * W1[None, :, c] + v).astype(np.float32).astype(np.float64)
    return v


def _edge_mlp(P, x):
    a1 = x @ P["W1"].T + P["b1"]
    z1 = _relu(a1)
    a2 = z1 @ P["W2"].T + P["b2"]
    z = _relu(a2)
    return a1, z1, a2, z


def _edge_mlp_decided(P, x, decide):
    """Kernel-MLP layers with the ReLU masks decided at the given precision.

    Returns float64 values (a1, z1, a2, z), the masks, the decision-path z
    (what the last-layer product sees) and the ambiguity flags of a1 and a2.
    """
    if decide is None:
        a1, z1, a2, z = _edge_mlp(P, x)
        m1, m2 = a1 > 0, a2 > 0
        none = np.zeros_like(m1), np.zeros_like(m2)
        return a1, z1, a2, z, m1, m2, z, none[0], none[1]
    a1d = a1_float32(P, x)
    s1 = np.abs(x) @ np.abs(P["W1"]).T + np.abs(P["b1"])
    m1 = a1d > 0
    amb1 = np.abs(a1d) <= _EPS_A1 * s1
    z1d = np.where(m1, a1d, 0.0)
    z1q = bf16(z1d) if decide == "bf16" else z1d
    a2d = z1q @ P["W2"].T + P["b2"]
    s2 = z1q @ np.abs(P["W2"]).T + np.abs(P["b2"])
    m2 = a2d > 0
    amb2 = np.abs(a2d) <= _EPS_A2 * s2
    zd = np.where(m2, a2d, 0.0)
    zq = bf16(zd) if decide == "bf16" else zd
    # float64 values under the decided masks
    a1 = x @ P["W1"].T + P["b1"]
    z1 = np.where(m1, a1, 0.0)
    a2 = z1 @ P["W2"].T + P["b2"]
    z = np.where(m2, a2, 0.0)
    return a1, z1, a2, z, m1, m2, zq, amb1, amb2


def _as64(P):
    return {k: np.asarray(v, dtype=np.float64) for k, v in P.items()}


def _edges_of_rows(row_ptr, rows):
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    if rows is None:
        return np.arange(row_ptr[-1], dtype=np.int64)
    parts = [np.arange(row_ptr[i], row_ptr[i + 1]) for i in rows]
    return np.concatenate(parts) if parts else np.zeros(0, np.int64)


def _forward_full(P, x_e, h, row_ptr, col, n_dst, act, residual, rows, decide):
    P = _as64(P)
    h = np.asarray(h, dtype=np.float64)
    x_e = np.asarray(x_e, dtype=np.float64)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    d = h.shape[1]
    deg = np.diff(row_ptr)[:n_dst]
    dst_all = np.repeat(np.arange(n_dst), deg)
    eids = _edges_of_rows(row_ptr, rows)
    need_dec = decide is not None and act == ACT_RELU
    msg_sum = np.zeros((n_dst, d))
    dec_sum = np.zeros((n_dst, d)) if need_dec else None
    abs_sum = np.zeros((n_dst, d)) if need_dec else None
    cs = _chunk_size(d)
    for s0 in range(0, eids.size, cs):
        e = eids[s0:s0 + cs]
        _, _, _, z, _, _, zq, _, _ = _edge_mlp_decided(P, x_e[e], decide)
        w = z @ P["W3"].T + P["b3"]                       # [n, d*d]
        theta = w.reshape(-1, d, d)                       # theta[e, p, q]
        m = np.einsum("epq,ep->eq", theta, h[col[e]])
        np.add.at(msg_sum, dst_all[e], m)
        if need_dec:
            thq = (zq @ P["W3"].T + P["b3"]).reshape(-1, d, d)
            np.add.at(dec_sum, dst_all[e], np.einsum("epq,ep->eq", thq, h[col[e]]))
            tha = (zq @ np.abs(P["W3"]).T + np.abs(P["b3"])).reshape(-1, d, d)
            np.add.at(abs_sum, dst_all[e], np.einsum("epq,ep->eq", tha, np.abs(h[col[e]])))
    sel = np.arange(n_dst) if rows is None else np.asarray(rows, dtype=np.int64)
    nz = sel[deg[sel] > 0]

    def finish(s):
        agg = np.zeros((n_dst, d))
        agg[nz] = s[nz] / deg[nz][:, None]
        y = np.zeros((n_dst, d))
        y[sel] = agg[sel] + h[sel] @ P["Wr"].T + P["br"]
        return y

    y = finish(msg_sum)
    if need_dec:
        y_dec = finish(dec_sum)
        scale = np.zeros((n_dst, d))
        scale[nz] = abs_sum[nz] / deg[nz][:, None]
        scale[sel] += np.abs(h[sel]) @ np.abs(P["Wr"]).T + np.abs(P["br"])
        amb_y = np.abs(y_dec) <= _EPS_Y * scale
    else:
        y_dec = y
        amb_y = np.zeros((n_dst, d), bool)
    my = y_dec > 0
    out = np.zeros((n_dst, d))
    a = np.where(my[sel], y[sel], 0.0) if act == ACT_RELU else y[sel]
    out[sel] = h[sel] + a if residual else a
    return out, y, my, amb_y


def forward(P, x_e, h, row_ptr, col, n_dst: int, act: int = ACT_IDENTITY,
            residual: bool = True, rows=None, decide=None, return_ambiguous: bool = False):
    """Layer output for destination rows (all rows, or only ``rows``).

    x_e: [E, de] edge attributes in CSR order; h: [n_src, d] input features.
    Returns (out, y): out and pre-activation y for the rows asked for, as
    [n_dst, d] arrays (rows not asked for are zero); with return_ambiguous
    also the [n_dst, d] flags of ReLU(y) decisions a float32 kernel could
    take either way.
    """
    out, y, _, amb_y = _forward_full(P, x_e, h, row_ptr, col, n_dst, act, residual, rows, decide)
    return (out, y, amb_y) if return_ambiguous else (out, y)


def backward(P, x_e, h, row_ptr, col, n_dst: int, grad_out, act: int = ACT_IDENTITY,
             residual: bool = True, rows=None, decide=None):
    """Gradients of sum(grad_out * out) with respect to h and every parameter.

    If ``rows`` is given, grad_out must vanish outside those rows; only their
    edges are visited, and the result is still exact.
    Returns a dict with grad_h [n_src, d], dW1, db1, dW2, db2, dW3, db3,
    dWr, dbr in the parameter layouts, grad_x [E, de] (the gradient with
    respect to the edge attributes, W1^T da1 per edge, zero for edges not
    visited), plus "allow": elementwise bounds on how far ambiguous a1/a2
    ReLU decisions can move dW1, db1, dW2, db2 and grad_x.
    """
    P = _as64(P)
    h = np.asarray(h, dtype=np.float64)
    x_e = np.asarray(x_e, dtype=np.float64)
    G = np.asarray(grad_out, dtype=np.float64)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    n_src, d = h.shape
    deg = np.diff(row_ptr)[:n_dst]
    dst_all = np.repeat(np.arange(n_dst), deg)
    _, y, my, _ = _forward_full(P, x_e, h, row_ptr, col, n_dst, act, residual, rows, decide)
    ybar = G * my if act == ACT_RELU else G.copy()
    if rows is not None:
        mask = np.zeros(n_dst, bool)
        mask[np.asarray(rows, dtype=np.int64)] = True
        ybar[~mask] = 0.0
    g_node = np.zeros_like(ybar)
    nz = deg > 0
    g_node[nz] = ybar[nz] / deg[nz][:, None]

    out = {k: np.zeros_like(P[k]) for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")}
    allow = {k: np.zeros_like(P[k]) for k in ("W1", "b1", "W2", "b2")}
    grad_h = np.zeros((n_src, d))
    grad_x = np.zeros_like(x_e)
    allow_x = np.zeros_like(x_e)
    # root, bias and residual terms (destinations are nodes [0, n_dst))
    out["Wr"] = ybar.T @ h[:n_dst]
    out["br"] = ybar.sum(0)
    grad_h[:n_dst] += ybar @ P["Wr"]
    if residual:
        grad_h[:n_dst] += G
    # edge terms
    eids = _edges_of_rows(row_ptr, rows)
    cs = _chunk_size(d)
    for s0 in range(0, eids.size, cs):
        e = eids[s0:s0 + cs]
        x = x_e[e]
        a1, z1, a2, z, m1, m2, _, amb1, amb2 = _edge_mlp_decided(P, x, decide)
        w = z @ P["W3"].T + P["b3"]
        theta = w.reshape(-1, d, d)
        g = g_node[dst_all[e]]                             # dL/dm_e
        hs = h[col[e]]
        np.add.at(grad_h, col[e], np.einsum("epq,eq->ep", theta, g))
        dw = (hs[:, :, None] * g[:, None, :]).reshape(-1, d * d)   # dL/dw_e
        out["W3"] += dw.T @ z
        out["b3"] += dw.sum(0)
        dz = dw @ P["W3"]
        da2 = dz * m2
        out["W2"] += da2.T @ z1
        out["b2"] += da2.sum(0)
        dz1 = da2 @ P["W2"]
        da1 = dz1 * m1
        out["W1"] += da1.T @ x
        out["b1"] += da1.sum(0)
        grad_x[e] = da1 @ P["W1"]
        if amb1.any() or amb2.any():
            # an ambiguous a2 decision moves da2[e,k] by dz[e,k]; an ambiguous a1
            # decision moves da1[e,j] by dz1[e,j]
            d2 = np.abs(dz) * amb2
            allow["W2"] += d2.T @ np.abs(z1)
            allow["b2"] += d2.sum(0)
            d1 = (d2 @ np.abs(P["W2"])) * m1 + np.abs(dz1) * amb1
            allow["W1"] += d1.T @ np.abs(x)
            allow["b1"] += d1.sum(0)
            allow_x[e] = d1 @ np.abs(P["W1"])
    res = {"grad_h": grad_h, "grad_x": grad_x}
    for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br"):
        res["d" + k] = out[k]
    res["allow"] = {"d" + k: v for k, v in allow.items()}
    res["allow"]["grad_x"] = allow_x
    return res
