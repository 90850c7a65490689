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

Pinned by: hand-computed messages on a 3-node graph, the constant kernel
(reduces to a neighbour mean), a constant matrix kernel (reduces to a mean of
A^T h_j, checked against a library matmul), linearity in h, node-permutation
equivariance, isolated nodes, central finite differences and the adjoint
(dot-product) identity for the backward pass.
"""

import numpy as np

ACT_IDENTITY = 0
ACT_RELU = 1


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


def _edge_mlp(P, x):
    a1 = x @ P["W1"].T + P["b1"]
    z1 = _relu(a1)
    a2 = z1 @ P["W2"].T + P["b2"]
    z = _relu(a2)
    return a1, z1, a2, z


def _as64(P):
    return {k: np.asarray(v, dtype=np.float64) for k, v in P.items()}


def _edges_of_rows(row_ptr, rows):
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    if rows is None:
        return np.arange(row_ptr[-1], dtype=np.int64)
    parts = [np.arange(row_ptr[i], row_ptr[i + 1]) for i in rows]
    return np.concatenate(parts) if parts else np.zeros(0, np.int64)


def forward(P, x_e, h, row_ptr, col, n_dst: int, act: int = ACT_IDENTITY,
            residual: bool = True, rows=None):
    """Layer output for destination rows (all rows, or only ``rows``).

    x_e: [E, de] edge attributes in CSR order; h: [n_src, d] input features.
    Returns (out, y): out and pre-activation y for the rows asked for, as
    [n_dst, d] arrays (rows not asked for are zero).
    """
    P = _as64(P)
    h = np.asarray(h, dtype=np.float64)
    x_e = np.asarray(x_e, dtype=np.float64)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    d = h.shape[1]
    deg = np.diff(row_ptr)[:n_dst]
    dst_all = np.repeat(np.arange(n_dst), deg)
    eids = _edges_of_rows(row_ptr, rows)
    msg_sum = np.zeros((n_dst, d))
    cs = _chunk_size(d)
    for s0 in range(0, eids.size, cs):
        e = eids[s0:s0 + cs]
        _, _, _, z = _edge_mlp(P, x_e[e])
        w = z @ P["W3"].T + P["b3"]                       # [n, d*d]
        theta = w.reshape(-1, d, d)                       # theta[e, p, q]
        m = np.einsum("epq,ep->eq", theta, h[col[e]])
        np.add.at(msg_sum, dst_all[e], m)
    sel = np.arange(n_dst) if rows is None else np.asarray(rows, dtype=np.int64)
    agg = np.zeros((n_dst, d))
    nz = sel[deg[sel] > 0]
    agg[nz] = msg_sum[nz] / deg[nz][:, None]
    y = np.zeros((n_dst, d))
    y[sel] = agg[sel] + h[sel] @ P["Wr"].T + P["br"]
    out = np.zeros((n_dst, d))
    a = _relu(y[sel]) if act == ACT_RELU else y[sel]
    out[sel] = h[sel] + a if residual else a
    return out, y


def backward(P, x_e, h, row_ptr, col, n_dst: int, grad_out, act: int = ACT_IDENTITY,
             residual: bool = True, rows=None):
    """Gradients of sum(grad_out * out) with respect to h and every parameter.

    If ``rows`` is given, grad_out must vanish outside those rows; only their
    edges are visited, and the result is still exact.
    Returns a dict with grad_h [n_src, d] and dW1, db1, dW2, db2, dW3, db3,
    dWr, dbr in the parameter layouts.
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
    _, y = forward(P, x_e, h, row_ptr, col, n_dst, act, residual, rows)
    ybar = G * (y > 0) if act == ACT_RELU else G.copy()
    if rows is not None:
        mask = np.zeros(n_dst, bool)
        mask[np.asarray(rows, dtype=np.int64)] = True
        ybar[~mask] = 0.0
    g_node = np.zeros_like(ybar)
    nz = deg > 0
    g_node[nz] = ybar[nz] / deg[nz][:, None]

    out = {k: np.zeros_like(P[k]) for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")}
    grad_h = np.zeros((n_src, d))
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
        a1, z1, a2, z = _edge_mlp(P, x)
        w = z @ P["W3"].T + P["b3"]
        theta = w.reshape(-1, d, d)
        g = g_node[dst_all[e]]                             # dL/dm_e
        hs = h[col[e]]
        np.add.at(grad_h, col[e], np.einsum("epq,eq->ep", theta, g))
        dw = (hs[:, :, None] * g[:, None, :]).reshape(-1, d * d)   # dL/dw_e
        out["W3"] += dw.T @ z
        out["b3"] += dw.sum(0)
        dz = dw @ P["W3"]
        da2 = dz * (a2 > 0)
        out["W2"] += da2.T @ z1
        out["b2"] += da2.sum(0)
        dz1 = da2 @ P["W2"]
        da1 = dz1 * (a1 > 0)
        out["W1"] += da1.T @ x
        out["b1"] += da1.sum(0)
    res = {"grad_h": grad_h}
    for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br"):
        res["d" + k] = out[k]
    return res
