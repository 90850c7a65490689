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

ReLU decisions and the precision model.  Every decision (the sign of a1,
a2, and of y when act is ReLU) is taken on the float64 values above.  A
kernel that computes with the operand precision a workload states (float32
throughout, or bfloat16 operands with float32 accumulation) reaches each
pre-activation up to rounding, so it may take a decision the other way where
the pre-activation is close to zero.  ``precision`` ("f32" or "bf16"; None
for exact arithmetic) turns on a first-order model of that rounding, written
from the operand types alone and not from any evaluation order:

* every operand of a product carries at most one rounding to its type, a
  relative error of at most u (u = 2^-24 for float32, 2^-8 for bfloat16):
  the caller's bfloat16 operands (h, W2, W3, b3, Wr) are exact, while the
  intermediate values that enter a bfloat16 product (z1, z, and the products
  z_k h_p or their sums over the edges of a destination) are not;
* every sum accumulates in float32 in some order: each partial sum carries a
  rounding of at most 2^-24 of itself, and no partial sum exceeds the sum of
  the absolute terms;
* rounding errors are independent, zero-mean and uniform within their bound
  (variance u^2/3 relative), so variances add (the probabilistic model of
  rounding error analysis; Higham and Mary, SIAM J. Sci. Comput. 41, 2019);
* errors carried by the inputs (``x_var``, ``h_var``: variances of the
  caller's values, e.g. the previous hop's outputs) propagate linearly.

This gives a variance for every pre-activation.  A decision is *ambiguous*
when |pre-activation| <= BAND_SIGMAS standard deviations; the probability
that a kernel decides the other way is modelled as 0.5 erfc(|a| / (sqrt(2)
sigma)).  The backward pass returns, for every gradient, the variance of the
change that such flips cause (each flip of a2 moves da2 by dz, each flip of
a1 moves da1 by dz1, each flip of y moves ybar by the upstream gradient),
plus the propagation of a variance of the upstream gradient (``grad_var``);
"allow" is ALLOW_SIGMAS standard deviations of it.  Forward returns the
variance of y and out.

Pinned by: hand-computed messages on a 3-node graph, the constant kernel
(reduces to a neighbour mean), a constant matrix kernel (reduces to a mean of
A^T h_j, checked against a library matmul), linearity in h, node-permutation
equivariance, isolated nodes, central finite differences and the adjoint
(dot-product) identity for the backward pass, torch float64 autograd; the
precision model against plain float32 and bfloat16 evaluations in several
summation orders (their deviations stay within the modelled spread and
their decisions agree outside the band) and against planted flips of the
ambiguous decisions (their effect stays within the allowance).
"""

import numpy as np

ACT_IDENTITY = 0
ACT_RELU = 1

U_F32 = 2.0 ** -24           # unit roundoff of float32 (24-bit significand)
U_BF16 = 2.0 ** -8           # unit roundoff of bfloat16 (8-bit significand)
BAND_SIGMAS = 6.0            # half-width of the ambiguity band, in standard deviations
ALLOW_SIGMAS = 4.0           # allowance of a gradient, in standard deviations of the flip effect


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
    """Round to the nearest bfloat16 (ties to even) via float32; returned as float64.
    Used for the caller-side operands a bfloat16 layer takes (e.g. node
    features handed from one hop to the next)."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
    return u.astype(np.uint32).view(np.float32).astype(np.float64).reshape(np.shape(x))


# ------------------------------------------------------------ precision model

def units(precision):
    """(u of a product operand, u of an accumulation) for a precision."""
    if precision is None:
        return 0.0, 0.0
    if precision == "f32":
        return U_F32, U_F32
    if precision == "bf16":
        return U_BF16, U_F32
    raise ValueError(precision)


def flip_probability(a, var) -> np.ndarray:
    """Probability that a value a carrying a zero-mean normal error of
    variance var is seen with the other sign: 0.5 erfc(|a| / sqrt(2 var));
    0 where var is 0."""
    from scipy.special import erfc
    a = np.asarray(a, dtype=np.float64)
    var = np.asarray(var, dtype=np.float64)
    s = np.sqrt(np.maximum(var, 0.0))
    with np.errstate(divide="ignore", invalid="ignore"):
        p = 0.5 * erfc(np.abs(a) / (np.sqrt(2.0) * s))
    return np.where(s > 0, p, 0.0)


def ambiguous(a, var) -> np.ndarray:
    """Decisions a kernel of the modelled precision may take either way."""
    return np.abs(a) <= BAND_SIGMAS * np.sqrt(np.maximum(var, 0.0))


def _acc_var(u_acc, n_terms, abs_sum):
    """Variance of a float32 accumulation of n_terms terms whose absolute
    values sum to abs_sum: one rounding per partial sum, each partial sum at
    most abs_sum."""
    return (u_acc * u_acc / 3.0) * n_terms * abs_sum * abs_sum


def edge_mlp(P, x, precision=None, x_var=None):
    """Kernel-MLP layers 1-2 on edge attribute rows x [n, de], float64.

    Returns a dict: a1, z1, a2, z (values), m1, m2 (float64 decisions
    a > 0) and, with a precision, v1, v2 (modelled error variances of a1, a2),
    amb1, amb2 (ambiguous decisions) and p1, p2 (flip probabilities)."""
    P = _as64(P)
    x = np.asarray(x, dtype=np.float64)
    a1 = x @ P["W1"].T + P["b1"]
    z1 = _relu(a1)
    a2 = z1 @ P["W2"].T + P["b2"]
    z = _relu(a2)
    r = {"a1": a1, "z1": z1, "a2": a2, "z": z, "m1": a1 > 0, "m2": a2 > 0}
    if precision is None:
        return r
    u_op, u_acc = units(precision)
    de, H1 = x.shape[1], a1.shape[1]
    # layer 1: float32 operands (attributes, W1, b1), float32 accumulation
    W1sq = P["W1"] ** 2
    s1 = np.abs(x) @ np.abs(P["W1"]).T + np.abs(P["b1"])
    v1 = (U_F32 * U_F32 / 3.0) * ((x * x) @ W1sq.T) + _acc_var(u_acc, de + 1, s1)
    if x_var is not None:
        v1 = v1 + np.asarray(x_var, dtype=np.float64) @ W1sq.T
    live1 = a1 > -BAND_SIGMAS * np.sqrt(v1)          # z1 may be nonzero in the kernel
    # layer 2: z1 enters the product as an operand of the layer's precision
    W2sq = P["W2"] ** 2
    s2 = z1 @ np.abs(P["W2"]).T + np.abs(P["b2"])
    v2 = (v1 * live1) @ W2sq.T + (u_op * u_op / 3.0) * ((z1 * z1) @ W2sq.T) + _acc_var(u_acc, H1 + 1, s2)
    r.update(v1=v1, v2=v2, amb1=ambiguous(a1, v1), amb2=ambiguous(a2, v2),
             p1=flip_probability(a1, v1), p2=flip_probability(a2, v2),
             vz=v2 * (a2 > -BAND_SIGMAS * np.sqrt(v2)))
    return r


def _as64(P):
    return {k: np.asarray(v, dtype=np.float64) for k, v in P.items()}


def _edges_of_rows(row_ptr, rows):
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    if rows is None:
        return np.arange(row_ptr[-1], dtype=np.int64)
    parts = [np.arange(row_ptr[i], row_ptr[i + 1]) for i in rows]
    return np.concatenate(parts) if parts else np.zeros(0, np.int64)


def _forward_full(P, x_e, h, row_ptr, col, n_dst, act, residual, rows, precision, x_var, h_var, want_var):
    P = _as64(P)
    h = np.asarray(h, dtype=np.float64)
    x_e = np.asarray(x_e, dtype=np.float64)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    d = h.shape[1]
    H2 = P["W2"].shape[0]
    deg = np.diff(row_ptr)[:n_dst]
    dst_all = np.repeat(np.arange(n_dst), deg)
    eids = _edges_of_rows(row_ptr, rows)
    need_var = precision is not None and (act == ACT_RELU or want_var)
    u_op, u_acc = units(precision)
    msg_sum = np.zeros((n_dst, d))
    if need_var:
        ve_sum = np.zeros((n_dst, d))      # propagated and z-rounding variance, summed over edges
        we_sum = np.zeros((n_dst, d))      # rounding of the products z_k h_p (or their edge sums)
        abs_sum = np.zeros((n_dst, d))     # sum of absolute terms
        W3r = P["W3"].reshape(d, d, H2)    # W3r[p, q, k] = W3[p*d + q, k]
        W3a = W3r.reshape(d, d * H2)
        W3s = (W3r ** 2).reshape(d, d * H2)
        b3s = P["b3"].reshape(d, d) ** 2
        absW3T = np.abs(P["W3"]).T
        absb3 = np.abs(P["b3"])
        hv = None if h_var is None else np.asarray(h_var, dtype=np.float64)
        xv = None if x_var is None else np.asarray(x_var, dtype=np.float64)
    cs = _chunk_size(d)
    if need_var:
        cs = max(1, min(cs, (1 << 23) // (d * H2)))
    for s0 in range(0, eids.size, cs):
        e = eids[s0:s0 + cs]
        em = edge_mlp(P, x_e[e], precision if need_var else None, None if not need_var or xv is None else xv[e])
        z = em["z"]
        w = z @ P["W3"].T + P["b3"]                       # [n, d*d]
        theta = w.reshape(-1, d, d)                       # theta[e, p, q]
        m = np.einsum("epq,ep->eq", theta, h[col[e]])
        np.add.at(msg_sum, dst_all[e], m)
        if need_var:
            hs = h[col[e]]
            A = (hs @ W3a).reshape(-1, d, H2)             # A[e, q, k] = sum_p W3[p*d+q, k] h_p
            B = ((hs * hs) @ W3s).reshape(-1, d, H2)      # B[e, q, k] = sum_p W3[p*d+q, k]^2 h_p^2
            ve = np.einsum("eqk,ek->eq", A * A, em["vz"] + (u_op * u_op / 3.0) * z * z)
            we = (u_op * u_op / 3.0) * (np.einsum("eqk,ek->eq", B, z * z) + (hs * hs) @ b3s)
            if hv is not None:
                ve = ve + np.einsum("epq,ep->eq", theta * theta, hv[col[e]])
            tha = (np.abs(z) @ absW3T + absb3).reshape(-1, d, d)
            np.add.at(ve_sum, dst_all[e], ve)
            np.add.at(we_sum, dst_all[e], we)
            np.add.at(abs_sum, dst_all[e], np.einsum("epq,ep->eq", tha, np.abs(hs)))
    sel = np.arange(n_dst) if rows is None else np.asarray(rows, dtype=np.int64)
    nz = sel[deg[sel] > 0]

    def finish(s):
        agg = np.zeros((n_dst, d))
        agg[nz] = s[nz] / deg[nz][:, None]
        y = np.zeros((n_dst, d))
        y[sel] = agg[sel] + h[sel] @ P["Wr"].T + P["br"]
        return y

    y = finish(msg_sum)
    y_var = np.zeros((n_dst, d))
    if need_var:
        dg = deg[nz][:, None].astype(np.float64)
        # the sum over edges of the product roundings is bounded (Cauchy-Schwarz)
        # by deg times the sum of their variances
        y_var[nz] = ve_sum[nz] / (dg * dg) + we_sum[nz] / dg
        S = np.zeros((n_dst, d))
        S[nz] = abs_sum[nz] / dg
        S[sel] += np.abs(h[sel]) @ np.abs(P["Wr"]).T + np.abs(P["br"])
        n_terms = (deg[:, None] * (H2 + 1) * d + d + 1).astype(np.float64)
        y_var[sel] += _acc_var(u_acc, n_terms[sel], S[sel])
        if hv is not None:
            y_var[sel] += hv[sel] @ (P["Wr"] ** 2).T
    my = y > 0
    out = np.zeros((n_dst, d))
    a = np.where(my[sel], y[sel], 0.0) if act == ACT_RELU else y[sel]
    out[sel] = h[sel] + a if residual else a
    stats = None
    if need_var:
        live = y > -BAND_SIGMAS * np.sqrt(y_var)
        out_var = np.zeros((n_dst, d))
        out_var[sel] = y_var[sel] * live[sel] if act == ACT_RELU else y_var[sel]
        if residual and hv is not None:
            out_var[sel] += hv[sel]
        stats = {"y_var": y_var, "out_var": out_var, "amb_y": ambiguous(y, y_var) & (act == ACT_RELU),
                 "p_y": flip_probability(y, y_var) if act == ACT_RELU else np.zeros_like(y)}
    return out, y, my, stats


def forward(P, x_e, h, row_ptr, col, n_dst: int, act: int = ACT_IDENTITY,
            residual: bool = True, rows=None, precision=None, x_var=None, h_var=None,
            return_stats: bool = False):
    """Layer output for destination rows (all rows, or only ``rows``).

    x_e: [E, de] edge attributes in CSR order; h: [n_src, d] input features.
    Returns (out, y): out and pre-activation y for the rows asked for, as
    [n_dst, d] arrays (rows not asked for are zero).  With a ``precision``
    and return_stats, also a dict: y_var and out_var (modelled error
    variances), amb_y (ReLU(y) decisions inside the band) and p_y (their
    flip probabilities); x_var [E, de] and h_var [n_src, d] are variances the
    inputs already carry.
    """
    out, y, _, st = _forward_full(P, x_e, h, row_ptr, col, n_dst, act, residual, rows, precision,
                                  x_var, h_var, return_stats)
    if not return_stats:
        return out, y
    if st is None:
        z = np.zeros_like(y)
        st = {"y_var": z, "out_var": z.copy(), "amb_y": np.zeros(y.shape, bool), "p_y": z.copy()}
    return out, y, st


GRAD_KEYS = ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")


def backward(P, x_e, h, row_ptr, col, n_dst: int, grad_out, act: int = ACT_IDENTITY,
             residual: bool = True, rows=None, precision=None, x_var=None, h_var=None,
             grad_var=None):
    """Gradients of sum(grad_out * out) with respect to h and every parameter.

    If ``rows`` is given, grad_out must vanish outside those rows; only their
    edges are visited, and the result is still exact.
    Returns a dict with grad_h [n_src, d], dW1, db1, dW2, db2, dW3, db3,
    dWr, dbr in the parameter layouts and grad_x [E, de] (the gradient with
    respect to the edge attributes, W1^T da1 per edge, zero for edges not
    visited).  With a ``precision``: "var", per gradient (and grad_h,
    grad_x) the modelled variance of the change that decisions taken the
    other way cause, plus the propagation of ``grad_var`` (a variance of
    grad_out); "allow" = ALLOW_SIGMAS * sqrt(var).
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
    model = precision is not None
    _, y, my, st = _forward_full(P, x_e, h, row_ptr, col, n_dst, act, residual, rows, precision,
                                 x_var, h_var, False)
    ybar = G * my if act == ACT_RELU else G.copy()
    if rows is not None:
        mask = np.zeros(n_dst, bool)
        mask[np.asarray(rows, dtype=np.int64)] = True
        ybar[~mask] = 0.0
    g_node = np.zeros_like(ybar)
    nz = deg > 0
    g_node[nz] = ybar[nz] / deg[nz][:, None]

    out = {k: np.zeros_like(P[k]) for k in GRAD_KEYS}
    grad_h = np.zeros((n_src, d))
    grad_x = np.zeros_like(x_e)
    # root, bias and residual terms (destinations are nodes [0, n_dst))
    out["Wr"] = ybar.T @ h[:n_dst]
    out["br"] = ybar.sum(0)
    grad_h[:n_dst] += ybar @ P["Wr"]
    if residual:
        grad_h[:n_dst] += G
    if model:
        V = {k: np.zeros_like(P[k]) for k in ("W3", "b3", "Wr", "br")}   # variances
        flips = FlipModel(P["W1"], P["W2"])
        gh_var = np.zeros((n_src, d))
        gx_var = np.zeros_like(x_e)
        gx_worst = np.zeros_like(x_e)
        Gv = np.zeros_like(G) if grad_var is None else np.asarray(grad_var, dtype=np.float64)
        if act == ACT_RELU:
            p_y = st["p_y"] if st is not None else np.zeros_like(G)
            yb_var = Gv * my + p_y * G * G
        else:
            yb_var = Gv.copy()
        if rows is not None:
            yb_var[~mask] = 0.0
        g_var = np.zeros_like(yb_var)
        g_var[nz] = yb_var[nz] / (deg[nz][:, None] ** 2)
        V["Wr"] = yb_var.T @ (h[:n_dst] ** 2)
        V["br"] = yb_var.sum(0)
        gh_var[:n_dst] += yb_var @ (P["Wr"] ** 2)
        if residual:
            gh_var[:n_dst] += Gv
        has_gvar = bool(np.any(g_var > 0))
        W3sq = P["W3"] ** 2
        xv = None if x_var is None else np.asarray(x_var, dtype=np.float64)
    # edge terms
    eids = _edges_of_rows(row_ptr, rows)
    cs = _chunk_size(d)
    for s0 in range(0, eids.size, cs):
        e = eids[s0:s0 + cs]
        x = x_e[e]
        em = edge_mlp(P, x, precision, None if not model or xv is None else xv[e])
        z1, z, m1, m2 = em["z1"], em["z"], em["m1"], em["m2"]
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
        if model:
            # a variance of g propagates with squared coefficients
            if has_gvar:
                gv = g_var[dst_all[e]]
                np.add.at(gh_var, col[e], np.einsum("epq,eq->ep", theta * theta, gv))
                dwv = ((hs * hs)[:, :, None] * gv[:, None, :]).reshape(-1, d * d)
                V["W3"] += dwv.T @ (z * z)
                V["b3"] += dwv.sum(0)
                dz_var = dwv @ W3sq
            else:
                dz_var = np.zeros_like(dz)
            gx_var[e], gx_worst[e] = flips.add(dz, dz_var, em, z1, x)
    res = {"grad_h": grad_h, "grad_x": grad_x}
    for k in GRAD_KEYS:
        res["d" + k] = out[k]
    if model:
        var = {"d" + k: v for k, v in V.items()}
        allow = {"d" + k: ALLOW_SIGMAS * np.sqrt(v) for k, v in V.items()}
        for k, part in flips.parts().items():
            var["d" + k] = part[0] + part[1] ** 2
            allow["d" + k] = bernstein_allowance(*part)
        var["grad_h"] = gh_var
        var["grad_x"] = gx_var
        res["var"] = var
        res["flip_parts"] = {"d" + k: v for k, v in flips.parts().items()}
        allow["grad_h"] = ALLOW_SIGMAS * np.sqrt(gh_var)
        allow["grad_x"] = gx_worst + ALLOW_SIGMAS * np.sqrt(gx_var)
        res["allow"] = allow
    else:
        res["allow"] = {}
    return res


class FlipModel:
    """Effect of ReLU decisions taken the other way in a two-layer chain
    da2 = dz * m2,  dz1 = W2^T da2,  da1 = dz1 * m1
    with weight gradients dW2 = sum da2 z1^T, db2 = sum da2, dW1 = sum da1 x^T,
    db1 = sum da1 and input gradient gx = W1^T da1 per row.  A flip of a2
    moves da2 by c2 = (1 - 2 m2) dz, a flip of a1 moves da1 by
    c1 = (1 - 2 m1) dz1, each with its flip probability; a variance of dz
    (from the upstream gradient) propagates with squared coefficients.

    Collects per weight gradient the variance, the expected shift and the
    largest single flip effect (the inputs of the Bernstein allowance)."""

    def __init__(self, W1, W2):
        self.W1, self.W2 = np.asarray(W1, np.float64), np.asarray(W2, np.float64)
        self.W1sq, self.W2sq = self.W1 ** 2, self.W2 ** 2
        self.aW1, self.aW2 = np.abs(self.W1), np.abs(self.W2)
        z = lambda a: np.zeros_like(a)
        shapes = {"W2": self.W2, "b2": self.W2[:, 0], "W1": self.W1, "b1": self.W1[:, 0]}
        self.V = {k: z(v) for k, v in shapes.items()}
        self.MEAN = {k: z(v) for k, v in shapes.items()}
        self.MX = {k: z(v) for k, v in shapes.items()}

    def add(self, dz, dz_var, em, z1, x):
        """One block of rows; returns (variance, worst case) of gx per row."""
        m1, m2, p1, p2, amb1, amb2 = em["m1"], em["m2"], em["p1"], em["p2"], em["amb1"], em["amb2"]
        dz1 = (dz * m2) @ self.W2
        c2 = np.where(m2, -dz, dz)
        c1 = np.where(m1, -dz1, dz1)
        v2 = dz_var * m2 + p2 * dz * dz
        V, MEAN, MX = self.V, self.MEAN, self.MX
        V["W2"] += v2.T @ (z1 * z1)
        V["b2"] += v2.sum(0)
        MEAN["W2"] += (p2 * c2).T @ z1
        MEAN["b2"] += (p2 * c2).sum(0)
        v1 = (v2 @ self.W2sq) * m1 + p1 * dz1 * dz1
        V["W1"] += v1.T @ (x * x)
        V["b1"] += v1.sum(0)
        sh1 = ((p2 * c2) @ self.W2) * m1 + p1 * c1
        MEAN["W1"] += sh1.T @ x
        MEAN["b1"] += sh1.sum(0)
        a2c = np.abs(c2) * amb2
        a1c = np.abs(c1) * amb1
        # worst case of a row: every ambiguous decision of the row flipped
        worst = ((a2c @ self.aW2) * m1 + a1c) @ self.aW1
        ea = np.nonzero(amb2.any(1) | amb1.any(1))[0]
        if ea.size:
            A2, A1 = a2c[ea], a1c[ea]
            MX["b2"] = np.maximum(MX["b2"], A2.max(0))
            MX["W2"] = np.maximum(MX["W2"], _max_outer(A2, np.abs(z1[ea])))
            # one a2 flip reaches da1[j] through W2[k, j] (where z1_j is live)
            T = np.maximum(np.max(A2[:, :, None] * self.aW2[None, :, :], axis=1) * m1[ea], A1)
            MX["b1"] = np.maximum(MX["b1"], T.max(0))
            MX["W1"] = np.maximum(MX["W1"], _max_outer(T, np.abs(x[ea])))
        return v1 @ self.W1sq, worst

    def parts(self):
        """{key: (variance, largest single flip, expected shift)}."""
        return {k: (self.V[k], self.MX[k], self.MEAN[k]) for k in self.V}


def _max_outer(a, b, chunk=256):
    """max over rows e of a[e, i] * b[e, j] (a, b >= 0), in pieces."""
    out = np.zeros((a.shape[1], b.shape[1]))
    for s0 in range(0, a.shape[0], chunk):
        out = np.maximum(out, np.max(a[s0:s0 + chunk, :, None] * b[s0:s0 + chunk, None, :], axis=0))
    return out


def bernstein_allowance(var, biggest, mean):
    """Bound on |sum of independent flip effects| that holds with probability
    at least 1 - 2 exp(-ALLOW_SIGMAS^2 / 2) (Bernstein's inequality): the
    expected shift plus t solving t^2 / 2 = L (var + biggest t / 3),
    L = ALLOW_SIGMAS^2 / 2."""
    L = 0.5 * ALLOW_SIGMAS * ALLOW_SIGMAS
    b = L * biggest / 3.0
    return np.abs(mean) + b + np.sqrt(b * b + 2.0 * L * var)
