"""Hop loop of DS-MPNN on one sub-domain (oracle; test infrastructure only).

One training step of Algorithm 1 without the optimiser update and the
communication steps, built on the edge-conditioned layer of ``oracle.nnconv``
and the model equations (i)-(iv) of Sec. 2.2:

    v_L^0     = N_e(v^0)                                   encoder, eq. (i)
    for l = 0 .. h-1:
        x_e^l     = v_i^l - v_j^l  (edge e = (i <- j))     edge attributes, eq. (iv);
                                                           l = 0 uses the input values
        v_L^{l+1} = v_L^l + K(x^l, v_L^l)                  graph convolution with the
                                                           residual hop update, eq. (ii)
        v^{l+1}   = N_d(v_L^{l+1})                         decoder, eq. (iii)
    loss      = mean over interior rows and components of (v^h - Y)^2

N_e and N_d are three-layer perceptrons, ReLU between layers and none after
the last: N(x) = W3 ReLU(W2 ReLU(W1 x + b1) + b2) + b3, in the [out, in]
layout of a linear layer.

Readings where the paper is silent:
* hidden widths of the encoder and decoder are parameters;
* the decoder output has the width of the input node values, so the edge
  attributes keep their width over the hops;
* the same encoder, decoder and convolution parameters serve every hop (one
  parameter set w in Algorithm 1), so their gradients sum over the hops;
* interior rows are given by a mask (the sub-domain's owned rows); the MSE
  averages over interior rows times output components;
* for bfloat16 layers the convolution takes its node features rounded to
  bfloat16 (its residual adds the rounded values, as the layer defines);
  encoder, decoder and loss are float64 here.

Everything is float64.  The backward pass is the chain rule written out by
hand.  ``margins`` reports, for every ReLU the step takes, the smallest
|pre-activation| relative to the sum of absolute terms that formed it, so a
test can check that no decision sits close enough to zero for a float32
evaluation to take it the other way.

Pinned by central finite differences of the loss (every parameter group and
the input values) and by torch float64 autograd of the same loop.
"""

import numpy as np

from . import nnconv


def _relu(a):
    return np.maximum(a, 0.0)


def mlp3_forward(P, x):
    """N(x) for rows x [n, d_in]; returns (y [n, d_out], cache)."""
    P = {k: np.asarray(v, dtype=np.float64) for k, v in P.items()}
    x = np.asarray(x, dtype=np.float64)
    a1 = x @ P["W1"].T + P["b1"]
    h1 = _relu(a1)
    a2 = h1 @ P["W2"].T + P["b2"]
    h2 = _relu(a2)
    y = h2 @ P["W3"].T + P["b3"]
    s1 = np.abs(x) @ np.abs(P["W1"]).T + np.abs(P["b1"])
    s2 = h1 @ np.abs(P["W2"]).T + np.abs(P["b2"])
    margin = min(_min_rel(a1, s1), _min_rel(a2, s2))
    return y, {"x": x, "h1": h1, "h2": h2, "m1": a1 > 0, "m2": a2 > 0, "margin": margin}


def mlp3_backward(P, cache, gy):
    """Gradients of sum(gy * y): returns (gx, {dW1, db1, dW2, db2, dW3, db3})."""
    P = {k: np.asarray(v, dtype=np.float64) for k, v in P.items()}
    gy = np.asarray(gy, dtype=np.float64)
    g = {"dW3": gy.T @ cache["h2"], "db3": gy.sum(0)}
    ga2 = (gy @ P["W3"]) * cache["m2"]
    g["dW2"] = ga2.T @ cache["h1"]
    g["db2"] = ga2.sum(0)
    ga1 = (ga2 @ P["W2"]) * cache["m1"]
    g["dW1"] = ga1.T @ cache["x"]
    g["db1"] = ga1.sum(0)
    return ga1 @ P["W1"], g


def masked_mse(pred, target, mask):
    """(loss, d loss / d pred): mean of (pred - target)^2 over interior rows
    (mask true) and all components; zero gradient on the other rows."""
    pred = np.asarray(pred, dtype=np.float64)
    diff = pred - np.asarray(target, dtype=np.float64)
    m = np.asarray(mask, dtype=bool)
    count = int(m.sum()) * pred.shape[1]
    if count == 0:
        return 0.0, np.zeros_like(pred)
    loss = float((diff[m] ** 2).sum() / count)
    grad = np.zeros_like(pred)
    grad[m] = 2.0 * diff[m] / count
    return loss, grad


def _min_rel(a, s):
    s = np.where(s > 0, s, 1.0)
    r = np.abs(a) / s
    return float(r.min()) if r.size else np.inf


def _bf16_features(v, dtype):
    return nnconv.bf16(v) if dtype == "bf16" else np.asarray(v, dtype=np.float64)


def train_step(Pe, Pk, Pd, v0, Y, mask, row_ptr, col, n_hops: int, dtype: str = "f32"):
    """Loss and gradients of one step of the hop loop on one sub-domain.

    Pe, Pd: encoder / decoder parameters (mlp3 layout); Pk: convolution
    parameters (``oracle.nnconv`` layout, with W1 [h1, dim+1]); v0 [n, dim+1]
    input node values; Y [n, dim+1] targets; mask [n] interior rows; the graph
    (row_ptr, col) joins the n nodes (every node is a destination).
    Returns a dict: loss, v (final decoder output), vL (final latent), the
    gradients "enc", "conv", "dec" (dicts keyed like the parameters with a
    leading "d"), "conv_allow" (per convolution gradient, the sum over the
    hops of the layer backward's bound on how far its ambiguous ReLU
    decisions can move it), "margin" (the smallest relative ReLU margin met)
    and "mlp_margin" (the same over the encoder and decoder only).
    """
    v0 = np.asarray(v0, dtype=np.float64)
    n = v0.shape[0]
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    decide = "bf16" if dtype == "bf16" else "f32"
    # forward
    vL, enc_cache = mlp3_forward(Pe, v0)
    mlp_margin = enc_cache["margin"]
    margin = mlp_margin
    v = v0
    hops = []
    for _ in range(n_hops):
        x = nnconv.edge_attr(v, row_ptr, col, mode="diff")
        h_in = _bf16_features(vL, dtype)
        out, _ = nnconv.forward(Pk, x, h_in, row_ptr, col, n, decide=decide)
        margin = min(margin, _conv_margin(Pk, x, dtype))
        v_new, dec_cache = mlp3_forward(Pd, out)
        margin = min(margin, dec_cache["margin"])
        mlp_margin = min(mlp_margin, dec_cache["margin"])
        hops.append({"x": x, "h_in": h_in, "out": out, "dec": dec_cache})
        vL, v = out, v_new
    loss, gv = masked_mse(v, Y, mask)
    # backward: gv is the gradient with respect to the decoder output v^{l+1},
    # g_lat the one with respect to the convolution output out^l through the
    # next hop's latent input
    g_conv = {"d" + k: np.zeros_like(np.asarray(Pk[k], dtype=np.float64))
              for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")}
    conv_allow = {k: np.zeros_like(v) for k, v in g_conv.items()}
    g_dec = None
    g_lat = np.zeros_like(hops[-1]["out"]) if hops else None
    dst = np.repeat(np.arange(n), np.diff(row_ptr))
    for l in reversed(range(n_hops)):
        hp = hops[l]
        g_out, gd = mlp3_backward(Pd, hp["dec"], gv)
        g_dec = gd if g_dec is None else {k: g_dec[k] + gd[k] for k in gd}
        gc = nnconv.backward(Pk, hp["x"], hp["h_in"], row_ptr, col, n, g_out + g_lat, decide=decide)
        for k in g_conv:
            g_conv[k] += gc[k]
            if k in gc["allow"]:
                conv_allow[k] += gc["allow"][k]
        g_lat = gc["grad_h"]                 # with respect to the latent input vL^l
        gv = np.zeros_like(v0)               # with respect to v^l, through x^l = v_i - v_j
        np.add.at(gv, dst, gc["grad_x"])
        np.add.at(gv, col, -gc["grad_x"])
    _, g_enc = mlp3_backward(Pe, enc_cache, g_lat if n_hops else np.zeros_like(vL))
    return {"loss": loss, "v": v, "vL": vL, "enc": g_enc, "conv": g_conv, "dec": g_dec, "conv_allow": conv_allow,
            "margin": margin, "mlp_margin": mlp_margin}


def _conv_margin(Pk, x, dtype):
    """Smallest relative margin of the kernel-MLP ReLUs (a1 as float32 computes it,
    a2 on the values the layer's second product sees)."""
    P = {k: np.asarray(v, dtype=np.float64) for k, v in Pk.items()}
    a1 = nnconv.a1_float32(P, x)
    s1 = np.abs(x) @ np.abs(P["W1"]).T + np.abs(P["b1"])
    z1 = _relu(a1)
    if dtype == "bf16":
        z1 = nnconv.bf16(z1)
    a2 = z1 @ P["W2"].T + P["b2"]
    s2 = z1 @ np.abs(P["W2"]).T + np.abs(P["b2"])
    return min(_min_rel(a1, s1), _min_rel(a2, s2))
