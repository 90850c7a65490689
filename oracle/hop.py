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
hand.

Precision model.  The step is what a kernel computes in float64; a kernel
that works in the configuration's precision (float32 perceptrons and loss,
the layer in float32 or with bfloat16 operands) deviates by rounding, and a
ReLU decision close to its kink may go the other way.  The step carries the
first-order model of ``oracle.nnconv`` through the loop: variances of every
value (the encoder output, the layer's input features after their rounding to
the layer type, its edge attributes v_i - v_j, its output, the decoder
output) propagate forward, so every decision of the perceptrons and of the
layer has a modelled spread, a band and a flip probability; the effects of
flips, and the variances of the gradients they feed, propagate backward
through every hop.  ``train_step`` returns, per gradient and per output, an
allowance: ALLOW_SIGMAS standard deviations, or the Bernstein bound of the
flip effects for the gradients that sum them directly.

Pinned by central finite differences of the loss (every parameter group and
the input values) and by torch float64 autograd of the same loop; the model
against a float32/bfloat16 evaluation of the loop whose decisions follow its
own rounded values.
"""

import numpy as np

from . import nnconv


def _relu(a):
    return np.maximum(a, 0.0)


def mlp3_forward(P, x, precision=None, x_var=None):
    """N(x) for rows x [n, d_in]; returns (y [n, d_out], cache).  With a
    precision (the perceptrons are float32: "f32") the cache also holds the
    modelled variances, bands and flip probabilities of both ReLU layers and
    cache["y_var"]; x_var is the variance the input already carries."""
    P = {k: np.asarray(v, dtype=np.float64) for k, v in P.items()}
    x = np.asarray(x, dtype=np.float64)
    em = nnconv.edge_mlp(P, x, precision, x_var)
    h1, h2 = em["z1"], em["z"]
    y = h2 @ P["W3"].T + P["b3"]
    cache = {"x": x, "h1": h1, "h2": h2, "m1": em["m1"], "m2": em["m2"], "em": em, "model": precision is not None}
    if precision is not None:
        u_op, u_acc = nnconv.units(precision)
        W3sq = P["W3"] ** 2
        s3 = np.abs(h2) @ np.abs(P["W3"]).T + np.abs(P["b3"])
        cache["y_var"] = (em["vz"] @ W3sq.T + (u_op * u_op / 3.0) * ((h2 * h2) @ W3sq.T)
                          + nnconv._acc_var(u_acc, h2.shape[1] + 1, s3))
        cache["n_amb"] = int(em["amb1"].sum() + em["amb2"].sum())
    return y, cache


def mlp3_backward(P, cache, gy, gy_var=None, return_model: bool = False):
    """Gradients of sum(gy * y): returns (gx, {dW1, db1, dW2, db2, dW3, db3}).
    With return_model (and a cache made with a precision) also a dict:
    "parts" {key: (variance, largest single flip, expected shift)} per
    parameter gradient, "gx_var" and "gx_worst" (variance and worst case of
    gx from flipped decisions and from gy_var, a variance of gy)."""
    P = {k: np.asarray(v, dtype=np.float64) for k, v in P.items()}
    gy = np.asarray(gy, dtype=np.float64)
    g = {"dW3": gy.T @ cache["h2"], "db3": gy.sum(0)}
    ga2 = (gy @ P["W3"]) * cache["m2"]
    g["dW2"] = ga2.T @ cache["h1"]
    g["db2"] = ga2.sum(0)
    ga1 = (ga2 @ P["W2"]) * cache["m1"]
    g["dW1"] = ga1.T @ cache["x"]
    g["db1"] = ga1.sum(0)
    gx = ga1 @ P["W1"]
    if not return_model:
        return gx, g
    gv = np.zeros_like(gy) if gy_var is None else np.asarray(gy_var, dtype=np.float64)
    h2 = cache["h2"]
    zero = lambda a: np.zeros_like(a)
    vW3 = gv.T @ (h2 * h2)
    vb3 = gv.sum(0)
    flips = nnconv.FlipModel(P["W1"], P["W2"])
    gx_var, gx_worst = flips.add(gy @ P["W3"], gv @ (P["W3"] ** 2), cache["em"], cache["h1"], cache["x"])
    parts = {"dW3": (vW3, zero(vW3), zero(vW3)), "db3": (vb3, zero(vb3), zero(vb3))}
    parts.update({"d" + k: v for k, v in flips.parts().items()})
    return gx, g, {"parts": parts, "gx_var": gx_var, "gx_worst": gx_worst}


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


def _features(v, v_var, dtype):
    """The layer's input features: v rounded to the layer type, and the
    variance of the difference between a kernel's rounding of its own value
    and this one (a value carrying variance v_var lands on a neighbouring
    bfloat16 value, one spacing away, with probability about 2 sigma /
    spacing)."""
    v = np.asarray(v, dtype=np.float64)
    if dtype != "bf16":
        return v, v_var
    q = nnconv.bf16(v)
    mag = np.maximum(np.abs(v), np.finfo(np.float32).tiny)
    ulp = 2.0 ** (np.floor(np.log2(mag)) - 7)
    sig = np.sqrt(v_var)
    return q, np.maximum(v_var, np.minimum(1.0, 2.0 * sig / ulp) * ulp * ulp)


def _sum_parts(acc, parts):
    for k, (v, mx, mean) in parts.items():
        if k in acc:
            a = acc[k]
            acc[k] = (a[0] + v, np.maximum(a[1], mx), a[2] + mean)
        else:
            acc[k] = (v.copy(), mx.copy(), mean.copy())


def train_step(Pe, Pk, Pd, v0, Y, mask, row_ptr, col, n_hops: int, dtype: str = "f32"):
    """Loss and gradients of one step of the hop loop on one sub-domain.

    Pe, Pd: encoder / decoder parameters (mlp3 layout); Pk: convolution
    parameters (``oracle.nnconv`` layout, with W1 [h1, dim+1]); v0 [n, dim+1]
    input node values; Y [n, dim+1] targets; mask [n] interior rows; the graph
    (row_ptr, col) joins the n nodes (every node is a destination); dtype:
    the layer's operand type ("f32" or "bf16"; the perceptrons are float32).
    Returns a dict: loss, v (final decoder output), vL (final latent), the
    gradients "enc", "conv", "dec" (dicts keyed like the parameters with a
    leading "d"), "allow" (the same three groups plus "loss", "v", "vL": the
    allowances of the precision model) and "ambiguous" (decisions inside
    their bands, a diagnostic).
    """
    v0 = np.asarray(v0, dtype=np.float64)
    n = v0.shape[0]
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    dst = np.repeat(np.arange(n), np.diff(row_ptr))
    A = nnconv.ALLOW_SIGMAS
    # forward, with the modelled variance of every value
    vL, enc_cache = mlp3_forward(Pe, v0, "f32")
    vL_var = enc_cache["y_var"]
    n_amb = enc_cache["n_amb"]
    v, v_var = v0, np.zeros_like(v0)
    hops = []
    for _ in range(n_hops):
        x = nnconv.edge_attr(v, row_ptr, col, mode="diff")
        x_var = v_var[dst] + v_var[col]
        h_in, h_var = _features(vL, vL_var, dtype)
        out, _, st = nnconv.forward(Pk, x, h_in, row_ptr, col, n, precision=dtype, x_var=x_var, h_var=h_var,
                                    return_stats=True)
        v_new, dec_cache = mlp3_forward(Pd, out, "f32", st["out_var"])
        n_amb += dec_cache["n_amb"] + int(nnconv.edge_mlp(Pk, x, dtype, x_var)["amb1"].sum())
        hops.append({"x": x, "x_var": x_var, "h_in": h_in, "h_var": h_var, "out": out, "dec": dec_cache})
        vL, vL_var, v, v_var = out, st["out_var"], v_new, dec_cache["y_var"]
    loss, gv = masked_mse(v, Y, mask)
    m = np.asarray(mask, dtype=bool)
    count = max(int(m.sum()) * v.shape[1], 1)
    gv_var = np.where(m[:, None], (2.0 / count) ** 2 * v_var, 0.0)
    loss_var = float((gv * gv * v_var).sum())
    # backward: gv is the gradient with respect to the decoder output v^{l+1},
    # g_lat the one with respect to the convolution output out^l through the
    # next hop's latent input; flips feed the variances of both upstream
    g_conv = {"d" + k: np.zeros_like(np.asarray(Pk[k], dtype=np.float64))
              for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")}
    p_conv, p_dec = {}, {}
    g_dec = None
    g_lat = np.zeros((n, np.asarray(Pk["Wr"]).shape[0]))
    g_lat_var = np.zeros_like(g_lat)
    for l in reversed(range(n_hops)):
        hp = hops[l]
        g_out, gd, md = mlp3_backward(Pd, hp["dec"], gv, gv_var, return_model=True)
        g_dec = gd if g_dec is None else {k: g_dec[k] + gd[k] for k in gd}
        _sum_parts(p_dec, md["parts"])
        g_out_var = md["gx_var"] + md["gx_worst"] ** 2
        gc = nnconv.backward(Pk, hp["x"], hp["h_in"], row_ptr, col, n, g_out + g_lat, precision=dtype,
                             x_var=hp["x_var"], h_var=hp["h_var"], grad_var=g_out_var + g_lat_var)
        for k in g_conv:
            g_conv[k] += gc[k]
        _sum_parts(p_conv, gc["flip_parts"])
        for k in ("dW3", "db3", "dWr", "dbr"):
            _sum_parts(p_conv, {k: (gc["var"][k], np.zeros_like(gc[k]), np.zeros_like(gc[k]))})
        g_lat, g_lat_var = gc["grad_h"], gc["var"]["grad_h"]
        gx_v = gc["var"]["grad_x"] + (gc["allow"]["grad_x"] - A * np.sqrt(gc["var"]["grad_x"])) ** 2
        gv = np.zeros_like(v0)               # with respect to v^l, through x^l = v_i - v_j
        np.add.at(gv, dst, gc["grad_x"])
        np.add.at(gv, col, -gc["grad_x"])
        gv_var = np.zeros_like(v0)
        np.add.at(gv_var, dst, gx_v)
        np.add.at(gv_var, col, gx_v)
    _, g_enc, me = mlp3_backward(Pe, enc_cache, g_lat if n_hops else np.zeros_like(vL), g_lat_var,
                                 return_model=True)
    allow = {"enc": {k: nnconv.bernstein_allowance(*p) for k, p in me["parts"].items()},
             "conv": {k: nnconv.bernstein_allowance(*p) for k, p in p_conv.items()},
             "dec": {k: nnconv.bernstein_allowance(*p) for k, p in p_dec.items()},
             "loss": A * np.sqrt(loss_var), "v": A * np.sqrt(v_var), "vL": A * np.sqrt(vL_var)}
    return {"loss": loss, "v": v, "vL": vL, "enc": g_enc, "conv": g_conv, "dec": g_dec, "allow": allow,
            "ambiguous": n_amb}
