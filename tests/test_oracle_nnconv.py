"""Pins for the oracle's NNConv layer, forward and backward (CPU only)."""

import inspect
import json
import os

import numpy as np
import pytest

from oracle import nnconv as nn
from oracle import radius_graph as rg

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _hand():
    with open(os.path.join(GOLDEN, "hand_3node.json")) as f:
        return json.load(f)


def _hand_params(c):
    return {k: np.array(c[k], dtype=np.float64) for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")}


def _hand_check(mod):
    """True when module ``mod`` reproduces every hand-worked value."""
    c = _hand()
    na = np.array(c["node_attr"], np.float32)
    rp, col = rg.radius_graph(na[:, :2], 3, c["r"])
    if rp.tolist() != c["row_ptr"] or col.tolist() != c["col"]:
        return False
    x = mod.edge_attr(na, rp, col)
    if not np.allclose(x, c["x_e"]):
        return False
    P = _hand_params(c)
    h = np.array(c["h"], np.float64)
    out, y = mod.forward(P, x, h, rp, col, 3, mod.ACT_IDENTITY, True)
    out_r, _ = mod.forward(P, x, h, rp, col, 3, mod.ACT_RELU, True)
    return (np.allclose(y, c["y"], atol=1e-12) and np.allclose(out, c["out_identity"], atol=1e-12)
            and np.allclose(out_r, c["out_relu"], atol=1e-12))


def test_hand_worked_three_node_graph():
    assert _hand_check(nn)


MUTANTS = {
    "theta_not_transposed": ('np.einsum("epq,ep->eq", theta, h[col[e]])', 'np.einsum("epq,eq->ep", theta, h[col[e]])'),
    "q_major_reshape": ("theta = w.reshape(-1, d, d)                       # theta[e, p, q]",
                        "theta = w.reshape(-1, d, d).transpose(0, 2, 1)"),
    "sum_not_mean": ("agg[nz] = s[nz] / deg[nz][:, None]", "agg[nz] = s[nz]"),
    "no_root": ('y[sel] = agg[sel] + h[sel] @ P["Wr"].T + P["br"]', 'y[sel] = agg[sel] + P["br"]'),
    "root_transposed": ('y[sel] = agg[sel] + h[sel] @ P["Wr"].T + P["br"]', 'y[sel] = agg[sel] + h[sel] @ P["Wr"] + P["br"]'),
    "no_kernel_bias": ('w = z @ P["W3"].T + P["b3"]                       # [n, d*d]', 'w = z @ P["W3"].T'),
    "no_residual": ("out[sel] = h[sel] + a if residual else a", "out[sel] = a"),
    "src_dst_swapped_attr": ("[na[dst, :D], na[src, :D], na[dst, D:D + 1], na[src, D:D + 1]]",
                             "[na[src, :D], na[dst, :D], na[src, D:D + 1], na[dst, D:D + 1]]"),
    "relu_dropped_layer2": ("z = _relu(a2)", "z = a2"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_hand_pin_catches_planted_mistakes(name):
    """Plant one plausible mistake in a copy of the oracle; the pin must fail."""
    old, new = MUTANTS[name]
    src = inspect.getsource(nn)
    assert old in src, name
    ns = {}
    exec(compile(src.replace(old, new), "mutant", "exec"), ns)
    mod = type("M", (), {k: staticmethod(v) if callable(v) else v for k, v in ns.items()})
    assert not _hand_check(mod)


def _random_case(seed, n=40, n_dst=None, D=2, d=4, H1=5, H2=3, r=0.35, cap=0):
    g = np.random.default_rng(seed)
    n_dst = n if n_dst is None else n_dst
    na = g.uniform(0, 1, (n, D + 1)).astype(np.float32)
    rp, col = rg.radius_graph(na[:, :D], n_dst, r, cap)
    de = 2 * D + 2
    P = {"W1": g.normal(size=(H1, de)), "b1": g.normal(size=H1), "W2": g.normal(size=(H2, H1)),
         "b2": g.normal(size=H2), "W3": g.normal(size=(d * d, H2)), "b3": g.normal(size=d * d),
         "Wr": g.normal(size=(d, d)), "br": g.normal(size=d)}
    h = g.normal(size=(n, d))
    x = nn.edge_attr(na, rp, col)
    return na, rp, col, P, h, x


def test_constant_kernel_is_neighbour_mean():
    na, rp, col, P, h, x = _random_case(1)
    d = h.shape[1]
    P["W3"][:] = 0
    P["b3"] = np.eye(d).ravel()
    P["Wr"][:] = 0
    P["br"][:] = 0
    out, _ = nn.forward(P, x, h, rp, col, len(rp) - 1, residual=False)
    for i in range(len(rp) - 1):
        nb = col[rp[i]:rp[i + 1]]
        want = h[nb].mean(0) if nb.size else np.zeros(d)
        assert np.allclose(out[i], want, atol=1e-12)


def test_constant_matrix_kernel_against_matmul():
    na, rp, col, P, h, x = _random_case(2)
    d = h.shape[1]
    A = np.random.default_rng(0).normal(size=(d, d))
    P["W3"][:] = 0
    P["b3"] = A.ravel()                      # Theta = A for every edge
    out, y = nn.forward(P, x, h, rp, col, len(rp) - 1, residual=False)
    M = h @ A                                # row j holds (A^T h_j)^T
    for i in range(len(rp) - 1):
        nb = col[rp[i]:rp[i + 1]]
        agg = M[nb].mean(0) if nb.size else 0.0
        assert np.allclose(out[i], agg + P["Wr"] @ h[i] + P["br"], atol=1e-10)


def test_affine_in_h():
    na, rp, col, P, h1, x = _random_case(3)
    h2 = np.random.default_rng(9).normal(size=h1.shape)
    nd = len(rp) - 1
    f = lambda h: nn.forward(P, x, h, rp, col, nd)[0] - P["br"]
    a, b = 0.7, -1.3
    assert np.allclose(f(a * h1 + b * h2), a * f(h1) + b * f(h2), atol=1e-9)


def test_permutation_equivariance():
    na, rp, col, P, h, x = _random_case(4, n=50)
    out, _ = nn.forward(P, x, h, rp, col, 50)
    perm = np.random.default_rng(1).permutation(50)
    na2, h2 = na[perm], h[perm]
    rp2, col2 = rg.radius_graph(na2[:, :2], 50, 0.35)
    out2, _ = nn.forward(P, nn.edge_attr(na2, rp2, col2), h2, rp2, col2, 50)
    assert np.allclose(out2, out[perm], atol=1e-10)


def test_isolated_node_gets_root_term_only():
    na, rp, col, P, h, x = _random_case(5)
    na = na.copy()
    na[0, :2] = 50.0                          # far from everyone
    rp, col = rg.radius_graph(na[:, :2], 40, 0.35)
    assert rp[1] - rp[0] == 0
    x = nn.edge_attr(na, rp, col)
    out, y = nn.forward(P, x, h, rp, col, 40)
    assert np.allclose(y[0], P["Wr"] @ h[0] + P["br"], atol=1e-12)
    assert np.allclose(out[0], h[0] + y[0], atol=1e-12)


def test_edge_attr_layouts():
    na = np.array([[0, 1, 5], [2, 3, 7]], np.float32)
    rp, col = np.array([0, 1, 2]), np.array([1, 0])
    assert nn.edge_attr(na, rp, col).tolist() == [[0, 1, 2, 3, 5, 7], [2, 3, 0, 1, 7, 5]]
    assert nn.edge_attr(na, rp, col, "diff").tolist() == [[-2, -2, -2], [2, 2, 2]]


def _loss(P, x, h, rp, col, nd, G, act, res):
    return float((nn.forward(P, x, h, rp, col, nd, act, res)[0] * G).sum())


@pytest.mark.parametrize("act,res", [(nn.ACT_IDENTITY, True), (nn.ACT_RELU, True), (nn.ACT_IDENTITY, False)])
def test_backward_central_differences(act, res):
    na, rp, col, P, h, x = _random_case(6, n=30, n_dst=24, r=0.4, cap=6)
    nd = 24
    G = np.random.default_rng(2).normal(size=(nd, h.shape[1]))
    grads = nn.backward(P, x, h, rp, col, nd, G, act, res)
    eps = 1e-6
    for key in ["h", "x", "W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br"]:
        base = {"h": h, "x": x}.get(key, P.get(key))
        gkey = {"h": "grad_h", "x": "grad_x"}.get(key, "d" + key)
        flat = base.reshape(-1)
        idx = np.random.default_rng(7).choice(flat.size, size=min(flat.size, 12), replace=False)
        for t in idx:
            old = flat[t]
            flat[t] = old + eps
            lp = _loss(P, x, h, rp, col, nd, G, act, res)
            flat[t] = old - eps
            lm = _loss(P, x, h, rp, col, nd, G, act, res)
            flat[t] = old
            fd = (lp - lm) / (2 * eps)
            an = grads[gkey].reshape(-1)[t]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (key, t, fd, an)


def test_backward_adjoint_identity():
    # out is affine in h: J v = out(h+v) - out(h); <J v, w> must equal <v, J^T w>
    na, rp, col, P, h, x = _random_case(7, n=60, n_dst=50, cap=8)
    g = np.random.default_rng(3)
    v = g.normal(size=h.shape)
    w = g.normal(size=(50, h.shape[1]))
    Jv = nn.forward(P, x, h + v, rp, col, 50)[0] - nn.forward(P, x, h, rp, col, 50)[0]
    JTw = nn.backward(P, x, h, rp, col, 50, w)["grad_h"]
    assert abs((Jv * w).sum() - (v * JTw).sum()) <= 1e-9 * abs((v * JTw).sum())


def test_constant_kernel_backward_closed_form():
    na, rp, col, P, h, x = _random_case(8)
    d = h.shape[1]
    P["W3"][:] = 0
    P["b3"] = np.eye(d).ravel()
    P["Wr"][:] = 0
    G = np.random.default_rng(4).normal(size=(40, d))
    gh = nn.backward(P, x, h, rp, col, 40, G, residual=False)["grad_h"]
    deg = np.diff(rp)
    want = np.zeros_like(h)
    for i in range(40):
        for j in col[rp[i]:rp[i + 1]]:
            want[j] += G[i] / deg[i]
    assert np.allclose(gh, want, atol=1e-12)


def test_rows_subset_matches_full():
    na, rp, col, P, h, x = _random_case(9, n=80, n_dst=70, cap=7)
    rows = [0, 5, 33, 69]
    full, _ = nn.forward(P, x, h, rp, col, 70)
    sub, _ = nn.forward(P, x, h, rp, col, 70, rows=rows)
    assert np.allclose(sub[rows], full[rows])
    G = np.zeros((70, h.shape[1]))
    G[rows] = np.random.default_rng(5).normal(size=(len(rows), h.shape[1]))
    a = nn.backward(P, x, h, rp, col, 70, G)
    b = nn.backward(P, x, h, rp, col, 70, G, rows=rows)
    for k in a:
        if k != "allow":
            assert np.allclose(a[k], b[k], atol=1e-12), k


def test_backward_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    na, rp, col, P, h, x = _random_case(10, n=35, n_dst=30, cap=5)
    nd = 30
    G = np.random.default_rng(6).normal(size=(nd, h.shape[1]))
    for act in (nn.ACT_IDENTITY, nn.ACT_RELU):
        T = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in P.items()}
        th = torch.tensor(h, dtype=torch.float64, requires_grad=True)
        tx = torch.tensor(x, dtype=torch.float64, requires_grad=True)
        dst = torch.tensor(rg.dst_of_edges(rp), dtype=torch.long)
        src = torch.tensor(col, dtype=torch.long)
        d = h.shape[1]
        z = torch.relu(torch.relu(tx @ T["W1"].T + T["b1"]) @ T["W2"].T + T["b2"])
        theta = (z @ T["W3"].T + T["b3"]).reshape(-1, d, d)
        m = torch.bmm(theta.transpose(1, 2).contiguous(), th[src].unsqueeze(2)).squeeze(2)
        s = torch.zeros(nd, d, dtype=torch.float64).index_add(0, dst, m)
        deg = torch.tensor(np.maximum(np.diff(rp), 1), dtype=torch.float64)[:, None]
        y = s / deg + th[:nd] @ T["Wr"].T + T["br"]
        out = th[:nd] + (torch.relu(y) if act == nn.ACT_RELU else y)
        (out * torch.tensor(G)).sum().backward()
        ref = nn.backward(P, x, h, rp, col, nd, G, act)
        assert np.allclose(out.detach().numpy(), nn.forward(P, x, h, rp, col, nd, act)[0], atol=1e-10)
        assert np.allclose(th.grad.numpy(), ref["grad_h"], atol=1e-9)
        assert np.allclose(tx.grad.numpy(), ref["grad_x"], atol=1e-9)
        for k in T:
            assert np.allclose(T[k].grad.numpy(), ref["d" + k], atol=1e-9), k


# ---------------------------------------------------------------- decision path

def test_bf16_rounding_known_values():
    torch = pytest.importorskip("torch")
    vals = np.array([1.0, 1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -2.5, 3.0e-39, 65504.0, 1e30], np.float32)
    want = [1.0, 1.0, 1 + 2.0 ** -6, -2.5]
    assert nn.bf16(vals)[:4].tolist() == want            # ties to even
    r = np.random.default_rng(0).normal(size=10000).astype(np.float32) * 10.0 ** np.random.default_rng(1).integers(-20, 20, 10000)
    lib = torch.from_numpy(r).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(nn.bf16(r), lib.astype(np.float64))


# A plain evaluation in the workloads' precision, written here for the pins
# only: float32 arithmetic, operands of bfloat16 products rounded to bfloat16
# where they are formed, sums in the order numpy's float32 routines take
# (forward) or in reverse attribute / neuron order.  It is one of the many
# evaluations a correct kernel may perform; the precision model must cover it.

def _bf(a):
    return nn.bf16(a).astype(np.float32)


def _eval_lowp(P, x, h, rp, col, n_dst, precision, reverse=False):
    f = np.float32
    P32 = {k: np.asarray(v, dtype=f) for k, v in P.items()}
    x32, h32 = np.asarray(x, dtype=f), np.asarray(h, dtype=f)
    rd = (lambda a: _bf(a)) if precision == "bf16" else (lambda a: a.astype(f))
    if reverse:
        a1 = np.broadcast_to(P32["b1"], (x32.shape[0], P32["b1"].size)).astype(f).copy()
        for c in reversed(range(x32.shape[1])):
            a1 = (a1 + x32[:, c:c + 1] * P32["W1"][None, :, c]).astype(f)
    else:
        a1 = (x32 @ P32["W1"].T + P32["b1"]).astype(f)
    z1 = rd(np.maximum(a1, f(0)))
    if reverse:
        a2 = np.broadcast_to(P32["b2"], (x32.shape[0], P32["b2"].size)).astype(f).copy()
        for j in reversed(range(z1.shape[1])):
            a2 = (a2 + z1[:, j:j + 1] * P32["W2"][None, :, j]).astype(f)
    else:
        a2 = (z1 @ P32["W2"].T + P32["b2"]).astype(f)
    z = rd(np.maximum(a2, f(0)))
    d = h32.shape[1]
    theta = (z @ P32["W3"].T + P32["b3"]).astype(f).reshape(-1, d, d)
    m = np.einsum("epq,ep->eq", theta, h32[col]).astype(f)
    deg = np.diff(rp)[:n_dst]
    agg = np.zeros((n_dst, d), f)
    np.add.at(agg, np.repeat(np.arange(n_dst), deg), m)
    agg[deg > 0] /= deg[deg > 0][:, None].astype(f)
    y = (agg + h32[:n_dst] @ P32["Wr"].T + P32["br"]).astype(f)
    return a1.astype(np.float64), a2.astype(np.float64), y.astype(np.float64)


def _lowp_case(seed, precision, n=300, d=16, H1=32, H2=32):
    from workloads import layer_params
    g = np.random.default_rng(seed)
    na = g.uniform(0, 1, (n, 3)).astype(np.float32)
    rp, col = rg.radius_graph(na[:, :2], n, 0.12, 16)
    P = layer_params(g, d, 6, H1, H2, precision)
    h = g.normal(size=(n, d)).astype(np.float32)
    if precision == "bf16":
        h = _bf(h)
    return na, rp, col, P, h.astype(np.float64), nn.edge_attr(na, rp, col)


@pytest.mark.parametrize("precision", ["f32", "bf16"])
@pytest.mark.parametrize("reverse", [False, True])
def test_precision_model_covers_a_low_precision_evaluation(precision, reverse):
    """The deviations of a float32 / bfloat16 evaluation from the float64
    values stay within the modelled spread (root mean square below one
    standard deviation, none beyond the band), and its decisions agree with
    the float64 decisions outside the band."""
    na, rp, col, P, h, x = _lowp_case(21 + reverse, precision)
    n = len(rp) - 1
    em = nn.edge_mlp(P, x, precision)
    _, y, st = nn.forward(P, x, h, rp, col, n, nn.ACT_RELU, precision=precision, return_stats=True)
    a1, a2, yl = _eval_lowp(P, x, h, rp, col, n, precision, reverse)
    for got, want, var in ((a1, em["a1"], em["v1"]), (a2, em["a2"], em["v2"]), (yl, y, st["y_var"])):
        t = (got - want) / np.sqrt(var)
        assert np.sqrt(np.mean(t * t)) <= 1.0
        assert np.abs(t).max() <= nn.BAND_SIGMAS
        band = nn.ambiguous(want, var)
        assert np.array_equal((got > 0)[~band], (want > 0)[~band])


def test_exact_arithmetic_has_no_band():
    na, rp, col, P, h, x = _lowp_case(23, "f32", n=80)
    em = nn.edge_mlp(P, x, None)
    assert "v1" not in em
    ref = nn.backward(P, x, h, rp, col, 80, np.ones((80, 16)))
    assert ref["allow"] == {}
    # a small-integer layer in float32 is computed exactly, and the model's
    # spread of a1 is within one rounding of its largest partial sum
    Pi = {"W1": np.arange(-6, 6).reshape(2, 6).astype(np.float64), "b1": np.array([1.0, -2.0]),
          "W2": np.eye(2), "b2": np.zeros(2)}
    xi = np.array([[1, 0, 2, 0, 1, 1], [0, 1, 1, 1, 0, 0]], np.float64)
    em = nn.edge_mlp(Pi, xi, "f32")
    s1 = np.abs(xi) @ np.abs(Pi["W1"]).T + np.abs(Pi["b1"])
    assert np.all(np.sqrt(em["v1"]) <= 7 * nn.U_F32 * s1)
    assert np.array_equal(em["a1"], xi @ Pi["W1"].T + Pi["b1"])


def test_flip_probability_closed_form():
    from math import erfc, sqrt
    assert nn.flip_probability(0.0, 1.0) == pytest.approx(0.5)
    assert nn.flip_probability(1.0, 1.0) == pytest.approx(0.5 * erfc(1 / sqrt(2)))
    assert nn.flip_probability(-3.0, 4.0) == pytest.approx(0.5 * erfc(1.5 / sqrt(2)))
    assert nn.flip_probability(1.0, 0.0) == 0.0
    assert nn.flip_probability(50.0, 1.0) < 1e-300 or nn.flip_probability(50.0, 1.0) == 0.0


def test_bernstein_allowance_closed_form():
    L = 0.5 * nn.ALLOW_SIGMAS ** 2
    # no single-flip bound: the Gaussian case, ALLOW_SIGMAS standard deviations
    assert nn.bernstein_allowance(np.array(4.0), np.array(0.0), np.array(0.0)) == pytest.approx(2 * nn.ALLOW_SIGMAS)
    # no variance: 2 L b / 3 (one flip of size b is covered for ALLOW_SIGMAS >= 2)
    assert nn.bernstein_allowance(np.array(0.0), np.array(3.0), np.array(-1.0)) == pytest.approx(1 + 2 * L)
    t = nn.bernstein_allowance(np.array(2.0), np.array(0.5), np.array(0.0))
    assert t * t / 2 == pytest.approx(L * (2.0 + 0.5 * t / 3))


@pytest.mark.parametrize("precision", ["f32", "bf16"])
def test_values_do_not_depend_on_the_model(precision):
    na, rp, col, P, h, x = _lowp_case(24, precision, n=120)
    G = np.random.default_rng(1).normal(size=(120, 16))
    a = nn.backward(P, x, h, rp, col, 120, G, nn.ACT_RELU)
    b = nn.backward(P, x, h, rp, col, 120, G, nn.ACT_RELU, precision=precision)
    for k in a:
        if k != "allow":
            assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(nn.forward(P, x, h, rp, col, 120)[0],
                          nn.forward(P, x, h, rp, col, 120, precision=precision)[0])


def _flipped_backward(monkeypatch, P, x, h, rp, col, n, G, precision, choose):
    """Backward with masks changed where ``choose(em)`` says (values kept):
    a kernel that took those decisions the other way."""
    orig = nn.edge_mlp

    def patched(P_, x_, precision_=None, x_var=None):
        em = orig(P_, x_, precision_, x_var)
        if precision_ is not None:
            f1, f2 = choose(em)
            em = dict(em, m1=em["m1"] ^ f1, m2=em["m2"] ^ f2)
        return em

    monkeypatch.setattr(nn, "edge_mlp", patched)
    try:
        return nn.backward(P, x, h, rp, col, n, G, precision=precision)
    finally:
        monkeypatch.setattr(nn, "edge_mlp", orig)


def test_allowance_covers_random_flips(monkeypatch):
    """Flip each decision with its modelled probability (several draws): the
    weight gradients move by less than their allowance."""
    na, rp, col, P, h, x = _lowp_case(25, "bf16", n=400, d=16, H1=64, H2=64)
    n = len(rp) - 1
    G = np.random.default_rng(3).normal(size=(n, 16))
    base = nn.backward(P, x, h, rp, col, n, G, precision="bf16")
    em = nn.edge_mlp(P, x, "bf16")
    assert em["amb1"].sum() + em["amb2"].sum() > 20        # the draws do flip decisions
    rng = np.random.default_rng(4)
    moved = 0
    for _ in range(4):
        alt = _flipped_backward(monkeypatch, P, x, h, rp, col, n, G, "bf16",
                                lambda e: (rng.uniform(size=e["p1"].shape) < e["p1"],
                                           rng.uniform(size=e["p2"].shape) < e["p2"]))
        for k in ("dW1", "db1", "dW2", "db2"):
            diff = np.abs(alt[k] - base[k])
            moved += int((diff > 0).sum())
            assert np.all(diff <= base["allow"][k]), k
    assert moved > 0


def test_worst_case_covers_every_ambiguous_flip(monkeypatch):
    """grad_x of an edge moves by at most its worst-case allowance when every
    ambiguous decision of the edge is flipped."""
    na, rp, col, P, h, x = _lowp_case(26, "bf16", n=300, d=16, H1=64, H2=64)
    n = len(rp) - 1
    G = np.random.default_rng(5).normal(size=(n, 16))
    base = nn.backward(P, x, h, rp, col, n, G, precision="bf16")
    alt = _flipped_backward(monkeypatch, P, x, h, rp, col, n, G, "bf16", lambda e: (e["amb1"], e["amb2"]))
    diff = np.abs(alt["grad_x"] - base["grad_x"])
    assert diff.max() > 0
    assert np.all(diff <= base["allow"]["grad_x"] * (1 + 1e-9) + 1e-15)


def test_allowance_propagates_an_upstream_variance():
    """A variance of grad_out reaches every gradient linear in it; with unit
    variance on one row the dWr allowance is ALLOW_SIGMAS * |h_i| per column."""
    na, rp, col, P, h, x = _lowp_case(27, "f32", n=60)
    G = np.random.default_rng(6).normal(size=(60, 16))
    Gv = np.zeros_like(G)
    Gv[7] = 1.0
    a = nn.backward(P, x, h, rp, col, 60, G, precision="f32")
    b = nn.backward(P, x, h, rp, col, 60, G, precision="f32", grad_var=Gv)
    assert np.allclose(b["var"]["dWr"] - a["var"]["dWr"], np.outer(Gv[7], h[7] ** 2))
    for k in ("dW3", "db3", "grad_h"):
        assert b["allow"][k].max() > a["allow"][k].max(), k


def test_model_pin_catches_a_dropped_rounding(monkeypatch):
    """Planted mistake: a model that forgets the bfloat16 rounding of the
    product operands underestimates the spread, and the coverage pin fails."""
    orig = nn.units
    monkeypatch.setattr(nn, "units", lambda p: (nn.U_F32, nn.U_F32) if p == "bf16" else orig(p))
    with pytest.raises(AssertionError):
        test_precision_model_covers_a_low_precision_evaluation("bf16", False)
