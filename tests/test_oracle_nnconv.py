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


def test_a1_float32_chain_bounds_and_exact_cases():
    g = np.random.default_rng(3)
    P = {"W1": g.normal(size=(16, 6)).astype(np.float32), "b1": g.normal(size=16).astype(np.float32)}
    x = g.uniform(0, 2, (500, 6)).astype(np.float32)
    a64 = x.astype(np.float64) @ P["W1"].astype(np.float64).T + P["b1"]
    a32 = nn.a1_float32(P, x)
    s1 = np.abs(x) @ np.abs(P["W1"]).T.astype(np.float64) + np.abs(P["b1"])
    assert np.all(np.abs(a32 - a64) <= 6 * 2.0 ** -24 * s1)
    assert np.all(a32 == a32.astype(np.float32))           # representable in float32
    # small integers: no rounding anywhere, so the chain is exact
    Pi = {"W1": g.integers(-3, 4, (8, 4)).astype(np.float32), "b1": g.integers(-3, 4, 8).astype(np.float32)}
    xi = g.integers(-3, 4, (50, 4)).astype(np.float32)
    assert np.array_equal(nn.a1_float32(Pi, xi), xi.astype(np.float64) @ Pi["W1"].T.astype(np.float64) + Pi["b1"])


@pytest.mark.parametrize("decide", ["f32", "bf16"])
def test_decided_layer_matches_float64_away_from_kinks(decide):
    na, rp, col, P, h, x = _random_case(12, n=60, n_dst=50, cap=8)
    P32 = {k: v.astype(np.float32) for k, v in P.items()}
    G = np.random.default_rng(1).normal(size=(50, h.shape[1]))
    ref = nn.backward(P32, x, h, rp, col, 50, G)
    got = nn.backward(P32, x, h, rp, col, 50, G, decide=decide)
    a1, z1, a2, z = nn._edge_mlp(nn._as64(P32), x)
    # the decided masks agree with float64 signs except within the rounding band
    a1d = nn.a1_float32(P32, x)
    assert np.all((a1d > 0) == (a1 > 0))
    if decide == "f32":
        for k in ref:
            if k != "allow":
                assert np.allclose(got[k], ref[k], rtol=1e-9, atol=1e-9), k


@pytest.mark.parametrize("layer", ["a1", "a2"])
def test_allowance_covers_flipped_decisions(monkeypatch, layer):
    """Plant flips of every decision of one layer that the oracle calls
    ambiguous (with that layer's band widened so there are many); the change
    must stay within the allowance.  Flipping a1 also moves z1 inside the
    band, a second-order effect on dW2 that is negligible at the real band
    width but not at this one, so that case checks dW1 and db1 only."""
    na, rp, col, P, h, x = _random_case(13, n=80, n_dst=70, cap=10)
    P32 = {k: v.astype(np.float32) for k, v in P.items()}
    G = np.random.default_rng(2).normal(size=(70, h.shape[1]))
    monkeypatch.setattr(nn, "_EPS_A1" if layer == "a1" else "_EPS_A2", 0.05)
    base = nn.backward(P32, x, h, rp, col, 70, G, decide="f32")
    orig = nn._edge_mlp_decided

    def flipped(P_, x_, decide):
        a1, z1, a2, z, m1, m2, zq, amb1, amb2 = orig(P_, x_, decide)
        m1 = np.where(amb1, ~m1, m1)
        m2 = np.where(amb2, ~m2, m2)
        z1 = np.where(m1, a1, 0.0)
        a2 = z1 @ P_["W2"].T + P_["b2"]
        z = np.where(m2, a2, 0.0)
        return a1, z1, a2, z, m1, m2, zq, amb1, amb2

    monkeypatch.setattr(nn, "_edge_mlp_decided", flipped)
    alt = nn.backward(P32, x, h, rp, col, 70, G, decide="f32")
    keys = ("dW2", "db2", "dW1", "db1") if layer == "a2" else ("dW1", "db1")
    nflip = 0
    for k in keys:
        diff = np.abs(alt[k] - base[k])
        nflip += int((diff > 1e-12).sum())
        assert np.all(diff <= base["allow"][k] + 1e-9 * np.abs(base[k]).max()), k
    assert nflip > 0
