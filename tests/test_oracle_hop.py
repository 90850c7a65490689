"""Pins for the oracle's hop loop: encoder/decoder perceptrons, masked MSE and
one training step of Algorithm 1 (CPU only)."""

import numpy as np
import pytest

from oracle import hop
from oracle import nnconv as nn
from oracle import radius_graph as rg


def _mlp_params(g, d_in, d_hid, d_out):
    return {"W1": g.normal(size=(d_hid, d_in)), "b1": g.normal(size=d_hid),
            "W2": g.normal(size=(d_hid, d_hid)) / np.sqrt(d_hid), "b2": g.normal(size=d_hid),
            "W3": g.normal(size=(d_out, d_hid)) / np.sqrt(d_hid), "b3": g.normal(size=d_out)}


def _case(seed, n=24, D=2, d=4, H1=5, H2=3, hid=6, r=0.4, cap=5):
    g = np.random.default_rng(seed)
    v0 = g.uniform(0, 1, (n, D + 1))
    rp, col = rg.radius_graph(v0[:, :D].astype(np.float32), n, r, cap)
    de = D + 1
    Pk = {"W1": g.normal(size=(H1, de)), "b1": g.normal(size=H1), "W2": g.normal(size=(H2, H1)),
          "b2": g.normal(size=H2), "W3": g.normal(size=(d * d, H2)) / d, "b3": g.normal(size=d * d) / d,
          "Wr": g.normal(size=(d, d)) / d, "br": g.normal(size=d)}
    Pe = _mlp_params(g, de, hid, d)
    Pd = _mlp_params(g, d, hid, de)
    Y = g.normal(size=(n, de))
    mask = g.uniform(size=n) < 0.7
    return Pe, Pk, Pd, v0, Y, mask, rp, col


def test_mlp3_known_values():
    # one hidden unit per layer, hand-computed
    P = {"W1": np.array([[2.0, -1.0]]), "b1": np.array([0.5]), "W2": np.array([[3.0]]), "b2": np.array([-1.0]),
         "W3": np.array([[1.0], [-2.0]]), "b3": np.array([0.25, 0.0])}
    y, _ = hop.mlp3_forward(P, np.array([[1.0, 1.0], [0.0, 1.0]]))
    # row 0: a1 = 2-1+0.5 = 1.5, a2 = 4.5-1 = 3.5, y = [3.75, -7]; row 1: a1 = -0.5 -> 0, a2 = -1 -> 0, y = b3
    assert np.allclose(y, [[3.75, -7.0], [0.25, 0.0]])


def test_mlp3_backward_central_differences():
    g = np.random.default_rng(1)
    P = _mlp_params(g, 3, 7, 4)
    x = g.normal(size=(9, 3))
    G = g.normal(size=(9, 4))
    y, cache = hop.mlp3_forward(P, x)
    gx, gr = hop.mlp3_backward(P, cache, G)
    eps = 1e-6

    def loss():
        return float((hop.mlp3_forward(P, x)[0] * G).sum())

    for key in ["x", "W1", "b1", "W2", "b2", "W3", "b3"]:
        base = x if key == "x" else P[key]
        an = gx if key == "x" else gr["d" + key]
        flat = base.reshape(-1)
        for t in range(flat.size):
            old = flat[t]
            flat[t] = old + eps
            lp = loss()
            flat[t] = old - eps
            lm = loss()
            flat[t] = old
            assert abs((lp - lm) / (2 * eps) - an.reshape(-1)[t]) <= 1e-6 * max(1.0, abs(an.reshape(-1)[t])), key


def test_masked_mse_closed_form():
    pred = np.array([[1.0, 2.0], [3.0, 5.0], [0.0, 0.0]])
    Y = np.array([[0.0, 2.0], [1.0, 1.0], [9.0, 9.0]])
    loss, grad = hop.masked_mse(pred, Y, [True, True, False])
    assert loss == pytest.approx((1 + 0 + 4 + 16) / 4)
    assert np.allclose(grad, [[0.5, 0.0], [1.0, 2.0], [0.0, 0.0]])
    assert hop.masked_mse(pred, Y, [False] * 3)[0] == 0.0


def _loss_only(Pe, Pk, Pd, v0, Y, mask, rp, col, hops):
    return hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, hops)["loss"]


@pytest.mark.parametrize("hops", [1, 3])
def test_train_step_central_differences(hops):
    Pe, Pk, Pd, v0, Y, mask, rp, col = _case(3)
    res = hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, hops)
    eps = 1e-6
    rng = np.random.default_rng(11)
    for group, P in (("enc", Pe), ("conv", Pk), ("dec", Pd)):
        for key in P:
            flat = P[key].reshape(-1)
            for t in rng.choice(flat.size, size=min(flat.size, 4), replace=False):
                old = flat[t]
                flat[t] = old + eps
                lp = _loss_only(Pe, Pk, Pd, v0, Y, mask, rp, col, hops)
                flat[t] = old - eps
                lm = _loss_only(Pe, Pk, Pd, v0, Y, mask, rp, col, hops)
                flat[t] = old
                fd = (lp - lm) / (2 * eps)
                an = res[group]["d" + key].reshape(-1)[t]
                assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (group, key, t, fd, an)


def test_train_step_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    Pe, Pk, Pd, v0, Y, mask, rp, col = _case(4, n=30)
    hops = 2
    res = hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, hops)
    T = {g: {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in P.items()}
         for g, P in (("enc", Pe), ("conv", Pk), ("dec", Pd))}
    n, d = v0.shape[0], Pe["W3"].shape[0]
    dst = torch.tensor(rg.dst_of_edges(rp), dtype=torch.long)
    src = torch.tensor(col, dtype=torch.long)
    deg = torch.tensor(np.maximum(np.diff(rp), 1), dtype=torch.float64)[:, None]

    def mlp(P, x):
        return torch.relu(torch.relu(x @ P["W1"].T + P["b1"]) @ P["W2"].T + P["b2"]) @ P["W3"].T + P["b3"]

    def conv(P, x, h):
        z = torch.relu(torch.relu(x @ P["W1"].T + P["b1"]) @ P["W2"].T + P["b2"])
        theta = (z @ P["W3"].T + P["b3"]).reshape(-1, d, d)
        m = torch.bmm(theta.transpose(1, 2).contiguous(), h[src].unsqueeze(2)).squeeze(2)
        s = torch.zeros(n, d, dtype=torch.float64).index_add(0, dst, m)
        return h + s / deg + h @ P["Wr"].T + P["br"]

    v = torch.tensor(v0)
    vL = mlp(T["enc"], v)
    for _ in range(hops):
        x = v[dst] - v[src]
        vL = conv(T["conv"], x, vL)
        v = mlp(T["dec"], vL)
    m = torch.tensor(mask)
    loss = ((v[m] - torch.tensor(Y)[m]) ** 2).mean()
    loss.backward()
    assert loss.item() == pytest.approx(res["loss"], rel=1e-12)
    assert np.allclose(v.detach().numpy(), res["v"], atol=1e-12)
    for g in T:
        for k, t in T[g].items():
            assert np.allclose(t.grad.numpy(), res[g]["d" + k], atol=1e-10), (g, k)


def test_ambiguous_decisions_are_counted_and_allowed_for():
    Pe, Pk, Pd, v0, Y, mask, rp, col = _case(5)
    res = hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, 2)
    base = res["ambiguous"]
    for g in ("enc", "conv", "dec"):
        for k, v in res[g].items():
            assert res["allow"][g][k].shape == v.shape and np.all(res["allow"][g][k] >= 0), (g, k)
    # pushing one encoder pre-activation onto its kink adds an ambiguous decision
    a1 = v0[0] @ Pe["W1"][0]
    Pe["b1"][0] = -a1
    res2 = hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, 2)
    assert res2["ambiguous"] >= base + 1
    assert res2["allow"]["enc"]["dW1"][0].max() > 0


def test_model_does_not_change_the_step():
    """The allowances ride along: a bfloat16 step differs from the float32
    one only in the rounding of the layer's input features."""
    Pe, Pk, Pd, v0, Y, mask, rp, col = _case(8)
    a = hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, 2, "f32")
    b = hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, 2, "bf16")
    assert abs(a["loss"] - b["loss"]) <= 1e-2 * abs(a["loss"])
    assert b["allow"]["loss"] > a["allow"]["loss"]


def test_zero_hops_is_decoder_free_encoder_loss():
    # with no hop the loss is on the input values themselves (no decoder ran)
    Pe, Pk, Pd, v0, Y, mask, rp, col = _case(6)
    res = hop.train_step(Pe, Pk, Pd, v0, Y, mask, rp, col, 0)
    assert res["loss"] == pytest.approx(hop.masked_mse(v0, Y, mask)[0])
    assert all(np.all(v == 0) for v in res["conv"].values())


def test_edge_gradient_enters_both_ends():
    # a single edge 0 <- 1: the attribute gradient adds at the destination and
    # subtracts at the source
    Pe, Pk, Pd, v0, Y, mask, _, _ = _case(7, n=2)
    rp, col = np.array([0, 1, 1]), np.array([1])
    base = hop.train_step(Pe, Pk, Pd, v0, Y, [True, True], rp, col, 2)
    x = nn.edge_attr(v0, rp, col, mode="diff")
    assert np.allclose(x, v0[0] - v0[1])
    assert np.isfinite(base["loss"])
