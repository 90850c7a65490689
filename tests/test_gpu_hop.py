"""GPU parity of the hop loop (Algorithm 1 on one sub-domain) against the
fp64 oracle: encoder/decoder perceptrons, masked MSE, the layer's attribute
gradient, and whole training steps.  Tolerance as for the layer: max
|gpu - oracle| / max |oracle| per tensor, 1e-4 (float32) or 2e-2 (bf16
layer operands)."""

import numpy as np
import pytest

from oracle import hop as ohop
from oracle import nnconv as onn
from oracle import radius_graph as org
from tests.helpers import TOL, announce, gpu_lib, rel_err
from workloads import layer_params

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    return gpu_lib()


def _mlp_params(g, d_in, d_hid, d_out):
    return {"W1": (g.normal(size=(d_hid, d_in)) / np.sqrt(d_in)).astype(np.float32),
            "b1": (0.1 * g.normal(size=d_hid)).astype(np.float32),
            "W2": (g.normal(size=(d_hid, d_hid)) / np.sqrt(d_hid)).astype(np.float32),
            "b2": (0.1 * g.normal(size=d_hid)).astype(np.float32),
            "W3": (g.normal(size=(d_out, d_hid)) / np.sqrt(d_hid)).astype(np.float32),
            "b3": (0.1 * g.normal(size=d_out)).astype(np.float32)}


def _dev(torch, a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    return t if dtype is None else t.to(dtype)


@pytest.mark.parametrize("n,d_in,d_hid,d_out", [(1000, 3, 64, 32), (257, 32, 64, 3), (5, 4, 8, 4), (0, 3, 16, 8)])
def test_mlp_forward_backward(env, n, d_in, d_hid, d_out):
    dm, lib, torch = env
    announce("mlp", n, d_in, d_hid, d_out)
    g = np.random.default_rng(n + d_in)
    P = _mlp_params(g, d_in, d_hid, d_out)
    x = g.normal(size=(n, d_in)).astype(np.float32)
    G = g.normal(size=(n, d_out)).astype(np.float32)
    desc = dm.MlpDesc(d_in, d_hid, d_out)
    tP = {k: _dev(torch, v) for k, v in P.items()}
    y, saved = lib.dsmp_mlp_forward(desc, tP, _dev(torch, x), y_bf16=torch.empty(n, d_out, dtype=torch.bfloat16,
                                                                                device="cuda"))
    gx = torch.empty(n, d_in, device="cuda")
    grads = lib.dsmp_mlp_backward(desc, tP, _dev(torch, x), saved, _dev(torch, G), grad_x=gx)
    torch.cuda.synchronize()
    ry, cache = ohop.mlp3_forward(P, x)
    rgx, rg = ohop.mlp3_backward(P, cache, G)
    assert rel_err(y.cpu().numpy(), ry) <= TOL["f32"]
    if n:
        assert rel_err(gx.cpu().numpy(), rgx) <= TOL["f32"]
    for k in rg:
        assert rel_err(grads[k].cpu().numpy(), rg[k]) <= TOL["f32"], k
    # accumulation: a second backward adds the same gradients (and input gradient)
    lib.dsmp_mlp_backward(desc, tP, _dev(torch, x), saved, _dev(torch, G), grad_x=gx, grads=grads,
                          flags=dm.GRAD_ACCUMULATE | dm.GRAD_X_ACCUMULATE)
    torch.cuda.synchronize()
    for k in rg:
        assert rel_err(grads[k].cpu().numpy(), 2 * rg[k]) <= TOL["f32"], k
    if n:
        assert rel_err(gx.cpu().numpy(), 2 * rgx) <= TOL["f32"]


@pytest.mark.parametrize("n,c,frac", [(3000, 3, 0.7), (300, 4, 1.0), (17, 2, 0.0), (0, 3, 1.0)])
def test_masked_mse(env, n, c, frac):
    dm, lib, torch = env
    announce("mse", n, c, frac)
    g = np.random.default_rng(n)
    pred = g.normal(size=(n, c)).astype(np.float32)
    Y = g.normal(size=(n, c)).astype(np.float32)
    mask = (g.uniform(size=n) < frac).astype(np.uint8)
    grad = torch.empty(n, c, device="cuda")
    loss, _ = lib.dsmp_masked_mse(_dev(torch, pred), _dev(torch, Y), _dev(torch, mask), grad=grad)
    torch.cuda.synchronize()
    rl, rgr = ohop.masked_mse(pred, Y, mask.astype(bool))
    assert abs(loss.item() - rl) <= TOL["f32"] * max(abs(rl), 1e-30) or (rl == 0.0 and loss.item() == 0.0)
    if n:
        assert rel_err(grad.cpu().numpy(), rgr) <= TOL["f32"]


ATTR_SHAPES = {"f32_32": ("f32", 32, 64, 64), "f32_64": ("f32", 64, 128, 128), "bf16_64": ("bf16", 64, 128, 128),
               "bf16_128": ("bf16", 128, 256, 256)}


@pytest.mark.parametrize("shape", sorted(ATTR_SHAPES))
@pytest.mark.parametrize("algo", ["per_edge", "aggregate"])
def test_layer_attribute_gradient(env, shape, algo):
    """dattr of a difference-attribute layer: W1^T da1 summed into the
    destination and subtracted from the source of every edge."""
    dm, lib, torch = env
    announce("dattr", shape, algo)
    dtype, d, h1, h2 = ATTR_SHAPES[shape]
    lib.dsmp_set_edge_algorithm(dm.EDGE_PER_EDGE if algo == "per_edge" else dm.EDGE_AGGREGATE)
    try:
        g = np.random.default_rng(h1 + d)
        n, D = (700 if d < 128 else 400), 2
        pos = g.uniform(0, 1, (n, D)).astype(np.float32)
        attr = np.concatenate([pos, g.uniform(0, 2, (n, 1)).astype(np.float32)], 1)
        rp, col = org.radius_graph(pos, n, 0.12, 24)
        cp, ceid = org.transpose(rp, col, n)
        i32 = lambda a: _dev(torch, a.astype(np.int32))
        G = dm.Graph(n, n, col.size, i32(rp), i32(col), i32(org.dst_of_edges(rp)), i32(cp), i32(ceid))
        P = layer_params(g, d, D + 1, h1, h2, dtype)
        h = g.normal(size=(n, d)).astype(np.float32)
        if dtype == "bf16":
            h = onn.bf16(h).astype(np.float32)
        Gout = g.normal(size=(n, d)).astype(np.float32)
        desc = dm.layer_desc(D, d, h1, h2, dm.BF16 if dtype == "bf16" else dm.F32, 0, 1, dm.ATTR_DIFF)
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        packed = lib.dsmp_nnconv_pack(desc, {k: torch.from_numpy(v) for k, v in P.items()})
        t_attr, t_h = _dev(torch, attr), _dev(torch, h, tdt)
        _, saved = lib.dsmp_nnconv_forward(desc, packed, G, t_attr, t_h)
        f32 = dict(dtype=torch.float32, device="cuda")
        grads = {"dW1": torch.empty(h1, D + 1, **f32), "db1": torch.empty(h1, **f32),
                 "dW2": torch.empty(h2, h1, **f32), "db2": torch.empty(h2, **f32),
                 "dW3": torch.empty(d * d, h2, **f32), "db3": torch.empty(d * d, **f32),
                 "dWr": torch.empty(d, d, **f32), "dbr": torch.empty(d, **f32),
                 "dattr": torch.empty(n, D + 1, **f32)}
        lib.dsmp_nnconv_backward(desc, packed, G, t_attr, t_h, saved, _dev(torch, Gout), grads=grads)
        torch.cuda.synchronize()
        x = onn.edge_attr(attr, rp, col, "diff")
        ref = onn.backward(P, x, h.astype(np.float64), rp, col, n, Gout, precision=dtype)
        dst = org.dst_of_edges(rp)
        want = np.zeros((n, D + 1))
        allow = np.zeros((n, D + 1))
        np.add.at(want, dst, ref["grad_x"])
        np.add.at(want, col, -ref["grad_x"])
        np.add.at(allow, dst, ref["allow"]["grad_x"])
        np.add.at(allow, col, ref["allow"]["grad_x"])
        err = rel_err(grads["dattr"].cpu().numpy(), want, allow)
        print("E=%d err=%.3e" % (col.size, err))
        assert err <= TOL[dtype], err
        # accumulation adds a second copy; the parameter flag alone leaves dattr overwritten
        lib.dsmp_nnconv_backward(desc, packed, G, t_attr, t_h, saved, _dev(torch, Gout), grads=grads,
                                 flags=dm.GRAD_ACCUMULATE)
        torch.cuda.synchronize()
        assert rel_err(grads["dattr"].cpu().numpy(), want, allow) <= TOL[dtype]
        lib.dsmp_nnconv_backward(desc, packed, G, t_attr, t_h, saved, _dev(torch, Gout), grads=grads,
                                 flags=dm.GRAD_ACCUMULATE | dm.GRAD_X_ACCUMULATE)
        torch.cuda.synchronize()
        assert rel_err(grads["dattr"].cpu().numpy(), 2 * want, 2 * allow) <= TOL[dtype]
    finally:
        lib.dsmp_set_edge_algorithm(dm.EDGE_AUTO)


def test_attribute_gradient_needs_difference_attributes(env):
    dm, lib, torch = env
    g = np.random.default_rng(0)
    n, D, d = 50, 2, 32
    pos = g.uniform(0, 1, (n, D)).astype(np.float32)
    attr = np.concatenate([pos, np.ones((n, 1), np.float32)], 1)
    rp, col = org.radius_graph(pos, n, 0.3, 8)
    cp, ceid = org.transpose(rp, col, n)
    i32 = lambda a: _dev(torch, a.astype(np.int32))
    G = dm.Graph(n, n, col.size, i32(rp), i32(col), i32(org.dst_of_edges(rp)), i32(cp), i32(ceid))
    desc = dm.layer_desc(D, d, 64, 64, dm.F32)
    P = layer_params(g, d, 2 * D + 2, 64, 64, "f32")
    packed = lib.dsmp_nnconv_pack(desc, {k: torch.from_numpy(v) for k, v in P.items()})
    t_attr, t_h = _dev(torch, attr), _dev(torch, g.normal(size=(n, d)).astype(np.float32))
    _, saved = lib.dsmp_nnconv_forward(desc, packed, G, t_attr, t_h)
    f32 = dict(dtype=torch.float32, device="cuda")
    grads = {k: torch.empty(1024, **f32) for k in ("dW1", "db1", "dW2", "db2", "dW3", "db3", "dWr", "dbr")}
    grads["dW3"] = torch.empty(d * d * 64, **f32)
    grads["dattr"] = torch.empty(n, D + 1, **f32)
    with pytest.raises(dm.DsmpError) as e:
        lib.dsmp_nnconv_backward(desc, packed, G, t_attr, t_h, saved, torch.zeros(n, d, **f32), grads=grads)
    assert e.value.status == dm.UNSUPPORTED


def _hop_case(seed, n, D, d, h1, h2, hid, dtype, r, cap):
    g = np.random.default_rng(seed)
    c = D + 1
    pos = g.uniform(0, 1, (n, D)).astype(np.float32)
    v0 = np.concatenate([pos, g.uniform(0, 1, (n, 1)).astype(np.float32)], 1)
    rp, col = org.radius_graph(pos, n, r, cap)
    Pk = layer_params(g, d, c, h1, h2, dtype)
    Pe = _mlp_params(g, c, hid, d)
    Pd = _mlp_params(g, d, hid, c)
    Y = g.normal(size=(n, c)).astype(np.float32)
    mask = (g.uniform(size=n) < 0.8).astype(np.uint8)
    return Pe, Pk, Pd, v0, Y, mask, rp, col


# (seed, n, D, d, h1, h2, hidden, dtype, r, cap, hops).
#
# Every step is compared in full: loss, outputs and every gradient, at the
# layer's bar (1e-4 float32, 2e-2 bf16) beyond the allowances of the oracle's
# precision model.  The model carries the spread of every value through the
# hops (from the second hop on, the edge attributes are differences of
# decoder outputs that a kernel rounds its own way), gives every ReLU
# decision of the perceptrons and the layer a band and a flip probability,
# and propagates the effect of flips back through the loop.  The number of
# decisions inside their bands and the size of the allowances are printed.
HOP_CASES = {
    "f32_32_1hop": (16, 120, 2, 32, 64, 64, 32, "f32", 0.2, 10, 1),
    "f32_32_2hops": (39, 96, 2, 32, 64, 64, 32, "f32", 0.2, 8, 2),
    "f32_32_3hops": (3, 80, 2, 32, 64, 64, 32, "f32", 0.25, 8, 3),
    "f32_64_3d_2hops": (9, 40, 3, 64, 128, 128, 16, "f32", 0.5, 6, 2),
    "bf16_32_1hop": (1, 200, 2, 32, 64, 64, 32, "bf16", 0.15, 16, 1),
    "bf16_64_3hops": (10, 300, 2, 64, 128, 128, 32, "bf16", 0.12, 24, 3),
    "bf16_64_3d_2hops": (2, 250, 3, 64, 128, 128, 32, "bf16", 0.25, 16, 2),
    "bf16_128_3d_2hops": (2, 160, 3, 128, 256, 256, 32, "bf16", 0.35, 16, 2),
}


@pytest.mark.parametrize("name", sorted(HOP_CASES))
def test_hop_train_step(env, name):
    dm, lib, torch = env
    seed, n, D, d, h1, h2, hid, dtype, r, cap, hops = HOP_CASES[name]
    announce("hop", name)
    Pe, Pk, Pd, v0, Y, mask, rp, col = _hop_case(seed, n, D, d, h1, h2, hid, dtype, r, cap)
    ref = ohop.train_step(Pe, Pk, Pd, v0, Y, mask.astype(bool), rp, col, hops, dtype)
    cp, ceid = org.transpose(rp, col, n)
    i32 = lambda a: _dev(torch, a.astype(np.int32))
    G = dm.Graph(n, n, col.size, i32(rp), i32(col), i32(org.dst_of_edges(rp)), i32(cp), i32(ceid))
    shapes = dm.HopShapes(n, D, d, h1, h2, hid, hid, dm.BF16 if dtype == "bf16" else dm.F32, hops)
    st = dm.HopStep(lib, G, shapes)
    desc = st.conv
    packed = lib.dsmp_nnconv_pack(desc, {k: torch.from_numpy(v) for k, v in Pk.items()})
    tPe = {k: _dev(torch, v) for k, v in Pe.items()}
    tPd = {k: _dev(torch, v) for k, v in Pd.items()}
    loss, grads = st.step(tPe, packed, tPd, _dev(torch, v0), _dev(torch, Y), _dev(torch, mask))
    torch.cuda.synchronize()
    tol = TOL[dtype]
    A = ref["allow"]
    print("E=%d loss gpu %.6e oracle %.6e (allowance %.2e), decisions inside their bands: %d"
          % (col.size, loss.item(), ref["loss"], A["loss"], ref["ambiguous"]))
    assert abs(loss.item() - ref["loss"]) <= A["loss"] + tol * abs(ref["loss"])
    assert rel_err(st.v[hops - 1].cpu().numpy(), ref["v"], A["v"]) <= tol
    assert rel_err(st.out[hops - 1].cpu().numpy(), ref["vL"], A["vL"]) <= tol
    for group in ("enc", "conv", "dec"):
        for k, want in ref[group].items():
            allow = A[group][k]
            err = rel_err(grads[group][k].cpu().numpy().reshape(want.shape), want, allow)
            print("  %s %s err %.3e (allowance/max %.3f)" % (group, k, err,
                                                            allow.max() / max(np.abs(want).max(), 1e-300)))
            assert err <= tol, (group, k, err)
