"""GPU parity: the NNConv layer (forward and backward) against the fp64 oracle.

The graph comes from the oracle and is uploaded, so these tests do not depend
on the GPU graph builder.  Tolerance: max |gpu - oracle| / max |oracle| per
tensor, 1e-4 for float32 layers and 2e-2 for bf16-operand layers.
"""

import zlib

import numpy as np
import pytest

import oracle
from oracle import nnconv as onn
from oracle import radius_graph as org
from tests.helpers import TOL, announce, gpu_lib, rel_err
from workloads import bf16_round, layer_params, make_config

pytestmark = pytest.mark.gpu

SHAPES = {"f32_32": ("f32", 32, 64, 64), "f32_64": ("f32", 64, 128, 128), "bf16_32": ("bf16", 32, 64, 64),
          "bf16_64": ("bf16", 64, 128, 128), "bf16_128": ("bf16", 128, 256, 256)}


@pytest.fixture(scope="module")
def env():
    return gpu_lib()


# Both evaluations of the edge contraction (per edge, and aggregate-first
# over the per-destination sums) are checked against the same oracle.
ALGOS = ("per_edge", "aggregate")


@pytest.fixture(params=ALGOS)
def algo(request, env):
    dm, lib, _ = env
    lib.dsmp_set_edge_algorithm(dm.EDGE_PER_EDGE if request.param == "per_edge" else dm.EDGE_AGGREGATE)
    yield request.param
    lib.dsmp_set_edge_algorithm(dm.EDGE_AUTO)


# Oracle results per case, shared by the tests of the two forms (the oracle
# does not depend on the form; the GPU runs each form afresh).
_ORACLE = {}


class Case:
    """A layer problem on the host plus its device copies."""

    def __init__(self, env, pos, attr, h, n_dst, r, cap, P, dtype, D, d, h1, h2, act=0, residual=1,
                 attr_mode=0, G=None, rows=None):
        dm, lib, torch = env
        self.dm, self.lib, self.torch = dm, lib, torch
        dev = torch.device("cuda", 0)
        self.rp, self.col = org.radius_graph(pos, n_dst, r, cap)
        rp, col = self.rp, self.col
        E = col.size
        cp, ceid = org.transpose(rp, col, pos.shape[0])
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
        pad = lambda a: np.concatenate([a, np.zeros(1, np.int32)]) if a.size == 0 else a
        self.g = dm.Graph(n_dst, pos.shape[0], E, i32(rp), i32(pad(col)), i32(pad(org.dst_of_edges(rp))),
                          i32(cp), i32(pad(ceid)))
        self.P, self.h, self.attr, self.n_dst = P, h, attr, n_dst
        self.act, self.residual, self.attr_mode = act, residual, attr_mode
        self.dtype = dtype
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.desc = dm.layer_desc(D, d, h1, h2, dm.BF16 if dtype == "bf16" else dm.F32, act, residual, attr_mode)
        self.t_attr = torch.from_numpy(attr).to(dev)
        self.t_h = torch.from_numpy(h).to(dev).to(tdt)
        self.packed = lib.dsmp_nnconv_pack(self.desc, {k: torch.from_numpy(v) for k, v in P.items()})
        self.x = onn.edge_attr(attr, rp, col, "concat" if attr_mode == 0 else "diff")
        self.G = G
        self.rows = rows
        self.key = None           # oracle results of keyed cases are shared by both forms

    def forward(self):
        out, saved = self.lib.dsmp_nnconv_forward(self.desc, self.packed, self.g, self.t_attr, self.t_h)
        self.torch.cuda.synchronize()
        self.saved = saved
        return out.cpu().numpy()

    def oracle_forward(self):
        if self.key is not None and ("fwd", self.key) in _ORACLE:
            return _ORACLE[("fwd", self.key)]
        out, _ = onn.forward(self.P, self.x, self.h.astype(np.float64), self.rp, self.col, self.n_dst,
                             self.act, bool(self.residual), rows=self.rows)
        if self.key is not None:
            _ORACLE[("fwd", self.key)] = out
        return out

    def clear_ambiguous_outputs(self):
        """Zero the upstream gradient where ReLU(y) is a decision inside the
        band of the layer's precision (a kernel may take it either way, and
        either choice is then correct)."""
        if self.act != onn.ACT_RELU:
            return 0
        _, _, st = onn.forward(self.P, self.x, self.h.astype(np.float64), self.rp, self.col, self.n_dst,
                               self.act, bool(self.residual), rows=self.rows, precision=self.dtype,
                               return_stats=True)
        amb = st["amb_y"]
        self.G = np.where(amb, 0.0, self.G).astype(np.float32)
        return int(amb.sum())

    def backward(self):
        dev = self.torch.device("cuda", 0)
        gh, grads = self.lib.dsmp_nnconv_backward(self.desc, self.packed, self.g, self.t_attr, self.t_h,
                                                  self.saved, self.torch.from_numpy(self.G).to(dev))
        self.torch.cuda.synchronize()
        return gh.cpu().numpy(), {k: v.cpu().numpy() for k, v in grads.items()}

    def oracle_backward(self):
        if self.key is not None and ("bwd", self.key) in _ORACLE:
            return _ORACLE[("bwd", self.key)]
        ref = onn.backward(self.P, self.x, self.h.astype(np.float64), self.rp, self.col, self.n_dst, self.G,
                           self.act, bool(self.residual), rows=self.rows, precision=self.dtype)
        if self.key is not None:
            _ORACLE[("bwd", self.key)] = ref
        return ref


def random_case(env, shape, n=900, n_dst=None, D=2, r=None, cap=0, act=0, residual=1, attr_mode=0, seed=0):
    dtype, d, h1, h2 = SHAPES[shape]
    g = np.random.default_rng(seed)
    n_dst = n if n_dst is None else n_dst
    pos = g.uniform(0, 1, (n, D)).astype(np.float32)
    attr = np.concatenate([pos, g.uniform(0, 2, (n, 1)).astype(np.float32)], 1)
    if r is None:
        r = (30.0 / n / (np.pi if D == 2 else 4.19)) ** (1.0 / D)   # ~30 neighbours
    h = g.normal(0, 1, (n, d)).astype(np.float32)
    if dtype == "bf16":
        h = bf16_round(h)
    de = 2 * D + 2 if attr_mode == 0 else D + 1
    P = layer_params(g, d, de, h1, h2, dtype)
    G = g.normal(0, 1, (n_dst, d)).astype(np.float32)
    return Case(env, pos, attr, h, n_dst, r, cap, P, dtype, D, d, h1, h2, act, residual, attr_mode, G)


FWD_CASES = {
    "f32_32_2d": dict(shape="f32_32"),
    "f32_64_3d": dict(shape="f32_64", D=3),
    "bf16_32_2d": dict(shape="bf16_32"),
    "bf16_64_2d": dict(shape="bf16_64"),
    "bf16_64_3d_knn": dict(shape="bf16_64", D=3, cap=12),
    "bf16_128_3d": dict(shape="bf16_128", D=3, cap=24, n=700),
    "bf16_128_3d_high_degree": dict(shape="bf16_128", D=3, n=300, r=0.35),
    "bf16_128_halo_isolated": dict(shape="bf16_128", D=3, n=600, n_dst=450, r=0.07),
    "bf16_64_relu_nores": dict(shape="bf16_64", act=1, residual=0),
    "bf16_64_diff_attr": dict(shape="bf16_64", attr_mode=1),
    "f32_32_halo": dict(shape="f32_32", n=1000, n_dst=700),
    "bf16_64_one_tile_ragged": dict(shape="bf16_64", n=37, r=0.3),
    "bf16_64_isolated": dict(shape="bf16_64", n=400, r=0.02),
    "bf16_64_high_degree": dict(shape="bf16_64", n=600, r=0.5),
}


@pytest.mark.parametrize("name", sorted(FWD_CASES))
def test_forward_parity(env, algo, name):
    kw = FWD_CASES[name]
    announce("forward", name, algo)
    c = random_case(env, seed=zlib.crc32(name.encode()) % 1000, **kw)
    c.key = name
    got = c.forward()
    ref = c.oracle_forward()
    err = rel_err(got, ref)
    print("E=%d err=%.3e" % (c.col.size, err))
    assert err <= TOL[c.dtype], err


def test_forward_no_edges(env, algo):
    announce("forward no edges", algo)
    c = random_case(env, "bf16_64", n=50, r=1e-6)
    assert c.col.size == 0
    assert rel_err(c.forward(), c.oracle_forward()) <= TOL["bf16"]


def test_forward_deterministic(env, algo):
    c = random_case(env, "bf16_64", n=3000, seed=5)
    a = c.forward()
    b = c.forward()
    assert np.array_equal(a, b)


def workload_case(env, k, layer=0, rows=None):
    w = make_config(k)
    pos, attr, h = [], [], []
    for p in w.parts:
        idx = oracle.sampling.sample_nodes(p.pos.shape[0], p.s, p.seed)
        pos.append(p.pos[idx]); attr.append(p.attr[idx]); h.append(p.h[idx])
    pos, attr, h = np.concatenate(pos), np.concatenate(attr), np.concatenate(h)
    G = np.zeros_like(w.grad_out)
    if rows is None:
        G = w.grad_out
    else:
        G[rows] = w.grad_out[rows]
    return Case(env, pos, attr, h, w.n_dst, w.r, w.cap, w.params[layer], w.dtype, w.D, w.d, w.H1, w.H2,
                G=G, rows=rows)


@pytest.mark.parametrize("k", [1, 2])
def test_forward_workload_full(env, algo, k):
    announce("forward workload", k, algo)
    c = workload_case(env, k)
    c.key = "workload%d" % k
    err = rel_err(c.forward(), c.oracle_forward())
    print("E=%d err=%.3e" % (c.col.size, err))
    assert err <= TOL[c.dtype]


@pytest.mark.parametrize("k", [3, 4, 5])
def test_forward_workload_rows(env, algo, k):
    announce("forward workload rows", k, algo)
    rows = np.sort(np.random.default_rng(k).choice(make_config(k).n_dst, 256, replace=False))
    c = workload_case(env, k, rows=rows)
    c.key = "workload%d-rows" % k
    got = c.forward()
    ref = c.oracle_forward()
    err = rel_err(got[rows], ref[rows])
    print("E=%d err=%.3e" % (c.col.size, err))
    assert err <= TOL[c.dtype]


GRAD_KEYS = ("dW1", "db1", "dW2", "db2", "dW3", "db3", "dWr", "dbr")


def _check_backward(c, label):
    namb = c.clear_ambiguous_outputs()
    c.forward()
    gh, grads = c.backward()
    ref = c.oracle_backward()
    errs = {"grad_h": rel_err(gh, ref["grad_h"], ref["allow"]["grad_h"])}
    for k in GRAD_KEYS:
        errs[k] = rel_err(grads[k], ref[k], ref["allow"][k])
    frac = {k: float(ref["allow"][k].max() / max(np.abs(ref[k]).max(), 1e-300)) for k in ("dW1", "dW2", "dW3")}
    print(label, "ambiguous-y=%d" % namb, " ".join("%s=%.2e" % kv for kv in errs.items()),
          "allowance/max:", " ".join("%s=%.3f" % kv for kv in frac.items()))
    for k, e in errs.items():
        assert e <= TOL[c.dtype], (k, e)


# Sizes at which the node kernels take the matrix-core form (at least 512
# steps of 128 / (d / 32) destinations) while the forward's per-destination
# sums still come in several K slices (2 at d = 64, 4 at d = 128); neither
# size is a whole number of 32-destination blocks.  The upstream gradient is
# nonzero on sampled rows only (the last rows among them), so the oracle
# visits only their edges.
NODE_SIZES = {"bf16_128": 16360, "bf16_64": 32760}


def _node_rows_case(env, shape):
    n = NODE_SIZES[shape]
    g = np.random.default_rng(n)
    rows = np.unique(np.concatenate([g.choice(n - 64, 96, replace=False), np.arange(n - 40, n)]))
    c = random_case(env, shape, n=n, D=3, seed=n % 997)
    G = np.zeros_like(c.G)
    G[rows] = c.G[rows]
    c.G, c.rows, c.key = G, rows, "node-%s" % shape
    return c, rows


@pytest.mark.parametrize("shape", sorted(NODE_SIZES))
def test_node_terms_sliced_sums(env, algo, shape):
    announce("node terms, sliced sums", shape, algo)
    c, rows = _node_rows_case(env, shape)
    err = rel_err(c.forward()[rows], c.oracle_forward()[rows])
    print("E=%d forward err=%.3e" % (c.col.size, err))
    assert err <= TOL[c.dtype]
    _check_backward(c, "E=%d" % c.col.size)


@pytest.mark.parametrize("name", sorted(FWD_CASES))
def test_backward_parity(env, algo, name):
    kw = FWD_CASES[name]
    announce("backward", name, algo)
    c = random_case(env, seed=zlib.crc32(name.encode()) % 1000, **kw)
    c.key = name
    _check_backward(c, "E=%d" % c.col.size)


def test_backward_no_edges(env, algo):
    announce("backward no edges", algo)
    c = random_case(env, "bf16_64", n=50, r=1e-6)
    _check_backward(c, "E=0")


def test_backward_accumulate_and_determinism(env, algo):
    announce("backward accumulate", algo)
    dm, lib, torch = env
    c = random_case(env, "bf16_64", n=2000, seed=11)
    c.forward()
    gh1, g1 = c.backward()
    gh2, g2 = c.backward()
    for k in GRAD_KEYS:
        assert np.array_equal(g1[k], g2[k]), k
    assert np.array_equal(gh1, gh2)
    dev = torch.device("cuda", 0)
    grads = {k: torch.from_numpy(v).to(dev) for k, v in g1.items()}
    lib.dsmp_nnconv_backward(c.desc, c.packed, c.g, c.t_attr, c.t_h, c.saved, torch.from_numpy(c.G).to(dev),
                             grads=grads, flags=dm.GRAD_ACCUMULATE)
    torch.cuda.synchronize()
    for k in GRAD_KEYS:
        assert np.array_equal(grads[k].cpu().numpy(), (g1[k] + g1[k]).astype(np.float32)), k


@pytest.mark.parametrize("k", [1, 2])
def test_backward_workload_full(env, algo, k):
    announce("backward workload", k, algo)
    c = workload_case(env, k)
    c.key = "workload%d" % k
    _check_backward(c, "E=%d" % c.col.size)


@pytest.mark.parametrize("k", [3, 4, 5])
def test_backward_workload_rows(env, algo, k):
    """Sparse upstream gradient (rows only): every gradient is an exact sum
    over those rows' edges, while the GPU runs the full-size kernels."""
    announce("backward workload rows", k, algo)
    rows = np.sort(np.random.default_rng(k + 10).choice(make_config(k).n_dst, 128, replace=False))
    c = workload_case(env, k, rows=rows)
    c.key = "workload%d-rows-bwd" % k
    _check_backward(c, "E=%d" % c.col.size)


# ---------------------------------------------------------------- kernel MLP
# What the forward keeps for the backward, read back from the saved buffer:
# the ReLU mask bits of both kernel-MLP layers (every layer shape), z1 and the
# bf16 high/low attribute parts (shapes whose backward reads them back), and
# z.  Layout of the saved buffer: y [n_dst][d] fp32, z [E][h2], z1 [E][h1],
# mask bits [E][(h1+h2)/8], split attributes [E][16] bf16, each section at a
# 256-byte boundary, the per-edge ones with E rounded up to whole 32-edge
# tiles (the mask bits with one tile more).  z1, z and their bits sit at packed positions: position
# p = 16 s + 8 g + t (fragment s, lane half g) holds neuron kperm(p) below.

def _kperm(p):
    n = (p // 16) * 8 + p % 8
    c, i, g = n // 16, n % 16, (p % 16) // 8
    return 32 * c + 8 * (i // 4) + 4 * g + i % 4


def _saved_sections(c):
    E, esz = c.col.size, 2
    E32 = (E + 31) // 32 * 32
    H1, H2 = c.P["W1"].shape[0], c.P["W2"].shape[0]
    off, out = 0, {}
    for name, nb in (("y", c.n_dst * c.h.shape[1] * 4), ("z", E32 * H2 * esz), ("z1", E32 * H1 * esz),
                     ("mask", (E32 + 32) * (H1 + H2) // 8), ("x", E32 * 32)):
        off = (off + 255) & ~255
        out[name] = (off, nb)
        off += nb
    return out


def _bits_natural(words, H):
    """[E][2 * H/64] uint32 (lane half 0 words, then half 1) -> [E][H] bool in neuron order."""
    E = words.shape[0]
    bits = np.unpackbits(words.view(np.uint8).reshape(E, -1), axis=1, bitorder="little").astype(bool)
    out = np.zeros((E, H), bool)
    for g in range(2):
        for b in range(H // 2):
            p = (b // 8) * 16 + 8 * g + b % 8
            out[:, _kperm(p)] = bits[:, g * (H // 2) + b]
    return out


def _positions_natural(vals, H):
    perm = np.array([_kperm(p) for p in range(H)])
    out = np.empty_like(vals)
    out[:, perm] = vals
    return out


def _bf16_bits_to_f64(u16):
    return (u16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("name", ["bf16_128_3d", "bf16_64_2d", "bf16_64_diff_attr", "bf16_32_2d",
                                  "bf16_64_one_tile_ragged"])
def test_kernel_mlp_saved(env, name):
    dm, lib, _ = env
    announce("kernel MLP saved outputs", name)
    lib.dsmp_set_edge_algorithm(dm.EDGE_AGGREGATE)
    try:
        c = random_case(env, seed=zlib.crc32(name.encode()) % 1000, **FWD_CASES[name])
        c.forward()
    finally:
        lib.dsmp_set_edge_algorithm(dm.EDGE_AUTO)
    E, H1, H2 = c.col.size, c.P["W1"].shape[0], c.P["W2"].shape[0]
    sv = c.saved.cpu().numpy().view(np.uint8)
    sec = _saved_sections(c)
    part = lambda k: sv[sec[k][0]:sec[k][0] + sec[k][1]]
    per_edge = {"z": H2 * 2, "z1": H1 * 2, "mask": (H1 + H2) // 8, "x": 32}
    part_e = lambda k: part(k)[:E * per_edge[k]]
    assert sv.size >= sec["x"][0] + sec["x"][1]
    words = part_e("mask").view(np.uint32).reshape(E, -1)
    m1 = _bits_natural(words[:, :H1 // 32], H1)
    m2 = _bits_natural(words[:, H1 // 32:], H2)
    # float64 decisions of the oracle; only those inside the band of the
    # layer's precision may differ
    em = onn.edge_mlp(c.P, c.x, c.dtype)
    amb1, amb2 = em["amb1"], em["amb2"]
    print("E=%d ambiguous a1 %d a2 %d" % (E, int(amb1.sum()), int(amb2.sum())))
    assert np.array_equal(m1[~amb1], em["m1"][~amb1])
    assert np.array_equal(m2[~amb2], em["m2"][~amb2])
    # z in bf16: one rounding of a value within the modelled spread of a2
    z = _positions_natural(_bf16_bits_to_f64(part_e("z").view(np.uint16).reshape(E, H2)), H2)
    ok = ~amb2
    zref = em["z"]
    assert np.all(np.abs(z - zref)[ok] <= 2.0 ** -8 * np.abs(zref)[ok] + onn.BAND_SIGMAS * np.sqrt(em["v2"])[ok])
    # the fused edge-gradient pass (h1 = h2 = 64, 128) recomputes z1 and the
    # split attributes; at h1 = h2 = 256 the dW2 pass recomputes z1 from the
    # stored split attributes
    fused = H1 == H2 and H1 in (64, 128)
    keeps_z1 = not fused and not (H1 == H2 == 256)
    if keeps_z1:
        # z1 within one rounding of the oracle's values
        z1 = _positions_natural(_bf16_bits_to_f64(part_e("z1").view(np.uint16).reshape(E, H1)), H1)
        z1ref = em["z1"]
        assert np.all(np.abs(z1 - z1ref) <= 2.0 ** -8 * np.abs(z1ref) + onn.BAND_SIGMAS * np.sqrt(em["v1"]))
    if not fused:
        # the attributes as bf16 high + low parts
        xs = part_e("x").view(np.uint16).reshape(E, 16)
        hi, lo = _bf16_bits_to_f64(xs[:, :8]), _bf16_bits_to_f64(xs[:, 8:])
        de = c.x.shape[1]
        x32 = c.x.astype(np.float32).astype(np.float64)
        assert np.array_equal(hi[:, :de], onn.bf16(x32))
        assert np.array_equal(lo[:, :de], onn.bf16(x32 - onn.bf16(x32)))
        assert not hi[:, de:].any() and not lo[:, de:].any()


# ------------------------------------------------------------- sign-definite kernel MLP
# Biases that dominate every pre-activation fix each kernel-MLP decision per
# neuron (half of the neurons of each layer always on, half always off), so no
# decision lies near its kink: every gradient, those of W1, b1, W2, b2 and the
# attribute gradient included, is held to the plain bar with no allowance.

def sign_definite_case(env, shape, seed, **kw):
    dm, lib, torch = env
    c = random_case(env, shape, seed=seed, **kw)
    P = {k: v.copy() for k, v in c.P.items()}
    x = c.x.astype(np.float32).astype(np.float64)
    H1, H2 = P["W1"].shape[0], P["W2"].shape[0]
    s1 = np.where(np.arange(H1) % 2 == 0, 1.0, -1.0)
    s2 = np.where(np.arange(H2) % 3 == 0, -1.0, 1.0)
    P["b1"] = (s1 * ((np.abs(x) @ np.abs(P["W1"]).T.astype(np.float64)).max(0) + 0.5)).astype(np.float32)
    z1 = np.maximum(x @ P["W1"].T.astype(np.float64) + P["b1"], 0.0)
    P["b2"] = (s2 * ((z1 @ np.abs(P["W2"]).T.astype(np.float64)).max(0) + 0.5)).astype(np.float32)
    c.P = P
    c.packed = lib.dsmp_nnconv_pack(c.desc, {k: torch.from_numpy(v) for k, v in P.items()})
    return c


@pytest.mark.parametrize("shape", ["f32_32", "bf16_64", "bf16_128"])
def test_backward_sign_definite_mlp(env, algo, shape):
    announce("backward sign-definite kernel MLP", shape, algo)
    kw = dict(n=700, D=3, cap=24) if shape == "bf16_128" else {}
    c = sign_definite_case(env, shape, 31, **kw)
    c.key = "sign-definite-" + shape
    em = onn.edge_mlp(c.P, c.x, c.dtype)
    assert not em["amb1"].any() and not em["amb2"].any()
    assert em["m1"].any() and not em["m1"].all() and em["m2"].any() and not em["m2"].all()
    c.forward()
    gh, grads = c.backward()
    ref = c.oracle_backward()
    errs = {"grad_h": rel_err(gh, ref["grad_h"])}
    for k in GRAD_KEYS:
        errs[k] = rel_err(grads[k], ref[k])
    print("E=%d" % c.col.size, " ".join("%s=%.2e" % kv for kv in errs.items()))
    for k, e in errs.items():
        assert e <= TOL[c.dtype], (k, e)
