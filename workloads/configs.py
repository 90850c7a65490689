"""Synthetic workload generators (inputs only; see the package docstring)."""

from dataclasses import dataclass, field
from typing import List

import numpy as np

CONFIG_IDS = (1, 2, 3, 4, 5)

# Cap modes understood by both sides: keep the nearest (d2, j) or a hashed
# random subset.
CAP_KNN = 0
CAP_RANDOM = 1


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as float32.

    Used to synthesise operands that are exactly representable in bfloat16,
    so both sides start from identical values.
    """
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32)
    # uint32 arithmetic: no finite value carries past bit 31
    out = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)).view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out.reshape(np.shape(x))


@dataclass
class Part:
    """A candidate point set the library samples from (owned nodes, or halo nodes)."""
    pos: np.ndarray        # [M, D] float32 candidate positions
    attr: np.ndarray       # [M, D+1] float32 (position, node scalar) for edge attributes
    h: np.ndarray          # [M, d] float32 latent features (bf16-representable for bf16 cases)
    s: int                 # number of nodes to sample from this part
    seed: int              # sampler seed handed to the library


@dataclass
class Workload:
    k: int
    name: str
    D: int
    d: int
    de: int
    H1: int
    H2: int
    layers: int
    dtype: str             # "f32" or "bf16": the type of the contraction operands
    r: float
    cap: int
    cap_mode: int
    parts: List[Part]
    params: List[dict]
    grad_out: np.ndarray   # [n_dst, d] float32 upstream gradient for the last layer
    act: int = 0
    residual: bool = True
    notes: dict = field(default_factory=dict)

    @property
    def n_dst(self) -> int:
        return self.parts[0].s

    @property
    def n_src(self) -> int:
        return sum(p.s for p in self.parts)


def _uniform(rng, shape, fan_in):
    b = 1.0 / np.sqrt(fan_in)
    return rng.uniform(-b, b, size=shape)


def layer_params(rng, d, de, H1, H2, dtype):
    """One layer's parameters, U(+-1/sqrt(fan_in)), torch Linear layout [out, in].

    For bf16 cases the operands the GPU feeds to bf16 matrix cores (W2, the
    last-layer matrix W3 with its bias column b3, and Wr) are rounded to
    bfloat16 here, so both sides use identical values.
    """
    P = {
        "W1": _uniform(rng, (H1, de), de), "b1": _uniform(rng, (H1,), de),
        "W2": _uniform(rng, (H2, H1), H1), "b2": _uniform(rng, (H2,), H1),
        "W3": _uniform(rng, (d * d, H2), H2), "b3": _uniform(rng, (d * d,), H2),
        "Wr": _uniform(rng, (d, d), d), "br": _uniform(rng, (d,), d),
    }
    P = {k: v.astype(np.float32) for k, v in P.items()}
    if dtype == "bf16":
        for k in ("W2", "W3", "b3", "Wr"):
            P[k] = bf16_round(P[k])
    return P


# ---------------------------------------------------------------- geometry

def _grid2d(n):
    t = np.linspace(0.0, 1.0, n)
    X, Y = np.meshgrid(t, t, indexing="ij")
    return np.stack([X.ravel(), Y.ravel()], axis=1)


def _grf_lognormal(n, ell, rng):
    """exp(g) with g a zero-mean, unit-variance field of squared-exponential
    covariance (length scale ell) on an n x n grid of [0,1]^2, by FFT
    filtering of white noise on a doubled periodic grid."""
    m = 2 * n
    hstep = 1.0 / (n - 1)
    k = np.fft.fftfreq(m, d=hstep)
    KX, KY = np.meshgrid(k, k, indexing="ij")
    spec = np.exp(-2.0 * np.pi ** 2 * ell ** 2 * (KX ** 2 + KY ** 2))
    noise = rng.standard_normal((m, m))
    g = np.fft.ifft2(np.fft.fft2(noise) * np.sqrt(spec)).real[:n, :n]
    g = (g - g.mean()) / g.std()
    return np.exp(g).ravel()


def _naca0012_half_thickness(x, t=0.12):
    x = np.clip(x, 0.0, 1.0)
    return 5.0 * t * (0.2969 * np.sqrt(x) - 0.1260 * x - 0.3516 * x ** 2
                      + 0.2843 * x ** 3 - 0.1015 * x ** 4)


def _airfoil_candidates(M, rng):
    from scipy.spatial import cKDTree
    th = np.linspace(0.0, np.pi, 3000)
    xc = 0.5 * (1.0 - np.cos(th))
    yt = _naca0012_half_thickness(xc)
    outline = np.concatenate([np.stack([xc, yt], 1), np.stack([xc[::-1], -yt[::-1]], 1)])
    tree = cKDTree(outline)
    out, wds = [], []
    got = 0
    while got < M:
        P = np.stack([rng.uniform(-2.0, 3.0, 1 << 20), rng.uniform(-1.5, 1.5, 1 << 20)], 1)
        inside = (P[:, 0] >= 0) & (P[:, 0] <= 1) & (np.abs(P[:, 1]) < _naca0012_half_thickness(P[:, 0]))
        P = P[~inside]
        u = rng.uniform(0.0, 1.0, P.shape[0])
        # distance to the airfoil's bounding box bounds the wall distance from
        # below, so most far points are rejected without a tree query
        bx = np.maximum(np.maximum(-P[:, 0], P[:, 0] - 1.0), 0.0)
        by = np.maximum(np.abs(P[:, 1]) - 0.061, 0.0)
        maybe = u < 0.01 / (0.01 + np.sqrt(bx * bx + by * by))
        P, u = P[maybe], u[maybe]
        wd, _ = tree.query(P)
        acc = u < 0.01 / (0.01 + wd)
        out.append(P[acc])
        wds.append(wd[acc])
        got += int(acc.sum())
    P = np.concatenate(out)[:M]
    wd = np.concatenate(wds)[:M]
    return P, wd


def _rect_dist(P, axis_fixed, value, lo, hi):
    """Distance from points P [n,3] to an axis-aligned rectangle lying in the
    plane {x[axis_fixed] = value}, spanning [lo, hi] in the other two axes."""
    d2 = (P[:, axis_fixed] - value) ** 2
    others = [a for a in range(3) if a != axis_fixed]
    for a, l, h in zip(others, lo, hi):
        c = np.clip(P[:, a], l, h)
        d2 = d2 + (P[:, a] - c) ** 2
    return np.sqrt(d2)


def _step_wall_distance(P):
    """Distance to the walls of the backward-facing step channel: y=0, y=1,
    z=1, the floor z=0 (x>=1), the step top z=0.5 (x<=1) and the step face
    x=1 (z<=0.5).  Inlet x=0 and outlet x=10 are not walls."""
    walls = [
        (1, 0.0, (0.0, 0.0), (10.0, 1.0)),
        (1, 1.0, (0.0, 0.0), (10.0, 1.0)),
        (2, 1.0, (0.0, 0.0), (10.0, 1.0)),
        (2, 0.0, (1.0, 0.0), (10.0, 1.0)),
        (2, 0.5, (0.0, 0.0), (1.0, 1.0)),
        (0, 1.0, (0.0, 0.0), (1.0, 0.5)),
    ]
    return np.min(np.stack([_rect_dist(P, *w) for w in walls], 0), axis=0)


def _step_lattice(h, x_lo_idx, x_hi_idx, rng):
    """Lattice points of spacing h with x index in [x_lo_idx, x_hi_idx], fluid
    region only, refined 4x near walls (all points with wall distance < 0.1,
    a seeded quarter of the others)."""
    ny = int(round(1.0 / h)) + 1
    ix = np.arange(x_lo_idx, x_hi_idx + 1)
    iy = np.arange(ny)
    IX, IY, IZ = np.meshgrid(ix, iy, iy, indexing="ij")
    IX, IY, IZ = IX.ravel(), IY.ravel(), IZ.ravel()
    solid = (IX * h < 1.0 - 1e-9) & (IZ * h < 0.5 - 1e-9)
    IX, IY, IZ = IX[~solid], IY[~solid], IZ[~solid]
    P = np.stack([IX * h, IY * h, IZ * h], 1)
    wd = _step_wall_distance(P)
    keep = (wd < 0.1) | (rng.uniform(0.0, 1.0, P.shape[0]) < 0.25)
    return P[keep], wd[keep], IX[keep]


# ---------------------------------------------------------------- configs

_SPECS = {
    1: dict(name="darcy64-f32", D=2, d=32, H1=64, H2=64, layers=2, dtype="f32", r=0.08, cap=0),
    2: dict(name="darcy256-bf16", D=2, d=64, H1=128, H2=128, layers=4, dtype="bf16", r=0.04, cap=0),
    3: dict(name="airfoil2d-bf16", D=2, d=64, H1=128, H2=128, layers=6, dtype="bf16", r=0.05, cap=32),
    4: dict(name="step3d-bf16", D=3, d=64, H1=128, H2=128, layers=4, dtype="bf16", r=0.06, cap=24),
    5: dict(name="step3d-slab-bf16", D=3, d=128, H1=256, H2=256, layers=4, dtype="bf16", r=0.06, cap=24),
}

_FULL_S = {1: 1024, 2: 8192, 3: 32768, 4: 100000, 5: 262144}

_cache = {}


def _geometry(k):
    """Candidate positions, node scalar and node features per part (cached)."""
    if k in _cache:
        return _cache[k]
    rng = np.random.Generator(np.random.PCG64(1000 + k))
    if k in (1, 2):
        n = 64 if k == 1 else 256
        P = _grid2d(n)
        a = _grf_lognormal(n, 0.1, rng)
        feat = np.concatenate([P, a[:, None]], 1)
        parts = [(P, a, feat)]
    elif k == 3:
        P, wd = _airfoil_candidates(3 * _FULL_S[3], rng)
        alpha = np.deg2rad(rng.uniform(-5.0, 15.0))
        uv = np.tile([np.cos(alpha), np.sin(alpha)], (P.shape[0], 1))
        feat = np.concatenate([P, wd[:, None], uv], 1)
        parts = [(P, wd, feat)]
    elif k == 4:
        P, wd, _ = _step_lattice(0.02, 0, 500, rng)
        feat = np.concatenate([P, wd[:, None]], 1)
        parts = [(P, wd, feat)]
    elif k == 5:
        h = 0.0125
        r = _SPECS[5]["r"]
        lo = int(np.ceil((2.5 - 2 * r) / h - 1e-9))
        hi = int(np.floor((5.0 + 2 * r) / h + 1e-9))
        P, wd, IX = _step_lattice(h, lo, hi, rng)
        own = (IX >= 200) & (IX <= 400)          # 2.5 <= x <= 5.0
        feat = np.concatenate([P, wd[:, None]], 1)
        parts = [(P[own], wd[own], feat[own]), (P[~own], wd[~own], feat[~own])]
    else:
        raise ValueError(k)
    _cache[k] = parts
    return parts


def make_config(k: int, n_sample: int = None, layers: int = None) -> Workload:
    """Workload k (1..5).  ``n_sample`` shrinks the sampled node count (the
    radius grows to keep the mean degree); ``layers`` overrides the depth."""
    spec = dict(_SPECS[k])
    D, d = spec["D"], spec["d"]
    de = 2 * D + 2
    geo = _geometry(k)
    s_full = _FULL_S[k]
    s_own = s_full if n_sample is None else int(n_sample)
    r = spec["r"]
    if n_sample is not None:
        r = float(r * (s_full / s_own) ** (1.0 / D))
    prng = np.random.Generator(np.random.PCG64(2000 + k))
    F = geo[0][2].shape[1]
    Wl = _uniform(prng, (d, F), F)
    bl = _uniform(prng, (d,), F)
    parts = []
    for pi, (P, s_attr, feat) in enumerate(geo):
        if pi == 0:
            s = s_own
        else:
            s = int(round(s_own * P.shape[0] / geo[0][0].shape[0]))
        hcand = (feat @ Wl.T + bl).astype(np.float32)
        if spec["dtype"] == "bf16":
            hcand = bf16_round(hcand)
        pos32 = P.astype(np.float32)
        attr = np.concatenate([pos32, s_attr.astype(np.float32)[:, None]], 1)
        parts.append(Part(pos=pos32, attr=np.ascontiguousarray(attr), h=hcand, s=s,
                          seed=4000 + k + 7919 * pi))
    L = spec["layers"] if layers is None else layers
    params = [layer_params(prng, d, de, spec["H1"], spec["H2"], spec["dtype"]) for _ in range(L)]
    grng = np.random.Generator(np.random.PCG64(3000 + k))
    G = grng.standard_normal((parts[0].s, d)).astype(np.float32)
    return Workload(k=k, name=spec["name"], D=D, d=d, de=de, H1=spec["H1"], H2=spec["H2"],
                    layers=L, dtype=spec["dtype"], r=r, cap=spec["cap"], cap_mode=CAP_KNN,
                    parts=parts, params=params, grad_out=G)


def hop_setup(w: Workload, hid: int = 64):
    """Parameters and targets of the hop-loop training step on workload w
    (seed 5000 + k): the encoder (dim+1 -> hid -> hid -> d) and decoder
    (d -> hid -> hid -> dim+1) perceptrons, U(+-1/sqrt(fan_in)); one layer with
    difference edge attributes (de = dim+1) serving every hop; targets
    Y ~ N(0, 1) for every node value.  Returns (enc, conv, dec, Y)."""
    rng = np.random.Generator(np.random.PCG64(5000 + w.k))
    c = w.D + 1

    def mlp(din, dout):
        return {"W1": _uniform(rng, (hid, din), din).astype(np.float32),
                "b1": _uniform(rng, (hid,), din).astype(np.float32),
                "W2": _uniform(rng, (hid, hid), hid).astype(np.float32),
                "b2": _uniform(rng, (hid,), hid).astype(np.float32),
                "W3": _uniform(rng, (dout, hid), hid).astype(np.float32),
                "b3": _uniform(rng, (dout,), hid).astype(np.float32)}

    enc = mlp(c, w.d)
    dec = mlp(w.d, c)
    conv = layer_params(rng, w.d, c, w.H1, w.H2, w.dtype)
    Y = rng.standard_normal((w.n_src, c)).astype(np.float32)
    return enc, conv, dec, Y


def subdomain_boxes(w: Workload, cuts_per_axis=None, seed_offset: int = 0):
    """Random sub-domains for the inference of workload w (seed 6000 + k):
    boxes [lo, hi) that tile space, cut at uniformly drawn positions inside
    the extent of the candidate points along each axis (the outermost sides
    are infinite, so every node has exactly one owning box).  cuts_per_axis
    [D] gives the number of cuts per axis (default: the 2-D squares 1 x 1, the
    3-D channels 7 cuts along x)."""
    rng = np.random.Generator(np.random.PCG64(6000 + w.k + seed_offset))
    if cuts_per_axis is None:
        cuts_per_axis = [1, 1] if w.D == 2 else [7, 0, 0]
    allpos = np.concatenate([p.pos for p in w.parts])
    lo_ext, hi_ext = allpos.min(0).astype(np.float64), allpos.max(0).astype(np.float64)
    edges = []
    for a in range(w.D):
        c = np.sort(rng.uniform(lo_ext[a], hi_ext[a], cuts_per_axis[a])).astype(np.float32)
        edges.append(np.concatenate([[-np.inf], c, [np.inf]]).astype(np.float32))
    boxes = []
    for cell in np.ndindex(*[len(e) - 1 for e in edges]):
        lo = [float(edges[a][cell[a]]) for a in range(w.D)]
        hi = [float(edges[a][cell[a] + 1]) for a in range(w.D)]
        boxes.append((lo, hi))
    return boxes
