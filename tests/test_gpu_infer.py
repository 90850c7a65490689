"""GPU parity of sub-domain inference with reassembly (Sec. 3, testing
procedure): node selection of a box with overlap (bit-exact), the row scatter
(bit-exact), and the reassembled output of the layer stack against the fp64
oracle (1e-4 float32, 2e-2 bf16 layer operands)."""

import numpy as np
import pytest

import oracle
from oracle import infer as oinf
from tests.helpers import TOL, announce, gpu_lib, rel_err
from workloads import make_config, subdomain_boxes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    return gpu_lib()


SELECT_CASES = {
    "2d": (2, 3000, [0.2, 0.1], [0.6, 0.55], 0.05),
    "3d": (3, 5000, [0.5, -np.inf, 0.25], [np.inf, 0.5, 0.75], 0.1),
    "3d_no_overlap": (3, 777, [0.0, 0.0, 0.0], [0.5, 0.5, 0.5], 0.0),
    "empty_box": (2, 500, [5.0, 5.0], [6.0, 6.0], 0.01),
    "everything": (2, 1000, [-np.inf, -np.inf], [np.inf, np.inf], 0.3),
    "one_node": (3, 1, [0.0, 0.0, 0.0], [1.0, 1.0, 1.0], 0.0),
    "large": (3, 300000, [2.0, 0.3, 0.0], [4.5, 0.8, 1.0], 0.12),
}


@pytest.mark.parametrize("name", sorted(SELECT_CASES))
def test_subdomain_select_bit_exact(env, name):
    dm, lib, torch = env
    D, n, lo, hi, l = SELECT_CASES[name]
    announce("subdomain select", name)
    g = np.random.default_rng(n)
    pos = (g.uniform(0, 1, (n, D)) * ([6.0] + [1.0] * (D - 1))).astype(np.float32)
    pos[: min(n, 10), 0] = np.float32(lo[0]) if np.isfinite(lo[0]) else pos[: min(n, 10), 0]   # on a bound
    own, ovl = oinf.subdomain_nodes(pos, lo, hi, l)
    idx, n_own = lib.dsmp_subdomain_select(torch.from_numpy(pos).cuda(), lo, hi, l)
    torch.cuda.synchronize()
    assert n_own == own.size
    assert np.array_equal(idx.cpu().numpy(), np.concatenate([own, ovl]))


def test_subdomain_select_empty_input(env):
    dm, lib, torch = env
    idx, n_own = lib.dsmp_subdomain_select(torch.zeros(0, 3, device="cuda"), [0, 0, 0], [1, 1, 1], 0.1)
    assert idx.numel() == 0 and n_own == 0


def test_scatter_rows_inverts_gather(env):
    dm, lib, torch = env
    g = np.random.default_rng(0)
    src = torch.from_numpy(g.normal(size=(1000, 24)).astype(np.float32)).cuda()
    perm = torch.from_numpy(g.permutation(5000)[:1000].astype(np.int32)).cuda()
    out = torch.zeros(5000, 24, device="cuda")
    lib.dsmp_scatter_rows(src, perm, out)
    back = lib.dsmp_gather_rows(out, perm)
    torch.cuda.synchronize()
    assert torch.equal(back, src)
    mask = np.ones(5000, bool)
    mask[perm.cpu().numpy()] = False
    assert not out.cpu().numpy()[mask].any()


def _workload_nodes(w):
    pos, attr, h = [], [], []
    for p in w.parts:
        idx = oracle.sampling.sample_nodes(p.pos.shape[0], p.s, p.seed)
        pos.append(p.pos[idx]); attr.append(p.attr[idx]); h.append(p.h[idx])
    return np.concatenate(pos), np.concatenate(attr), np.concatenate(h)


def _gpu_infer(env, w, pos, attr, h, boxes, overlap):
    dm, lib, torch = env
    dev = torch.device("cuda", 0)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    desc = dm.layer_desc(w.D, w.d, w.H1, w.H2, dm.BF16 if w.dtype == "bf16" else dm.F32)
    packed = [lib.dsmp_nnconv_pack(desc, {k: torch.from_numpy(v) for k, v in P.items()}) for P in w.params]
    inf = dm.SubdomainInference(lib, desc, packed, w.r, w.cap, w.cap_mode)
    out = inf.run(torch.from_numpy(pos).to(dev), torch.from_numpy(attr).to(dev),
                  torch.from_numpy(h).to(dev).to(tdt), boxes, overlap)
    torch.cuda.synchronize()
    return out.cpu().numpy(), inf.stats


@pytest.mark.parametrize("k,boxes_checked", [(1, None), (2, None), (4, (0, 3))])
def test_subdomain_inference_parity(env, k, boxes_checked):
    """Random boxes with the paper's overlap l = r; the GPU reassembles every
    box, the oracle runs the boxes checked (all, or a subset at workload 4)."""
    announce("subdomain inference", k, boxes_checked)
    w = make_config(k)
    pos, attr, h = _workload_nodes(w)
    boxes = subdomain_boxes(w)
    got, stats = _gpu_infer(env, w, pos, attr, h, boxes, w.r)
    want, ostats = oinf.infer(w.params, pos, attr, h, boxes, w.r, w.r, w.cap, w.cap_mode, w.dtype,
                              only=boxes_checked)
    rows = np.concatenate([oinf.subdomain_nodes(pos, *boxes[b], w.r)[0]
                           for b in (boxes_checked or range(len(boxes)))])
    for b in (boxes_checked or range(len(boxes))):
        assert stats[b] == ostats[b], (b, stats[b], ostats[b])     # nodes and edges of the box
    assert sum(s[0] for s in stats) == pos.shape[0]
    err = rel_err(got[rows], want[rows])
    print("boxes %d, checked rows %d, err %.3e" % (len(boxes), rows.size, err))
    assert err <= TOL[w.dtype]


def test_receptive_overlap_matches_whole_domain_on_gpu(env):
    """With overlap layers * r the GPU's reassembled output equals its own
    forward over the whole domain up to summation order."""
    dm, lib, torch = env
    announce("subdomain inference vs whole domain")
    w = make_config(2, n_sample=3000)
    pos, attr, h = _workload_nodes(w)
    boxes = subdomain_boxes(w, [2, 1])
    got, _ = _gpu_infer(env, w, pos, attr, h, boxes, w.layers * w.r)
    whole, _ = _gpu_infer(env, w, pos, attr, h, [([-np.inf] * 2, [np.inf] * 2)], 0.0)
    err = rel_err(got, whole)
    print("err %.3e" % err)
    assert err <= TOL[w.dtype]
