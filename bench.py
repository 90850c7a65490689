"""Benchmark of the DS-MPNN hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input,
all inputs resident in HBM before timing starts:
  sample the nodes (every part of the workload), gather their positions,
  attributes and latent features, build the radius graph (count, cap, CSR,
  transpose), then for every layer pack its parameters and run the NNConv
  forward, then the backward through every layer in reverse (the feature
  gradient of layer l is the upstream gradient of layer l-1).

Default workload: one GPU's share of the 3-D step domain decomposition -- a
262,144-node slab plus a halo of ghost nodes (23,420 sampled), r = 0.06,
kNN cap 24, d = 128, kernel MLP 8->256->256->16384, 4 layers, bf16 operands
with fp32 accumulation (the largest workload that fits one GPU).  Prints one
JSON line.

value = edges/s = E * layers / (seconds per step), i.e. edge-layer passes
(forward + backward) per second, sampling and graph build included.

Per kernel class the line carries the algorithmic work of one launch (flops,
and the compulsory HBM bytes: inputs read once, outputs written once), the
rates these give over the HIP-event launch time (mean, median and minimum over
the steps of a second, profiled pass), and the bound (MFMA or HBM by
arithmetic intensity).  `roofline` is that of the class taking the most time
per step.  `executed_tflops_step` is the flops the kernels of the step
actually perform (the modelled classes) over the step time, and
`executed_frac_peak` its fraction of the dense MFMA peak.  The nominal work of
eq. (1) per edge (one kernel evaluation per retained edge, as a per-edge
implementation performs it) is given as a count, `nominal_flops_per_edge_layer`,
not as a rate: the aggregate form reaches the same result with far fewer
operations.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA (2.5 PFLOP/s published)
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 (matrix and vector)
METRIC = "edges/sec and achieved TFLOP/s per NNConv layer fwd+bwd on 1 MI355X"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5, help="workload 1..5 (default 5)")
    ap.add_argument("--algo", choices=["auto", "per_edge", "aggregate"], default="auto",
                    help="edge-contraction form (default: the library's automatic choice)")
    ap.add_argument("--model", choices=["layer", "hop", "infer"], default="layer",
                    help="layer: the NNConv layer stack (default); hop: the hop-loop training step "
                         "(encoder, layer + decoder per hop, masked MSE, backward); infer: sub-domain "
                         "inference (random boxes with overlap r, the layer stack forward on each, "
                         "owned outputs reassembled)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=None,
                    help="destination rows of the oracle's timed sample (default: about 10-30 s of host work)")
    return ap.parse_args()


CPU_ROWS = {1: 1024, 2: 4096, 3: 2048, 4: 2048, 5: 4096}
SRC_CORE = ["core.hip", "common.hpp"]
SRC_GRAPH = ["graph.hip", "common.hpp"]
SRC_FWD = ["nnconv_fwd.hip", "nnconv.hpp", "common.hpp"]
SRC_BWD = ["nnconv_bwd.hip", "nnconv.hpp", "common.hpp"]
SRC_AGG = ["nnconv_agg.hip", "nnconv.hpp", "common.hpp"]
KERNEL_SOURCES = {
    "sample": SRC_CORE, "gather": SRC_CORE, "graph": SRC_GRAPH,
    "edge_fwd": SRC_FWD, "edge_dh": SRC_FWD, "edge_mlp": SRC_FWD,
    "dz": SRC_BWD, "u_gemm": SRC_BWD, "dW2": SRC_BWD, "dW1": SRC_BWD, "dh_u": SRC_BWD, "dh_final": SRC_BWD,
    "da1": SRC_BWD, "node_bwd": SRC_BWD, "node_fwd": SRC_FWD,
    "dW3": SRC_BWD + ["nnconv_agg.hip"],
    "outer_fwd": SRC_AGG, "gemm_fwd": SRC_AGG, "outer_dh": SRC_AGG, "gemm_dh": SRC_AGG,
}
HBM_TBPS = 8.0                 # MI355X HBM3E peak (8 TB/s published)
RIDGE = PEAK_BF16_TFLOPS / HBM_TBPS   # flop/byte where the two rooflines meet (bf16)


def source_digest(cls):
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[cls]:
        with open(os.path.join(ROOT, "paper_2402_15106_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_table(workload):
    return os.path.join(ROOT, "profiles", workload.replace("-", "_") + "_traffic.md")


def measured_traffic(cls, workload):
    """HBM bytes per launch of kernel class ``cls`` from the committed
    rocprofv3 FETCH_SIZE/WRITE_SIZE table of this workload, or None when
    there is none or the kernel's sources changed since it was taken."""
    table = traffic_table(workload)
    if cls not in KERNEL_SOURCES or not os.path.exists(table):
        return None
    digest = source_digest(cls)
    for line in open(table):
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) == 6 and cells[0] == cls:
            return int(float(cells[5])) if cells[2] == digest else None
    return None


def method_flops_per_edge(w):
    """Nominal work of eq. (1) per retained edge, forward + backward, as the
    per-edge evaluation does it (the aggregate form reaches the same result
    with far fewer operations; this is the yardstick, not its count)."""
    d, H1, H2, de = w.d, w.H1, w.H2, w.de
    return (8 * H2 + 6) * d * d + 6 * H1 * H2 + 4 * de * H1


def gemm_slices(n_rows):
    """K slices of the library's W3 GEMM over segment sums (agg_gemm_slices)."""
    waves = max(1, -(-n_rows // 32))
    return max(1, min(16, 2048 // waves))


def work_model(w, E, n_src, fused=False, n_dst=None):
    """Algorithmic work of one launch of each kernel class: flops and the
    compulsory HBM bytes (every input read once, every output written once).
    With ``fused`` (the one-pass edge gradients) the kernel-MLP pass stores z
    and the mask bits only: the backward recomputes z1."""
    d, H1, H2, de, D = w.d, w.H1, w.H2, w.de, w.D
    n = w.n_dst if n_dst is None else n_dst
    esz = 2 if w.dtype == "bf16" else 4
    kt = (H2 + 1) * d                  # length of a segment-sum row
    mask = (H1 + H2) // 8              # ReLU mask bytes per edge
    # z1 rows are kept for the backward unless it recomputes them: the fused
    # edge-gradient pass, or the dW2 pass at d = 128, h1 = h2 = 256 (bf16)
    keeps_z1 = not fused and not (w.dtype == "bf16" and (d, H1, H2) == (128, 256, 256))
    idx = 8                            # two int32 indices per edge
    attr = 2 * (D + 1) * 4             # node attribute rows of both ends
    m = {
        # per-edge form
        "edge_fwd": (2 * E * (de * H1 + H1 * H2) + 2 * E * (H2 + 1) * d * d,
                     E * (idx + attr + d * esz + (H1 + H2) * esz + mask) + n * d * 4),
        "edge_dh": (2 * E * (H2 + 1) * d * d, E * (idx + d * esz + H2 * esz) + n_src * d * 4),
        # aggregate form
        # the split attributes (32 bytes) are stored for the unfused backward, z1
        # too where the dW2 pass does not recompute it (d = 128, h = 256)
        "edge_mlp": (2 * E * (de * H1 + H1 * H2),
                     E * (idx + attr + H2 * esz + mask + (0 if fused else 32) + (H1 * esz if keeps_z1 else 0))),
        "outer_fwd": (2 * E * H2 * d, E * (4 + H2 * esz + d * esz) + n * kt * esz),
        "gemm_fwd": (2 * n * kt * d, n * kt * esz + gemm_slices(n) * n * d * 4),
        "outer_dh": (2 * E * H2 * d, E * (idx + H2 * esz + d * esz) + n_src * kt * esz),
        "gemm_dh": (2 * n_src * kt * d, n_src * kt * esz + gemm_slices(n_src) * n_src * d * 4),
        "u_gemm": (2 * n * d * H2 * d, n * d * esz + n * H2 * d * esz),
        "dW2": (2 * E * H1 * H2, E * ((H1 if keeps_z1 else 0) + H2) * esz + (0 if keeps_z1 else 32 * E)),
    }
    return m


def agg_work(w, E, n_src, fused=False):
    """Work of the classes whose kernels differ between the two forms.  With
    ``fused`` the dz class is the one-pass kernel that also forms the dW2 and
    dW1 sums: it reads U_i, the gathered rows, the ReLU mask bits and both
    endpoints' node attributes, and writes no per-edge array (its per-workgroup
    partial sums are not counted)."""
    d, H1, H2, D, de = w.d, w.H1, w.H2, w.D, w.de
    n = w.n_dst
    esz = 2 if w.dtype == "bf16" else 4
    kt = (H2 + 1) * d
    mask = (H1 + H2) // 8
    dz_m = w.dtype == "bf16" and not fused and (d, H1, H2) == (128, 256, 256)
    if fused:
        dz = (2 * E * (d * H2 + H1 * H2 + H1 * H2 + H1 * de),
              n * H2 * d * esz + E * (4 + d * esz + mask + 2 * (D + 1) * 4))
    elif dz_m:
        # dz masked into da2 and the feature-gradient terms m_e from one read
        # of U_i and g_i: reads the source index, h_j, z and z's mask bits,
        # writes da2 and m_e
        dz = (2 * E * (d * H2 + H2 * d) + 2 * n * d * d,
              n * (H2 * d + d) * esz + E * (4 + d * esz + H2 * esz + H2 // 8 + H2 * esz + d * esz))
    else:
        dz = (2 * E * (d * H2 + H1 * H2), n * H2 * d * esz + E * (4 + d * esz + mask + (H1 + H2) * esz))
    out = {
        "dz": dz,
        "dW3": (2 * n * kt * d, n * kt * esz + n * d * esz),
    }
    if dz_m:
        # da1 = [z1 > 0] W2^T da2 from the stored da2 rows and the dW1/db1 sums
        # from it (x as bf16 high and low parts, 32 bytes per edge); da1 itself
        # stays on chip
        out["da1"] = (2 * E * H1 * H2 + 2 * E * H1 * (2 * de + 1), E * (H2 * esz + H1 // 8 + 32))
    if w.dtype == "bf16":
        # the feature gradient from U: per-edge terms from U_i, z_e and the bias
        # row, then their sums over the edges leaving each source
        if not dz_m:
            out["dh_u"] = (2 * E * H2 * d + 2 * n * d * d,
                           n * H2 * d * esz + E * (H2 * esz + d * esz) + n * (d * esz + 4))
        out["dh_final"] = (0, E * (d * esz + 4) + n_src * (d * 4 + 4) + n * d * 4)
    return out


def boxes_view(w, n_box):
    """The workload's shape with the inference boxes' nodes as its nodes
    (n_dst = n_src = n_box), for the work model of the inference mode."""
    import dataclasses
    return dataclasses.replace(w, parts=[dataclasses.replace(w.parts[0], s=n_box)])


def prep_work_step(w, E):
    """Algorithmic work per step of the data-preparation classes (no flops):
    sampling writes the kept indices (the keys are recomputed, nothing is
    read); the gathers read and write every sampled row of positions,
    attributes and features plus its index; the graph build reads the
    positions once and writes row_ptr, col, dst, csc_ptr and csc_eid."""
    esz = 2 if w.dtype == "bf16" else 4
    s_all = sum(p.s for p in w.parts)
    row = 4 * w.D + 4 * (w.D + 1) + w.d * esz
    return {
        "sample": (0, 4 * s_all),
        "gather": (0, s_all * (2 * row + 3 * 4)),
        "graph": (0, w.n_src * 4 * w.D + 12 * E + 4 * (w.n_dst + 1) + 4 * (w.n_src + 1)),
    }


def per_edge_work(w, E, n_src):
    d, H1, H2 = w.d, w.H1, w.H2
    n = w.n_dst
    esz = 2 if w.dtype == "bf16" else 4
    mask = (H1 + H2) // 8
    return {
        "dz": (2 * E * (H2 * d * d + H1 * H2), E * (8 + d * esz + mask + (H1 + H2) * esz) + n * d * 4),
        "dW3": (2 * E * H2 * d * d, E * (8 + d * esz + H2 * esz) + n * d * 4),
    }


class Pipeline:
    def __init__(self, w, lib, dm, torch):
        self.w, self.lib, self.dm, self.torch = w, lib, dm, torch
        dev = torch.device("cuda", 0)
        tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.tdt = tdt
        self.parts = []
        for p in w.parts:
            self.parts.append(dict(
                M=p.pos.shape[0], s=p.s, seed=p.seed,
                pos=torch.from_numpy(p.pos).to(dev), attr=torch.from_numpy(p.attr).to(dev),
                h=torch.from_numpy(p.h).to(dev).to(tdt),
                idx=torch.empty(p.s, dtype=torch.int32, device=dev)))
        n_src, n_dst, d = w.n_src, w.n_dst, w.d
        self.pos = torch.empty(n_src, w.D, dtype=torch.float32, device=dev)
        self.attr = torch.empty(n_src, w.D + 1, dtype=torch.float32, device=dev)
        self.h = [torch.empty(n_src, d, dtype=tdt, device=dev) for _ in range(w.layers + 1)]
        self.desc = dm.layer_desc(w.D, d, w.H1, w.H2, dm.BF16 if w.dtype == "bf16" else dm.F32)
        self.params = [{k: torch.from_numpy(v).to(dev) for k, v in P.items()} for P in w.params]
        self.G = torch.from_numpy(w.grad_out).to(dev)
        # size the graph once (E is fixed for this input) and preallocate everything
        self.sample_and_gather()
        E = lib.dsmp_radius_graph_count(self.pos, n_dst, w.r, w.cap, w.cap_mode)
        self.graph = lib.dsmp_radius_graph_build(self.pos, n_dst, w.r, w.cap, w.cap_mode, capacity=E)
        self.E = E
        sb, fb, bb = lib.dsmp_nnconv_workspace(self.desc, self.graph)
        self.saved = [torch.empty(max(sb, 256), dtype=torch.uint8, device=dev) for _ in range(w.layers)]
        self.fws = torch.empty(max(fb, 256), dtype=torch.uint8, device=dev)
        self.bws = torch.empty(max(bb, 256), dtype=torch.uint8, device=dev)
        self.packed = [lib.dsmp_nnconv_pack(self.desc, P) for P in self.params]
        self.out = [torch.empty(n_dst, d, dtype=torch.float32, device=dev) for _ in range(w.layers)]
        self.grad_h = [torch.empty(n_src, d, dtype=torch.float32, device=dev) for _ in range(w.layers)]
        f32 = dict(dtype=torch.float32, device=dev)
        de, H1, H2 = w.de, w.H1, w.H2
        self.grads = [{"dW1": torch.empty(H1, de, **f32), "db1": torch.empty(H1, **f32),
                       "dW2": torch.empty(H2, H1, **f32), "db2": torch.empty(H2, **f32),
                       "dW3": torch.empty(d * d, H2, **f32), "db3": torch.empty(d * d, **f32),
                       "dWr": torch.empty(d, d, **f32), "dbr": torch.empty(d, **f32)} for _ in range(w.layers)]

    def sample_and_gather(self):
        lib = self.lib
        off = 0
        for p in self.parts:
            lib.dsmp_sample_nodes(p["M"], p["s"], p["seed"], out=p["idx"])
            sl = slice(off, off + p["s"])
            lib.dsmp_gather_rows(p["pos"], p["idx"], out=self.pos[sl])
            lib.dsmp_gather_rows(p["attr"], p["idx"], out=self.attr[sl])
            lib.dsmp_gather_rows(p["h"], p["idx"], out=self.h[0][sl])
            off += p["s"]

    def step(self):
        w, lib = self.w, self.lib
        n_dst = w.n_dst
        self.sample_and_gather()
        lib.dsmp_radius_graph_build(self.pos, n_dst, w.r, w.cap, w.cap_mode, capacity=self.E, out=self.graph)
        for l in range(w.layers):
            if n_dst < w.n_src:      # halo rows keep their input features at every layer
                self.h[l + 1][n_dst:].copy_(self.h[0][n_dst:])
            lib.dsmp_nnconv_pack(self.desc, self.params[l], out=self.packed[l])
            lib.dsmp_nnconv_forward(self.desc, self.packed[l], self.graph, self.attr, self.h[l],
                                    h_out=self.out[l], h_out_lp=self.h[l + 1][:n_dst], saved=self.saved[l],
                                    ws=self.fws)
        G = self.G
        for l in reversed(range(w.layers)):
            lib.dsmp_nnconv_backward(self.desc, self.packed[l], self.graph, self.attr, self.h[l], self.saved[l],
                                     G, grad_h=self.grad_h[l], grads=self.grads[l], ws=self.bws)
            G = self.grad_h[l][:n_dst]


class HopPipeline:
    """The hop-loop training step on a workload: sample, gather, radius graph,
    then encoder, (layer with difference attributes + decoder) per hop, the
    masked MSE on the owned rows and the backward through all of it."""

    def __init__(self, w, lib, dm, torch):
        from workloads import hop_setup
        self.w, self.lib, self.dm, self.torch = w, lib, dm, torch
        if w.n_src != w.n_dst:
            raise SystemExit("the hop-loop step runs on workloads without halo rows (1-4)")
        dev = torch.device("cuda", 0)
        self.parts = [dict(M=p.pos.shape[0], s=p.s, seed=p.seed, pos=torch.from_numpy(p.pos).to(dev),
                           attr=torch.from_numpy(p.attr).to(dev), idx=torch.empty(p.s, dtype=torch.int32, device=dev))
                      for p in w.parts]
        n = w.n_dst
        self.pos = torch.empty(n, w.D, dtype=torch.float32, device=dev)
        self.attr = torch.empty(n, w.D + 1, dtype=torch.float32, device=dev)
        enc, conv, dec, Y = hop_setup(w)
        self.enc = {k: torch.from_numpy(v).to(dev) for k, v in enc.items()}
        self.dec = {k: torch.from_numpy(v).to(dev) for k, v in dec.items()}
        self.conv = {k: torch.from_numpy(v).to(dev) for k, v in conv.items()}
        self.Y = torch.from_numpy(Y).to(dev)
        self.mask = torch.ones(n, dtype=torch.uint8, device=dev)
        self.sample_and_gather()
        E = lib.dsmp_radius_graph_count(self.pos, n, w.r, w.cap, w.cap_mode)
        self.graph = lib.dsmp_radius_graph_build(self.pos, n, w.r, w.cap, w.cap_mode, capacity=E)
        self.E = E
        shapes = dm.HopShapes(n, w.D, w.d, w.H1, w.H2, 64, 64, dm.BF16 if w.dtype == "bf16" else dm.F32, w.layers)
        self.st = dm.HopStep(lib, self.graph, shapes)
        self.packed = lib.dsmp_nnconv_pack(self.st.conv, self.conv)

    def sample_and_gather(self):
        off = 0
        for p in self.parts:
            self.lib.dsmp_sample_nodes(p["M"], p["s"], p["seed"], out=p["idx"])
            sl = slice(off, off + p["s"])
            self.lib.dsmp_gather_rows(p["pos"], p["idx"], out=self.pos[sl])
            self.lib.dsmp_gather_rows(p["attr"], p["idx"], out=self.attr[sl])
            off += p["s"]

    def step(self):
        w, lib = self.w, self.lib
        self.sample_and_gather()
        lib.dsmp_radius_graph_build(self.pos, w.n_dst, w.r, w.cap, w.cap_mode, capacity=self.E, out=self.graph)
        lib.dsmp_nnconv_pack(self.st.conv, self.conv, out=self.packed)
        self.st.step(self.enc, self.packed, self.dec, self.attr, self.Y, self.mask)


class InferPipeline:
    """Sub-domain inference on a workload: sample and gather the nodes, then
    for every random box (overlap r) select its nodes, build its radius graph,
    run the layer stack forward and scatter the owned outputs back."""

    def __init__(self, w, lib, dm, torch):
        from workloads import subdomain_boxes
        self.w, self.lib, self.dm, self.torch = w, lib, dm, torch
        self.layer = Pipeline.__new__(Pipeline)
        Pipeline.__init__(self.layer, w, lib, dm, torch)
        self.boxes = subdomain_boxes(w)
        self.inf = dm.SubdomainInference(lib, self.layer.desc, self.layer.packed, w.r, w.cap, w.cap_mode)
        self.out = torch.zeros(w.n_src, w.d, dtype=torch.float32, device=torch.device("cuda", 0))
        self.step()
        self.E = sum(st[2] for st in self.inf.stats)

    def step(self):
        self.layer.sample_and_gather()
        self.inf.run(self.layer.pos, self.layer.attr, self.layer.h[0], self.boxes, self.w.r, out=self.out)


def infer_cpu_baseline(w, E_gpu):
    """The oracle's sub-domain inference on the smallest box of the workload,
    extrapolated to all boxes by their share of the edges."""
    import numpy as np
    import oracle
    from threadpoolctl import threadpool_info
    from workloads import subdomain_boxes
    pos, attr, h = [], [], []
    for p in w.parts:
        idx = oracle.sampling.sample_nodes(p.pos.shape[0], p.s, p.seed)
        pos.append(p.pos[idx]); attr.append(p.attr[idx]); h.append(p.h[idx])
    pos, attr, h = np.concatenate(pos), np.concatenate(attr), np.concatenate(h)
    boxes = subdomain_boxes(w)
    sizes = [oracle.infer.subdomain_nodes(pos, lo, hi, w.r)[0].size for lo, hi in boxes]
    b = int(np.argmin(sizes))
    t = time.perf_counter()
    _, st = oracle.infer.infer(w.params, pos, attr, h, boxes, w.r, w.r, w.cap, w.cap_mode, w.dtype, only=[b])
    sec = time.perf_counter() - t
    E_b = st[b][2]
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    return {"value": E_b * w.layers / sec, "unit": "edges/s", "cores": int(threads), "kind": "oracle",
            "sample": "subset-extrapolated: the oracle's inference of the smallest of %d boxes (%d edges, %d layers, "
                      "%.2f s); the rate carries to all boxes' %d edges" % (len(boxes), E_b, w.layers, sec, E_gpu),
            "seconds": round(sec, 2)}


def hop_cpu_baseline(w, E_gpu, m=1536):
    """The oracle's hop-loop step on the sub-graph of the first m sampled nodes
    (hops couple every row, so rows cannot be subsampled), extrapolated to the
    workload's edges."""
    import numpy as np
    import oracle
    from threadpoolctl import threadpool_info
    from workloads import hop_setup
    p = w.parts[0]
    idx = oracle.sampling.sample_nodes(p.pos.shape[0], p.s, p.seed)[:m]
    pos, v0 = p.pos[idx], p.attr[idx].astype(np.float64)
    rp, col = oracle.radius_graph.radius_graph(pos, m, w.r, w.cap, w.cap_mode)
    enc, conv, dec, Y = hop_setup(w)
    t = time.perf_counter()
    oracle.hop.train_step(enc, conv, dec, v0, Y[:m], np.ones(m, bool), rp, col, w.layers, w.dtype)
    sec = time.perf_counter() - t
    E_sub = int(rp[-1])
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    return {"value": E_sub * w.layers / sec, "unit": "edges/s", "cores": int(threads), "kind": "oracle",
            "sample": "hop-loop step of the oracle on the graph of the first %d sampled nodes (%d edges, %d hops, "
                      "%.2f s); the rate carries to the workload's %d edges as edges per second"
                      % (m, E_sub, w.layers, sec, E_gpu),
            "seconds": round(sec, 2)}


def cpu_baseline(w, rows_n, E_gpu):
    """Time the oracle, as it stands, on the host, on a bounded sample of the
    workload: the sampling of every part (whole), then, for a fixed set of
    destination rows, their radius-graph rows and one layer forward+backward
    (sparse upstream gradient: only their edges are visited).  The per-step
    time of the whole workload is extrapolated from the sample by its share
    of the edges: t_sample + (t_graph_rows + layers * t_layer_rows) * E / E_rows."""
    import numpy as np
    import oracle
    from threadpoolctl import threadpool_info
    t = time.perf_counter()
    pos, attr, h = [], [], []
    for p in w.parts:
        idx = oracle.sampling.sample_nodes(p.pos.shape[0], p.s, p.seed)
        pos.append(p.pos[idx]); attr.append(p.attr[idx]); h.append(p.h[idx])
    t_sample = time.perf_counter() - t
    pos, attr, h = np.concatenate(pos), np.concatenate(attr), np.concatenate(h).astype(np.float64)
    rows = np.sort(np.random.default_rng(0).choice(w.n_dst, min(rows_n, w.n_dst), replace=False))
    t = time.perf_counter()
    lists = oracle.radius_graph.rows_subset(pos, rows, w.n_dst, w.r, w.cap, w.cap_mode)
    t_graph = time.perf_counter() - t
    deg = np.zeros(w.n_dst, np.int64)
    deg[rows] = [len(c) for c in lists]
    rp = np.zeros(w.n_dst + 1, np.int64)
    np.cumsum(deg, out=rp[1:])
    col = np.concatenate(lists) if lists else np.zeros(0, np.int32)
    E_sub = int(rp[-1])
    G = np.zeros((w.n_dst, w.d))
    G[rows] = w.grad_out[rows]
    t = time.perf_counter()
    x = oracle.nnconv.edge_attr(attr, rp, col)
    oracle.nnconv.forward(w.params[0], x, h, rp, col, w.n_dst, rows=rows)
    oracle.nnconv.backward(w.params[0], x, h, rp, col, w.n_dst, G, rows=rows)
    t_layer_sub = time.perf_counter() - t
    t_step = t_sample + (t_graph + w.layers * t_layer_sub) * E_gpu / max(E_sub, 1)
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    return {
        "value": E_gpu * w.layers / t_step, "unit": "edges/s", "cores": int(threads), "kind": "oracle",
        "sample": ("subset-extrapolated: sampling of every part (%.2f s), then %d fixed destination rows "
                   "(%d of the %d edges): their radius-graph rows (%.2f s) and one layer forward+backward "
                   "(%.2f s); the step time of the whole workload extrapolated by the edge share to %d layers; "
                   "%d BLAS threads, %d cores in affinity"
                   % (t_sample, len(rows), E_sub, E_gpu, t_graph, t_layer_sub, w.layers, threads,
                      len(os.sched_getaffinity(0)))),
        "seconds": round(t_sample + t_graph + t_layer_sub, 2),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build runs the hot path on one MI355X "
              "(one sub-domain's share); --gpus %d is not supported." % max(args.gpus, world), file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2402_15106_amd as dm
    from workloads import make_config
    assert torch.cuda.is_available(), "bench.py needs a GPU"

    w = make_config(args.config)
    lib = dm.Dsmp(0)
    lib.dsmp_set_edge_algorithm({"auto": dm.EDGE_AUTO, "per_edge": dm.EDGE_PER_EDGE,
                                 "aggregate": dm.EDGE_AGGREGATE}[args.algo])
    hop = args.model == "hop"
    infer = args.model == "infer"
    pipe = HopPipeline(w, lib, dm, torch) if hop else InferPipeline(w, lib, dm, torch) if infer \
        else Pipeline(w, lib, dm, torch)
    print("workload %s: n_dst=%d n_src=%d E=%d layers=%d" % (w.name, w.n_dst, w.n_src, pipe.E, w.layers),
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        pipe.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        pipe.step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    print("timed %d steps: %.3f ms/step" % (args.steps, ms), file=sys.stderr, flush=True)

    # per-kernel durations: HIP events recorded by the library on its stream,
    # read after every step of a second pass (mean, median and minimum)
    import statistics
    lib.dsmp_profile_enable(True)
    per_step = []
    for _ in range(args.steps):
        lib.dsmp_profile_reset()
        pipe.step()
        per_step.append(lib.dsmp_profile_read())
    lib.dsmp_profile_enable(False)

    E, L = pipe.E, w.layers
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_TFLOPS
    prof = {k: (sum(p[k][0] for p in per_step), sum(p[k][1] for p in per_step)) for k in per_step[0]}
    agg = "edge_mlp" in prof and prof["edge_mlp"][1] > 0
    if hop:   # the layer of the hop loop reads difference attributes (dim+1 per edge)
        import dataclasses
        w = dataclasses.replace(w, de=w.D + 1)
    fused = agg and not ("dW2" in prof and prof["dW2"][1] > 0)
    if infer:   # no backward ran: the forward's stores follow the shape's backward
        fused = agg and w.dtype == "bf16" and w.H1 == w.H2 and w.H1 in (64, 128)
    if infer:
        # every box is a graph of its own and each layer launch runs over one
        # box: a launch's work is the boxes' total over the number of boxes
        # (time and work are then both averages over the boxes)
        n_box = sum(st[1] for st in pipe.inf.stats)
        nb = sum(1 for st in pipe.inf.stats if st[1] > 0)
        wb = boxes_view(w, n_box)
        work = work_model(wb, E, n_box, fused, n_dst=n_box)
        work.update(agg_work(wb, E, n_box, fused) if agg else per_edge_work(wb, E, n_box))
        work = {k: (fl / nb, by / nb) for k, (fl, by) in work.items()}
    else:
        work = work_model(w, E, w.n_src, fused)
        work.update(agg_work(w, E, w.n_src, fused) if agg else per_edge_work(w, E, w.n_src))
    for name, (fl, by) in prep_work_step(w, E).items():
        if name in prof and prof[name][1] > 0:
            nper = prof[name][1] / args.steps
            work[name] = (fl / nper, by / nper)
    kernels = {}
    for name, (tot, n) in prof.items():
        if n == 0:
            continue
        avg = tot / n
        launch_ms = [p[name][0] / p[name][1] for p in per_step if p[name][1] > 0]
        ent = {"ms_avg": round(avg, 5), "ms_median": round(statistics.median(launch_ms), 5),
               "ms_min": round(min(launch_ms), 5), "launches_per_step": n / args.steps,
               "ms_per_step": round(tot / args.steps, 4)}
        if name in work:
            fl, by = work[name]
            tf = fl / (avg * 1e-3) / 1e12
            gbs = by / (avg * 1e-3) / 1e9
            bound = "mfma" if fl / by > (peak / HBM_TBPS) else "hbm"
            ent.update({"flops": fl, "bytes": by, "tflops": round(tf, 2), "gbps": round(gbs, 1), "bound": bound,
                        "frac": round(tf / peak if bound == "mfma" else gbs / (HBM_TBPS * 1e3), 4)})
        kernels[name] = ent
    modeled = {k: v for k, v in kernels.items() if "bound" in v}
    dom = max(modeled, key=lambda k: modeled[k]["ms_per_step"])
    dk = kernels[dom]
    if dk["bound"] == "mfma":
        roof = {"bound": "mfma", "achieved": dk["tflops"], "peak": peak, "unit": "TFLOP/s", "frac": dk["frac"],
                "algorithmic": dk["flops"]}
    else:
        roof = {"bound": "hbm", "achieved": dk["gbps"], "peak": HBM_TBPS * 1e3, "unit": "GB/s", "frac": dk["frac"],
                "algorithmic": dk["bytes"]}
    # the traffic tables record the layer bench in the aggregate form
    traffic = measured_traffic(dom, w.name) if agg and not hop and not infer else None
    roof.update({"kernel": dom, "traffic": traffic, "ms_per_launch": dk["ms_avg"],
                 "ms_per_launch_median": dk["ms_median"], "ms_per_launch_min": dk["ms_min"]})
    executed = sum(v["flops"] * v["launches_per_step"] for v in modeled.values())
    if hop:
        METRIC_RUN = ("edges/sec of the hop-loop training step (encoder, layer + decoder per hop, masked MSE, "
                      "backward) on 1 MI355X")
    elif infer:
        METRIC_RUN = ("edges/sec of sub-domain inference (the layer stack forward on random boxes with overlap r, "
                      "owned outputs reassembled) on 1 MI355X")
    else:
        METRIC_RUN = METRIC
    res = {
        "metric": METRIC_RUN,
        "value": round(E * L / (ms * 1e-3), 1),
        "unit": "edges/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded stand-in for the paper's mesh datasets)",
        "config": {"workload": "%s: %d nodes sampled from %d candidates%s, radius %.3g, cap %s, d=%d, kernel MLP "
                               "%d->%d->%d->%d, %d %s, %s per step"
                               % (w.name, w.n_dst, sum(p.pos.shape[0] for p in w.parts),
                                  " (plus %d halo nodes)" % (w.n_src - w.n_dst) if w.n_src > w.n_dst else "",
                                  w.r, w.cap or "none",
                                  w.d, w.de, w.H1, w.H2, w.d * w.d, L,
                                  "hops (encoder and decoder 64 wide, difference attributes)" if hop else "layers",
                                  "sample, then for each of %d random boxes with overlap r: select, gather, "
                                  "graph, forward, scatter" % len(pipe.boxes) if infer
                                  else "sample+graph+forward+backward"),
                   "n_dst": w.n_dst, "n_src": w.n_src, "edges": E, "layers": L, "d": w.d, "h1": w.H1,
                   "h2": w.H2, "nominal_flops_per_edge_layer": method_flops_per_edge(w)},
        "edge_algorithm": "aggregate" if agg else "per_edge",
        "executed_tflops_step": round(executed / (ms * 1e-3) / 1e12, 2),
        "executed_frac_peak": round(executed / (ms * 1e-3) / 1e12 / peak, 4),
        "roofline": roof,
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        rows_n = args.cpu_rows if args.cpu_rows is not None else CPU_ROWS[args.config]
        res["cpu_baseline"] = (hop_cpu_baseline(w, E) if hop else infer_cpu_baseline(w, E) if infer
                               else cpu_baseline(w, rows_n, E))
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
