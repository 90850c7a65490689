"""ctypes binding of libdsmpnn (the C ABI declared in include/dsmpnn.h).

Argument marshalling only: every step of the hot path runs in the HIP
library.  Tensors are PyTorch device tensors (device memory and streams are
the only things PyTorch provides); the caller's current stream is bound to the
handle before every call.  Output and scratch buffers are allocated here with
torch when the caller does not pass them.  If the shared library is missing
the import fails: there is no fallback.
"""

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libdsmpnn.so")

OK, INVALID_ARG, CAPACITY, HIP_ERROR, UNSUPPORTED, WORKSPACE_TOO_SMALL = range(6)
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "CAPACITY", 3: "HIP_ERROR", 4: "UNSUPPORTED",
                5: "WORKSPACE_TOO_SMALL"}
CAP_KNN, CAP_RANDOM = 0, 1
F32, BF16 = 0, 1
ACT_IDENTITY, ACT_RELU = 0, 1
ATTR_CONCAT, ATTR_DIFF = 0, 1
GRAD_ACCUMULATE = 1
GRAD_X_ACCUMULATE = 2
EDGE_AUTO, EDGE_PER_EDGE, EDGE_AGGREGATE = 0, 1, 2

EXPORTED = ["dsmp_version", "dsmp_create", "dsmp_destroy", "dsmp_set_stream", "dsmp_last_error",
            "dsmp_sample_workspace", "dsmp_sample_nodes", "dsmp_sample_nodes_noalloc", "dsmp_gather_rows",
            "dsmp_scatter_rows",
            "dsmp_subdomain_workspace", "dsmp_subdomain_select",
            "dsmp_radius_graph_workspace", "dsmp_radius_graph_count", "dsmp_radius_graph_build",
            "dsmp_nnconv_packed_bytes", "dsmp_nnconv_pack", "dsmp_nnconv_workspace",
            "dsmp_nnconv_forward", "dsmp_nnconv_backward", "dsmp_profile_enable", "dsmp_profile_reset",
            "dsmp_profile_read", "dsmp_set_edge_algorithm", "dsmp_mlp_workspace", "dsmp_mlp_forward",
            "dsmp_mlp_backward", "dsmp_masked_mse_workspace", "dsmp_masked_mse"]

# kernel classes of the opt-in timing (dsmp_profile_*)
KERNEL_CLASSES = ["sample", "gather", "graph", "edge_fwd", "node_fwd", "node_bwd", "edge_dh", "dh_final",
                  "dz", "dW3", "dW2", "dW1", "reduce", "edge_mlp", "outer_fwd", "gemm_fwd", "outer_dh",
                  "gemm_dh", "u_gemm", "attr", "mlp", "loss", "dh_u", "da1"]


class DsmpError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), msg))
        self.status = status


class GraphQuery(ctypes.Structure):
    _fields_ = [("pos", ctypes.c_void_p), ("n_src", ctypes.c_int64), ("n_dst", ctypes.c_int64),
                ("dim", ctypes.c_int32), ("r", ctypes.c_float), ("cap", ctypes.c_int32),
                ("cap_mode", ctypes.c_int32), ("seed", ctypes.c_uint64)]


class CGraph(ctypes.Structure):
    _fields_ = [("n_dst", ctypes.c_int64), ("n_src", ctypes.c_int64), ("n_edges", ctypes.c_int64),
                ("row_ptr", ctypes.c_void_p), ("col", ctypes.c_void_p), ("dst", ctypes.c_void_p),
                ("csc_ptr", ctypes.c_void_p), ("csc_eid", ctypes.c_void_p)]


class LayerDesc(ctypes.Structure):
    _fields_ = [("dim", ctypes.c_int32), ("d", ctypes.c_int32), ("h1", ctypes.c_int32),
                ("h2", ctypes.c_int32), ("dtype", ctypes.c_int32), ("act", ctypes.c_int32),
                ("residual", ctypes.c_int32), ("attr_mode", ctypes.c_int32)]


class LayerParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")]


class LayerGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("dW1", "db1", "dW2", "db2", "dW3", "db3", "dWr", "dbr", "dattr")]


class MlpDesc(ctypes.Structure):
    _fields_ = [("d_in", ctypes.c_int32), ("d_hid", ctypes.c_int32), ("d_out", ctypes.c_int32)]


class MlpParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("W1", "b1", "W2", "b2", "W3", "b3")]


class MlpGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("dW1", "db1", "dW2", "db2", "dW3", "db3")]


_P = ctypes.c_void_p
_SIG = {
    "dsmp_version": (ctypes.c_int, []),
    "dsmp_create": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int]),
    "dsmp_destroy": (ctypes.c_int, [_P]),
    "dsmp_set_stream": (ctypes.c_int, [_P, _P]),
    "dsmp_set_edge_algorithm": (ctypes.c_int, [_P, ctypes.c_int32]),
    "dsmp_last_error": (ctypes.c_char_p, [_P]),
    "dsmp_sample_workspace": (ctypes.c_int, [ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]),
    "dsmp_sample_nodes": (ctypes.c_int, [_P, ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64, _P, _P,
                                         ctypes.c_size_t]),
    "dsmp_sample_nodes_noalloc": (ctypes.c_int, [_P, ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64, _P]),
    "dsmp_gather_rows": (ctypes.c_int, [_P, _P, ctypes.c_int64, ctypes.c_int64, _P, ctypes.c_int64, _P]),
    "dsmp_scatter_rows": (ctypes.c_int, [_P, _P, ctypes.c_int64, ctypes.c_int64, _P, _P, ctypes.c_int64]),
    "dsmp_subdomain_workspace": (ctypes.c_int, [ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]),
    "dsmp_subdomain_select": (ctypes.c_int, [_P, _P, ctypes.c_int64, ctypes.c_int32, ctypes.POINTER(ctypes.c_float),
                                             ctypes.POINTER(ctypes.c_float), ctypes.c_float, _P, _P, ctypes.c_size_t,
                                             ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]),
    "dsmp_radius_graph_workspace": (ctypes.c_int, [ctypes.POINTER(GraphQuery), ctypes.POINTER(ctypes.c_size_t)]),
    "dsmp_radius_graph_count": (ctypes.c_int, [_P, ctypes.POINTER(GraphQuery), _P, ctypes.c_size_t,
                                               ctypes.POINTER(ctypes.c_int64)]),
    "dsmp_radius_graph_build": (ctypes.c_int, [_P, ctypes.POINTER(GraphQuery), _P, ctypes.c_size_t,
                                               ctypes.c_int64, ctypes.POINTER(CGraph)]),
    "dsmp_nnconv_packed_bytes": (ctypes.c_int, [ctypes.POINTER(LayerDesc), ctypes.POINTER(ctypes.c_size_t)]),
    "dsmp_nnconv_pack": (ctypes.c_int, [_P, ctypes.POINTER(LayerDesc), ctypes.POINTER(LayerParams), _P]),
    "dsmp_nnconv_workspace": (ctypes.c_int, [ctypes.POINTER(LayerDesc), ctypes.POINTER(CGraph),
                                             ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t),
                                             ctypes.POINTER(ctypes.c_size_t)]),
    "dsmp_nnconv_forward": (ctypes.c_int, [_P, ctypes.POINTER(LayerDesc), _P, ctypes.POINTER(CGraph), _P, _P,
                                           _P, _P, _P, ctypes.c_size_t, _P, ctypes.c_size_t]),
    "dsmp_nnconv_backward": (ctypes.c_int, [_P, ctypes.POINTER(LayerDesc), _P, ctypes.POINTER(CGraph), _P, _P,
                                            _P, ctypes.c_size_t, _P, _P, ctypes.POINTER(LayerGrads),
                                            ctypes.c_int32, _P, ctypes.c_size_t]),
    "dsmp_mlp_workspace": (ctypes.c_int, [ctypes.POINTER(MlpDesc), ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t),
                                          ctypes.POINTER(ctypes.c_size_t)]),
    "dsmp_mlp_forward": (ctypes.c_int, [_P, ctypes.POINTER(MlpDesc), ctypes.POINTER(MlpParams), _P, ctypes.c_int64,
                                        _P, _P, _P, ctypes.c_size_t]),
    "dsmp_mlp_backward": (ctypes.c_int, [_P, ctypes.POINTER(MlpDesc), ctypes.POINTER(MlpParams), _P, ctypes.c_int64,
                                         _P, ctypes.c_size_t, _P, _P, ctypes.POINTER(MlpGrads), ctypes.c_int32, _P,
                                         ctypes.c_size_t]),
    "dsmp_masked_mse_workspace": (ctypes.c_int, [ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]),
    "dsmp_masked_mse": (ctypes.c_int, [_P, _P, _P, _P, ctypes.c_int64, ctypes.c_int32, _P, _P, _P, ctypes.c_size_t]),
    "dsmp_profile_enable": (ctypes.c_int, [_P, ctypes.c_int]),
    "dsmp_profile_reset": (ctypes.c_int, [_P]),
    "dsmp_profile_read": (ctypes.c_int, [_P, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_int64)]),
}

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libdsmpnn.so and declare every exported signature (no GPU needed)."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise ImportError("libdsmpnn.so is not built (%s); run __graft_entry__.build()" % path)
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIG.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path == LIB_PATH:
        _lib = lib
    return lib


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


@dataclass
class Graph:
    """A radius graph held in device tensors (int32)."""
    n_dst: int
    n_src: int
    n_edges: int
    row_ptr: torch.Tensor
    col: torch.Tensor
    dst: torch.Tensor
    csc_ptr: torch.Tensor
    csc_eid: torch.Tensor

    def c(self) -> CGraph:
        return CGraph(self.n_dst, self.n_src, self.n_edges, self.row_ptr.data_ptr(),
                      self.col.data_ptr(), self.dst.data_ptr(), self.csc_ptr.data_ptr(),
                      self.csc_eid.data_ptr())


def layer_desc(dim, d, h1, h2, dtype, act=ACT_IDENTITY, residual=1, attr_mode=ATTR_CONCAT) -> LayerDesc:
    return LayerDesc(dim, d, h1, h2, dtype, act, residual, attr_mode)


def _torch_dtype(desc: LayerDesc):
    return torch.bfloat16 if desc.dtype == BF16 else torch.float32


class Dsmp:
    """A library handle on one device, with methods named after the C calls."""

    def __init__(self, device: int = 0):
        self.lib = load_library()
        self.device = torch.device("cuda", device)
        h = ctypes.c_void_p()
        self._check(self.lib.dsmp_create(ctypes.byref(h), device), None)
        self.h = h
        self._ws = {}

    def close(self):
        if getattr(self, "h", None) is not None:
            self.lib.dsmp_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------ helpers
    def _check(self, st, h):
        if st != OK:
            msg = self.lib.dsmp_last_error(h).decode() if h is not None else ""
            raise DsmpError(st, msg)

    def _bind(self):
        s = torch.cuda.current_stream(self.device).cuda_stream
        self._check(self.lib.dsmp_set_stream(self.h, ctypes.c_void_p(s)), self.h)

    def dsmp_set_edge_algorithm(self, algorithm: int):
        """Edge-contraction form for later layer calls (EDGE_AUTO / EDGE_PER_EDGE / EDGE_AGGREGATE)."""
        self._check(self.lib.dsmp_set_edge_algorithm(self.h, int(algorithm)), self.h)

    def workspace(self, key: str, nbytes: int) -> torch.Tensor:
        """A cached uint8 device buffer of at least nbytes for scratch use."""
        buf = self._ws.get(key)
        if buf is None or buf.numel() < nbytes:
            buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
            self._ws[key] = buf
        return buf

    # ------------------------------------------------------------ timing
    def dsmp_profile_enable(self, on: bool = True):
        self._check(self.lib.dsmp_profile_enable(self.h, int(bool(on))), self.h)

    def dsmp_profile_reset(self):
        self._check(self.lib.dsmp_profile_reset(self.h), self.h)

    def dsmp_profile_read(self) -> dict:
        """{kernel class: (total ms, launches)} since the last reset (synchronises)."""
        out = {}
        for i, name in enumerate(KERNEL_CLASSES):
            ms, n = ctypes.c_double(), ctypes.c_int64()
            self._check(self.lib.dsmp_profile_read(self.h, i, ctypes.byref(ms), ctypes.byref(n)), self.h)
            out[name] = (ms.value, n.value)
        return out

    # ------------------------------------------------------------ sampling
    def dsmp_sample_nodes(self, M: int, s: int, seed: int, out: Optional[torch.Tensor] = None):
        out = torch.empty(s, dtype=torch.int32, device=self.device) if out is None else out
        nb = ctypes.c_size_t()
        self._check(self.lib.dsmp_sample_workspace(M, ctypes.byref(nb)), None)
        ws = self.workspace("sample", nb.value)
        self._bind()
        self._check(self.lib.dsmp_sample_nodes(self.h, M, s, ctypes.c_uint64(seed & (2 ** 64 - 1)),
                                               _ptr(out), _ptr(ws), ws.numel()), self.h)
        return out

    def dsmp_sample_nodes_noalloc(self, M: int, s: int, seed: int, out: torch.Tensor):
        """dsmp_sample_nodes on the library's own scratch (no workspace); out
        is the caller's int32 [s] device buffer."""
        self._bind()
        self._check(self.lib.dsmp_sample_nodes_noalloc(self.h, M, s, seed & (2 ** 64 - 1), _ptr(out)), self.h)
        return out

    def dsmp_gather_rows(self, src: torch.Tensor, idx: torch.Tensor, out: Optional[torch.Tensor] = None):
        src = src.contiguous()
        n = idx.numel()
        out = torch.empty((n,) + tuple(src.shape[1:]), dtype=src.dtype, device=self.device) if out is None else out
        row_bytes = src[0].numel() * src.element_size() if src.shape[0] > 0 else out[0].numel() * out.element_size()
        self._bind()
        self._check(self.lib.dsmp_gather_rows(self.h, _ptr(src), src.shape[0], row_bytes, _ptr(idx), n,
                                              _ptr(out)), self.h)
        return out

    def dsmp_scatter_rows(self, src: torch.Tensor, idx: torch.Tensor, out: torch.Tensor):
        """out[idx[i]] = src[i] (the inverse of dsmp_gather_rows)."""
        src = src.contiguous()
        n = idx.numel()
        row_bytes = out[0].numel() * out.element_size() if out.shape[0] > 0 else 4
        self._bind()
        self._check(self.lib.dsmp_scatter_rows(self.h, _ptr(src), n, row_bytes, _ptr(idx), _ptr(out),
                                               out.shape[0]), self.h)
        return out

    # ------------------------------------------------------------ sub-domains
    def dsmp_subdomain_select(self, pos: torch.Tensor, lo, hi, overlap: float,
                              out: Optional[torch.Tensor] = None):
        """Nodes of the box [lo, hi) with overlap: (idx [n_total] int32 with the
        owned nodes first, n_owned).  Synchronises."""
        pos = pos.contiguous()
        n, D = pos.shape
        out = torch.empty(max(n, 1), dtype=torch.int32, device=self.device) if out is None else out
        nb = ctypes.c_size_t()
        self._check(self.lib.dsmp_subdomain_workspace(n, ctypes.byref(nb)), None)
        ws = self.workspace("subdomain", nb.value)
        clo = (ctypes.c_float * D)(*[float(v) for v in lo])
        chi = (ctypes.c_float * D)(*[float(v) for v in hi])
        n_own, n_tot = ctypes.c_int64(), ctypes.c_int64()
        self._bind()
        self._check(self.lib.dsmp_subdomain_select(self.h, _ptr(pos), n, D, clo, chi, float(overlap), _ptr(out),
                                                   _ptr(ws), ws.numel(), ctypes.byref(n_own),
                                                   ctypes.byref(n_tot)), self.h)
        return out[:n_tot.value], n_own.value

    # ------------------------------------------------------------ graph
    def _query(self, pos, n_dst, r, cap, cap_mode, seed):
        pos = pos.contiguous()
        return GraphQuery(pos.data_ptr() if pos.numel() else 0, pos.shape[0], n_dst, pos.shape[1],
                          float(r), int(cap), int(cap_mode), seed & (2 ** 64 - 1)), pos

    def _graph_ws(self, q):
        nb = ctypes.c_size_t()
        self._check(self.lib.dsmp_radius_graph_workspace(ctypes.byref(q), ctypes.byref(nb)), None)
        return self.workspace("graph", nb.value)

    def dsmp_radius_graph_count(self, pos, n_dst, r, cap=0, cap_mode=CAP_KNN, seed=0) -> int:
        q, pos = self._query(pos, n_dst, r, cap, cap_mode, seed)
        ws = self._graph_ws(q)
        E = ctypes.c_int64()
        self._bind()
        self._check(self.lib.dsmp_radius_graph_count(self.h, ctypes.byref(q), _ptr(ws), ws.numel(),
                                                     ctypes.byref(E)), self.h)
        return E.value

    def dsmp_radius_graph_build(self, pos, n_dst, r, cap=0, cap_mode=CAP_KNN, seed=0,
                                capacity: Optional[int] = None, out: Optional[Graph] = None) -> Graph:
        q, pos = self._query(pos, n_dst, r, cap, cap_mode, seed)
        if out is None:
            if capacity is None:
                capacity = self.dsmp_radius_graph_count(pos, n_dst, r, cap, cap_mode, seed)
            i32 = dict(dtype=torch.int32, device=self.device)
            out = Graph(n_dst, pos.shape[0], 0, torch.empty(n_dst + 1, **i32),
                        torch.empty(max(capacity, 1), **i32), torch.empty(max(capacity, 1), **i32),
                        torch.empty(pos.shape[0] + 1, **i32), torch.empty(max(capacity, 1), **i32))
        cap_e = out.col.numel() if capacity is None else capacity
        ws = self._graph_ws(q)
        cg = out.c()
        self._bind()
        st = self.lib.dsmp_radius_graph_build(self.h, ctypes.byref(q), _ptr(ws), ws.numel(), cap_e,
                                              ctypes.byref(cg))
        out.n_edges = cg.n_edges
        out.n_dst, out.n_src = cg.n_dst, cg.n_src
        self._check(st, self.h)
        return out

    # ------------------------------------------------------------ layer
    def dsmp_nnconv_pack(self, desc: LayerDesc, params: dict, out: Optional[torch.Tensor] = None):
        nb = ctypes.c_size_t()
        self._check(self.lib.dsmp_nnconv_packed_bytes(ctypes.byref(desc), ctypes.byref(nb)), None)
        out = torch.empty(nb.value, dtype=torch.uint8, device=self.device) if out is None else out
        P = {k: params[k].to(device=self.device, dtype=torch.float32).contiguous() for k in
             ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")}
        lp = LayerParams(*[P[k].data_ptr() for k in ("W1", "b1", "W2", "b2", "W3", "b3", "Wr", "br")])
        self._bind()
        self._check(self.lib.dsmp_nnconv_pack(self.h, ctypes.byref(desc), ctypes.byref(lp), _ptr(out)), self.h)
        out._keepalive = P   # the pack is asynchronous: keep inputs alive with the output
        return out

    def dsmp_nnconv_workspace(self, desc: LayerDesc, g: Graph):
        s, f, b = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        cg = g.c()
        self._check(self.lib.dsmp_nnconv_workspace(ctypes.byref(desc), ctypes.byref(cg), ctypes.byref(s),
                                                   ctypes.byref(f), ctypes.byref(b)), None)
        return s.value, f.value, b.value

    def dsmp_nnconv_forward(self, desc: LayerDesc, packed, g: Graph, node_attr, h_in, h_out=None,
                            h_out_lp=None, saved=None, ws=None):
        sb, fb, _ = self.dsmp_nnconv_workspace(desc, g)
        if h_out is None:
            h_out = torch.empty(g.n_dst, desc.d, dtype=torch.float32, device=self.device)
        if saved is None:
            saved = torch.empty(max(sb, 256), dtype=torch.uint8, device=self.device)
        if ws is None:
            ws = self.workspace("fwd", fb)
        cg = g.c()
        self._bind()
        self._check(self.lib.dsmp_nnconv_forward(self.h, ctypes.byref(desc), _ptr(packed), ctypes.byref(cg),
                                                 _ptr(node_attr), _ptr(h_in), _ptr(h_out), _ptr(h_out_lp),
                                                 _ptr(saved), saved.numel(), _ptr(ws), ws.numel()), self.h)
        return h_out, saved

    def dsmp_nnconv_backward(self, desc: LayerDesc, packed, g: Graph, node_attr, h_in, saved, grad_out,
                             grad_h=None, grads: Optional[dict] = None, flags: int = 0, ws=None):
        _, _, bb = self.dsmp_nnconv_workspace(desc, g)
        d, h1, h2 = desc.d, desc.h1, desc.h2
        de = 2 * desc.dim + 2 if desc.attr_mode == ATTR_CONCAT else desc.dim + 1
        f32 = dict(dtype=torch.float32, device=self.device)
        if grad_h is None:
            grad_h = torch.empty(g.n_src, d, **f32)
        if grads is None:
            grads = {"dW1": torch.empty(h1, de, **f32), "db1": torch.empty(h1, **f32),
                     "dW2": torch.empty(h2, h1, **f32), "db2": torch.empty(h2, **f32),
                     "dW3": torch.empty(d * d, h2, **f32), "db3": torch.empty(d * d, **f32),
                     "dWr": torch.empty(d, d, **f32), "dbr": torch.empty(d, **f32)}
        lg = LayerGrads(*[grads[k].data_ptr() for k in ("dW1", "db1", "dW2", "db2", "dW3", "db3", "dWr", "dbr")],
                        grads["dattr"].data_ptr() if grads.get("dattr") is not None else None)
        if ws is None:
            ws = self.workspace("bwd", bb)
        cg = g.c()
        self._bind()
        self._check(self.lib.dsmp_nnconv_backward(self.h, ctypes.byref(desc), _ptr(packed), ctypes.byref(cg),
                                                  _ptr(node_attr), _ptr(h_in), _ptr(saved), saved.numel(),
                                                  _ptr(grad_out), _ptr(grad_h), ctypes.byref(lg), flags,
                                                  _ptr(ws), ws.numel()), self.h)
        return grad_h, grads

    # ------------------------------------------------------------ encoder / decoder and loss
    def dsmp_mlp_workspace(self, desc: "MlpDesc", n: int):
        sb, wb = ctypes.c_size_t(), ctypes.c_size_t()
        self._check(self.lib.dsmp_mlp_workspace(ctypes.byref(desc), n, ctypes.byref(sb), ctypes.byref(wb)), None)
        return sb.value, wb.value

    def dsmp_mlp_forward(self, desc: "MlpDesc", params: dict, x, y=None, y_bf16=None, saved=None):
        """Three-layer perceptron on the rows of x (float32 [n, d_in]); returns (y, saved)."""
        n = x.shape[0]
        sb, _ = self.dsmp_mlp_workspace(desc, n)
        if y is None:
            y = torch.empty(n, desc.d_out, dtype=torch.float32, device=self.device)
        if saved is None:
            saved = torch.empty(max(sb, 256), dtype=torch.uint8, device=self.device)
        mp = MlpParams(*[params[k].data_ptr() for k in ("W1", "b1", "W2", "b2", "W3", "b3")])
        self._bind()
        self._check(self.lib.dsmp_mlp_forward(self.h, ctypes.byref(desc), ctypes.byref(mp), _ptr(x), n, _ptr(y),
                                              _ptr(y_bf16), _ptr(saved), saved.numel()), self.h)
        return y, saved

    def dsmp_mlp_backward(self, desc: "MlpDesc", params: dict, x, saved, grad_y, grad_x=None,
                          grads: Optional[dict] = None, flags: int = 0, ws=None):
        """Gradients of sum(grad_y * y); grad_x optional (None: not computed).  Returns grads."""
        n = x.shape[0]
        _, wb = self.dsmp_mlp_workspace(desc, n)
        f32 = dict(dtype=torch.float32, device=self.device)
        if grads is None:
            grads = {"dW1": torch.empty(desc.d_hid, desc.d_in, **f32), "db1": torch.empty(desc.d_hid, **f32),
                     "dW2": torch.empty(desc.d_hid, desc.d_hid, **f32), "db2": torch.empty(desc.d_hid, **f32),
                     "dW3": torch.empty(desc.d_out, desc.d_hid, **f32), "db3": torch.empty(desc.d_out, **f32)}
        mp = MlpParams(*[params[k].data_ptr() for k in ("W1", "b1", "W2", "b2", "W3", "b3")])
        mg = MlpGrads(*[grads[k].data_ptr() for k in ("dW1", "db1", "dW2", "db2", "dW3", "db3")])
        if ws is None:
            ws = self.workspace("mlp_bwd", wb)
        self._bind()
        self._check(self.lib.dsmp_mlp_backward(self.h, ctypes.byref(desc), ctypes.byref(mp), _ptr(x), n, _ptr(saved),
                                               saved.numel(), _ptr(grad_y), _ptr(grad_x), ctypes.byref(mg), flags,
                                               _ptr(ws), ws.numel()), self.h)
        return grads

    def dsmp_masked_mse(self, pred, target, mask, loss=None, grad=None):
        """Mean squared error over interior rows (mask uint8 [n]); returns (loss [1] device, grad)."""
        n, c = pred.shape
        nb = ctypes.c_size_t()
        self._check(self.lib.dsmp_masked_mse_workspace(n, ctypes.byref(nb)), None)
        ws = self.workspace("mse", nb.value)
        if loss is None:
            loss = torch.empty(1, dtype=torch.float32, device=self.device)
        self._bind()
        self._check(self.lib.dsmp_masked_mse(self.h, _ptr(pred), _ptr(target), _ptr(mask), n, c, _ptr(loss),
                                             _ptr(grad), _ptr(ws), ws.numel()), self.h)
        return loss, grad
