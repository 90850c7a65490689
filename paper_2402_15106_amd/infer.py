"""Sub-domain inference with reassembly, composed from library calls.

At test time the paper cuts the domain into smaller sub-domains, each with an
overlap region, feeds them through the trained model one after another, and
reassembles the outputs over the whole domain (Sec. 3, Methodology, testing
procedure).  For every box this class calls, in order:

  dsmp_subdomain_select   owned nodes of the box, then its overlap nodes
  dsmp_gather_rows        their positions, attributes and input features
  dsmp_radius_graph_*     the sub-domain's own radius graph (every node a
                          destination, the same radius and cap)
  dsmp_nnconv_forward     the layer stack (each layer's output, rounded to the
                          layer type, is the next layer's input)
  dsmp_scatter_rows       the final outputs of the owned nodes into the
                          output over the whole domain

Call order and buffers only: no arithmetic happens here.
"""

from typing import List, Optional, Sequence, Tuple

import torch

from ._lib import CAP_KNN, BF16, Dsmp, LayerDesc


class SubdomainInference:
    def __init__(self, lib: Dsmp, desc: LayerDesc, packed: Sequence[torch.Tensor], r: float, cap: int = 0,
                 cap_mode: int = CAP_KNN, seed: int = 0):
        self.lib, self.desc, self.packed = lib, desc, list(packed)
        self.r, self.cap, self.cap_mode, self.seed = r, cap, cap_mode, seed
        self.stats: List[Tuple[int, int, int]] = []

    def run(self, pos: torch.Tensor, attr: torch.Tensor, h0: torch.Tensor,
            boxes: Sequence[Tuple[Sequence[float], Sequence[float]]], overlap: float,
            out: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Reassembled output [n, d] (float32) of the layer stack over the
        boxes; rows of nodes no box owns are left as they are in ``out``
        (zero when ``out`` is not given).  self.stats receives per box
        (owned nodes, sub-domain nodes, edges)."""
        lib, desc = self.lib, self.desc
        n = pos.shape[0]
        dev = lib.device
        if out is None:
            out = torch.zeros(n, desc.d, dtype=torch.float32, device=dev)
        tdt = torch.bfloat16 if desc.dtype == BF16 else torch.float32
        self.stats = []
        for lo, hi in boxes:
            idx, n_own = lib.dsmp_subdomain_select(pos, lo, hi, overlap)
            m = idx.numel()
            if m == 0:
                self.stats.append((0, 0, 0))
                continue
            p = lib.dsmp_gather_rows(pos, idx)
            a = lib.dsmp_gather_rows(attr, idx)
            h = lib.dsmp_gather_rows(h0, idx)
            g = lib.dsmp_radius_graph_build(p, m, self.r, self.cap, self.cap_mode, self.seed)
            y = None
            for packed in self.packed:
                nxt = torch.empty(m, desc.d, dtype=tdt, device=dev)
                y, _ = lib.dsmp_nnconv_forward(desc, packed, g, a, h, h_out_lp=nxt)
                h = nxt
            lib.dsmp_scatter_rows(y[:n_own], idx[:n_own], out)
            self.stats.append((n_own, m, g.n_edges))
        return out
