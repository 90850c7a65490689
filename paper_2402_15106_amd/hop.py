"""One training step of the hop loop of Algorithm 1 on one sub-domain,
composed from the library's calls (binding level: buffers and call order
only; every arithmetic step runs in the HIP library).

    v_L   = N_e(v0)                                encoder (eq. (i))
    for each hop l:
        edge attributes x_e = v_i - v_j of the current values (eq. (iv);
        the input values at the first hop), read by the layer itself
        v_L   = v_L + K(x, v_L)                     layer with residual (eq. (ii))
        v     = N_d(v_L)                            decoder (eq. (iii))
    loss  = MSE over the interior rows of v against Y

The backward pass runs the hops in reverse: decoder backward (its input
gradient added onto the latent gradient coming back from the next hop), layer
backward (parameter gradients summed over the hops, the attribute gradient
becoming the previous hop's decoder output gradient), and the encoder
backward last.  The graph joins the n nodes with every node a destination.
"""

from dataclasses import dataclass

import torch

from . import _lib as L


@dataclass
class HopShapes:
    n: int            # nodes (all destinations)
    dim: int          # spatial dimension; node values have dim + 1 components
    d: int            # latent width
    h1: int
    h2: int
    hid_enc: int      # encoder hidden width
    hid_dec: int      # decoder hidden width
    dtype: int        # F32 or BF16 layer operands
    hops: int


class HopStep:
    """Buffers for one sub-domain and one hop count; ``step`` runs forward,
    loss and backward and returns (loss [1] device tensor, grads)."""

    def __init__(self, lib: "L.Dsmp", graph: "L.Graph", s: HopShapes):
        self.lib, self.g, self.s = lib, graph, s
        dev = lib.device
        f32 = dict(dtype=torch.float32, device=dev)
        tdt = torch.bfloat16 if s.dtype == L.BF16 else torch.float32
        c = s.dim + 1
        self.conv = L.layer_desc(s.dim, s.d, s.h1, s.h2, s.dtype, L.ACT_IDENTITY, 1, L.ATTR_DIFF)
        self.enc = L.MlpDesc(c, s.hid_enc, s.d)
        self.dec = L.MlpDesc(s.d, s.hid_dec, c)
        n = s.n
        self.vL0 = torch.empty(n, s.d, **f32)
        self.h_in = [torch.empty(n, s.d, dtype=tdt, device=dev) for _ in range(s.hops)]
        self.out = [torch.empty(n, s.d, **f32) for _ in range(s.hops)]
        self.v = [torch.empty(n, c, **f32) for _ in range(s.hops)]
        sb, fb, bb = lib.dsmp_nnconv_workspace(self.conv, graph)
        self.saved = [torch.empty(max(sb, 256), dtype=torch.uint8, device=dev) for _ in range(s.hops)]
        self.fws = torch.empty(max(fb, 256), dtype=torch.uint8, device=dev)
        self.bws = torch.empty(max(bb, 256), dtype=torch.uint8, device=dev)
        es, _ = lib.dsmp_mlp_workspace(self.enc, n)
        ds, _ = lib.dsmp_mlp_workspace(self.dec, n)
        self.enc_saved = torch.empty(max(es, 256), dtype=torch.uint8, device=dev)
        self.dec_saved = [torch.empty(max(ds, 256), dtype=torch.uint8, device=dev) for _ in range(s.hops)]
        self.gv = [torch.empty(n, c, **f32) for _ in range(2)]
        self.glat = [torch.empty(n, s.d, **f32) for _ in range(2)]
        self.loss = torch.empty(1, **f32)

    def forward(self, enc_params: dict, packed, dec_params: dict, v0):
        lib, s = self.lib, self.s
        bf = s.dtype == L.BF16
        lib.dsmp_mlp_forward(self.enc, enc_params, v0, y=self.vL0, y_bf16=self.h_in[0] if bf else None,
                             saved=self.enc_saved)
        if not bf and s.hops:
            self.h_in[0] = self.vL0
        attr = v0
        for l in range(s.hops):
            nxt = self.h_in[l + 1] if (bf and l + 1 < s.hops) else None
            lib.dsmp_nnconv_forward(self.conv, packed, self.g, attr, self.h_in[l], h_out=self.out[l], h_out_lp=nxt,
                                    saved=self.saved[l], ws=self.fws)
            if not bf and l + 1 < s.hops:
                self.h_in[l + 1] = self.out[l]
            lib.dsmp_mlp_forward(self.dec, dec_params, self.out[l], y=self.v[l], saved=self.dec_saved[l])
            attr = self.v[l]
        return self.v[s.hops - 1] if s.hops else v0

    def step(self, enc_params: dict, packed, dec_params: dict, v0, Y, mask):
        """Forward, loss, backward.  mask: uint8 [n] interior rows."""
        lib, s = self.lib, self.s
        v = self.forward(enc_params, packed, dec_params, v0)
        gv = self.gv[0]
        lib.dsmp_masked_mse(v, Y, mask, loss=self.loss, grad=gv)
        f32 = dict(dtype=torch.float32, device=lib.device)
        d, c = s.d, s.dim + 1
        de = c
        conv_g = {"dW1": torch.empty(s.h1, de, **f32), "db1": torch.empty(s.h1, **f32),
                  "dW2": torch.empty(s.h2, s.h1, **f32), "db2": torch.empty(s.h2, **f32),
                  "dW3": torch.empty(d * d, s.h2, **f32), "db3": torch.empty(d * d, **f32),
                  "dWr": torch.empty(d, d, **f32), "dbr": torch.empty(d, **f32)}
        dec_g = enc_g = None
        glat = None          # gradient with respect to the next hop's latent input
        for l in reversed(range(s.hops)):
            G = self.glat[l % 2]
            first = l == s.hops - 1
            # decoder of hop l: its input gradient goes into G (added onto the latent gradient)
            if first:
                dec_g = lib.dsmp_mlp_backward(self.dec, dec_params, self.out[l], self.dec_saved[l], gv, grad_x=G)
            else:
                lib.dsmp_mlp_backward(self.dec, dec_params, self.out[l], self.dec_saved[l], gv, grad_x=glat,
                                      grads=dec_g, flags=L.GRAD_ACCUMULATE | L.GRAD_X_ACCUMULATE)
                G = glat
            attr = self.v[l - 1] if l > 0 else v0
            gnext = self.gv[(s.hops - l) % 2]
            conv_g["dattr"] = gnext if l > 0 else None
            gh = self.glat[(l + 1) % 2]
            lib.dsmp_nnconv_backward(self.conv, packed, self.g, attr, self.h_in[l], self.saved[l], G, grad_h=gh,
                                     grads=conv_g, flags=0 if first else L.GRAD_ACCUMULATE, ws=self.bws)
            glat, gv = gh, gnext
        conv_g.pop("dattr", None)
        if s.hops:
            enc_g = lib.dsmp_mlp_backward(self.enc, enc_params, v0, self.enc_saved, glat)
        return self.loss, {"enc": enc_g, "conv": conv_g, "dec": dec_g}
