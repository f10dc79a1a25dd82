"""BERT-base encoder linear stack on n:m:g weights (the fp16 workload).

Each of the 12 layers holds four sparse projections: QKV (2304 x 768),
attention-out (768 x 768), FFN up (3072 x 768) and FFN down (768 x 3072),
packed by ``nmg.compress``.  Attention itself is omitted: the attention-out
projection reads the V third of the QKV output.  Residual sums follow BERT's
encoder block (without LayerNorm):

    h  = x + AO(V(x))
    x' = h + Down(GELU(Up(h)))

Activations are features x tokens (768 x 4096), binary16 in memory, binary32
inside every kernel.  Every step runs in libnmg's kernels; torch only holds
the buffers.  By default GELU and the residual sums are folded into the
products (``nmg_spmm_epilogue``); with a trace every step runs on its own so
that each intermediate can be checked, and both give the same bits.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import synth

NAMES = ("qkv", "ao", "up", "down")


@dataclass
class StackLayer:
    packed: dict = field(default_factory=dict)   # name -> (values, indices, layout)
    dense: dict = field(default_factory=dict)    # name -> dense weight (kept on request)


class LinearStack:
    def __init__(self, nmg, layers):
        self.nmg = nmg
        self.layers = layers

    @classmethod
    def from_workload(cls, workload: int, nmg, n=2, m=8, g=8, n_layers=synth.BERT_LAYERS,
                      tokens=synth.BERT_TOKENS, keep_dense=True, device="cuda:0"):
        lins = synth.bert_stack_layers(tokens, n, m, g)
        layers = []
        for li in range(n_layers):
            layer = StackLayer()
            for j, lin in enumerate(lins):
                W = synth.normal((lin.M, lin.K), synth.seed_for(workload, 4 * li + j, "W"),
                                 synth.W_STD, lin.dtype).to(device)
                layer.packed[lin.name] = nmg.compress(W, lin.n, lin.m, lin.g)
                if keep_dense:
                    layer.dense[lin.name] = W
            layers.append(layer)
        return cls(nmg, layers)

    def linear(self, layer: StackLayer, name: str, x: torch.Tensor, out=None):
        v, idx, L = layer.packed[name]
        if out is None:
            return self.nmg.spmm(v, idx, x, L)
        self.nmg.spmm_into(L, v, idx, x, out)
        return out

    def fused(self, layer: StackLayer, name: str, x: torch.Tensor, epilogue: str, r=None):
        v, idx, L = layer.packed[name]
        return self.nmg.spmm_epilogue(v, idx, x, L, epilogue, r)

    def forward_layer(self, layer: StackLayer, x: torch.Tensor, trace: dict | None = None):
        nmg = self.nmg
        d = x.shape[0]
        qkv = self.linear(layer, "qkv", x)
        vpart = qkv[2 * d:3 * d]                 # rows of V: a contiguous view
        if trace is None:                        # GELU and residuals fused into the products
            h = self.fused(layer, "ao", vpart, "add", x)
            gl = self.fused(layer, "up", h, "gelu")
            return self.fused(layer, "down", gl, "add", h)
        a = self.linear(layer, "ao", vpart)
        h = nmg.add(x, a)
        u = self.linear(layer, "up", h)
        gl = nmg.gelu(u)
        dn = self.linear(layer, "down", gl)
        out = nmg.add(h, dn)
        trace["linear"] = {"qkv": (x, qkv), "ao": (vpart, a), "up": (h, u), "down": (gl, dn)}
        trace["gelu"] = (u, gl)
        trace["add"] = [(x, a, h), (h, dn, out)]
        return out

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        for layer in self.layers:
            x = self.forward_layer(layer, x)
        return x
