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
products (``nmg_spmm_epilogue``, ``nmg_spmm_x16_epilogue``); with a trace
every step runs on its own so that each intermediate can be checked, and both
give the same bits.

Each projection runs on a kernel family of its own (``kernels``, name ->
family).  A family that works on prepared operands (``nmg.X16_KERNELS``) gets
them once, when the stack is built, like the packing itself.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import synth

NAMES = ("qkv", "ao", "up", "down")

# the 16 x 16 x 32 binary16 product everywhere (residual sums folded into its
# output stores, GELU as a pass of its own)
DEFAULT_KERNELS = dict.fromkeys(NAMES, "mfma_wide")


@dataclass
class StackLayer:
    packed: dict = field(default_factory=dict)   # name -> (values, indices, layout)
    dense: dict = field(default_factory=dict)    # name -> dense weight (kept on request)
    prepared: dict = field(default_factory=dict)  # name -> prepared operands (x16 families)


class LinearStack:
    def __init__(self, nmg, layers, kernels=None):
        self.nmg = nmg
        self.layers = layers
        self.kernels = dict.fromkeys(NAMES, "auto") if kernels is None else dict(kernels)
        for layer in layers:
            for name, kernel in self.kernels.items():
                if kernel in nmg.X16_KERNELS and name not in layer.prepared:
                    v, idx, L = layer.packed[name]
                    layer.prepared[name] = nmg.x16_prepare(v, idx, L)

    @classmethod
    def from_workload(cls, workload: int, nmg, n=2, m=8, g=8, n_layers=synth.BERT_LAYERS,
                      tokens=synth.BERT_TOKENS, keep_dense=True, device="cuda:0",
                      kernels=DEFAULT_KERNELS):
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
        return cls(nmg, layers, kernels)

    def linear(self, layer: StackLayer, name: str, x: torch.Tensor):
        v, idx, L = layer.packed[name]
        if name in layer.prepared:
            return self.nmg.spmm_x16_epilogue(L, layer.prepared[name], x)
        return self.nmg.spmm(v, idx, x, L, self.kernels[name])

    def fused(self, layer: StackLayer, name: str, x: torch.Tensor, epilogue: str, r=None):
        v, idx, L = layer.packed[name]
        if name in layer.prepared:
            if epilogue == "gelu":
                # measured: the product, then the table GELU on its output
                # while that is still in the caches, is at least as fast as
                # the GELU folded into the product's stores
                p = self.linear(layer, name, x)
                return self.nmg.gelu(p, out=p)
            return self.nmg.spmm_x16_epilogue(L, layer.prepared[name], x, epilogue, r)
        return self.nmg.spmm_epilogue(v, idx, x, L, epilogue, r, self.kernels[name])

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

    def capture(self, x: torch.Tensor):
        """The forward on x captured in a HIP graph: returns (graph, y), where
        graph.replay() recomputes y from the current contents of x with no
        host-side launches.  Every step is a library kernel that allocates
        nothing and writes no memory with a memset; torch's graph pool holds
        the intermediate buffers."""
        side = torch.cuda.Stream(device=x.device)
        side.wait_stream(torch.cuda.current_stream(x.device))
        with torch.cuda.stream(side):
            for _ in range(2):   # launch shapes cached, torch's pool warmed
                self.forward(x)
        torch.cuda.current_stream(x.device).wait_stream(side)
        torch.cuda.synchronize(x.device)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            y = self.forward(x)
        return graph, y
