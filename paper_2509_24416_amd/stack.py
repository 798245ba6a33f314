"""A stack of DiT-block linears on the hot path, optionally replayed as one
HIP graph.

Every linear is clq_rotate_quant_act + clq_w4a4_linear (argument marshalling
only; the arithmetic runs in the library's kernels).  Blocks chain
qkv -> proj -> fc1 -> fc2 -> next block's qkv; proj reads the first `hidden`
columns of the qkv output through a row stride (the attention between them
is not part of this path).  Weights are quantized once at construction and
stay resident; activation buffers are allocated once and reused by every
block, so a captured graph replays the whole stack (2 launches per linear)
with no host work and no allocation.

Paper: "CLQ" (arXiv 2509.24416) -- the method quantizes every linear of the
DiT blocks (Sec. 4.1, W4A4), with the online rotation of Sec. 3.3 in front of
each.
"""
import torch

from . import (clq_act_bytes, clq_quantize_weights, clq_rotate_quant_act, clq_w4a4_linear)

LAYERS = ("qkv", "proj", "fc1", "fc2")


class DiTStack:
    """weights: one dict per block, {"qkv": (W, b), "proj": ..., "fc1": ...,
    "fc2": ...}, fp16 device tensors in torch Linear layout (b may be None).
    M tokens per step, Hadamard block size `block`."""

    def __init__(self, weights, M, block=64, perm=None):
        self.M, self.block = M, block
        W0 = weights[0]["qkv"][0]
        self.hidden = W0.shape[1]
        self.mlp = weights[0]["fc1"][0].shape[0]
        dev = W0.device
        self.blocks = []
        for blk in weights:
            q = {}
            for name in LAYERS:
                W, b = blk[name]
                q[name] = (clq_quantize_weights(W, block, perm=perm), b)
            self.blocks.append(q)
        self.perm = perm
        h, f = self.hidden, self.mlp
        f16 = dict(dtype=torch.float16, device=dev)
        self.x_in = torch.empty((M, h), **f16)
        self.out = {"qkv": torch.empty((M, 3 * h), **f16), "proj": torch.empty((M, h), **f16),
                    "fc1": torch.empty((M, f), **f16), "fc2": torch.empty((M, h), **f16)}
        self.xq = {h: torch.empty(clq_act_bytes(M, h), dtype=torch.uint8, device=dev),
                   f: torch.empty(clq_act_bytes(M, f), dtype=torch.uint8, device=dev)}
        self.xs = torch.empty(M, dtype=torch.float32, device=dev)
        self.graph = None

    def _input(self, j, name):
        if name == "qkv":
            return self.x_in if j == 0 else self.out["fc2"]
        if name == "proj":
            return self.out["qkv"][:, :self.hidden]
        if name == "fc1":
            return self.out["proj"]
        return self.out["fc1"]

    def _run(self, taps=None):
        for j, blk in enumerate(self.blocks):
            for name in LAYERS:
                qw, b = blk[name]
                x = self._input(j, name)
                xq = self.xq[qw.K]
                clq_rotate_quant_act(x, self.block, perm=self.perm, out=xq, scale_out=self.xs)
                clq_w4a4_linear(xq, self.xs, qw, b, out=self.out[name])
                if taps is not None and (j, name) in taps:
                    taps[(j, name)] = (x.clone(), self.out[name].clone())

    def forward(self, x=None, taps=None):
        """Eager run.  x: fp16 [M, hidden] copied to the stack input (None:
        keep the current input).  taps: optional dict whose keys (block,
        layer) receive (input, output) copies.  Returns the last fc2 output
        buffer."""
        if x is not None:
            self.x_in.copy_(x)
        self._run(taps)
        return self.out["fc2"]

    def capture(self):
        """Captures the whole stack as one graph (after an eager run, so that
        every kernel is loaded and every one-time attribute set)."""
        self._run()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self._run()
        self.graph = g
        return g

    def replay(self, x=None):
        if x is not None:
            self.x_in.copy_(x)
        self.graph.replay()
        return self.out["fc2"]

    @property
    def ops(self):
        """Integer ops of one pass: sum over the linears of 2 M N K."""
        h, f, M = self.hidden, self.mlp, self.M
        return len(self.blocks) * 2 * M * (h * 3 * h + h * h + h * f + f * h)
