"""A stack of DiT-block linears on the hot path, optionally replayed as one
HIP graph.

Every linear is clq_rotate_quant_act + clq_w4a4_linear (argument marshalling
only; the arithmetic runs in the library's kernels).  Blocks chain
qkv -> proj -> fc1 -> fc2 -> next block's qkv; proj reads the first `hidden`
columns of the qkv output through a row stride (the attention between them
is not part of this path).  Weights are quantized once at construction and
stay resident; activation buffers are allocated once and reused by every
block, so a captured graph replays the whole stack with no host work and no
allocation: two launches per linear, or one where the rotate+quantize of the
layer's input is folded into its GEMM launch (clq_w4a4_rq_linear).

Swap vectors (the `s` of G = S.H, Sec. 3.3, one per layer input) are either
gathered by each rotate+quant, or folded upstream: the layer that produces an
input gets its output channels (weight rows and bias) reordered by that
input's `s` once, at construction, so its output already comes out gathered
and the consumer's rotate+quant reads it in order.  Each output channel is
computed independently, so the folded stack produces the same bits.  The
stack's first input has no producer inside the stack and keeps its gather.

codes="fp6" runs every linear on the fp6 storage of the same codes
(clq_rotate_quant_act_f6 + clq_w4a4_linear_f6); the fp16 outputs are the
same bits as with int4 storage.

Paper: "CLQ" (arXiv 2509.24416) -- the method quantizes every linear of the
DiT blocks (Sec. 4.1, W4A4), with the online rotation of Sec. 3.3 in front of
each.
"""
import torch

from . import (clq_act_bytes, clq_act_bytes_f6, clq_quantize_weights, clq_quantize_weights_f6,
               clq_rotate_quant_act, clq_rotate_quant_act_f6, clq_w4a4_linear, clq_w4a4_linear_f6,
               clq_w4a4_rq_linear, clq_w4a4_workspace_bytes)

LAYERS = ("qkv", "proj", "fc1", "fc2")


class DiTStack:
    """weights: one dict per block, {"qkv": (W, b), "proj": ..., "fc1": ...,
    "fc2": ...}, fp16 device tensors in torch Linear layout (b may be None).
    M tokens per step, Hadamard block size `block`.  perm: one swap vector
    (int32 [K]) for every layer input, or perms: one dict per block mapping a
    layer name to its input's swap vector (or None).  fold: reorder each
    producer's output channels by its consumer's swap vector instead of
    gathering in the consumer's rotate+quant.  codes: "int4" (default) or
    "fp6" (the codes stored as fp6 for the fp6 matrix instructions; not with
    fuse)."""

    def __init__(self, weights, M, block=64, perm=None, perms=None, fold=False, fuse=False, codes="int4"):
        if codes not in ("int4", "fp6"):
            raise ValueError(f"codes must be 'int4' or 'fp6', not {codes!r}")
        if codes == "fp6" and fuse:
            raise ValueError("the fused launch takes int4 codes only")
        self.codes = codes
        self.M, self.block = M, block
        # fuse: each layer's rotate+quantize and GEMM through clq_w4a4_rq_linear
        # (one launch where its schedule allows; inputs that still gather by
        # a swap vector take the two launches).  Off by default: on MI355X the
        # separate launches are faster at every stack size measured.
        self.fuse = fuse
        W0 = weights[0]["qkv"][0]
        self.hidden = W0.shape[1]
        self.mlp = weights[0]["fc1"][0].shape[0]
        dev = W0.device
        nb = len(weights)
        if perms is None:
            perms = [{name: perm for name in LAYERS} for _ in range(nb)]
        self.fold = fold
        # the swap vector each layer's rotate+quant still gathers by
        self.gather = [{name: perms[j][name] for name in LAYERS} for j in range(nb)]
        # output-channel order of each layer (None: natural)
        rows = [{name: None for name in LAYERS} for _ in range(nb)]
        if fold:
            for j in range(nb):
                for name in LAYERS:
                    s = perms[j][name]
                    if s is None or (j == 0 and name == "qkv"):
                        continue
                    pj, pname = self._producer(j, name)
                    if pname == "qkv":   # proj reads the first `hidden` qkv columns
                        rest = torch.arange(self.hidden, 3 * self.hidden, dtype=s.dtype, device=s.device)
                        rows[pj][pname] = torch.cat([s, rest])
                    else:
                        rows[pj][pname] = s
                    self.gather[j][name] = None
        self.blocks = []
        for j, blk in enumerate(weights):
            q = {}
            for name in LAYERS:
                W, b = blk[name]
                r = rows[j][name]
                if r is not None:   # one-time reorder of the layer's parameters
                    W = W.index_select(0, r.long()).contiguous()
                    b = None if b is None else b.index_select(0, r.long()).contiguous()
                quant = clq_quantize_weights_f6 if codes == "fp6" else clq_quantize_weights
                q[name] = (quant(W, block, perm=perms[j][name]), b)
            self.blocks.append(q)
        h, f = self.hidden, self.mlp
        f16 = dict(dtype=torch.float16, device=dev)
        self.x_in = torch.empty((M, h), **f16)
        self.out = {"qkv": torch.empty((M, 3 * h), **f16), "proj": torch.empty((M, h), **f16),
                    "fc1": torch.empty((M, f), **f16), "fc2": torch.empty((M, h), **f16)}
        act_bytes = clq_act_bytes_f6 if codes == "fp6" else clq_act_bytes
        self.xq = {h: torch.empty(act_bytes(M, h), dtype=torch.uint8, device=dev),
                   f: torch.empty(act_bytes(M, f), dtype=torch.uint8, device=dev)}
        self.xs = torch.empty(M, dtype=torch.float32, device=dev)
        # the GEMM workspace of this stack: every launch (eager or replayed)
        # runs in the order of one stream, so one is enough
        self.ws = torch.zeros(clq_w4a4_workspace_bytes(), dtype=torch.uint8, device=dev)
        self.graph = None

    @staticmethod
    def _producer(j, name):
        """The layer whose output is the input of (j, name) (j >= 0)."""
        if name == "qkv":
            return j - 1, "fc2"
        return j, {"proj": "qkv", "fc1": "proj", "fc2": "fc1"}[name]

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
                if self.codes == "fp6":
                    clq_rotate_quant_act_f6(x, self.block, perm=self.gather[j][name], out=xq, scale_out=self.xs)
                    clq_w4a4_linear_f6(xq, self.xs, qw, b, out=self.out[name])
                elif self.fuse and self.gather[j][name] is None:
                    clq_w4a4_rq_linear(x, self.block, qw, b, Xq_out=xq, scale_out=self.xs, out=self.out[name],
                                       workspace=self.ws)
                else:
                    clq_rotate_quant_act(x, self.block, perm=self.gather[j][name], out=xq, scale_out=self.xs)
                    clq_w4a4_linear(xq, self.xs, qw, b, out=self.out[name], workspace=self.ws)
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
