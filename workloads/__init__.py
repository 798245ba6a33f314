"""Seeded synthetic inputs and layer shapes for the W4A4 DiT linear.

This module holds the input recipe only: no step of the method's arithmetic
lives here.  It is the one module that both the GPU-side tests/bench and the
CPU oracle use, so that both see the very same fp16 tensors.

The trained PixArt-alpha / Open-Sora weights and their calibration data are
not available, so seeded draws stand in for them.  The paper evaluates
PixArt-alpha and Open-Sora 1.2 (Sec. 4.1) but states neither their depth nor
their width; the shapes here are the workload definitions this library is
measured on (hidden 1152 with 28 blocks for the PixArt-style and video
blocks, a FLUX-style width 3072 block), not figures from the paper.
Activation laws plant the per-channel outliers that motivate OBS
(Sec. 1 and Sec. 3.3: a few channels with much larger magnitude, stable
across tokens).

Laws (all sampled in fp32 with numpy's PCG64, then rounded to fp16 with
round-to-nearest-even):
  L1  Z ~ N(0, 1); round(frac * K) channels, drawn without replacement, are
      multiplied by exp(U(ln lo, ln hi)) (frac 1%, factor 20-100x).
  L2  as L1 with frac 0.5%, factor 50-200x, and each token row multiplied by
      exp(0.5 * N(0, 1)) (a per-token lognormal(0, 0.5) scale).
  W   N(0, 1) / sqrt(K)      bias  0.1 * N(0, 1)
"""
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Layer:
    name: str
    M: int
    K: int
    N: int
    block: int
    law: str = "L1"
    seed: int = 0


@dataclass(frozen=True)
class Workload:
    name: str
    layers: tuple = field(default_factory=tuple)

    @property
    def ops(self):
        return sum(2 * l.M * l.N * l.K for l in self.layers)


def _dit_block(prefix, M, hidden, mlp, block, law, seed0):
    shapes = [("qkv", hidden, 3 * hidden), ("proj", hidden, hidden),
              ("fc1", hidden, mlp), ("fc2", mlp, hidden)]
    return tuple(Layer(f"{prefix}.{n}", M, K, N, block, law, seed0 + 10 * i)
                 for i, (n, K, N) in enumerate(shapes))


# single linear, 256 tokens, PixArt width
C1 = Workload("single_linear_m256_k1152_n1152_b64",
              (Layer("lin", 256, 1152, 1152, 64, "L1", 0),))
# PixArt-style block linears: 1024^2 image (4096 tokens) x CFG batch 2
C2 = Workload("pixart_block_m8192_h1152_b64",
              _dit_block("pixart", 8192, 1152, 4608, 64, "L1", 200))
# FLUX-style width 3072: 4096 image + 512 text tokens
C3 = Workload("flux_block_m4608_h3072_b128",
              _dit_block("flux", 4608, 3072, 12288, 128, "L2", 300))
# video DiT: 16 latent frames x 30 x 45 patches x batch 2
C4 = Workload("video_block_m43200_h1152_b64",
              _dit_block("video", 43200, 1152, 4608, 64, "L1", 400))

WORKLOADS = {w.name: w for w in (C1, C2, C3, C4)}


def dit_stack(nblocks=28, M=4096, block=64, hidden=1152, mlp=4608):
    """A stack of DiT blocks' linears (qkv, proj, fc1, fc2 per block) for the
    multi-layer path: layer i (block i // 4) draws its weights with seed
    500 + 10 i + 1 and bias with 500 + 10 i + 2; the stack input is L1 with
    seed 500.  Between layers the previous output feeds the next input (proj
    reads the first `hidden` columns of the qkv output, standing in for the
    attention that is not part of this path), so only the stack input has
    planted outliers."""
    shapes = [("qkv", hidden, 3 * hidden), ("proj", hidden, hidden),
              ("fc1", hidden, mlp), ("fc2", mlp, hidden)]
    layers = []
    for j in range(nblocks):
        for t, (n, K, N) in enumerate(shapes):
            i = 4 * j + t
            layers.append(Layer(f"blk{j}.{n}", M, K, N, block, "L1", 500 + 10 * i))
    return Workload(f"dit_stack_{nblocks}x4_m{M}_h{hidden}_b{block}", tuple(layers))


def law_params(law):
    if law == "L1":
        return dict(frac=0.01, lo=20.0, hi=100.0, token_sigma=0.0)
    if law == "L2":
        return dict(frac=0.005, lo=50.0, hi=200.0, token_sigma=0.5)
    if law == "N":
        return dict(frac=0.0, lo=1.0, hi=1.0, token_sigma=0.0)
    raise ValueError(law)


def activations(M, K, law="L1", seed=0):
    """fp16 [M][K] activations with planted outlier channels."""
    p = law_params(law)
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, K), dtype=np.float32)
    n_out = int(round(p["frac"] * K))
    if n_out:
        ch = rng.choice(K, size=n_out, replace=False)
        fac = np.exp(rng.uniform(np.log(p["lo"]), np.log(p["hi"]), size=n_out)).astype(np.float32)
        x[:, ch] *= fac[None, :]
    if p["token_sigma"]:
        tok = np.exp(p["token_sigma"] * rng.standard_normal(M, dtype=np.float32))
        x *= tok[:, None]
    return x.astype(np.float16)


def weights(N, K, seed=1):
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((N, K), dtype=np.float32) / np.float32(np.sqrt(K))
    return w.astype(np.float16)


def bias(N, seed=2):
    rng = np.random.default_rng(seed)
    return (np.float32(0.1) * rng.standard_normal(N, dtype=np.float32)).astype(np.float16)


def calibration(B, N, D, law="L1", seed=0):
    """fp16 [B][N][D] calibration activations for the OBS derivation: the
    outlier channels and their factors are drawn once and shared by every
    sample and token (the paper observes statistics that are stable along
    the batch); the Gaussian body (and, for L2, the per-token scale) is drawn
    per sample."""
    p = law_params(law)
    rng = np.random.default_rng(seed)
    n_out = int(round(p["frac"] * D))
    ch = rng.choice(D, size=n_out, replace=False) if n_out else np.zeros(0, np.int64)
    fac = np.exp(rng.uniform(np.log(p["lo"]), np.log(p["hi"]), size=n_out)).astype(np.float32)
    out = np.empty((B, N, D), np.float16)
    for b in range(B):
        x = rng.standard_normal((N, D), dtype=np.float32)
        x[:, ch] *= fac[None, :]
        if p["token_sigma"]:
            x *= np.exp(p["token_sigma"] * rng.standard_normal(N, dtype=np.float32))[:, None]
        out[b] = x.astype(np.float16)
    return out


def calibration_outliers(D, law="L1", seed=0):
    """The planted outlier channels of calibration(B, N, D, law, seed)."""
    p = law_params(law)
    rng = np.random.default_rng(seed)
    n_out = int(round(p["frac"] * D))
    return np.sort(rng.choice(D, size=n_out, replace=False)) if n_out else np.zeros(0, np.int64)


def random_perm(K, seed=3):
    """A seeded gather vector s (a permutation of 0..K-1) for tests of the
    optional column swap."""
    rng = np.random.default_rng(seed)
    return rng.permutation(K).astype(np.int32)


def layer_inputs(layer):
    """(X fp16 [M][K], W fp16 [N][K], bias fp16 [N]) for one layer."""
    return (activations(layer.M, layer.K, layer.law, layer.seed),
            weights(layer.N, layer.K, layer.seed + 1),
            bias(layer.N, layer.seed + 2))
