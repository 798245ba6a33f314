"""Single-layer CLPS clip search on the CPU.

TEST INFRASTRUCTURE ONLY (same rule as the rest of ``oracle``): only
``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use it; it shares no code with the GPU path.

Paper: "CLQ" (arXiv 2509.24416), Sec. 3.4 (Cross-Layer Parameter Searching):
a grid search over the quantizer bounds of the layer being optimised, between
quantiles of its weights (beta = 0, gamma = 0.01 in Sec. 4.1, one percentile
for all channels of a matrix), minimising the squared Frobenius norm of the
output error, Eq. (3).  The single-layer form here takes the layer's own
output as the target (the cross-layer target needs a whole model).

Readings (where the paper is silent):
  * Symmetric bounds: the searched quantity is the clip ratio alpha of the
    hot path's weight quantizer (row bound = alpha * max|w~_row|).
  * Window: alpha in [alpha_lo, 1], alpha_lo = min over rows of
    Q / max|w~_row|, Q the order statistic of |w~_row| with
    l = floor(gamma (K - 1)) values above it (beta = 0 gives the top, 1).
  * Grid: G points, alpha_i = 1 - ((1 - alpha_lo) * (G - 1 - i)) / (G - 1) in
    fp32, left to right (alpha_{G-1} = 1 exactly); G = 1 gives alpha = 1.
  * Objective: e(alpha) = sum over (m, n) of (Y0 - acc * x_scale * w_scale)^2
    in fp64, Y0 = X W^T the unquantised output (bias cancels), acc the exact
    integer sum of the quantized codes.
  * Choice: the smallest e, ties to the lower index.
"""
import math

import numpy as np

import oracle


def order_index(K, gamma):
    """Position (ascending, 0-based) of the upper gamma order statistic of K
    values: l = floor(gamma (K - 1)) values lie above it, gamma taken as an
    fp32 value and the product formed in fp64."""
    return K - 1 - int(math.floor(float(np.float32(gamma)) * (K - 1)))


def alpha_floor(W, block, perm=None, gamma=0.01):
    """min over rows of Q_row / max_row on the rotated rows (1 for an all-zero
    row), fp32."""
    wt = np.abs(oracle.rotate(W, block, perm))
    K = wt.shape[1]
    srt = np.sort(wt, axis=1)
    q = srt[:, order_index(K, gamma)]
    mx = srt[:, K - 1]
    with np.errstate(divide="ignore", invalid="ignore"):
        r = (q / mx).astype(np.float32)
    r = np.where(mx == 0, np.float32(1.0), r).astype(np.float32)
    return np.float32(r.min())


def alpha_grid(alpha_lo, G):
    """The G candidate clip ratios (fp32, ascending, the last exactly 1)."""
    if G == 1:
        return np.ones(1, np.float32)
    lo = np.float32(alpha_lo)
    t = np.float32(1.0) - lo
    out = np.empty(G, np.float32)
    for i in range(G):
        u = np.float32(t * np.float32(G - 1 - i))
        v = np.float32(u / np.float32(G - 1))
        out[i] = np.float32(np.float32(1.0) - v)
    return out


def errors(X, W, Y0, block, alphas, perm=None, wbits=4, abits=4):
    """e(alpha) for every candidate (fp64), with the activations quantized
    once."""
    _, xc, xs = oracle.quantize_act(X, block, perm, abits)
    Y0 = np.asarray(Y0, np.float64)
    out = np.empty(len(alphas), np.float64)
    for i, a in enumerate(alphas):
        _, wc, ws = oracle.quantize_weights(W, block, perm, float(a), wbits)
        acc = oracle.gemm_i32(xc, wc).astype(np.float64)
        p = acc * xs.astype(np.float64)[:, None] * ws.astype(np.float64)[None, :]
        out[i] = float(np.sum((Y0 - p) ** 2))
    return out


def search(X, W, Y0, block, perm=None, gamma=0.01, G=20, wbits=4, abits=4):
    """The whole single-layer search: returns (alphas, errors, best index)."""
    al = alpha_grid(alpha_floor(W, block, perm, gamma), G)
    e = errors(X, W, Y0, block, al, perm, wbits, abits)
    return al, e, int(np.argmin(e))
