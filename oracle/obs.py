"""OBS calibration on the CPU: channel outlier scores and the column swap.

TEST INFRASTRUCTURE ONLY (same rule as the rest of ``oracle``): only
``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use it; it shares no code with the GPU path.

Paper: "CLQ" (arXiv 2509.24416), Sec. 3.3 (Orthogonal-Based Smoothing):
  * Data preparing: calibration activations X [B, N, D] are averaged over the
    batch, giving a mean matrix of N tokens x D channels.
  * Outlier detection: one outlier score per channel (the paper keeps the
    absolute maximum; its ablation, Sec. 4.2 "Choice of Outlier Metric",
    also tries percentile (1%, 99%), top-k mean with k = 1%, range and peak
    average ratio); channels are ranked by score, the top half moves to the
    left half of the columns and the rest to the right.  No full descending
    order is needed inside a half, so each half keeps the channels' original
    order.  The swap is stored as a gather vector s: x'[k] = x[s[k]].

Arithmetic (the readings where the paper is silent): every value is IEEE
fp32.  The batch mean adds the B samples in batch order and divides the sum
by B once (correctly rounded).  Sums over tokens use pairwise summation: the
values, zero-padded to a power-of-two count, are added as a balanced binary
tree (element i + element i + half, halving until one value is left).
Percentiles are order statistics (no interpolation).  Ranking: higher score
first, equal scores by lower channel index.
"""
import numpy as np

METRICS = ("absmax", "range", "par", "topk_mean", "percentile")
ABSMAX, RANGE, PAR, TOPK_MEAN, PERCENTILE = range(5)


def batch_mean(X):
    """Mean over the batch of X [B, N, D] (fp16 or fp32) as fp32 [N, D]: the
    B samples added one after another in fp32, then one division by B."""
    X = np.asarray(X)
    B = X.shape[0]
    acc = np.zeros(X.shape[1:], np.float32)
    for b in range(B):
        acc = (acc + X[b].astype(np.float32)).astype(np.float32)
    return (acc / np.float32(B)).astype(np.float32)


def pairwise_sum(v, axis=0):
    """fp32 sum along ``axis`` by a balanced binary tree: zero-pad to a power
    of two, then repeatedly add the upper half onto the lower half."""
    v = np.moveaxis(np.asarray(v, np.float32), axis, 0)
    n = v.shape[0]
    p = 1
    while p < n:
        p *= 2
    w = np.zeros((p,) + v.shape[1:], np.float32)
    w[:n] = v
    while p > 1:
        p //= 2
        w = (w[:p] + w[p:2 * p]).astype(np.float32)
    return w[0]


def topk_count(N):
    """k of the top-k mean: 1% of the tokens, rounded half up, at least 1."""
    return max(1, (N + 50) // 100)


def percentile_ranks(N):
    """Ascending order-statistic positions of the 1% and 99% percentiles:
    floor(0.01 (N - 1)) and its mirror N - 1 - floor(0.01 (N - 1))."""
    lo = (N - 1) // 100
    return lo, N - 1 - lo


def channel_scores(S, metric):
    """Outlier score per channel of the mean matrix S [N, D] (fp32):
      absmax      max_n |S[n, d]|
      range       max_n S[n, d] - min_n S[n, d]
      par         max_n |S| / (pairwise_sum_n |S| / N)      (0 if the sum is 0)
      topk_mean   pairwise sum of the k largest |S|, in descending order, / k
      percentile  S at the 99% order statistic - S at the 1% one
    Returns fp32 [D]."""
    S = np.asarray(S, np.float32)
    N, D = S.shape
    if isinstance(metric, str):
        metric = METRICS.index(metric)
    A = np.abs(S)
    if metric == ABSMAX:
        return A.max(axis=0).astype(np.float32)
    if metric == RANGE:
        return (S.max(axis=0) - S.min(axis=0)).astype(np.float32)
    if metric == PAR:
        peak = A.max(axis=0)
        mean = (pairwise_sum(A, 0) / np.float32(N)).astype(np.float32)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = (peak / mean).astype(np.float32)
        return np.where(mean == 0, np.float32(0), r).astype(np.float32)
    if metric == TOPK_MEAN:
        k = topk_count(N)
        top = -np.sort(-A, axis=0)[:k]          # descending
        return (pairwise_sum(top, 0) / np.float32(k)).astype(np.float32)
    if metric == PERCENTILE:
        lo, hi = percentile_ranks(N)
        srt = np.sort(S, axis=0)
        return (srt[hi] - srt[lo]).astype(np.float32)
    raise ValueError(f"unknown metric {metric}")


def permutation(scores):
    """The gather vector s of the column swap: the D/2 channels of highest
    score (equal scores: lower channel index first) fill positions 0..D/2-1
    in ascending channel order, the others positions D/2..D-1, also in
    ascending order.  Returns int32 [D]."""
    scores = np.asarray(scores, np.float32)
    D = scores.shape[0]
    order = np.lexsort((np.arange(D), -scores.astype(np.float64)))   # rank order
    top = np.zeros(D, bool)
    top[order[:D // 2]] = True
    return np.concatenate([np.nonzero(top)[0], np.nonzero(~top)[0]]).astype(np.int32)


def obs(X, metric="absmax"):
    """Whole OBS derivation from calibration activations X [B, N, D]:
    returns (mean fp32 [N, D], scores fp32 [D], s int32 [D])."""
    S = batch_mean(X)
    sc = channel_scores(S, metric)
    return S, sc, permutation(sc)
