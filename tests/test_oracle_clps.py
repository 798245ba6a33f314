"""Pins of the single-layer CLPS clip search oracle.

Paper: "CLQ" (arXiv 2509.24416), Sec. 3.4 (grid search of the quantizer
bounds between weight quantiles, squared Frobenius objective, Eq. (3)) and
Sec. 4.1 (beta = 0, gamma = 0.01, one percentile for all channels).  Each
test checks the oracle against hand-worked values, an independent way of
computing the objective, or invariants of the definition.
"""
import numpy as np
import pytest

import oracle
from oracle import clps
import workloads


def sylvester(b):
    H = np.ones((1, 1))
    while H.shape[0] < b:
        H = np.block([[H, H], [H, -H]])
    return H


def test_order_index():
    assert clps.order_index(1152, 0.01) == 1152 - 1 - 11
    assert clps.order_index(64, 0.0) == 63
    assert clps.order_index(64, 0.05) == 60


def test_alpha_floor_on_designed_rows():
    # rows built so that their rotation is known exactly: w = H v / b per
    # block gives FWHT(w) = v (H H = b I); |v| is a permutation of 1..32 per
    # block, so the sorted magnitudes are 1,1,2,2,...,32,32
    b, K = 32, 64
    H = sylvester(b)
    rng = np.random.default_rng(0)
    rows = []
    for scale in (1.0, 0.5):
        v = np.concatenate([rng.permutation(np.arange(1, 33)) * rng.choice([-1, 1], 32) for _ in range(2)])
        v = v * scale
        w = np.concatenate([H @ v[i * b:(i + 1) * b] / b for i in range(2)])
        rows.append(w)
    W = np.array(rows).astype(np.float16)
    assert np.array_equal(np.abs(oracle.rotate(W, b)), np.abs(np.array([r for r in [
        np.concatenate([H @ W[j, i * b:(i + 1) * b].astype(np.float64) for i in range(2)]) for j in range(2)]])))
    # gamma = 0.05: l = 3 values above -> ascending position 60 -> 31 (of 32)
    assert clps.alpha_floor(W, b, gamma=0.05) == np.float32(31.0 / 32.0)
    # an all-zero row counts as ratio 1
    Wz = np.vstack([W, np.zeros((1, K), np.float16)])
    assert clps.alpha_floor(Wz, b, gamma=0.05) == np.float32(31.0 / 32.0)


def test_alpha_grid_hand():
    g = clps.alpha_grid(0.5, 6)
    assert g[0] == np.float32(0.5) and g[-1] == np.float32(1.0)
    assert np.allclose(g, [0.5, 0.6, 0.7, 0.8, 0.9, 1.0], atol=1e-7)
    assert np.all(np.diff(g) > 0)
    assert clps.alpha_grid(0.3, 1).tolist() == [1.0]
    g = clps.alpha_grid(np.float32(0.3), 7)
    assert g[-1] == 1.0 and np.all(g > 0) and np.all(g <= 1.0)


def test_objective_against_dequantised_matmul():
    # e(alpha) from the integer sums equals ||Y0 - Xhat What^T||^2 computed by
    # dequantising both operands and multiplying in fp64
    K, b = 1152, 64
    X = workloads.activations(48, K, "L1", 71)
    W = workloads.weights(40, K, 72)
    Y0 = oracle.linear_fp64(X, W).astype(np.float32)
    alphas = np.array([0.8, 0.9, 1.0], np.float32)
    e = clps.errors(X, W, Y0, b, alphas)
    _, xc, xs = oracle.quantize_act(X, b)
    for i, a in enumerate(alphas):
        _, wc, ws = oracle.quantize_weights(W, b, None, float(a))
        Xh = xc.astype(np.float64) * xs.astype(np.float64)[:, None]
        Wh = wc.astype(np.float64) * ws.astype(np.float64)[:, None]
        ref = np.sum((Y0.astype(np.float64) - Xh @ Wh.T) ** 2)
        assert abs(e[i] - ref) <= 1e-9 * ref


def test_search_picks_the_minimum_and_clipping_helps_gaussian_weights():
    K, b = 1152, 64
    X = workloads.activations(64, K, "L1", 81)
    W = workloads.weights(48, K, 82)
    Y0 = oracle.linear_fp64(X, W).astype(np.float32)
    al, e, best = clps.search(X, W, Y0, b, G=12)
    assert al[-1] == 1.0 and best == int(np.argmin(e))
    assert e[best] <= e[-1]
    # Gaussian rows: the max is an outlier of the row, so some clipping wins
    assert best < len(al) - 1


@pytest.mark.parametrize("k", [1, 2])   # upward: no fp16 subnormals
def test_weight_scaling_invariance(k):
    K, b = 1152, 64
    X = workloads.activations(32, K, "L1", 91)
    W = workloads.weights(24, K, 92)
    Ws = (W.astype(np.float32) * np.float32(2.0 ** k)).astype(np.float16)
    assert np.array_equal(Ws.astype(np.float32), W.astype(np.float32) * np.float32(2.0 ** k))
    Y0 = oracle.linear_fp64(X, W).astype(np.float32)
    Y0s = (Y0 * np.float32(2.0 ** k)).astype(np.float32)
    a0, e0, b0 = clps.search(X, W, Y0, b, G=8)
    a1, e1, b1 = clps.search(X, Ws, Y0s, b, G=8)
    assert np.array_equal(a0, a1) and b0 == b1
    assert np.allclose(e1, e0 * 4.0 ** k, rtol=1e-12)
