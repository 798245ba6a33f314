"""Pins of the oracle's 8-bit quantizer (the W4A8 and W8A8 settings).

Paper: "CLQ" (arXiv 2509.24416), Sec. 3.1 Eq. (1) with n = 8 bits, and the
three bit settings of Sec. 4.1 (W8A8, W4A8, W4A4).  Reading: the symmetric
mid-tread grid of the 4-bit path with qmax = 2^(n-1) - 1 = 127, s = a/127.
Each test checks the oracle against hand-worked values, bounds that follow
from the definition, invariants, or an error bound derived from Eq. (1).
"""
import numpy as np
import pytest

import oracle
import workloads


def test_qmax():
    assert oracle.qmax(4) == 7 and oracle.qmax(8) == 127


def test_quantizer8_hand_examples():
    # a = 127 -> s = 1, r = 1: ties to even
    row = np.array([[127.0, 2.5, 3.5, -0.5, 0.5, -126.5, 100.0]], np.float32)
    q, s, n = oracle.quantize(row, bits=8)
    assert q.tolist() == [[127, 2, 4, 0, 0, -126, 100]]
    assert s.tolist() == [1.0] and n.tolist() == [0]
    # a = 2 -> r = 63.5: 2 -> 127, -1 -> -63.5 -> -64 (tie to even), 0.5 -> 31.75 -> 32
    row = np.array([[2.0, -1.0, 0.5, 0.0]], np.float32)
    q, s, _ = oracle.quantize(row, bits=8)
    assert q.tolist() == [[127, -64, 32, 0]]
    assert s[0] == np.float32(2.0) / np.float32(127.0)
    q, s, _ = oracle.quantize(np.zeros((1, 8), np.float32), bits=8)
    assert q.tolist() == [[0] * 8] and s.tolist() == [0.0]


def test_quantizer8_bounds():
    xr = oracle.rotate(workloads.activations(64, 1152, "L1", seed=121), 64)
    q, s, n = oracle.quantize(xr, bits=8)
    assert q.min() >= -127 and q.max() <= 127 and n.sum() == 0
    idx = np.abs(xr).argmax(axis=1)
    assert np.all(q[np.arange(64), idx] == np.sign(xr[np.arange(64), idx]) * 127)
    a = np.abs(xr).max(axis=1).astype(np.float64)
    assert np.all(np.abs(s.astype(np.float64) * 127 - a) <= a * 2.0 ** -23)
    err = np.abs(xr.astype(np.float64) - q * s.astype(np.float64)[:, None])
    assert np.all(err <= (s.astype(np.float64)[:, None] / 2) * (1 + 2.0 ** -20))
    # 8 bits are 127/7 times finer than 4
    q4, s4, _ = oracle.quantize(xr, bits=4)
    assert np.allclose(s4 / s, 127.0 / 7.0, rtol=1e-6)


def test_quantizer8_clip_ratio():
    xr = oracle.rotate(workloads.weights(32, 1152, seed=122), 64)
    alpha = 0.7
    q, s, n = oracle.quantize(xr, alpha, bits=8)
    ac = (np.float32(alpha) * np.abs(xr).max(axis=1)).astype(np.float64)
    far = np.abs(xr) >= (ac * (127.5 / 127.0))[:, None] * (1 + 1e-6)
    assert far.any()
    assert np.all(q[far] == 127 * np.sign(xr[far]))
    assert n.sum() >= far.sum()
    inside = np.abs(xr) <= ac[:, None]
    err = np.abs(xr.astype(np.float64) - q * s.astype(np.float64)[:, None])
    assert np.all(err[inside] <= np.broadcast_to(s[:, None] / 2 * (1 + 2.0 ** -20), err.shape)[inside])


@pytest.mark.parametrize("k", [-2, 1, 3])
def test_power_of_two_scaling8(k):
    X = workloads.activations(16, 1152, "L1", seed=131)
    X[np.abs(X) < 2.0 ** -10] = 0
    Xs = (X.astype(np.float32) * np.float32(2.0 ** k)).astype(np.float16)
    _, q0, s0 = oracle.quantize_act(X, 64, bits=8)
    _, q1, s1 = oracle.quantize_act(Xs, 64, bits=8)
    assert np.array_equal(q0, q1) and np.array_equal(s1, s0 * np.float32(2.0 ** k))
    _, qn, sn = oracle.quantize_act(-X, 64, bits=8)
    assert np.array_equal(qn, -q0) and np.array_equal(sn, s0)


@pytest.mark.parametrize("wbits,abits", [(4, 8), (8, 8)])
@pytest.mark.parametrize("b,law", [(64, "L1"), (128, "L2")])
def test_error_bound_8bit(wbits, abits, b, law):
    # |y - y_fp| <= sum_k (|x~| s_w/2 + |w~| s_a/2 + s_a s_w/4) / b, the
    # bound of Eq. (1)'s rounding on both operands of the rotated product
    K = 1152 if b == 64 else 1536
    X = workloads.activations(24, K, law, 141)
    W = workloads.weights(20, K, 142)
    bias = workloads.bias(20, 143)
    r = oracle.linear(X, W, bias, b, wbits=wbits, abits=abits)
    y_fp = oracle.linear_fp64(X, W, bias)
    G = oracle.rotation_dense(K, b)
    xt = np.abs(X.astype(np.float64) @ G)
    wt = np.abs(W.astype(np.float64) @ G)
    sa = r["x_scale"].astype(np.float64)
    sw = r["w_scale"].astype(np.float64) * b
    bound = (xt.sum(1)[:, None] * sw[None, :] / 2 + sa[:, None] * wt.sum(1)[None, :] / 2
             + K * sa[:, None] * sw[None, :] / 4) / b
    slack = 1e-5 * (xt.sum(1)[:, None] * wt.max(1)[None, :]) / b
    assert np.all(np.abs(r["y64"] - y_fp) <= bound + slack)
    assert np.abs(r["xcodes"]).max() <= oracle.qmax(abits)
    assert np.abs(r["wcodes"]).max() <= oracle.qmax(wbits)


def test_more_bits_less_error():
    # Sec. 4.1's three settings, ordered by error on the same data
    K = 1152
    X = workloads.activations(64, K, "L1", 151)
    W = workloads.weights(64, K, 152)
    y_fp = oracle.linear_fp64(X, W)
    e = {}
    for wb, ab in [(4, 4), (4, 8), (8, 8)]:
        e[(wb, ab)] = np.linalg.norm(oracle.linear(X, W, None, 64, wbits=wb, abits=ab)["y64"] - y_fp)
    assert e[(8, 8)] < e[(4, 8)] < e[(4, 4)]
