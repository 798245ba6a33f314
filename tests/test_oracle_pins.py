"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, an independent construction, brute force on tiny inputs, hand-worked
examples, invariants of the method, or an error bound derived from it.
Paper: "CLQ" (arXiv 2509.24416), Sec. 3.1 Eq. (1) and Sec. 3.3.
"""
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def sylvester(b):
    """H_1 = [1]; H_2n = [[H, H], [H, -H]] (independent of the popcount
    formula the oracle uses)."""
    H = np.ones((1, 1))
    while H.shape[0] < b:
        H = np.block([[H, H], [H, -H]])
    return H


BLOCKS = [2, 4, 8, 16, 32, 64, 128]


# ---- P1: the block Hadamard matrix (Sec. 3.3: +-1 entries, G G^T = I) ------

@pytest.mark.parametrize("b", BLOCKS)
def test_hadamard_closed_form(b):
    H = oracle.hadamard_dense(b)
    assert np.array_equal(H, sylvester(b))
    assert np.array_equal(H @ H.T, b * np.eye(b))
    assert set(np.unique(H)) == {-1.0, 1.0}


def test_hadamard_2():
    assert np.array_equal(oracle.hadamard_dense(2), np.array([[1.0, 1.0], [1.0, -1.0]]))


@pytest.mark.parametrize("b", [32, 64, 128])
def test_rotation_orthogonal(b):
    K = 4 * b
    perm = workloads.random_perm(K, seed=b)
    G = oracle.rotation_dense(K, b, perm, normalised=True)
    assert np.abs(G @ G.T - np.eye(K)).max() < 1e-12


# ---- P2: the fast transform equals the dense matrix ------------------------

@pytest.mark.parametrize("b", BLOCKS)
def test_fwht_unit_vectors(b):
    K = 2 * b
    E = np.eye(K, dtype=np.float16)
    out = oracle.rotate(E, b)
    expect = np.kron(np.eye(2), sylvester(b))
    assert np.array_equal(out.astype(np.float64), expect)


@pytest.mark.parametrize("b", [32, 64, 128])
def test_fwht_involution_on_integers(b):
    rng = np.random.default_rng(b)
    K = 3 * b
    X = rng.integers(-8, 9, size=(5, K)).astype(np.float16)
    once = oracle.rotate(X, b)
    # exact: integer inputs, |values| * b < 2^24
    assert np.array_equal(once.astype(np.float64),
                          X.astype(np.float64) @ np.kron(np.eye(3), sylvester(b)))
    twice = oracle.rotate(once, b)
    assert np.array_equal(twice, b * X.astype(np.float32))


@pytest.mark.parametrize("b", [32, 64, 128])
def test_fwht_fp32_close_to_fp64(b):
    X = workloads.activations(16, 4 * b, "L1", seed=7)
    out = oracle.rotate(X, b).astype(np.float64)
    ref = X.astype(np.float64) @ np.kron(np.eye(4), sylvester(b))
    # each of log2(b) stages adds at most one fp32 rounding per partial sum
    mag = np.abs(X.astype(np.float64)).reshape(16, 4, b).sum(-1).repeat(b, axis=1)
    assert np.all(np.abs(out - ref) <= np.log2(b) * 2.0 ** -24 * mag * 1.01)


def test_gather_reading():
    """s is a gather: x'[k] = x[s[k]] (reading of Sec. 3.3's vector s)."""
    b, K = 32, 128
    rng = np.random.default_rng(11)
    X = rng.integers(-8, 9, size=(4, K)).astype(np.float16)
    perm = workloads.random_perm(K, seed=5)
    out = oracle.rotate(X, b, perm).astype(np.float64)
    ref = X.astype(np.float64)[:, perm] @ np.kron(np.eye(K // b), sylvester(b))
    assert np.array_equal(out, ref)
    G = oracle.rotation_dense(K, b, perm)
    assert np.array_equal(X.astype(np.float64) @ G, ref)


# ---- P3: lossless smoothing (Sec. 3.3: G G^T = I, W absorbs G) -------------

@pytest.mark.parametrize("b", [32, 64, 128])
@pytest.mark.parametrize("with_perm", [False, True])
def test_rotation_invariance_exact(b, with_perm):
    rng = np.random.default_rng(100 + b)
    K, M, N = 2 * b, 6, 5
    X = rng.integers(-6, 7, size=(M, K)).astype(np.float16)
    W = rng.integers(-6, 7, size=(N, K)).astype(np.float16)
    perm = workloads.random_perm(K, seed=b) if with_perm else None
    Xr = oracle.rotate(X, b, perm).astype(np.float64)
    Wr = oracle.rotate(W, b, perm).astype(np.float64)
    lhs = Xr @ Wr.T
    rhs = b * (X.astype(np.float64) @ W.astype(np.float64).T)
    assert np.array_equal(lhs, rhs)


def test_rotation_invariance_fp64_real_data():
    b, K = 64, 1152
    X = workloads.activations(8, K, "L1", seed=3).astype(np.float64)
    W = workloads.weights(4, K, seed=4).astype(np.float64)
    G = oracle.rotation_dense(K, b, workloads.random_perm(K, 9), normalised=True)
    d = np.abs((X @ G) @ (W @ G).T - X @ W.T).max()
    assert d <= 1e-12 * np.abs(X).max() * np.abs(W).max() * K


# ---- P4: the quantizer of Eq. (1), symmetric int4 ---------------------------

def test_quantizer_hand_examples():
    # a = 7 -> s = 1, r = 1: rounding half to even on exact ties
    row = np.array([[7.0, 2.5, 3.5, -0.5, 0.5, 1.5, -2.5, 6.5]], np.float32)
    q, s, n = oracle.quantize(row)
    assert q.tolist() == [[7, 2, 4, 0, 0, 2, -2, 6]]
    assert s.tolist() == [1.0] and n.tolist() == [0]
    # a = 14 -> s = 2, r = 0.5
    row = np.array([[14.0, 3.0, -5.0, 1.0]], np.float32)
    q, s, _ = oracle.quantize(row)
    assert q.tolist() == [[7, 2, -2, 0]] and s.tolist() == [2.0]
    # zero row: s = 0 and every code 0
    q, s, _ = oracle.quantize(np.zeros((1, 8), np.float32))
    assert q.tolist() == [[0] * 8] and s.tolist() == [0.0]


def test_quantizer_bounds():
    xr = oracle.rotate(workloads.activations(64, 1152, "L1", seed=21), 64)
    q, s, n = oracle.quantize(xr)
    assert q.min() >= -7 and q.max() <= 7 and n.sum() == 0
    a = np.abs(xr).max(axis=1)
    # the abs-max element maps to +-7
    idx = np.abs(xr).argmax(axis=1)
    assert np.all(np.abs(q[np.arange(64), idx]) == 7)
    assert np.all(q[np.arange(64), idx] == np.sign(xr[np.arange(64), idx]) * 7)
    # s = a/7 to fp32 rounding
    assert np.all(np.abs(s.astype(np.float64) * 7 - a) <= a * 2.0 ** -23)
    err = np.abs(xr.astype(np.float64) - q * s.astype(np.float64)[:, None])
    assert np.all(err <= (s.astype(np.float64)[:, None] / 2) * (1 + 2.0 ** -20))


def test_quantizer_clip_ratio():
    xr = oracle.rotate(workloads.weights(32, 1152, seed=22), 64)
    alpha = 0.8
    q, s, n = oracle.quantize(xr, alpha)
    a = np.abs(xr).max(axis=1).astype(np.float64)
    ac = (np.float32(alpha) * np.abs(xr).max(axis=1)).astype(np.float64)
    assert np.all(np.abs(s * 7.0 - ac) <= ac * 2.0 ** -23)
    inside = np.abs(xr) <= ac[:, None]
    err = np.abs(xr.astype(np.float64) - q * s.astype(np.float64)[:, None])
    assert np.all(err[inside] <= np.broadcast_to(s[:, None] / 2 * (1 + 2.0 ** -20), err.shape)[inside])
    # beyond the clip bound (by more than half a step) the code saturates
    far = np.abs(xr) >= (ac * (7.5 / 7.0))[:, None] * (1 + 1e-6)
    assert far.any()
    assert np.all(q[far] == 7 * np.sign(xr[far]))
    assert n.sum() >= far.sum()
    assert np.all(a >= ac)


# ---- P5: metamorphic properties ---------------------------------------------

@pytest.mark.parametrize("k", [-3, -1, 1, 2])
def test_power_of_two_scaling(k):
    X = workloads.activations(16, 1152, "L1", seed=31)
    X[np.abs(X) < 2.0 ** -10] = 0  # keep the scaled copy out of fp16 subnormals
    Xs = (X.astype(np.float32) * np.float32(2.0 ** k)).astype(np.float16)
    assert np.array_equal(Xs.astype(np.float32), X.astype(np.float32) * np.float32(2.0 ** k))
    _, q0, s0 = oracle.quantize_act(X, 64)
    _, q1, s1 = oracle.quantize_act(Xs, 64)
    assert np.array_equal(q0, q1)
    assert np.array_equal(s1, s0 * np.float32(2.0 ** k))


def test_negation():
    X = workloads.activations(16, 1152, "L1", seed=32)
    _, q0, s0 = oracle.quantize_act(X, 64)
    _, q1, s1 = oracle.quantize_act(-X, 64)
    assert np.array_equal(q1, -q0) and np.array_equal(s0, s1)


def test_shared_perm_leaves_linear_unchanged():
    b, K = 64, 1152
    X = workloads.activations(8, K, "L1", seed=33)
    W = workloads.weights(6, K, seed=34)
    perm = workloads.random_perm(K, 35)
    Xr = oracle.rotate(X, b, perm).astype(np.float64)
    Wr = oracle.rotate(W, b, perm).astype(np.float64)
    y = Xr @ Wr.T / b
    y_fp = oracle.linear_fp64(X, W)
    assert np.abs(y - y_fp).max() <= 1e-5 * np.abs(X.astype(np.float64)).max() * np.abs(W.astype(np.float64)).max() * np.sqrt(K)


# ---- P6: nibble packing (hand examples) --------------------------------------

def _golden_pairs():
    rows = []
    with open(os.path.join(GOLDEN, "pack_examples.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                a, b, h = line.split()
                rows.append((int(a), int(b), int(h, 16)))
    return rows


def test_pack_golden():
    rows = _golden_pairs()
    assert len(rows) >= 8
    codes = np.array([[a, b] for a, b, _ in rows], np.int8)
    packed = oracle.pack(codes)
    assert packed[:, 0].tolist() == [h for _, _, h in rows]
    # one long row: the pairs side by side
    long_row = codes.reshape(1, -1)
    assert oracle.pack(long_row)[0].tolist() == [h for _, _, h in rows]


def test_pack_roundtrip_all_pairs():
    v = np.arange(-7, 8)
    codes = np.stack(np.meshgrid(v, v, indexing="ij"), -1).reshape(1, -1).astype(np.int8)
    assert np.array_equal(oracle.unpack(oracle.pack(codes), codes.shape[1]), codes)


# ---- P7: integer GEMM against brute force -----------------------------------

@pytest.mark.parametrize("M,N,K", [(1, 1, 64), (3, 8, 64), (8, 5, 128), (7, 2, 128)])
def test_gemm_bruteforce(M, N, K):
    rng = np.random.default_rng(M * 100 + N * 10 + K)
    qa = rng.integers(-7, 8, size=(M, K)).astype(np.int8)
    qw = rng.integers(-7, 8, size=(N, K)).astype(np.int8)
    acc = oracle.gemm_i32(qa, qw)
    assert acc.shape == (M, N)
    for m in range(M):
        for n in range(N):
            ref = 0
            for k in range(K):
                ref += int(qa[m, k]) * int(qw[n, k])
            assert acc[m, n] == ref


def test_gemm_special_cases():
    K = 128
    seven = np.full((2, K), 7, np.int8)
    assert np.all(oracle.gemm_i32(seven, seven) == 49 * K)
    rng = np.random.default_rng(3)
    qw = rng.integers(-7, 8, size=(4, K)).astype(np.int8)
    onehot = np.zeros((K, K), np.int8)
    onehot[np.arange(K), np.arange(K)] = 1
    assert np.array_equal(oracle.gemm_i32(onehot, qw), qw.T.astype(np.int32))


# ---- P8: the dequantising epilogue --------------------------------------------

def test_epilogue_special_cases():
    acc = np.array([[3]], np.int32)
    y, p = oracle.epilogue(acc, np.array([0.5], np.float32), np.array([0.25], np.float32),
                           np.array([1.0], np.float16))
    assert y.tolist() == [[1.375]] and p.tolist() == [[0.375]]
    zeros = np.zeros((4, 6), np.int32)
    bias = workloads.bias(6, 1)
    y, p = oracle.epilogue(zeros, np.ones(4, np.float32), np.ones(6, np.float32), bias)
    assert np.array_equal(y, np.broadcast_to(bias.astype(np.float64), (4, 6)))
    y, p = oracle.epilogue(np.full((2, 3), 5, np.int32), np.ones(2, np.float32),
                           np.ones(3, np.float32), None)
    assert np.array_equal(y, p)


def test_epilogue_equals_dequantise_then_matmul():
    X = workloads.activations(16, 1152, "L1", 41)
    W = workloads.weights(12, 1152, 42)
    bias = workloads.bias(12, 43)
    r = oracle.linear(X, W, bias, 64)
    Xd = r["xcodes"].astype(np.float64) * r["x_scale"].astype(np.float64)[:, None]
    Wd = r["wcodes"].astype(np.float64) * r["w_scale"].astype(np.float64)[:, None]
    ref = Xd @ Wd.T + bias.astype(np.float64)
    assert np.abs(r["y64"] - ref).max() <= 1e-12 * np.abs(ref).max()


# ---- P9: end-to-end error bound (derived from Eq. (1)) ------------------------

@pytest.mark.parametrize("b,law", [(64, "L1"), (128, "L2"), (32, "L1")])
@pytest.mark.parametrize("with_perm", [False, True])
def test_end_to_end_error_bound(b, law, with_perm):
    K = 1152 if b != 128 else 1536
    X = workloads.activations(24, K, law, 51)
    W = workloads.weights(20, K, 52)
    bias = workloads.bias(20, 53)
    perm = workloads.random_perm(K, 54) if with_perm else None
    r = oracle.linear(X, W, bias, b, perm)
    y_fp = oracle.linear_fp64(X, W, bias)
    G = oracle.rotation_dense(K, b, perm)
    xt = np.abs(X.astype(np.float64) @ G)
    wt = np.abs(W.astype(np.float64) @ G)
    sa = r["x_scale"].astype(np.float64)
    sw = r["w_scale"].astype(np.float64) * b
    bound = (xt.sum(1)[:, None] * sw[None, :] / 2 + sa[:, None] * wt.sum(1)[None, :] / 2
             + K * sa[:, None] * sw[None, :] / 4) / b
    slack = 1e-5 * (xt.sum(1)[:, None] * wt.max(1)[None, :]) / b
    assert np.all(np.abs(r["y64"] - y_fp) <= bound + slack)


def test_smoothing_reduces_error():
    """Sec. 3.3 / Sec. 4.2: rotating before quantizing lowers the W4A4 error on
    activations with outlier channels (information; the paper's ~90% figure is
    for real models and is not asserted)."""
    K = 1152
    X = workloads.activations(64, K, "L1", 61)
    W = workloads.weights(64, K, 62)
    y_fp = oracle.linear_fp64(X, W)
    rot = oracle.linear(X, W, None, 64)["y64"]
    # block size 1 would be no rotation: quantize the raw rows instead
    qa, sa, _ = oracle.quantize(X.astype(np.float32))
    qw, sw, _ = oracle.quantize(W.astype(np.float32))
    plain, _ = oracle.epilogue(oracle.gemm_i32(qa, qw), sa, sw, None)
    e_rot = np.linalg.norm(rot - y_fp)
    e_plain = np.linalg.norm(plain - y_fp)
    assert e_rot < e_plain


# ---- adversarial fp16 inputs ---------------------------------------------------

def test_extreme_fp16_rows():
    K, b = 256, 128
    X = np.zeros((4, K), np.float16)
    X[0, :] = np.float16(65504)
    X[1, ::2] = np.float16(-65504)
    X[2, :] = np.float16(-0.0)
    X[3, 5] = np.float16(6e-8)  # fp16 subnormal
    xq, q, s = oracle.quantize_act(X, b)
    assert np.all(np.abs(q) <= 7)
    assert s[2] == 0 and np.all(q[2] == 0)
    assert s[3] > 0 and np.abs(q[3]).max() == 7
    assert np.isfinite(s).all()


# ---- Eq. (1) Round(.): one rounding of the exact product ---------------------
# Round(.) maps the scaled value to its nearest integer.  The scaled value is
# the exact product x~ * r with r = fl32(qmax / a) the per-row reciprocal.
# The cases below were chosen so that rounding that product to fp32 first
# lands exactly on k + 1/2 while the exact product lies just off the tie: an
# oracle that rounded twice (to fp32, then to an integer) gets the other
# integer.  Expected codes come from exact rational arithmetic here, not from
# the oracle's formula.
from fractions import Fraction  # noqa: E402

ROUNDING_CASES = [
    # (qmax, abs-max a, element x) as fp32 hex; the exact product's nearest integer
    (7.0, "0x1.448a1cp+0", "0x1.fdfd98p-1", 5),
    (7.0, "0x1.ec480ap+0", "0x1.a5f49ap-2", 1),
    (7.0, "0x1.228eaep+0", "0x1.9f14fap-2", 3),
    (127.0, "0x1.4ea5a4p+0", "0x1.f749bep-1", 95),
    (127.0, "0x1.a023dap+0", "0x1.b713aep-2", 33),
    (127.0, "0x1.d4a706p-1", "0x1.555762p-1", 93),
]


def _f32_correctly_rounded_quotient(num, den):
    """fl32(num / den) from the exact rational quotient, rounding half to
    even, without using a floating-point division."""
    q = Fraction(float(num)) / Fraction(float(den))
    lo = np.float32(float(q))            # within one fp32 step of q
    cands = [np.nextafter(lo, np.float32(-np.inf)), lo, np.nextafter(lo, np.float32(np.inf))]
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - q),
                                     int(np.frombuffer(np.float32(c).tobytes(), np.uint32)[0]) & 1))
    return np.float32(best)


@pytest.mark.parametrize("qm,a_hex,x_hex,expect", ROUNDING_CASES)
def test_quantizer_single_rounding(qm, a_hex, x_hex, expect):
    a = np.float32(float.fromhex(a_hex))
    x = np.float32(float.fromhex(x_hex))
    r = _f32_correctly_rounded_quotient(qm, a)
    exact = Fraction(float(x)) * Fraction(float(r))
    # the case is a discriminating one: fp32 rounding of the product is a tie
    # that rounds (half to even) to the other integer
    f32 = np.float32(float(exact))  # exact product (fits a double) rounded once to fp32
    assert Fraction(float(f32)).denominator == 2
    assert round(exact) == expect and abs(exact - expect) < Fraction(1, 2)
    assert int(np.rint(f32)) != expect
    row = np.array([[a, x, -x, 0.0]], np.float32)
    bits = 4 if qm == 7.0 else 8
    q, s, n = oracle.quantize(row, bits=bits)
    assert q.tolist() == [[int(qm), expect, -expect, 0]]
    assert n.tolist() == [0]
    assert Fraction(float(s[0])) == Fraction(float(_f32_correctly_rounded_quotient(a, qm)))


# ---- the fp16 error metric of the 2e-3 bound (hand-computed cases) -----------

def test_err_metric_identity_and_empty():
    y64 = np.array([[1.5, -2.0], [0.25, 8.0]])
    assert oracle.err_metric(y64.astype(np.float16), y64, y64) == 0.0
    assert oracle.err_metric(np.zeros((0, 3)), np.zeros((0, 3)), np.zeros((0, 3))) == 0.0


def test_err_metric_one_element_off():
    p64 = np.array([[2.0, -4.0, 0.5]])
    y = p64.copy()
    y[0, 1] += 2.0 ** -7          # error d = 2^-7 on |p| = 4
    assert oracle.err_metric(y, p64, p64) == 2.0 ** -9


def test_err_metric_cancelling_bias():
    # p = 3, bias = -3: y64 = 0; the denominator is |p| + |bias| = 6, not |y64|
    p64 = np.array([[3.0, 1.0]])
    bias = np.array([-3.0, 1.0])
    y64 = p64 + bias[None, :]
    y = y64.copy()
    y[0, 0] = 0.5
    assert oracle.err_metric(y, y64, p64, bias) == 0.5 / 6.0
    # without the bias term the same deviation is measured against |p| only
    assert oracle.err_metric(y, y64, p64) == 0.5 / 3.0


def test_err_metric_floor():
    # p = bias = 0: the denominator is the 2^-24 floor
    z = np.zeros((1, 2))
    y = np.array([[2.0 ** -30, 0.0]])
    assert oracle.err_metric(y, z, z, np.zeros(2)) == 2.0 ** -6


def test_err_metric_worst_element_wins():
    p64 = np.array([[10.0, 10.0, 10.0]])
    y = np.array([[11.0, 10.0, 7.0]])   # relative errors 0.1, 0, 0.3
    assert oracle.err_metric(y, p64, p64) == pytest.approx(0.3, abs=0, rel=1e-15)
    assert oracle.err_metric(y, p64, p64) > 0.3 - 1e-15
