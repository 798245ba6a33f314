"""GPU parity of the fp6-stored W4A4 path against the CPU oracle.

The codes are the 4-bit grid's (Eq. (1)); only their storage differs (fp6
e2m3 in the layout the fp6 matrix instructions read).  Codes (after
clq_unswizzle_f6) and scales must match the oracle bit for bit, the integer
sums too (the fp32 accumulation of integer products is exact), and the fp16
output must lie within 2e-3 of the oracle's fp64 dequantised result.  Each
fp6 buffer must also equal, byte for byte, the int4 buffer of the same codes
converted by clq_f6_from_int4, and the integer sums must equal the int4
path's on the whole output.
"""
import numpy as np
import pytest

import oracle
import workloads

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

TOL = 2e-3


@pytest.fixture(scope="module")
def clq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2509_24416_amd as m
    return m


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


# ---- codes ----------------------------------------------------------------------

# every activation kernel: the batched one (K <= 2048 or b != 64), the 8-row
# one (b = 64, 2048 <= K <= 5120) and the one-shot one (rows of more than 256
# blocks); ragged row counts; laws L1 / L2
@pytest.mark.parametrize("M,K,block", [
    (1, 64, 32), (7, 128, 64), (255, 1152, 64), (257, 1152, 32), (64, 1152, 128),
    (33, 4608, 64), (20, 3072, 128), (5, 12288, 128), (3, 64, 64), (9, 256, 128), (41, 16384, 32)])
@pytest.mark.parametrize("law", ["L1", "L2"])
def test_f6_act_codes_bitexact(clq, M, K, block, law):
    X = workloads.activations(M, K, law, seed=M + K + block + 1)
    Xq6, xs = clq.clq_rotate_quant_act_f6(dev(X), block)
    ref_q, _, ref_s = oracle.quantize_act(X, block)
    assert Xq6.numel() == clq.clq_act_bytes_f6(M, K) == (M + 31) // 32 * 32 * K * 3 // 4
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_f6(Xq6, M, K, False)), ref_q)
    Xq4, _ = clq.clq_rotate_quant_act(dev(X), block)
    assert torch.equal(clq.clq_f6_from_int4(Xq4, M, K, False), Xq6)


def test_f6_act_perm_and_stride(clq):
    M, K, block = 300, 1152, 64
    Xw = workloads.activations(M, K + 64, "L2", seed=4)
    perm = workloads.random_perm(K, seed=5)
    X = dev(Xw)[:, :K]
    Xq6, xs = clq.clq_rotate_quant_act_f6(X, block, dev(perm))
    ref_q, _, ref_s = oracle.quantize_act(Xw[:, :K], block, perm)
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_f6(Xq6, M, K, False)), ref_q)


@pytest.mark.parametrize("N,K,block,clip", [
    (1, 64, 32, 1.0), (8, 1152, 64, 1.0), (72, 1152, 64, 0.9), (200, 4608, 64, 1.0),
    (1152, 1152, 64, 1.0), (100, 3072, 128, 0.75), (3, 128, 128, 0.5)])
def test_f6_weight_codes_bitexact(clq, N, K, block, clip):
    W = workloads.weights(N, K, seed=N + K + 1)
    qw6 = clq.clq_quantize_weights_f6(dev(W), block, clip_ratio=clip)
    ref_q, _, ref_s = oracle.quantize_weights(W, block, None, clip)
    assert qw6.bits == 6 and qw6.wq.numel() == clq.clq_weight_bytes_f6(N, K)
    assert np.array_equal(host(qw6.w_scale), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_f6(qw6.wq, N, K, True)), ref_q)
    qw4 = clq.clq_quantize_weights(dev(W), block, clip_ratio=clip)
    assert torch.equal(clq.clq_qweight_f6(qw4).wq, qw6.wq)


def test_f6_weights_perm(clq):
    N, K, block = 96, 1152, 64
    W = workloads.weights(N, K, seed=7)
    perm = workloads.random_perm(K, seed=8)
    qw6 = clq.clq_quantize_weights_f6(dev(W), block, dev(perm))
    ref_q, _, ref_s = oracle.quantize_weights(W, block, perm)
    assert np.array_equal(host(qw6.w_scale), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_f6(qw6.wq, N, K, True)), ref_q)


# ---- GEMM -------------------------------------------------------------------------

# few and many tiles, ragged tokens and channels, k loops from 2 to 72 stages,
# one tile per workgroup and several
F6_GEMM_SHAPES = [(1, 1, 128), (7, 8, 128), (129, 72, 192), (257, 200, 1152), (64, 1152, 1152),
                  (300, 130, 640), (513, 264, 4608), (100, 1001, 320), (33, 48, 256), (5, 3, 256),
                  (2049, 1030, 640), (4000, 2000, 576), (8193, 1030, 576), (600, 700, 4608),
                  (9000, 2000, 1152)]


@pytest.mark.parametrize("M,N,K", F6_GEMM_SHAPES)
def test_f6_accum_exact(clq, M, N, K):
    block = 64
    X = workloads.activations(M, K, "L1", seed=M + 2)
    W = workloads.weights(N, K, seed=N + 2)
    qw6 = clq.clq_quantize_weights_f6(dev(W), block)
    Xq6, xs = clq.clq_rotate_quant_act_f6(dev(X), block)
    acc = host(clq.clq_w4a4_accum_f6(Xq6, xs, qw6))
    rows = np.unique(np.r_[0:min(M, 40), M // 2, M - 3:M].clip(0, M - 1))
    _, xc, _ = oracle.quantize_act(X[rows], block)
    _, wc, _ = oracle.quantize_weights(W, block)
    assert np.array_equal(acc[rows], oracle.gemm_i32(xc, wc))
    # the int4 path's sums, whole output
    qw4 = clq.clq_quantize_weights(dev(W), block)
    Xq4, _ = clq.clq_rotate_quant_act(dev(X), block)
    assert np.array_equal(acc, host(clq.clq_w4a4_accum_i32(Xq4, xs, qw4)))


@pytest.mark.parametrize("M,N,K", F6_GEMM_SHAPES)
@pytest.mark.parametrize("with_bias", [True, False])
def test_f6_linear_tolerance(clq, M, N, K, with_bias):
    block = 64
    X = workloads.activations(M, K, "L1", seed=M + 3)
    W = workloads.weights(N, K, seed=N + 3)
    b = workloads.bias(N, seed=N + 4) if with_bias else None
    qw6 = clq.clq_quantize_weights_f6(dev(W), block)
    Xq6, xs = clq.clq_rotate_quant_act_f6(dev(X), block)
    Y = host(clq.clq_w4a4_linear_f6(Xq6, xs, qw6, dev(b) if b is not None else None))
    rows = np.unique(np.r_[0:min(M, 24), M // 2, M - 2:M].clip(0, M - 1))
    r = oracle.linear(X[rows], W, b, block)
    assert oracle.err_metric(Y[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL


def test_f6_linear_row_stride_and_zero_rows(clq):
    M, N, K, block = 300, 520, 1152, 64
    X = workloads.activations(M, K, "L1", seed=11)
    X[[0, 77, 299]] = 0
    W = workloads.weights(N, K, seed=12)
    b = workloads.bias(N, seed=13)
    qw6 = clq.clq_quantize_weights_f6(dev(W), block)
    Xq6, xs = clq.clq_rotate_quant_act_f6(dev(X), block)
    big = torch.full((M, N + 40), 7.0, dtype=torch.float16, device="cuda")
    out = big[:, :N]
    clq.clq_w4a4_linear_f6(Xq6, xs, qw6, dev(b), out=out)
    Y = host(big)
    assert np.all(Y[:, N:] == 7.0)
    assert np.array_equal(Y[[0, 77, 299], :N], np.tile(b, (3, 1)))
    r = oracle.linear(X[:16], W, b, block)
    assert oracle.err_metric(Y[:16, :N].astype(np.float64), r["y64"], r["p64"], b) <= TOL


# 256-token tiles (the first shape) and 128-token tiles (fewer 256-token
# tiles than compute units), against the int4 persistent and two-halves
# kernels
@pytest.mark.parametrize("M,N,K", [(4096, 3456, 1152), (1024, 3456, 1152), (1000, 1152, 4608)])
def test_f6_matches_int4_fp16_output(clq, M, N, K):
    # the same sums and the same epilogue arithmetic: the int4 path's sums
    # are 256 times the fp6 path's, exact in fp32 below 2^24 codes' worth,
    # and its scale is x_scale / 256, so every product is the same real
    # number rounded once: equal outputs
    block = 64
    X = workloads.activations(M, K, "L1", seed=21)
    W = workloads.weights(N, K, seed=22)
    b = workloads.bias(N, seed=23)
    qw4 = clq.clq_quantize_weights(dev(W), block)
    Xq4, xs = clq.clq_rotate_quant_act(dev(X), block)
    y4 = host(clq.clq_w4a4_linear(Xq4, xs, qw4, dev(b)))
    y6 = host(clq.clq_w4a4_linear_f6(clq.clq_f6_from_int4(Xq4, M, K, False), xs, clq.clq_qweight_f6(qw4), dev(b)))
    assert np.array_equal(y4.view(np.uint16), y6.view(np.uint16))


FULL = [l for wl in (workloads.C2, workloads.C3, workloads.C4) for l in wl.layers]


@pytest.mark.parametrize("layer", FULL, ids=[l.name for l in FULL])
def test_f6_full_size_layer_sampled(clq, layer):
    l = layer
    X = workloads.activations(l.M, l.K, "L1", l.seed)
    W = workloads.weights(l.N, l.K, l.seed + 1)
    b = workloads.bias(l.N, l.seed + 2)
    qw6 = clq.clq_quantize_weights_f6(dev(W), l.block)
    Xq6, xs = clq.clq_rotate_quant_act_f6(dev(X), l.block)
    Y = host(clq.clq_w4a4_linear_f6(Xq6, xs, qw6, dev(b)))
    rows = np.unique(np.r_[0:4, l.M // 3, l.M // 2, l.M - 4:l.M])
    r = oracle.linear(X[rows], W, b, l.block)
    assert np.array_equal(host(xs)[rows], oracle.quantize_act(X[rows], l.block)[2])
    acc = host(clq.clq_w4a4_accum_f6(Xq6, xs, qw6))
    assert np.array_equal(acc[rows], r["acc"])
    assert oracle.err_metric(Y[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL


def test_f6_argument_errors(clq):
    W = dev(workloads.weights(64, 128, seed=1))
    qw4 = clq.clq_quantize_weights(W, 64)
    X = dev(workloads.activations(8, 128, "L1", seed=2))
    Xq6, xs = clq.clq_rotate_quant_act_f6(X, 64)
    with pytest.raises(ValueError):
        clq.clq_w4a4_linear_f6(Xq6, xs, qw4)          # int4 weights
    qw6 = clq.clq_quantize_weights_f6(W, 64)
    with pytest.raises(ValueError):
        clq.clq_w4a4_linear(Xq6, xs, qw6)             # fp6 weights into the int4 GEMM
    W64 = dev(workloads.weights(64, 64, seed=3))
    X64 = dev(workloads.activations(8, 64, "L1", seed=4))
    qw64 = clq.clq_quantize_weights_f6(W64, 64)
    Xq64, xs64 = clq.clq_rotate_quant_act_f6(X64, 64)
    with pytest.raises(clq.ClqError):
        clq.clq_w4a4_linear_f6(Xq64, xs64, qw64)      # K < 128


# every fp6 GEMM schedule (the persistent kernel, the two-halves kernel on
# 128- and 64-token tiles) on few and many tiles, ragged shapes and short and
# long k loops: the same integer sums and the same fp16 bits
F6_FORCED = [(1024, 1152, 1152), (300, 1000, 640), (1000, 1152, 4608), (4096, 3456, 1152), (8192, 1152, 4608),
             (65, 200, 256), (2, 16, 128), (777, 3072, 3072)]


@pytest.mark.parametrize("M,N,K", F6_FORCED)
def test_f6_forced_schedules_agree(clq, M, N, K):
    block = 64
    X = workloads.activations(M, K, "L1", seed=M + 5)
    W = workloads.weights(N, K, seed=N + 5)
    b = workloads.bias(N, seed=N + 6)
    qw = clq.clq_quantize_weights_f6(dev(W), block)
    Xq, xs = clq.clq_rotate_quant_act_f6(dev(X), block)
    rows = np.unique(np.r_[0:3, M // 2, M - 3:M].clip(0, M - 1))
    r = oracle.linear(X[rows], W, b, block)
    ref = None
    try:
        for force in (1, 2, 3):
            clq.clq_debug_set(clq.CLQ_DEBUG_F6_SCHEDULE, force)
            acc = host(clq.clq_w4a4_accum_f6(Xq, xs, qw))
            Y = host(clq.clq_w4a4_linear_f6(Xq, xs, qw, dev(b)))
            if ref is None:
                ref, refY = acc, Y
                assert np.array_equal(acc[rows], r["acc"])
                assert oracle.err_metric(Y[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL
            else:
                assert np.array_equal(acc, ref), force
                assert np.array_equal(Y.view(np.uint16), refY.view(np.uint16)), force
    finally:
        clq.clq_debug_set(clq.CLQ_DEBUG_F6_SCHEDULE, 0)
