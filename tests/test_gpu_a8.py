"""GPU parity of the 8-bit settings (W4A8, W8A8) against the CPU oracle.

Paper: "CLQ" (arXiv 2509.24416), Sec. 4.1 (the method at W8A8, W4A8 and
W4A4) and Sec. 3.1 Eq. (1) with n = 8.  Codes, scales and integer sums must
match bit for bit; the fp16 output lies within 2e-3 of the oracle's fp64
dequantised result (the metric of the W4A4 tests).
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


@pytest.mark.parametrize("M,K,block", [
    (1, 64, 32), (7, 128, 64), (255, 1152, 64), (257, 1152, 32), (64, 1152, 128),
    (33, 4608, 64), (20, 3072, 128), (5, 12288, 128), (1000, 1152, 64)])
@pytest.mark.parametrize("law", ["L1", "L2"])
def test_rotate_quant_act8_bitexact(clq, M, K, block, law):
    X = workloads.activations(M, K, law, seed=M + K + block + 7)
    Xq8, xs = clq.clq_rotate_quant_act8(dev(X), block)
    _, ref_c, ref_s = oracle.quantize_act(X, block, bits=8)
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_act8(Xq8, M, K)), ref_c)
    assert Xq8.numel() == clq.clq_act8_bytes(M, K)


def test_rotate_quant_act8_perm_and_stride(clq):
    M, K, block, ld = 300, 1152, 64, 1280
    X = workloads.activations(M, K, "L1", seed=17)
    wide = np.zeros((M, ld), np.float16)
    wide[:, :K] = X
    perm = workloads.random_perm(K, seed=18)
    Xq8, xs = clq.clq_rotate_quant_act8(dev(wide)[:, :K], block, perm=dev(perm))
    _, ref_c, ref_s = oracle.quantize_act(X, block, perm, bits=8)
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_act8(Xq8, M, K)), ref_c)


@pytest.mark.parametrize("M,K,with_perm", [(1000, 4608, False), (777, 4608, True), (13, 2048, False)])
def test_rotate_quant_act8_long_rows(clq, M, K, with_perm):
    # the 8-aligned-row batches of long rows (b = 64), int8 codes
    X = workloads.activations(M, K, "L2", seed=M + K)
    perm = workloads.random_perm(K, seed=M + 1) if with_perm else None
    Xq8, xs = clq.clq_rotate_quant_act8(dev(X), 64, perm=None if perm is None else dev(perm))
    _, ref_c, ref_s = oracle.quantize_act(X, 64, perm, bits=8)
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_act8(Xq8, M, K)), ref_c)


@pytest.mark.parametrize("N,K,block,clip", [
    (1, 64, 32, 1.0), (65, 1152, 64, 1.0), (200, 1152, 64, 0.8), (96, 3072, 128, 0.9),
    (40, 4608, 64, 0.5)])
def test_quantize_weights8_bitexact(clq, N, K, block, clip):
    W = workloads.weights(N, K, seed=N + K)
    qw = clq.clq_quantize_weights8(dev(W), block, clip_ratio=clip)
    _, ref_c, ref_ws = oracle.quantize_weights(W, block, None, clip, bits=8)
    assert np.array_equal(host(qw.w_scale), ref_ws)
    assert np.array_equal(host(clq.clq_unswizzle_weights8(qw)), ref_c)
    assert qw.wq.numel() == clq.clq_weight8_bytes(N, K)


# the last shape: several token-tile groups of 8 per XCD run, ragged token
# rows and channels
SHAPES = [(1, 1, 64), (7, 9, 128), (100, 200, 1152), (257, 129, 1152), (130, 520, 640),
          (300, 1000, 4608), (512, 256, 64), (1000, 384, 3072), (4100, 1030, 640)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("wbits", [4, 8])
def test_a8_accum_exact(clq, M, N, K, wbits):
    block = 64 if K % 64 == 0 and K >= 64 else 32
    X = workloads.activations(M, K, "L1", seed=M * 7 + K)
    W = workloads.weights(N, K, seed=N * 3 + K)
    Xq8, xs = clq.clq_rotate_quant_act8(dev(X), block)
    qw = (clq.clq_quantize_weights if wbits == 4 else clq.clq_quantize_weights8)(dev(W), block)
    _, xc, _ = oracle.quantize_act(X, block, bits=8)
    _, wc, _ = oracle.quantize_weights(W, block, bits=wbits)
    acc = host(clq.clq_a8_accum_i32(Xq8, xs, qw))
    assert np.array_equal(acc, oracle.gemm_i32(xc, wc))


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("wbits", [4, 8])
@pytest.mark.parametrize("with_bias", [True, False])
def test_a8_linear_tolerance(clq, M, N, K, wbits, with_bias):
    block = 64
    X = workloads.activations(M, K, "L2", seed=M + 3 * K)
    W = workloads.weights(N, K, seed=N + 5 * K)
    b = workloads.bias(N, seed=N) if with_bias else None
    Xq8, xs = clq.clq_rotate_quant_act8(dev(X), block)
    qw = (clq.clq_quantize_weights if wbits == 4 else clq.clq_quantize_weights8)(dev(W), block)
    Y = host(clq.clq_a8_linear(Xq8, xs, qw, None if b is None else dev(b)))
    r = oracle.linear(X, W, b, block, wbits=wbits, abits=8)
    assert oracle.err_metric(Y.astype(np.float64), r["y64"], r["p64"], b) <= TOL


@pytest.mark.parametrize("layer", workloads.C2.layers, ids=lambda l: l.name)
@pytest.mark.parametrize("wbits", [4, 8])
def test_full_size_layer_sampled(clq, layer, wbits):
    # the PixArt block's linears at full size (M = 8192); the oracle checks
    # a sample of token rows (codes, scales, sums, fp16 output)
    X, W, b = workloads.layer_inputs(layer)
    Xq8, xs = clq.clq_rotate_quant_act8(dev(X), layer.block)
    qw = (clq.clq_quantize_weights if wbits == 4 else clq.clq_quantize_weights8)(dev(W), layer.block)
    bd = dev(b)
    Y = host(clq.clq_a8_linear(Xq8, xs, qw, bd))
    acc = host(clq.clq_a8_accum_i32(Xq8, xs, qw))
    rows = np.r_[0:3, layer.M // 2:layer.M // 2 + 3, layer.M - 3:layer.M]
    r = oracle.linear(X[rows], W, b, layer.block, wbits=wbits, abits=8)
    assert np.array_equal(host(xs)[rows], r["x_scale"])
    assert np.array_equal(acc[rows], r["acc"])
    assert oracle.err_metric(Y[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL
