"""GPU parity: the HIP path (through the C ABI binding) against the CPU oracle.

Integer results -- activation codes and scales, weight codes (after
unswizzling) and scales, int32 accumulators -- must match bit for bit; the
fp16 output must lie within 2e-3 of the oracle's fp64 dequantised result
(err = max |y - y64| / max(|p64| + |bias|, 2^-24)).  Small shapes span
several tiles and ragged tails; full-size layers are checked on sampled
token rows the oracle can afford.
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


# ---- rotate + quantize ---------------------------------------------------------

@pytest.mark.parametrize("M,K,block", [
    (1, 64, 32), (7, 128, 64), (255, 1152, 64), (257, 1152, 32), (64, 1152, 128),
    (33, 4608, 64), (20, 3072, 128), (5, 12288, 128), (3, 64, 64), (9, 256, 128)])
@pytest.mark.parametrize("law", ["L1", "L2"])
def test_rotate_quant_bitexact(clq, M, K, block, law):
    X = workloads.activations(M, K, law, seed=M + K + block)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    ref_q, _, ref_s = oracle.quantize_act(X, block)
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_act(Xq, M, K)), ref_q)
    # padding rows of the packed buffer hold zero codes
    assert Xq.numel() == clq.clq_act_bytes(M, K)


# Long rows (b = 64, 2048 <= K <= 5120) are handled in batches of 8 aligned
# rows; ragged row counts, a gather vector and a wider row stride included.
@pytest.mark.parametrize("M,K,ld,with_perm", [
    (1000, 4608, 4608, False), (777, 4608, 4672, True), (9, 2048, 2048, True), (1001, 5120, 5120, False),
    (8, 4608, 4608, False)])
def test_rotate_quant_long_rows(clq, M, K, ld, with_perm):
    X = workloads.activations(M, K, "L1", seed=M + K + 11)
    wide = np.zeros((M, ld), np.float16)
    wide[:, :K] = X
    perm = workloads.random_perm(K, seed=M) if with_perm else None
    Xq, xs = clq.clq_rotate_quant_act(dev(wide)[:, :K], 64, perm=None if perm is None else dev(perm))
    ref_q, _, ref_s = oracle.quantize_act(X, 64, perm)
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_act(Xq, M, K)), ref_q)


@pytest.mark.parametrize("block", [32, 64, 128])
def test_rotate_quant_perm_and_stride(clq, block):
    M, K, ld = 37, 1152 if block != 128 else 1536, 2048
    X = workloads.activations(M, K, "L1", seed=block)
    wide = np.zeros((M, ld), np.float16)
    wide[:, :K] = X
    wide[:, K:] = np.float16(1000.0)          # must never be read
    perm = workloads.random_perm(K, seed=block + 1)
    Xd = dev(wide)[:, :K]
    Xq, xs = clq.clq_rotate_quant_act(Xd, block, dev(perm))
    ref_q, _, ref_s = oracle.quantize_act(X, block, perm)
    assert np.array_equal(host(xs), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_act(Xq, M, K)), ref_q)


def test_rotate_quant_adversarial_rows(clq):
    K, block = 256, 64
    X = np.zeros((8, K), np.float16)
    X[0, :] = np.float16(65504)
    X[1, ::2] = np.float16(-65504)
    X[2, :] = np.float16(-0.0)
    X[3, 17] = np.float16(6e-8)                   # one subnormal
    X[4, :] = np.float16(0.5)                     # exact ties after scaling
    X[4, 0] = np.float16(3.5)
    X[5, :64] = np.arange(64, dtype=np.float16) - np.float16(32)
    X[6, 3] = np.float16(-1.0)                    # single non-zero
    X[7, :] = workloads.activations(1, K, "L1", 3)[0]
    for block in (32, 64, 128):
        Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
        ref_q, _, ref_s = oracle.quantize_act(X, block)
        assert np.array_equal(host(xs), ref_s), block
        assert np.array_equal(host(clq.clq_unswizzle_act(Xq, 8, K)), ref_q), block


def test_act_padding_rows_are_zero(clq):
    M, K, block = 45, 256, 64                 # 45 rows -> 64 rows of storage
    X = workloads.activations(M, K, "L1", seed=4)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    assert Xq.numel() == 64 * K // 2
    full = host(clq.clq_unswizzle_act(Xq, 64, K))
    assert np.array_equal(full[:M], oracle.quantize_act(X, block)[0])
    assert not full[M:].any()


# ---- weights -------------------------------------------------------------------

@pytest.mark.parametrize("N,K,block,clip", [
    (1, 64, 32, 1.0), (8, 1152, 64, 1.0), (72, 1152, 64, 0.9), (200, 4608, 64, 1.0),
    (1152, 1152, 64, 1.0), (100, 3072, 128, 0.75), (3, 128, 128, 0.5)])
def test_quantize_weights_bitexact(clq, N, K, block, clip):
    W = workloads.weights(N, K, seed=N + K)
    qw = clq.clq_quantize_weights(dev(W), block, clip_ratio=clip)
    ref_q, _, ref_s = oracle.quantize_weights(W, block, None, clip)
    assert np.array_equal(host(qw.w_scale), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_weights(qw)), ref_q)


def test_quantize_weights_perm(clq):
    N, K, block = 96, 1152, 64
    W = workloads.weights(N, K, seed=5)
    perm = workloads.random_perm(K, seed=6)
    qw = clq.clq_quantize_weights(dev(W), block, dev(perm))
    ref_q, _, ref_s = oracle.quantize_weights(W, block, perm)
    assert np.array_equal(host(qw.w_scale), ref_s)
    assert np.array_equal(host(clq.clq_unswizzle_weights(qw)), ref_q)


# ---- GEMM: exact accumulators and the fp16 epilogue ------------------------------

# few tiles and at least 4 k-stages go through the two-halves kernel (the k
# loop split in two, the halves' sums added in LDS), including odd stage
# counts (one half a stage shorter) and ragged channels.  Its tiles have 128
# tokens, or 64 while the 128-token tiles would fill at most half the compute
# units: 64 for the small shapes, 128 for the last four (the last three at
# one to 2.5 tiles per compute unit, 8193 x 1030 in two rounds)
GEMM_SHAPES = [(1, 1, 64), (7, 8, 128), (129, 72, 192), (257, 200, 1152), (64, 1152, 1152),
               (300, 130, 640), (128, 128, 128), (513, 264, 4608), (257, 200, 576), (100, 1001, 320),
               (33, 48, 256), (5, 3, 256), (2049, 1030, 640), (4097, 1030, 640), (4000, 2000, 576),
               (8193, 1030, 576)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("workspace", [None, False], ids=["ws", "nows"])
def test_accum_i32_bitexact(clq, M, N, K, workspace):
    block = 64
    X = workloads.activations(M, K, "L1", seed=M)
    W = workloads.weights(N, K, seed=N)
    qw = clq.clq_quantize_weights(dev(W), block)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    acc = clq.clq_w4a4_accum_i32(Xq, xs, qw, workspace=workspace)
    _, xc, _ = oracle.quantize_act(X, block)
    _, wc, _ = oracle.quantize_weights(W, block)
    assert np.array_equal(host(acc), oracle.gemm_i32(xc, wc))


# Few tiles and a long k loop (the eight-wave kernel at these sizes), called
# repeatedly with a shared workspace.
SPLIT_SHAPES = [(2048, 1152, 4608), (2000, 1000, 4608), (2048, 640, 8192), (1024, 1152, 4608), (300, 520, 8192)]


@pytest.mark.parametrize("M,N,K", SPLIT_SHAPES)
def test_split_k_exact_and_repeatable(clq, M, N, K):
    block = 64
    X = workloads.activations(M, K, "L1", seed=M + 7)
    W = workloads.weights(N, K, seed=N + 7)
    b = workloads.bias(N, seed=8)
    qw = clq.clq_quantize_weights(dev(W), block)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    ref = oracle.linear(X, W, b, block)
    ws = torch.zeros(clq.clq_w4a4_workspace_bytes(), dtype=torch.uint8, device="cuda")
    for rep in range(3):          # the workspace is left ready for the next call
        acc = clq.clq_w4a4_accum_i32(Xq, xs, qw, workspace=ws)
        assert np.array_equal(host(acc), ref["acc"]), rep
        Y = clq.clq_w4a4_linear(Xq, xs, qw, dev(b), workspace=ws)
        assert oracle.err_metric(host(Y).astype(np.float64), ref["y64"], ref["p64"], b) <= TOL, rep
    groups = clq.clq_w4a4_workspace_bytes() // (128 * 256 * 4 + 4 * 4)
    assert not host(ws[:groups * 4 * 4]).any()     # every flag back at zero


def test_persistent_tail_split_exact(clq):
    # more tiles than compute units (the persistent kernel), a last round
    # split along k over every workgroup: the split sums equal the
    # whole-tile sums bit for bit and the oracle's on sampled rows
    M, N, K, block = 4352, 2048, 2432, 64     # 17 x 16 tiles, 38 k-stages
    X = workloads.activations(M, K, "L1", seed=61)
    W = workloads.weights(N, K, seed=62)
    qw = clq.clq_quantize_weights(dev(W), block)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    ws = torch.zeros(clq.clq_w4a4_workspace_bytes(), dtype=torch.uint8, device="cuda")
    split = host(clq.clq_w4a4_accum_i32(Xq, xs, qw, workspace=ws))
    whole = host(clq.clq_w4a4_accum_i32(Xq, xs, qw, workspace=False))
    assert np.array_equal(split, whole)
    rows = np.r_[0:3, 2047:2051, M - 3:M]
    _, xc, _ = oracle.quantize_act(X[rows], block)
    _, wc, _ = oracle.quantize_weights(W, block)
    assert np.array_equal(split[rows], oracle.gemm_i32(xc, wc))
    groups = clq.clq_w4a4_workspace_bytes() // (128 * 256 * 4 + 4 * 4)
    assert not host(ws[:groups * 4 * 4]).any()


def test_accum_i32_extremes(clq):
    """All codes +7 and alternating signs: |acc| reaches 49 K."""
    M, N, K, block = 48, 80, 4608, 64
    X = np.zeros((M, K), np.float16)
    X[:, 0] = np.float16(1.0)                 # a delta: every rotated entry is +-1
    X[1::2, 0] = np.float16(-1.0)
    W = np.zeros((N, K), np.float16)
    W[:, 0] = np.float16(1.0)
    qw = clq.clq_quantize_weights(dev(W), block)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    acc = host(clq.clq_w4a4_accum_i32(Xq, xs, qw))
    _, xc, _ = oracle.quantize_act(X, block)
    _, wc, _ = oracle.quantize_weights(W, block)
    ref = oracle.gemm_i32(xc, wc)
    assert np.array_equal(acc, ref)
    assert np.abs(ref).max() == 49 * block


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("with_bias", [True, False])
def test_linear_fp16_tolerance(clq, M, N, K, with_bias):
    block = 64
    X = workloads.activations(M, K, "L1", seed=M + 1)
    W = workloads.weights(N, K, seed=N + 1)
    b = workloads.bias(N, seed=3) if with_bias else None
    qw = clq.clq_quantize_weights(dev(W), block)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    Y = clq.clq_w4a4_linear(Xq, xs, qw, None if b is None else dev(b))
    ref = oracle.linear(X, W, b, block)
    err = oracle.err_metric(host(Y).astype(np.float64), ref["y64"], ref["p64"], b)
    assert err <= TOL, err


def test_linear_row_stride_and_zero_rows(clq):
    M, N, K, block, ldy = 70, 136, 1152, 64, 256
    X = workloads.activations(M, K, "L1", seed=9)
    X[5] = 0
    X[66] = 0
    W = workloads.weights(N, K, seed=10)
    b = workloads.bias(N, seed=11)
    qw = clq.clq_quantize_weights(dev(W), block)
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
    Ybig = torch.full((M, ldy), float("nan"), dtype=torch.float16, device="cuda")
    clq.clq_w4a4_linear(Xq, xs, qw, dev(b), out=Ybig[:, :N])
    Yh = host(Ybig)
    assert np.isnan(Yh[:, N:].astype(np.float32)).all()        # untouched padding
    ref = oracle.linear(X, W, b, block)
    assert oracle.err_metric(Yh[:, :N].astype(np.float64), ref["y64"], ref["p64"], b) <= TOL
    assert np.array_equal(Yh[5, :N], b) and np.array_equal(Yh[66, :N], b)   # zero rows -> bias


def test_linear_block128_perm(clq):
    M, N, K, block = 96, 192, 3072, 128
    X = workloads.activations(M, K, "L2", seed=12)
    W = workloads.weights(N, K, seed=13)
    b = workloads.bias(N, seed=14)
    perm = workloads.random_perm(K, seed=15)
    qw = clq.clq_quantize_weights(dev(W), block, dev(perm))
    Xq, xs = clq.clq_rotate_quant_act(dev(X), block, dev(perm))
    acc = clq.clq_w4a4_accum_i32(Xq, xs, qw)
    Y = clq.clq_w4a4_linear(Xq, xs, qw, dev(b))
    ref = oracle.linear(X, W, b, block, perm)
    assert np.array_equal(host(acc), ref["acc"])
    assert oracle.err_metric(host(Y).astype(np.float64), ref["y64"], ref["p64"], b) <= TOL


# ---- full-size layers (the shapes the benchmark times), sampled rows --------------

FULL = [l for w in (workloads.C2, workloads.C3, workloads.C4) for l in w.layers]


@pytest.mark.parametrize("layer", FULL, ids=[l.name for l in FULL])
def test_full_size_layer_sampled(clq, layer):
    X, W, b = workloads.layer_inputs(layer)
    qw = clq.clq_quantize_weights(dev(W), layer.block)
    Xd = dev(X)
    Xq, xs = clq.clq_rotate_quant_act(Xd, layer.block)
    Y = clq.clq_w4a4_linear(Xq, xs, qw, dev(b))
    rng = np.random.default_rng(layer.seed)
    rows = np.unique(np.concatenate([[0, layer.M - 1], rng.choice(layer.M, 30, replace=False)]))
    rows_t = torch.from_numpy(rows).cuda()
    Xq_s = host(clq.clq_unswizzle_act(Xq, layer.M, layer.K)[rows_t])
    xs_s, Y_s = host(xs[rows_t]), host(Y[rows_t])
    ref_xq, xc, ref_xs = oracle.quantize_act(X[rows], layer.block)
    assert np.array_equal(xs_s, ref_xs)
    assert np.array_equal(Xq_s, ref_xq)
    wq_ref, wc, ws_ref = oracle.quantize_weights(W, layer.block)
    assert np.array_equal(host(qw.w_scale), ws_ref)
    acc = oracle.gemm_i32(xc, wc)
    y64, p64 = oracle.epilogue(acc, ref_xs, ws_ref, b)
    assert oracle.err_metric(Y_s.astype(np.float64), y64, p64, b) <= TOL
    # the exact accumulators on the same rows, through the int32 variant
    acc_gpu = clq.clq_w4a4_accum_i32(Xq, xs, qw)
    assert np.array_equal(host(acc_gpu[rows_t]), acc)
