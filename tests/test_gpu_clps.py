"""GPU parity of the single-layer CLPS clip search against the CPU oracle.

Paper: "CLQ" (arXiv 2509.24416), Sec. 3.4, Eq. (3) and Sec. 4.1 (beta = 0,
gamma = 0.01).  The candidate clip ratios must match bit for bit (integer
order statistics and fp32 arithmetic in the same order); the fp64 errors
agree to 1e-12 relative (sums in different orders); the chosen candidate
must be the oracle's, or carry the same error to that precision (a tie).
"""
import numpy as np
import pytest

import oracle
from oracle import clps
import workloads

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


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


def check(clq, X, W, block, perm=None, gamma=0.01, G=12):
    Y0 = oracle.linear_fp64(X, W).astype(np.float32)
    al, er, best = clq.clq_clps_search(dev(X), dev(W), dev(Y0), block,
                                       perm=None if perm is None else dev(perm), gamma=gamma, grid=G)
    ral, rer, rbest = clps.search(X, W, Y0, block, perm, gamma, G)
    assert np.array_equal(host(al), ral)
    e = host(er)
    assert np.allclose(e, rer, rtol=1e-12, atol=0)
    b = int(host(best)[0])
    assert b == rbest or abs(rer[b] - rer[rbest]) <= 1e-12 * rer[rbest]
    return b, ral


@pytest.mark.parametrize("M,N,K,block", [(64, 48, 1152, 64), (100, 70, 4608, 64), (33, 130, 3072, 128),
                                         (256, 256, 1152, 32), (1, 1, 64, 64)])
def test_search_matches_oracle(clq, M, N, K, block):
    X = workloads.activations(M, K, "L1", seed=M + K)
    W = workloads.weights(N, K, seed=N + K)
    check(clq, X, W, block)


def test_search_with_swap_and_l2(clq):
    K = 1152
    X = workloads.activations(80, K, "L2", seed=3)
    W = workloads.weights(60, K, seed=4)
    check(clq, X, W, 64, perm=workloads.random_perm(K, 5), G=20)


def test_degenerate_windows(clq):
    K = 1152
    X = workloads.activations(40, K, "L1", seed=6)
    W = workloads.weights(30, K, seed=7)
    # gamma = 0: the window is the max itself, every candidate is 1 -> ties,
    # the first wins
    b, al = check(clq, X, W, 64, gamma=0.0, G=5)
    assert np.all(al == 1.0) and b == 0
    # one candidate
    b, al = check(clq, X, W, 64, G=1)
    assert al.tolist() == [1.0] and b == 0
    # a row of zeros counts as ratio 1
    Wz = W.copy()
    Wz[3] = 0
    check(clq, X, Wz, 64, G=6)
    # weights on a coarse lattice: the rotated rows repeat their magnitudes
    # many times, so the order statistic falls inside runs of equal values
    Wl = (np.round(W.astype(np.float32) * 64.0) / 64.0).astype(np.float16)
    check(clq, X, Wl, 64, gamma=0.05, G=6)
    check(clq, X, Wl, 32, gamma=0.2, G=6)


def test_calibration_sized_layer(clq):
    # PixArt qkv width: 1024 calibration tokens, 1152 -> 1152 channels
    K, N = 1152, 1152
    X = workloads.activations(1024, K, "L1", seed=11)
    W = workloads.weights(N, K, seed=12)
    b, al = check(clq, X, W, 64, G=20)
    assert b < len(al) - 1     # clipping helps Gaussian weight rows


@pytest.mark.parametrize("pad", [4, 3])   # aligned rows (vector loads), misaligned rows (element loads)
def test_search_strided_target(clq, pad):
    # the target as a column slice of a wider fp32 tensor: the fused error
    # epilogue reads it through its row stride
    M, N, K, b = 96, 256, 1152, 64
    X = workloads.activations(M, K, "L1", seed=41)
    W = workloads.weights(N, K, seed=42)
    Y0 = oracle.linear_fp64(X, W).astype(np.float32)
    wide = np.full((M, N + pad), np.nan, np.float32)
    wide[:, :N] = Y0
    al, er, best = clq.clq_clps_search(dev(X), dev(W), dev(wide)[:, :N], b, grid=8)
    ral, rer, rbest = clps.search(X, W, Y0, b, G=8)
    assert np.array_equal(host(al), ral)
    assert np.allclose(host(er), rer, rtol=1e-12, atol=0)
    bb = int(host(best)[0])
    assert bb == rbest or abs(rer[bb] - rer[rbest]) <= 1e-12 * rer[rbest]
