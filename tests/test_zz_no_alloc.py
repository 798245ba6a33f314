"""The allocation-free linear (clq_w4a4_linear_noalloc) against
clq_w4a4_linear, through the C ABI.

Same kernels, so the fp16 outputs must be identical bit for bit (and within
the 2e-3 bound of the oracle, which the linear's own tests establish); two
calls in a row share the library's per-device scratch, the second with a
smaller input, both on shapes whose schedule splits the k loop (the scratch
is in use), then one that does not split.
"""
import ctypes

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
    L = m.lib()
    p, i64 = ctypes.c_void_p, ctypes.c_int64
    L.clq_w4a4_linear_noalloc.argtypes = [p, p, p, p, p, i64, i64, i64, p, i64, p, p]
    L.clq_w4a4_linear_noalloc.restype = ctypes.c_int
    return m


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def test_noalloc_matches_linear(clq):
    L = clq.lib()
    stream = torch.cuda.current_stream()
    block = 64
    # (11264, 3200, 1536): one whole round then a split one; (6300, 3000,
    # 1536): smaller, ragged, both rounds split; (300, 520, 1152): no split
    shapes = [(11264, 3200, 1536, 80), (6300, 3000, 1536, 81), (300, 520, 1152, 82)]
    status = torch.full((3,), -1, dtype=torch.int32, device="cuda")
    for M, N, K, seed in shapes:
        split = clq.clq_w4a4_schedule(M, N, K)["split_stages"] > 0
        assert split == (M > 1000)
        X = workloads.activations(M, K, "L1", seed=seed)
        W = workloads.weights(N, K, seed=seed + 100)
        b = workloads.bias(N, seed=seed + 200)
        qw = clq.clq_quantize_weights(dev(W), block)
        Xq, xs = clq.clq_rotate_quant_act(dev(X), block)
        bd = dev(b)
        ws = torch.zeros(clq.clq_w4a4_workspace_bytes(), dtype=torch.uint8, device="cuda")
        ref = clq.clq_w4a4_linear(Xq, xs, qw, bd, workspace=ws)
        Y = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda")
        rc = L.clq_w4a4_linear_noalloc(_ptr(Xq), _ptr(xs), _ptr(qw.wq), _ptr(qw.w_scale), _ptr(bd), M, N, K,
                                       _ptr(Y), Y.stride(0), _ptr(status), ctypes.c_void_p(stream.cuda_stream))
        assert rc == 0, clq.lib().clq_status_string(rc)
        torch.cuda.synchronize()
        assert status.cpu().tolist() == [0, 0, 0]
        Yh, Rh = Y.cpu().numpy(), ref.cpu().numpy()
        assert np.array_equal(Yh.view(np.uint16), Rh.view(np.uint16)), (M, N, K)
        # and within the bound of the oracle on sampled rows
        rows = np.r_[0:2, M // 2, M - 2:M]
        r = oracle.linear(X[rows], W, b, block)
        assert oracle.err_metric(Yh[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL


def test_noalloc_validation(clq):
    L = clq.lib()
    A = ctypes.c_void_p(0x10000)
    # NULL pointers and misaligned status are rejected before any launch
    assert L.clq_w4a4_linear_noalloc(None, A, A, A, None, 8, 8, 64, A, 8, None, None) == 1
    assert L.clq_w4a4_linear_noalloc(A, A, A, A, None, 8, 8, 64, A, 8, ctypes.c_void_p(0x10002), None) == 4
    assert L.clq_w4a4_linear_noalloc(A, A, A, A, None, 8, 8, 96, A, 8, None, None) == 2
