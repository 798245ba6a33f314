"""The fused inter-layer path: clq_w4a4_rq_linear, the consumer's
rotate+quantize folded into the W4A4 GEMM launch.

The fused launch runs the same arithmetic as clq_rotate_quant_act followed by
clq_w4a4_linear, so its codes, scales and fp16 output must equal theirs bit
for bit (and, through them, the oracle: codes and scales exactly, the output
within 2e-3 on sampled rows).  Paper: "CLQ" (arXiv 2509.24416), Sec. 3.3
(online block-Hadamard rotation) and Sec. 3.1 Eq. (1) (per-token quantizer),
applied in front of every linear of a DiT stack (Sec. 4.1).
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


# (M, N, K, block): 64-token tiles (1024 x 1152), 128-token tiles (1024 x
# 3456), ragged token counts, long rows (4 rows per item at K = 2048),
# every Hadamard block, and a shape on the persistent grid (two launches)
SHAPES = [(1024, 1152, 1152, 64), (1024, 3456, 1152, 64), (1000, 3456, 1152, 32), (777, 1152, 1152, 128),
          (1024, 1152, 2048, 64), (2048, 1152, 4608, 64), (4096, 1152, 1152, 64), (300, 4608, 1152, 128),
          (33, 1152, 1152, 64), (8192, 3456, 1152, 64)]
# two launches: the persistent grid (8192 x 3456), items of fewer than 4
# rows (K = 4608 at 64-token tiles)
TWO_LAUNCHES = {(8192, 3456, 1152), (2048, 1152, 4608)}


@pytest.mark.parametrize("M,N,K,block", SHAPES)
@pytest.mark.parametrize("with_bias", [True, False], ids=["bias", "nobias"])
def test_fused_equals_two_launches_and_oracle(clq, M, N, K, block, with_bias):
    plan = clq.clq_w4a4_rq_schedule(M, N, K, block)
    assert plan["fused"] == (0 if (M, N, K) in TWO_LAUNCHES else 1), plan
    assert plan["fused"] == 0 or plan["rows_per_item"] >= 4, plan
    X = workloads.activations(M, K, "L1", seed=M + N + K)
    W = workloads.weights(N, K, seed=N + 5)
    b = workloads.bias(N, seed=6) if with_bias else None
    qw = clq.clq_quantize_weights(dev(W), block)
    bd = None if b is None else dev(b)
    Xd = dev(X)
    Xq_ref, xs_ref = clq.clq_rotate_quant_act(Xd, block)
    Y_ref = clq.clq_w4a4_linear(Xq_ref, xs_ref, qw, bd, workspace=False)
    ws = torch.zeros(clq.clq_w4a4_workspace_bytes(), dtype=torch.uint8, device="cuda")
    Yr, Xqr, xsr = host(Y_ref), host(Xq_ref), host(xs_ref)
    for rep in range(3):   # the workspace's queue state carries over between calls
        Xq = torch.full_like(Xq_ref, 0x5A)
        xs = torch.full_like(xs_ref, float("nan"))
        Y, _, _ = clq.clq_w4a4_rq_linear(Xd, block, qw, bd, Xq_out=Xq, scale_out=xs, workspace=ws)
        assert np.array_equal(host(Xq), Xqr), rep
        assert np.array_equal(host(xs), xsr), rep
        assert np.array_equal(host(Y).view(np.uint16), Yr.view(np.uint16)), rep
    assert clq.clq_w4a4_workspace_status(ws) == [0, 0, 0]
    rows = np.unique(np.r_[0:2, M // 2, M - 2:M])
    r = oracle.linear(X[rows], W, b, block)
    assert np.array_equal(xsr[rows], r["x_scale"])
    assert np.array_equal(host(clq.clq_unswizzle_act(Xq_ref, M, K))[rows], r["xq"])
    assert oracle.err_metric(Yr[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL


def test_fused_strided_input_and_next_call(clq):
    # a column slice of a wider tensor (the proj input read out of qkv's
    # output), then a different input through the same workspace
    M, N, K, block, ld = 1024, 1152, 1152, 64, 3456
    W = workloads.weights(N, K, seed=41)
    qw = clq.clq_quantize_weights(dev(W), block)
    ws = torch.zeros(clq.clq_w4a4_workspace_bytes(), dtype=torch.uint8, device="cuda")
    for seed in (42, 43):
        wide = dev(workloads.activations(M, ld, "L1", seed=seed))
        X = wide[:, :K]
        Xq_ref, xs_ref = clq.clq_rotate_quant_act(X, block)
        Y_ref = clq.clq_w4a4_linear(Xq_ref, xs_ref, qw, workspace=False)
        Y, Xq, xs = clq.clq_w4a4_rq_linear(X, block, qw, workspace=ws)
        assert np.array_equal(host(Xq), host(Xq_ref)) and np.array_equal(host(xs), host(xs_ref))
        assert np.array_equal(host(Y).view(np.uint16), host(Y_ref).view(np.uint16))


@pytest.mark.parametrize("M,block", [(1024, 64), (300, 32), (512, 128)])
def test_fused_stack_equals_unfused_and_replays(clq, M, block):
    from paper_2509_24416_amd.stack import DiTStack
    nb = 3
    wl = workloads.dit_stack(nb, M, block)
    weights = [{} for _ in range(nb)]
    for j in range(nb):
        for l in wl.layers[4 * j:4 * j + 4]:
            weights[j][l.name.split(".")[1]] = (dev(workloads.weights(l.N, l.K, l.seed + 1)),
                                                dev(workloads.bias(l.N, l.seed + 2)))
    x = dev(workloads.activations(M, 1152, "L1", 500))
    a = DiTStack(weights, M, block, fuse=False)
    f = DiTStack(weights, M, block, fuse=True)
    ya = host(a.forward(x)).copy()
    yf = host(f.forward(x)).copy()
    assert np.array_equal(ya.view(np.uint16), yf.view(np.uint16))
    f.capture()
    other = dev(workloads.activations(M, 1152, "L1", 77))
    for _ in range(3):
        f.forward(other)
        torch.cuda.synchronize()
        got = host(f.replay(x))
        assert np.array_equal(got.view(np.uint16), ya.view(np.uint16))
    assert clq.clq_w4a4_workspace_status(f.ws) == [0, 0, 0]
