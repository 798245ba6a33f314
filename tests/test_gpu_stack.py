"""The multi-layer path: a stack of DiT-block linears on the GPU, eager and
as one replayed HIP graph.

Paper: "CLQ" (arXiv 2509.24416), Sec. 4.1 (every linear of the DiT blocks
quantized W4A4) with Sec. 3.3's online rotation before each.  Parity is per
layer, against the oracle applied to that layer's actual GPU fp16 input (so
quantization errors do not compound into the comparison); graph replays
must reproduce the eager result bit for bit (every kernel is deterministic).
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


def build(nblocks, M, block):
    from paper_2509_24416_amd.stack import DiTStack
    wl = workloads.dit_stack(nblocks, M, block)
    weights, host_w = [], {}
    for j in range(nblocks):
        blk = {}
        for l in wl.layers[4 * j:4 * j + 4]:
            W, b = workloads.weights(l.N, l.K, l.seed + 1), workloads.bias(l.N, l.seed + 2)
            host_w[l.name] = (W, b)
            blk[l.name.split(".")[1]] = (dev(W), dev(b))
        weights.append(blk)
    x = workloads.activations(M, wl.layers[0].K, "L1", wl.layers[0].seed)
    return DiTStack(weights, M, block), host_w, x


@pytest.mark.parametrize("M,block", [(1024, 64), (300, 32), (512, 128)])
def test_layers_match_oracle_on_their_inputs(clq, M, block):
    st, host_w, x = build(3, M, block)
    taps = {(0, "qkv"): None, (0, "proj"): None, (1, "fc1"): None, (1, "fc2"): None, (2, "qkv"): None,
            (2, "fc2"): None}
    st.forward(dev(x), taps=taps)
    rows = np.r_[0:4, M // 2:M // 2 + 4, M - 4:M]
    for (j, name), (xin, y) in taps.items():
        W, b = host_w[f"blk{j}.{name}"]
        xin_h = host(xin)[rows]
        assert np.isfinite(xin_h.astype(np.float32)).all()
        r = oracle.linear(xin_h, W, b, block)
        assert oracle.err_metric(host(y)[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL, (j, name)


def test_graph_replays_match_eager(clq):
    M, block = 1024, 64
    st, _, x = build(4, M, block)
    ref = host(st.forward(dev(x))).copy()
    st.capture()
    other = dev(workloads.activations(M, 1152, "L1", 77))
    for _ in range(3):
        # eager work between replays (a different input through the same
        # buffers), then the graph on the original input
        st.forward(other)
        torch.cuda.synchronize()
        got = host(st.replay(dev(x)))
        assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


def test_full_depth_stack_is_finite_and_replays(clq):
    # 28 blocks (112 linears) at M = 1024: outputs stay finite through the
    # chain and one graph replay equals the eager pass
    M = 1024
    st, _, x = build(28, M, 64)
    ref = host(st.forward(dev(x))).copy()
    assert np.isfinite(ref.astype(np.float32)).all()
    st.capture()
    got = host(st.replay())
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))
