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


_HOST_W = {}


def stack_weights(nblocks, M, block):
    """Host weights and biases of the stack's linears (they do not depend on
    M or the block size; drawn once per process)."""
    wl = workloads.dit_stack(nblocks, M, block)
    host_w = {}
    for l in wl.layers:
        if l.name not in _HOST_W:
            _HOST_W[l.name] = (workloads.weights(l.N, l.K, l.seed + 1), workloads.bias(l.N, l.seed + 2))
        host_w[l.name] = _HOST_W[l.name]
    return wl, host_w


def build(nblocks, M, block, codes="int4"):
    from paper_2509_24416_amd.stack import DiTStack
    wl, host_w = stack_weights(nblocks, M, block)
    weights = []
    for j in range(nblocks):
        blk = {}
        for l in wl.layers[4 * j:4 * j + 4]:
            W, b = host_w[l.name]
            blk[l.name.split(".")[1]] = (dev(W), dev(b))
        weights.append(blk)
    x = workloads.activations(M, wl.layers[0].K, "L1", wl.layers[0].seed)
    return DiTStack(weights, M, block, codes=codes), host_w, x


@pytest.mark.parametrize("M,block,codes", [(1024, 64, "int4"), (300, 32, "int4"), (512, 128, "int4"),
                                           (300, 32, "fp6"), (512, 128, "fp6")])
def test_layers_match_oracle_on_their_inputs(clq, M, block, codes):
    st, host_w, x = build(3, M, block, codes)
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


@pytest.mark.parametrize("block", [32, 64, 128])
def test_full_depth_stack_layers_match_oracle(clq, block):
    # the 28-block stack (112 linears) at M = 4096: every linear of blocks 0,
    # 13 and 27 against the oracle on that linear's actual fp16 input, on
    # sampled token rows -- activation codes and scales bit for bit, the fp16
    # output within the tolerance
    M, nb = 4096, 28
    st, host_w, x = build(nb, M, block)
    taps = {(j, n): None for j in (0, 13, 27) for n in ("qkv", "proj", "fc1", "fc2")}
    st.forward(dev(x), taps=taps)
    rng = np.random.default_rng(block)
    rows = np.unique(np.concatenate([[0, 1, M - 1], rng.choice(M, 13, replace=False)]))
    rows_t = torch.from_numpy(rows).cuda()
    for (j, name), (xin, y) in taps.items():
        W, b = host_w[f"blk{j}.{name}"]
        xin_h = host(xin)[rows]
        assert np.isfinite(xin_h.astype(np.float32)).all(), (j, name)
        r = oracle.linear(xin_h, W, b, block)
        Xq, xs = clq.clq_rotate_quant_act(xin, block)
        K = xin.shape[1]
        assert np.array_equal(host(xs)[rows], r["x_scale"]), (j, name)
        assert np.array_equal(host(clq.clq_unswizzle_act(Xq, M, K)[rows_t]), r["xq"]), (j, name)
        assert oracle.err_metric(host(y)[rows].astype(np.float64), r["y64"], r["p64"], b) <= TOL, (j, name)
    del st
    torch.cuda.empty_cache()


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


@pytest.mark.parametrize("M,block", [(300, 64), (256, 128)])
def test_swap_folded_upstream_matches_gather(clq, M, block):
    # one swap vector per layer input (Sec. 3.3's s): gathering it in every
    # rotate+quant and folding it into the producing layer's output channels
    # give the same bits; the folded producers' outputs come out gathered
    from paper_2509_24416_amd.stack import DiTStack, LAYERS
    nb = 3
    wl = workloads.dit_stack(nb, M, block)
    x = workloads.activations(M, wl.layers[0].K, "L1", wl.layers[0].seed)
    weights = [{} for _ in range(nb)]
    for j in range(nb):
        for l in wl.layers[4 * j:4 * j + 4]:
            weights[j][l.name.split(".")[1]] = (dev(workloads.weights(l.N, l.K, l.seed + 1)),
                                                dev(workloads.bias(l.N, l.seed + 2)))
    perms = [{name: dev(workloads.random_perm(weights[j][name][0].shape[1], 100 * j + i))
              for i, name in enumerate(LAYERS)} for j in range(nb)]
    a = DiTStack(weights, M, block, perms=perms, fold=False)
    f = DiTStack(weights, M, block, perms=perms, fold=True)
    ta = {(j, n): None for j in range(nb) for n in LAYERS}
    tf = dict(ta)
    ya = host(a.forward(dev(x), taps=ta)).copy()
    yf = host(f.forward(dev(x), taps=tf)).copy()
    assert np.array_equal(ya.view(np.uint16), yf.view(np.uint16))
    for (j, name), (xa, _) in ta.items():
        xf = host(tf[(j, name)][0])
        s = host(perms[j][name]).astype(np.int64)
        want = host(xa) if (j, name) == (0, "qkv") else host(xa)[:, s]
        assert np.array_equal(xf.view(np.uint16), want.view(np.uint16)), (j, name)
    # the folded stack gathers only at its first input
    assert [f.gather[j][n] is None for j in range(nb) for n in LAYERS].count(False) == 1


def test_fp6_stack_matches_int4_stack(clq):
    # the same codes in either storage give the same fp16 outputs layer by
    # layer, so the whole chain stays bit-identical; the fp6 stack also
    # replays as a graph
    M, block = 1024, 64
    st4, _, x = build(6, M, block, "int4")
    y4 = host(st4.forward(dev(x))).copy()
    del st4
    st6, _, _ = build(6, M, block, "fp6")
    y6 = host(st6.forward(dev(x))).copy()
    assert np.array_equal(y4.view(np.uint16), y6.view(np.uint16))
    st6.capture()
    for _ in range(2):
        got = host(st6.replay(dev(x)))
        assert np.array_equal(got.view(np.uint16), y6.view(np.uint16))


def test_fp6_stack_rejects_fuse(clq):
    # checked before any weight is touched
    from paper_2509_24416_amd.stack import DiTStack
    with pytest.raises(ValueError):
        DiTStack([], 64, 64, fuse=True, codes="fp6")
    with pytest.raises(ValueError):
        DiTStack([], 64, 64, codes="int8")
