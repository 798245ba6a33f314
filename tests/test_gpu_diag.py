"""The diagnostic matrix-core probe behind the benchmark's measured ceiling:
it runs, is deterministic, and its work is not optimised away."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def clq():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2509_24416_amd as m
    return m


def test_mfma_probe_runs_and_is_deterministic(clq):
    g = torch.Generator(device="cpu").manual_seed(5)
    ops = torch.randint(0, 256, (clq.clq_diag_mfma_probe_bytes(),), dtype=torch.uint8, generator=g).cuda()
    grid = 8
    s1 = torch.zeros(grid * 256, dtype=torch.int32, device="cuda")
    s2 = torch.zeros_like(s1)
    n = clq.clq_diag_mfma_probe(ops, 3, grid, s1)
    clq.clq_diag_mfma_probe(ops, 3, grid, s2)
    torch.cuda.synchronize()
    assert n == grid * 3 * 64 * 2 * 32 ** 3
    a, b = s1.cpu().numpy(), s2.cpu().numpy()
    assert np.array_equal(a, b) and np.count_nonzero(a) > a.size // 2
    # a different iteration count changes the sums
    clq.clq_diag_mfma_probe(ops, 4, grid, s2)
    torch.cuda.synchronize()
    assert not np.array_equal(a, s2.cpu().numpy())


def test_mfma_probe_f6_runs_and_is_deterministic(clq):
    g = torch.Generator(device="cpu").manual_seed(6)
    ops = torch.randint(0, 256, (clq.clq_diag_mfma_probe_bytes(),), dtype=torch.uint8, generator=g).cuda()
    grid = 8
    s1 = torch.zeros(grid * 256, dtype=torch.int32, device="cuda")
    s2 = torch.zeros_like(s1)
    n = clq.clq_diag_mfma_probe_f6(ops, 3, grid, s1)
    clq.clq_diag_mfma_probe_f6(ops, 3, grid, s2)
    torch.cuda.synchronize()
    assert n == grid * 3 * 64 * 2 * 32 * 32 * 64
    a, b = s1.cpu().numpy(), s2.cpu().numpy()
    # each lane stores the float sum of its accumulators: integer-valued
    # (products of codes on the integer grid, exact in fp32) and finite
    f = a.view(np.float32)
    assert np.array_equal(a, b) and np.count_nonzero(a) > a.size // 2
    assert np.all(np.isfinite(f)) and np.array_equal(f, np.round(f))
    clq.clq_diag_mfma_probe_f6(ops, 4, grid, s2)
    torch.cuda.synchronize()
    assert not np.array_equal(a, s2.cpu().numpy())
