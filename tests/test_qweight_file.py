"""Serialised quantized weights (host side, no GPU): the file format carries
the library version of the packed layout, and a file from another version or
with mismatched sizes is refused."""
import os

import pytest

torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2509_24416_amd", "libclq.so")


@pytest.fixture(scope="module")
def clq():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    import paper_2509_24416_amd as m
    return m


def _write(path, meta, wq, ws):
    from safetensors.torch import save_file
    save_file({"wq": wq, "w_scale": ws}, path, metadata=meta)


def test_version_and_size_checks(clq, tmp_path):
    N, K = 64, 128
    good = {"format": "clq-qweight", "clq_version": str(clq.clq_version()), "N": str(N), "K": str(K),
            "block": "64", "clip_ratio": "1.0", "bits": "4"}
    wq = torch.zeros(clq.clq_weight_bytes(N, K), dtype=torch.uint8)
    ws = torch.ones(N, dtype=torch.float32)
    p = str(tmp_path / "a.safetensors")
    _write(p, dict(good, clq_version=str(clq.clq_version() - 1)), wq, ws)
    with pytest.raises(ValueError, match="version"):
        clq.load_qweight(p, device="cpu")
    _write(p, good, wq[:-1].clone(), ws)
    with pytest.raises(ValueError, match="sizes"):
        clq.load_qweight(p, device="cpu")
    _write(p, dict(good, format="other"), wq, ws)
    with pytest.raises(ValueError, match="not a CLQ"):
        clq.load_qweight(p, device="cpu")
    _write(p, good, wq, ws)
    qw = clq.load_qweight(p, device="cpu")
    assert (qw.N, qw.K, qw.block, qw.bits) == (N, K, 64, 4) and qw.perm is None
