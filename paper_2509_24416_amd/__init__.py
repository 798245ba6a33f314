"""Python binding of libclq.so: the W4A4 DiT linear hot path on MI355X.

Argument marshalling only.  Every step of the path runs in the library's HIP
kernels; torch supplies device memory and the current stream.  The functions
carry the names of the C entry points declared in ``include/clq.h``:

    clq_quantize_weights(W, block, perm=None, clip_ratio=1.0) -> QWeight
    clq_rotate_quant_act(X, block, perm=None)                 -> (Xq, x_scale)
    clq_w4a4_linear(Xq, x_scale, qw, bias=None)               -> Y
    clq_w4a4_accum_i32(Xq, x_scale, qw)                        -> acc
    clq_unswizzle_weights(qw)                                  -> canonical codes
    clq_unswizzle_act(Xq, M, K)                                -> canonical codes
    clq_obs_channel_scores(X, metric="absmax")                 -> scores [D]
    clq_obs_permutation(scores)                                -> perm [D]
    clq_rotate_quant_act8(X, block, perm=None)                 -> (Xq8, x_scale)
    clq_quantize_weights8(W, block, perm=None, clip_ratio=1.0) -> QWeight (8-bit)
    clq_a8_linear(Xq8, x_scale, qw, bias=None)                 -> Y   (W4A8 / W8A8)
    clq_a8_accum_i32(Xq8, x_scale, qw)                         -> acc
    clq_unswizzle_act8(Xq8, M, K), clq_unswizzle_weights8(qw)  -> int8 codes
    clq_clps_search(X, W, Y0, block, perm=None, gamma=0.01, grid=20)
                                                               -> (alphas, errors, best)

Paper: "CLQ" (arXiv 2509.24416) -- Sec. 3.3 (online block-Hadamard rotation,
weights absorb it offline) and Sec. 3.1 Eq. (1) (4-bit quantizer; dynamic
per-token activations, per-channel weights).

Importing this package fails loudly if ``libclq.so`` has not been built;
there is no fallback path.
"""
import ctypes
import os
from dataclasses import dataclass

import torch  # loads the HIP runtime that libclq.so then shares

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libclq.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'` "
        "(or python paper_2509_24416_amd/build.py)")

_lib = ctypes.CDLL(LIB_PATH)

_i64, _i32, _f32, _p = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
_lib.clq_version.restype = ctypes.c_int
_lib.clq_status_string.restype = ctypes.c_char_p
_lib.clq_status_string.argtypes = [ctypes.c_int]
_lib.clq_weight_bytes.restype = ctypes.c_size_t
_lib.clq_weight_bytes.argtypes = [_i64, _i64]
_lib.clq_act_bytes.restype = ctypes.c_size_t
_lib.clq_act_bytes.argtypes = [_i64, _i64]
_lib.clq_quantize_weights.argtypes = [_p, _p, _i64, _i64, _i32, _f32, _p, _p, _p]
_lib.clq_rotate_quant_act.argtypes = [_p, _i64, _p, _i64, _i64, _i32, _p, _p, _p]
_lib.clq_w4a4_workspace_bytes.restype = ctypes.c_size_t
_lib.clq_w4a4_workspace_bytes.argtypes = []
_lib.clq_w4a4_linear.argtypes = [_p, _p, _p, _p, _p, _i64, _i64, _i64, _p, _i64, _p, ctypes.c_size_t, _p]
_lib.clq_w4a4_accum_i32.argtypes = [_p, _p, _i64, _i64, _i64, _p, _i64, _p, ctypes.c_size_t, _p]
_lib.clq_unswizzle_weights.argtypes = [_p, _i64, _i64, _p, _p]
_lib.clq_unswizzle_act.argtypes = [_p, _i64, _i64, _p, _p]
_lib.clq_obs_workspace_bytes.restype = ctypes.c_size_t
_lib.clq_obs_workspace_bytes.argtypes = [_i64, _i64, _i32]
_lib.clq_obs_channel_scores.argtypes = [_p, _i64, _i64, _i64, _i64, _i32, _p, ctypes.c_size_t, _p, _p]
_lib.clq_obs_permutation.argtypes = [_p, _i64, _p, _p]
_lib.clq_act8_bytes.restype = ctypes.c_size_t
_lib.clq_act8_bytes.argtypes = [_i64, _i64]
_lib.clq_weight8_bytes.restype = ctypes.c_size_t
_lib.clq_weight8_bytes.argtypes = [_i64, _i64]
_lib.clq_rotate_quant_act8.argtypes = [_p, _i64, _p, _i64, _i64, _i32, _p, _p, _p]
_lib.clq_quantize_weights8.argtypes = [_p, _p, _i64, _i64, _i32, _f32, _p, _p, _p]
_lib.clq_a8_linear.argtypes = [_p, _p, _p, _p, _i32, _p, _i64, _i64, _i64, _p, _i64, _p]
_lib.clq_a8_accum_i32.argtypes = [_p, _p, _i32, _i64, _i64, _i64, _p, _i64, _p]
_lib.clq_unswizzle_act8.argtypes = [_p, _i64, _i64, _p, _p]
_lib.clq_unswizzle_weights8.argtypes = [_p, _i64, _i64, _p, _p]
_lib.clq_clps_workspace_bytes.restype = ctypes.c_size_t
_lib.clq_clps_workspace_bytes.argtypes = [_i64, _i64, _i64]
_lib.clq_clps_search.argtypes = [_p, _i64, _p, _p, _i64, _p, _i64, _i64, _i64, _i32, _f32, _i32, _p,
                                 ctypes.c_size_t, _p, _p, _p, _p]
_lib.clq_w4a4_workspace_status.argtypes = [_p, ctypes.c_size_t, _p, _p]
_lib.clq_debug_set.argtypes = [_i32, _i64]
_lib.clq_w4a4_schedule.argtypes = [_i64, _i64, _i64, _i32, _p]
_lib.clq_w4a4_linear_noalloc.argtypes = [_p, _p, _p, _p, _p, _i64, _i64, _i64, _p, _i64, _p, _p]
_lib.clq_w4a4_rq_linear.argtypes = [_p, _i64, _i32, _p, _p, _p, _p, _p, _i64, _i64, _i64, _p, _i64, _p,
                                    ctypes.c_size_t, _p]
_lib.clq_w4a4_rq_schedule.argtypes = [_i64, _i64, _i64, _i32, _i32, _p]
_lib.clq_diag_mfma_probe_bytes.restype = ctypes.c_size_t
_lib.clq_diag_mfma_probe_bytes.argtypes = []
_lib.clq_diag_mfma_probe.argtypes = [_p, ctypes.c_size_t, _i32, _i32, _p, _p]
_lib.clq_diag_mfma_probe_f6.argtypes = [_p, ctypes.c_size_t, _i32, _i32, _p, _p]
_lib.clq_debug_get.argtypes = [_i32]
_lib.clq_debug_get.restype = _i64
_lib.clq_weight_bytes_f6.restype = ctypes.c_size_t
_lib.clq_weight_bytes_f6.argtypes = [_i64, _i64]
_lib.clq_act_bytes_f6.restype = ctypes.c_size_t
_lib.clq_act_bytes_f6.argtypes = [_i64, _i64]
_lib.clq_quantize_weights_f6.argtypes = [_p, _p, _i64, _i64, _i32, _f32, _p, _p, _p]
_lib.clq_rotate_quant_act_f6.argtypes = [_p, _i64, _p, _i64, _i64, _i32, _p, _p, _p]
_lib.clq_w4a4_linear_f6.argtypes = [_p, _p, _p, _p, _p, _i64, _i64, _i64, _p, _i64, _p]
_lib.clq_w4a4_accum_f6.argtypes = [_p, _p, _i64, _i64, _i64, _p, _i64, _p]
_lib.clq_unswizzle_f6.argtypes = [_p, _i64, _i64, _i32, _p, _p]
_lib.clq_f6_from_int4.argtypes = [_p, _i64, _i64, _i32, _p, _p]
_lib.clq_w4a4_schedule_f6.argtypes = [_i64, _i64, _i64, _p]
for _f in ("clq_quantize_weights", "clq_rotate_quant_act", "clq_w4a4_linear",
           "clq_w4a4_accum_i32", "clq_unswizzle_weights", "clq_unswizzle_act",
           "clq_obs_channel_scores", "clq_obs_permutation", "clq_rotate_quant_act8",
           "clq_quantize_weights8", "clq_a8_linear", "clq_a8_accum_i32", "clq_unswizzle_act8",
           "clq_unswizzle_weights8", "clq_clps_search", "clq_w4a4_workspace_status", "clq_debug_set",
           "clq_w4a4_schedule", "clq_w4a4_linear_noalloc", "clq_diag_mfma_probe",
           "clq_w4a4_rq_linear", "clq_w4a4_rq_schedule", "clq_quantize_weights_f6",
           "clq_rotate_quant_act_f6", "clq_w4a4_linear_f6", "clq_w4a4_accum_f6", "clq_unswizzle_f6",
           "clq_f6_from_int4", "clq_diag_mfma_probe_f6", "clq_w4a4_schedule_f6"):
    getattr(_lib, _f).restype = ctypes.c_int

EXPORTS = ("clq_version", "clq_status_string", "clq_weight_bytes", "clq_act_bytes",
           "clq_quantize_weights", "clq_rotate_quant_act", "clq_w4a4_workspace_bytes",
           "clq_w4a4_linear", "clq_w4a4_accum_i32", "clq_unswizzle_weights", "clq_unswizzle_act",
           "clq_obs_workspace_bytes", "clq_obs_channel_scores", "clq_obs_permutation",
           "clq_act8_bytes", "clq_weight8_bytes", "clq_rotate_quant_act8", "clq_quantize_weights8",
           "clq_a8_linear", "clq_a8_accum_i32", "clq_unswizzle_act8", "clq_unswizzle_weights8",
           "clq_clps_workspace_bytes", "clq_clps_search", "clq_w4a4_workspace_status",
           "clq_debug_set", "clq_debug_get", "clq_w4a4_schedule", "clq_w4a4_linear_noalloc",
           "clq_diag_mfma_probe_bytes", "clq_diag_mfma_probe", "clq_w4a4_rq_linear",
           "clq_w4a4_rq_schedule", "clq_weight_bytes_f6", "clq_act_bytes_f6", "clq_quantize_weights_f6",
           "clq_rotate_quant_act_f6", "clq_w4a4_linear_f6", "clq_w4a4_accum_f6", "clq_unswizzle_f6",
           "clq_f6_from_int4", "clq_diag_mfma_probe_f6", "clq_w4a4_schedule_f6")

CLQ_DEBUG_SYNC, CLQ_DEBUG_SPLIT_SPIN_LIMIT, CLQ_DEBUG_SPLIT_DROP_SIGNAL = 0, 1, 2
CLQ_DEBUG_GEMM_SCHEDULE, CLQ_DEBUG_F6_SCHEDULE = 3, 4

OBS_METRICS = ("absmax", "range", "par", "topk_mean", "percentile")

(CLQ_OK, CLQ_ERR_NULL, CLQ_ERR_SHAPE, CLQ_ERR_BLOCK, CLQ_ERR_ALIGN, CLQ_ERR_ARG, CLQ_ERR_HIP,
 CLQ_ERR_WORKSPACE) = range(8)


class ClqError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {_lib.clq_status_string(status).decode()}")


def lib():
    """The raw ctypes handle (for tests that drive the C ABI directly)."""
    return _lib


def _check(status, where):
    if status != CLQ_OK:
        raise ClqError(status, where)


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def clq_debug_set(knob, value):
    """Sets a process-wide debug knob (CLQ_DEBUG_*)."""
    _check(_lib.clq_debug_set(int(knob), int(value)), "clq_debug_set")


def clq_debug_get(knob):
    return int(_lib.clq_debug_get(int(knob)))


def clq_diag_mfma_probe_bytes():
    return int(_lib.clq_diag_mfma_probe_bytes())


def clq_diag_mfma_probe(ops, iters, grid, sink, stream=None):
    """Enqueues the matrix-core ceiling loop (diagnostic): ops a uint8
    device tensor of clq_diag_mfma_probe_bytes() random bytes, sink an int32
    device tensor of grid * 256 elements.  Returns the int8 ops it performs."""
    _dev(ops, "ops", torch.uint8)
    _dev(sink, "sink", torch.int32)
    if sink.numel() < grid * 256:
        raise ValueError("sink needs grid * 256 elements")
    _check(_lib.clq_diag_mfma_probe(_ptr(ops), ops.numel(), iters, grid, _ptr(sink), _stream(stream)),
           "clq_diag_mfma_probe")
    return grid * iters * 64 * 2 * 32 ** 3


def clq_diag_mfma_probe_f6(ops, iters, grid, sink, stream=None):
    """clq_diag_mfma_probe on the fp6 matrix instruction; returns the ops it
    performs (2 x 32 x 32 x 64 per instruction)."""
    _dev(ops, "ops", torch.uint8)
    _dev(sink, "sink", torch.int32)
    if sink.numel() < grid * 256:
        raise ValueError("sink needs grid * 256 elements")
    _check(_lib.clq_diag_mfma_probe_f6(_ptr(ops), ops.numel(), iters, grid, _ptr(sink), _stream(stream)),
           "clq_diag_mfma_probe_f6")
    return grid * iters * 64 * 2 * 32 * 32 * 64


F6_SCHEDULES = {1: "f6_gemm_kernel", 2: "f6_gemm_halves_kernel (128-token tiles)",
                3: "f6_gemm_halves_kernel (64-token tiles)"}


def clq_w4a4_schedule_f6(M, N, K):
    """The fp6 GEMM kernel choice for an M x N x K product: 1 persistent
    (256-token tiles), 2 / 3 two halves of the k loop (128- / 64-token tiles)."""
    c = ctypes.c_int32()
    _check(_lib.clq_w4a4_schedule_f6(M, N, K, ctypes.byref(c)), "clq_w4a4_schedule_f6")
    return c.value


def clq_w4a4_schedule(M, N, K, with_workspace=True):
    """The GEMM schedule for an M x N x K product on the current device:
    dict(kernel=0 persistent / 1 halves-128 / 2 halves-64, tiles, whole,
    split_stages, grid)."""
    info = (ctypes.c_int64 * 5)()
    _check(_lib.clq_w4a4_schedule(M, N, K, 1 if with_workspace else 0, ctypes.cast(info, ctypes.c_void_p)),
           "clq_w4a4_schedule")
    return dict(kernel=info[0], tiles=info[1], whole=info[2], split_stages=info[3], grid=info[4])


def _dev(t, name, dtype):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _perm(perm, K):
    if perm is None:
        return None
    _dev(perm, "perm", torch.int32)
    if perm.shape != (K,) or not perm.is_contiguous():
        raise ValueError(f"perm must be a contiguous int32 [K={K}] tensor")
    return perm


def clq_version():
    return int(_lib.clq_version())


def clq_weight_bytes(N, K):
    return int(_lib.clq_weight_bytes(N, K))


def clq_act_bytes(M, K):
    return int(_lib.clq_act_bytes(M, K))


@dataclass
class QWeight:
    """A weight matrix quantized by clq_quantize_weights."""
    wq: torch.Tensor        # uint8 [clq_weight_bytes(N, K)], opaque layout
    w_scale: torch.Tensor   # fp32 [N], includes the 1/block factor
    N: int
    K: int
    block: int
    perm: torch.Tensor = None
    clip_ratio: float = 1.0
    bits: int = 4           # 4: clq_quantize_weights, 6: clq_quantize_weights_f6, 8: clq_quantize_weights8


def clq_quantize_weights(W, block, perm=None, clip_ratio=1.0, stream=None):
    """Offline: rotate each weight row by G = S.H and quantize it to int4 with
    one scale per output channel."""
    _dev(W, "W", torch.float16)
    if W.dim() != 2 or not W.is_contiguous():
        raise ValueError("W must be a contiguous 2-D [N, K] tensor")
    N, K = W.shape
    perm = _perm(perm, K)
    nbytes = clq_weight_bytes(N, K)
    if nbytes == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_quantize_weights")
    wq = torch.empty(nbytes, dtype=torch.uint8, device=W.device)
    ws = torch.empty(N, dtype=torch.float32, device=W.device)
    _check(_lib.clq_quantize_weights(_ptr(W), _ptr(perm), N, K, block, clip_ratio,
                                     _ptr(wq), _ptr(ws), _stream(stream)), "clq_quantize_weights")
    return QWeight(wq, ws, N, K, block, perm, clip_ratio)


def save_qweight(path, qw):
    """Writes a quantized weight to a safetensors file: the opaque packed
    codes, the scales (1/block included), the swap vector if any, and the
    metadata (N, K, block, clip ratio, bits) keyed to the library version
    whose layout the codes use."""
    from safetensors.torch import save_file
    tensors = {"wq": qw.wq.detach().cpu().contiguous(), "w_scale": qw.w_scale.detach().cpu().contiguous()}
    if qw.perm is not None:
        tensors["perm"] = qw.perm.detach().cpu().contiguous()
    meta = {"format": "clq-qweight", "clq_version": str(clq_version()), "N": str(qw.N), "K": str(qw.K),
            "block": str(qw.block), "clip_ratio": repr(float(qw.clip_ratio)), "bits": str(qw.bits)}
    save_file(tensors, path, metadata=meta)


def load_qweight(path, device="cuda"):
    """Reads a file written by save_qweight onto `device`.  Raises ValueError
    if it was written by a library version with another packed layout or its
    sizes do not match that layout."""
    from safetensors import safe_open
    with safe_open(path, framework="pt") as f:
        meta = f.metadata() or {}
        if meta.get("format") != "clq-qweight":
            raise ValueError(f"{path}: not a CLQ quantized weight")
        if int(meta["clq_version"]) != clq_version():
            raise ValueError(f"{path}: written by library version {meta['clq_version']}, "
                             f"this is version {clq_version()} (the packed layouts differ)")
        N, K, block, bits = int(meta["N"]), int(meta["K"]), int(meta["block"]), int(meta["bits"])
        wq = f.get_tensor("wq")
        ws = f.get_tensor("w_scale")
        perm = f.get_tensor("perm") if "perm" in f.keys() else None
    need = clq_weight_bytes(N, K) if bits == 4 else clq_weight8_bytes(N, K)
    if wq.dtype != torch.uint8 or wq.numel() != need or ws.dtype != torch.float32 or ws.numel() != N or \
            (perm is not None and (perm.dtype != torch.int32 or perm.numel() != K)):
        raise ValueError(f"{path}: tensor sizes do not match N={N}, K={K}, bits={bits}")
    dev = torch.device(device)
    return QWeight(wq.to(dev), ws.to(dev), N, K, block, None if perm is None else perm.to(dev),
                   float(meta["clip_ratio"]), bits)


def clq_rotate_quant_act(X, block, perm=None, out=None, scale_out=None, stream=None):
    """Online: x~ = FWHT(gather(x, perm)) per token, quantized to int4 codes
    with one fp32 scale per token.  Returns (Xq, x_scale): Xq is the opaque
    packed buffer (uint8 [clq_act_bytes(M, K)]).  X may have a row stride
    larger than K (a column slice of a wider tensor)."""
    _dev(X, "X", torch.float16)
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D [M, K] with unit column stride")
    M, K = X.shape
    perm = _perm(perm, K)
    nbytes = clq_act_bytes(M, K)
    if nbytes == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_rotate_quant_act")
    Xq = out if out is not None else torch.empty(nbytes, dtype=torch.uint8, device=X.device)
    xs = scale_out if scale_out is not None else torch.empty(M, dtype=torch.float32, device=X.device)
    _dev(Xq, "Xq", torch.uint8)
    _dev(xs, "x_scale", torch.float32)
    if Xq.numel() < nbytes or not Xq.is_contiguous() or xs.numel() < M:
        raise ValueError("Xq / x_scale buffers are too small")
    _check(_lib.clq_rotate_quant_act(_ptr(X), X.stride(0), _ptr(perm), M, K, block, _ptr(Xq),
                                     _ptr(xs), _stream(stream)), "clq_rotate_quant_act")
    return Xq, xs


def clq_w4a4_workspace_bytes():
    return int(_lib.clq_w4a4_workspace_bytes())


_workspaces = {}


def _workspace(device, workspace, stream=None):
    """The GEMM workspace: the caller's tensor, False for none, or (default)
    one zero-filled buffer per (device, stream), allocated on first use and
    zero-filled on that stream, so calls sharing it run in stream order and
    calls on different streams never share one."""
    if workspace is False:
        return None, 0
    if workspace is None:
        workspace = default_workspace(device, stream)
    _dev(workspace, "workspace", torch.uint8)
    return workspace, workspace.numel()


def default_workspace(device=None, stream=None):
    """The default GEMM workspace of (device, stream) (the current stream if
    None): created on first use, zero-filled on that stream."""
    device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    idx = device.index if device.index is not None else torch.cuda.current_device()
    s = torch.cuda.current_stream(idx) if stream is None else stream
    key = (idx, s.cuda_stream)
    ws = _workspaces.get(key)
    if ws is None:
        with torch.cuda.device(idx), torch.cuda.stream(s):
            ws = torch.empty(clq_w4a4_workspace_bytes(), dtype=torch.uint8, device=device)
            ws.zero_()   # a fill kernel on the stream that will use it
        _workspaces[key] = ws
    return ws


def clq_w4a4_workspace_status(workspace=None, device=None, stream=None):
    """The split-k status words of a GEMM workspace (the default one of
    (device, stream) if None), as host ints [gave_up, first_tile, rank]:
    gave_up == 0 means every split tile was summed completely.  Synchronises
    with the stream."""
    if workspace is None:
        workspace = default_workspace(device, stream)
    _dev(workspace, "workspace", torch.uint8)
    s = torch.cuda.current_stream(workspace.device) if stream is None else stream
    with torch.cuda.stream(s):
        out = torch.empty(3, dtype=torch.int32, device=workspace.device)
        _check(_lib.clq_w4a4_workspace_status(_ptr(workspace), workspace.numel(), _ptr(out),
                                              ctypes.c_void_p(s.cuda_stream)), "clq_w4a4_workspace_status")
        s.synchronize()
        return [int(v) for v in out.cpu()]


def _check_xq(Xq, x_scale, K):
    _dev(Xq, "Xq", torch.uint8)
    _dev(x_scale, "x_scale", torch.float32)
    M = x_scale.shape[0]
    if not Xq.is_contiguous() or Xq.numel() < clq_act_bytes(M, K):
        raise ValueError("Xq must be the contiguous buffer clq_rotate_quant_act produced for "
                         "these M and K")
    return M


def clq_w4a4_linear(Xq, x_scale, qw, bias=None, out=None, stream=None, workspace=None):
    """Y = dequant(Xq . Wq^T) + bias as fp16 [M, N] (M = len(x_scale)).
    workspace: None (the per-device default), False (none), or a zero-filled
    uint8 tensor of clq_w4a4_workspace_bytes() bytes."""
    M = _check_xq(Xq, x_scale, qw.K)
    if qw.bits != 4:
        raise ValueError("qw must come from clq_quantize_weights (use clq_w4a4_linear_f6 for fp6 weights)")
    if bias is not None:
        _dev(bias, "bias", torch.float16)
        if bias.shape != (qw.N,) or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous fp16 [N] tensor")
    if out is None:  # rows padded to a multiple of 8 elements (16-byte aligned rows)
        out = torch.empty((M, (qw.N + 7) // 8 * 8), dtype=torch.float16, device=Xq.device)[:, :qw.N]
    Y = out
    _dev(Y, "Y", torch.float16)
    if Y.dim() != 2 or Y.stride(1) != 1 or Y.shape != (M, qw.N):
        raise ValueError("Y must be 2-D [M, N] with unit column stride")
    wsp, wsb = _workspace(Xq.device, workspace, stream)
    _check(_lib.clq_w4a4_linear(_ptr(Xq), _ptr(x_scale), _ptr(qw.wq), _ptr(qw.w_scale), _ptr(bias),
                                M, qw.N, qw.K, _ptr(Y), Y.stride(0), _ptr(wsp), wsb, _stream(stream)),
           "clq_w4a4_linear")
    return Y


def clq_w4a4_linear_noalloc(Xq, x_scale, qw, bias=None, out=None, status=None, stream=None):
    """clq_w4a4_linear without a workspace argument: the split schedule uses
    the library's own per-device scratch (nothing is allocated by the call
    when `out` is given).  status: None or a device int32 [3] tensor that
    receives the call's split-k status words.  Calls on one device must not
    overlap."""
    M = _check_xq(Xq, x_scale, qw.K)
    if bias is not None:
        _dev(bias, "bias", torch.float16)
        if bias.shape != (qw.N,) or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous fp16 [N] tensor")
    if out is None:
        out = torch.empty((M, (qw.N + 7) // 8 * 8), dtype=torch.float16, device=Xq.device)[:, :qw.N]
    Y = out
    _dev(Y, "Y", torch.float16)
    if Y.dim() != 2 or Y.stride(1) != 1 or Y.shape != (M, qw.N):
        raise ValueError("Y must be 2-D [M, N] with unit column stride")
    if status is not None:
        _dev(status, "status", torch.int32)
        if status.numel() < 3 or not status.is_contiguous():
            raise ValueError("status must be a contiguous int32 tensor of at least 3 elements")
    _check(_lib.clq_w4a4_linear_noalloc(_ptr(Xq), _ptr(x_scale), _ptr(qw.wq), _ptr(qw.w_scale), _ptr(bias),
                                        M, qw.N, qw.K, _ptr(Y), Y.stride(0), _ptr(status), _stream(stream)),
           "clq_w4a4_linear_noalloc")
    return Y


def clq_w4a4_rq_schedule(M, N, K, block, with_workspace=True):
    """Whether clq_w4a4_rq_linear runs this shape as one launch: dict(fused,
    rows_per_item, items, tiles)."""
    info = (ctypes.c_int64 * 4)()
    _check(_lib.clq_w4a4_rq_schedule(M, N, K, block, 1 if with_workspace else 0, ctypes.cast(info, ctypes.c_void_p)),
           "clq_w4a4_rq_schedule")
    return dict(fused=info[0], rows_per_item=info[1], items=info[2], tiles=info[3])


def clq_w4a4_rq_linear(X, block, qw, bias=None, Xq_out=None, scale_out=None, out=None, stream=None,
                       workspace=None):
    """Rotate+quantize X (fp16 [M, K], row stride allowed) and run the W4A4
    linear against qw, in one launch when clq_w4a4_rq_schedule says so (else
    the two launches).  X is not gathered: if qw was quantized with a swap
    vector, X must already be in that column order (gathered upstream).  Returns (Y, Xq, x_scale), each exactly what
    clq_rotate_quant_act and clq_w4a4_linear would write.  workspace: None
    (the default of (device, stream)), False (none: two launches), or a
    zero-filled uint8 tensor of clq_w4a4_workspace_bytes() bytes."""
    _dev(X, "X", torch.float16)
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D [M, K] with unit column stride")
    M, K = X.shape
    if K != qw.K or qw.bits != 4 or qw.block != block:
        raise ValueError("qw must be a 4-bit weight of the same K and block")
    nbytes = clq_act_bytes(M, K)
    Xq = Xq_out if Xq_out is not None else torch.empty(nbytes, dtype=torch.uint8, device=X.device)
    xs = scale_out if scale_out is not None else torch.empty(M, dtype=torch.float32, device=X.device)
    _dev(Xq, "Xq", torch.uint8)
    _dev(xs, "x_scale", torch.float32)
    if Xq.numel() < nbytes or not Xq.is_contiguous() or xs.numel() < M:
        raise ValueError("Xq / x_scale buffers are too small")
    if bias is not None:
        _dev(bias, "bias", torch.float16)
        if bias.shape != (qw.N,) or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous fp16 [N] tensor")
    if out is None:
        out = torch.empty((M, (qw.N + 7) // 8 * 8), dtype=torch.float16, device=X.device)[:, :qw.N]
    Y = out
    _dev(Y, "Y", torch.float16)
    if Y.dim() != 2 or Y.stride(1) != 1 or Y.shape != (M, qw.N):
        raise ValueError("Y must be 2-D [M, N] with unit column stride")
    wsp, wsb = _workspace(X.device, workspace, stream)
    _check(_lib.clq_w4a4_rq_linear(_ptr(X), X.stride(0), block, _ptr(Xq), _ptr(xs), _ptr(qw.wq), _ptr(qw.w_scale),
                                   _ptr(bias), M, qw.N, K, _ptr(Y), Y.stride(0), _ptr(wsp), wsb, _stream(stream)),
           "clq_w4a4_rq_linear")
    return Y, Xq, xs


def clq_w4a4_accum_i32(Xq, x_scale, qw, out=None, stream=None, workspace=None):
    """The exact int32 accumulators sum_k qx * qw, [M, N] (diagnostic); the
    scales only give M."""
    M = _check_xq(Xq, x_scale, qw.K)
    if out is None:  # rows padded to a multiple of 4 elements (16-byte aligned rows)
        out = torch.empty((M, (qw.N + 3) // 4 * 4), dtype=torch.int32, device=Xq.device)[:, :qw.N]
    acc = out
    _dev(acc, "acc", torch.int32)
    wsp, wsb = _workspace(Xq.device, workspace, stream)
    _check(_lib.clq_w4a4_accum_i32(_ptr(Xq), _ptr(qw.wq), M, qw.N, qw.K, _ptr(acc), acc.stride(0),
                                   _ptr(wsp), wsb, _stream(stream)), "clq_w4a4_accum_i32")
    return acc


def clq_unswizzle_weights(qw, stream=None):
    """Canonical packed codes uint8 [N, K/2] of a QWeight (diagnostic)."""
    out = torch.empty((qw.N, qw.K // 2), dtype=torch.uint8, device=qw.wq.device)
    _check(_lib.clq_unswizzle_weights(_ptr(qw.wq), qw.N, qw.K, _ptr(out), _stream(stream)),
           "clq_unswizzle_weights")
    return out


def clq_unswizzle_act(Xq, M, K, stream=None):
    """Canonical packed codes uint8 [M, K/2] of an activation buffer (diagnostic)."""
    _dev(Xq, "Xq", torch.uint8)
    out = torch.empty((M, K // 2), dtype=torch.uint8, device=Xq.device)
    _check(_lib.clq_unswizzle_act(_ptr(Xq), M, K, _ptr(out), _stream(stream)), "clq_unswizzle_act")
    return out


def clq_obs_workspace_bytes(N, D, metric):
    return int(_lib.clq_obs_workspace_bytes(N, D, _metric(metric)))


def _metric(metric):
    if isinstance(metric, str):
        if metric not in OBS_METRICS:
            raise ValueError(f"metric must be one of {OBS_METRICS}")
        return OBS_METRICS.index(metric)
    return int(metric)


def clq_obs_channel_scores(X, metric="absmax", workspace=None, out=None, stream=None):
    """OBS outlier score per channel of calibration activations X, fp16
    [B, N, D] (tokens with unit channel stride; the batch stride must be N
    token rows).  Returns fp32 [D].  A workspace passed in for abs-max or
    range must be zero-filled before its first use (each call leaves it so)."""
    _dev(X, "X", torch.float16)
    if X.dim() != 3 or X.stride(2) != 1 or X.stride(0) != X.shape[1] * X.stride(1):
        raise ValueError("X must be [B, N, D] with unit channel stride and batch stride N * ldx")
    B, N, D = X.shape
    m = _metric(metric)
    need = clq_obs_workspace_bytes(N, D, m)
    if need == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_obs_channel_scores")
    if workspace is None:   # abs-max / range need it zero-filled; calls leave it so
        workspace = torch.zeros(need, dtype=torch.uint8, device=X.device)
    _dev(workspace, "workspace", torch.uint8)
    scores = out if out is not None else torch.empty(D, dtype=torch.float32, device=X.device)
    _dev(scores, "scores", torch.float32)
    _check(_lib.clq_obs_channel_scores(_ptr(X), X.stride(1), B, N, D, m, _ptr(workspace),
                                       workspace.numel(), _ptr(scores), _stream(stream)),
           "clq_obs_channel_scores")
    return scores


def clq_obs_permutation(scores, out=None, stream=None):
    """The gather vector s (int32 [D]) that moves the top-scoring half of the
    channels to the left half, each half in ascending channel order."""
    _dev(scores, "scores", torch.float32)
    if scores.dim() != 1 or not scores.is_contiguous():
        raise ValueError("scores must be a contiguous fp32 [D] tensor")
    D = scores.shape[0]
    perm = out if out is not None else torch.empty(D, dtype=torch.int32, device=scores.device)
    _dev(perm, "perm", torch.int32)
    _check(_lib.clq_obs_permutation(_ptr(scores), D, _ptr(perm), _stream(stream)), "clq_obs_permutation")
    return perm


# ---- 8-bit activations: W4A8 and W8A8 -------------------------------------------

def clq_act8_bytes(M, K):
    return int(_lib.clq_act8_bytes(M, K))


def clq_weight8_bytes(N, K):
    return int(_lib.clq_weight8_bytes(N, K))


def clq_rotate_quant_act8(X, block, perm=None, out=None, scale_out=None, stream=None):
    """clq_rotate_quant_act with 8-bit codes (x_scale = max|x~| / 127).
    Returns (Xq8 uint8 [clq_act8_bytes(M, K)], x_scale fp32 [M])."""
    _dev(X, "X", torch.float16)
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D [M, K] with unit column stride")
    M, K = X.shape
    perm = _perm(perm, K)
    nbytes = clq_act8_bytes(M, K)
    if nbytes == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_rotate_quant_act8")
    Xq = out if out is not None else torch.empty(nbytes, dtype=torch.uint8, device=X.device)
    xs = scale_out if scale_out is not None else torch.empty(M, dtype=torch.float32, device=X.device)
    _dev(Xq, "Xq8", torch.uint8)
    _dev(xs, "x_scale", torch.float32)
    if Xq.numel() < nbytes or not Xq.is_contiguous() or xs.numel() < M:
        raise ValueError("Xq8 / x_scale buffers are too small")
    _check(_lib.clq_rotate_quant_act8(_ptr(X), X.stride(0), _ptr(perm), M, K, block, _ptr(Xq),
                                      _ptr(xs), _stream(stream)), "clq_rotate_quant_act8")
    return Xq, xs


def clq_quantize_weights8(W, block, perm=None, clip_ratio=1.0, stream=None):
    """clq_quantize_weights with 8-bit codes (w_scale = alpha max|w~| / 127 / b)."""
    _dev(W, "W", torch.float16)
    if W.dim() != 2 or not W.is_contiguous():
        raise ValueError("W must be a contiguous 2-D [N, K] tensor")
    N, K = W.shape
    perm = _perm(perm, K)
    nbytes = clq_weight8_bytes(N, K)
    if nbytes == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_quantize_weights8")
    wq = torch.empty(nbytes, dtype=torch.uint8, device=W.device)
    ws = torch.empty(N, dtype=torch.float32, device=W.device)
    _check(_lib.clq_quantize_weights8(_ptr(W), _ptr(perm), N, K, block, clip_ratio, _ptr(wq), _ptr(ws),
                                      _stream(stream)), "clq_quantize_weights8")
    return QWeight(wq, ws, N, K, block, perm, clip_ratio, 8)


# ---- W4A4 with the codes stored as fp6 (e2m3) --------------------------------------

def clq_weight_bytes_f6(N, K):
    return int(_lib.clq_weight_bytes_f6(N, K))


def clq_act_bytes_f6(M, K):
    return int(_lib.clq_act_bytes_f6(M, K))


def clq_quantize_weights_f6(W, block, perm=None, clip_ratio=1.0, stream=None):
    """clq_quantize_weights with the codes stored as fp6 (QWeight.bits == 6):
    the same codes and scales."""
    _dev(W, "W", torch.float16)
    if W.dim() != 2 or not W.is_contiguous():
        raise ValueError("W must be a contiguous 2-D [N, K] tensor")
    N, K = W.shape
    perm = _perm(perm, K)
    nbytes = clq_weight_bytes_f6(N, K)
    if nbytes == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_quantize_weights_f6")
    wq = torch.empty(nbytes, dtype=torch.uint8, device=W.device)
    ws = torch.empty(N, dtype=torch.float32, device=W.device)
    _check(_lib.clq_quantize_weights_f6(_ptr(W), _ptr(perm), N, K, block, clip_ratio,
                                        _ptr(wq), _ptr(ws), _stream(stream)), "clq_quantize_weights_f6")
    return QWeight(wq, ws, N, K, block, perm, clip_ratio, bits=6)


def clq_rotate_quant_act_f6(X, block, perm=None, out=None, scale_out=None, stream=None):
    """clq_rotate_quant_act with the codes stored as fp6: (Xq, x_scale), Xq
    uint8 [clq_act_bytes_f6(M, K)]."""
    _dev(X, "X", torch.float16)
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be 2-D [M, K] with unit column stride")
    M, K = X.shape
    perm = _perm(perm, K)
    nbytes = clq_act_bytes_f6(M, K)
    if nbytes == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_rotate_quant_act_f6")
    Xq = out if out is not None else torch.empty(nbytes, dtype=torch.uint8, device=X.device)
    xs = scale_out if scale_out is not None else torch.empty(M, dtype=torch.float32, device=X.device)
    _dev(Xq, "Xq", torch.uint8)
    _dev(xs, "x_scale", torch.float32)
    if Xq.numel() < nbytes or not Xq.is_contiguous() or xs.numel() < M:
        raise ValueError("Xq / x_scale buffers are too small")
    _check(_lib.clq_rotate_quant_act_f6(_ptr(X), X.stride(0), _ptr(perm), M, K, block, _ptr(Xq),
                                        _ptr(xs), _stream(stream)), "clq_rotate_quant_act_f6")
    return Xq, xs


def _check_f6(Xq, x_scale, qw):
    _dev(Xq, "Xq", torch.uint8)
    _dev(x_scale, "x_scale", torch.float32)
    if qw.bits != 6:
        raise ValueError("qw must come from clq_quantize_weights_f6 or clq_qweight_f6")
    M = x_scale.shape[0]
    if not Xq.is_contiguous() or Xq.numel() < clq_act_bytes_f6(M, qw.K):
        raise ValueError("Xq must be the contiguous buffer clq_rotate_quant_act_f6 produced for "
                         "these M and K")
    return M


def clq_w4a4_linear_f6(Xq, x_scale, qw, bias=None, out=None, stream=None):
    """clq_w4a4_linear on the fp6 layouts (no workspace): fp16 [M, N]."""
    M = _check_f6(Xq, x_scale, qw)
    if bias is not None:
        _dev(bias, "bias", torch.float16)
        if bias.shape != (qw.N,) or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous fp16 [N] tensor")
    if out is None:
        out = torch.empty((M, (qw.N + 7) // 8 * 8), dtype=torch.float16, device=Xq.device)[:, :qw.N]
    Y = out
    _dev(Y, "Y", torch.float16)
    if Y.dim() != 2 or Y.stride(1) != 1 or Y.shape != (M, qw.N):
        raise ValueError("Y must be 2-D [M, N] with unit column stride")
    _check(_lib.clq_w4a4_linear_f6(_ptr(Xq), _ptr(x_scale), _ptr(qw.wq), _ptr(qw.w_scale), _ptr(bias),
                                   M, qw.N, qw.K, _ptr(Y), Y.stride(0), _stream(stream)), "clq_w4a4_linear_f6")
    return Y


def clq_w4a4_accum_f6(Xq, x_scale, qw, out=None, stream=None):
    """The exact integer sums of the fp6 operands, int32 [M, N] (diagnostic)."""
    M = _check_f6(Xq, x_scale, qw)
    if out is None:
        out = torch.empty((M, (qw.N + 3) // 4 * 4), dtype=torch.int32, device=Xq.device)[:, :qw.N]
    _dev(out, "acc", torch.int32)
    _check(_lib.clq_w4a4_accum_f6(_ptr(Xq), _ptr(qw.wq), M, qw.N, qw.K, _ptr(out), out.stride(0),
                                  _stream(stream)), "clq_w4a4_accum_f6")
    return out


def clq_unswizzle_f6(q6, rows, K, weights, stream=None):
    """Canonical packed codes uint8 [rows, K/2] of an fp6 buffer (diagnostic)."""
    out = torch.empty((rows, K // 2), dtype=torch.uint8, device=q6.device)
    _check(_lib.clq_unswizzle_f6(_ptr(q6), rows, K, 1 if weights else 0, _ptr(out), _stream(stream)),
           "clq_unswizzle_f6")
    return out


def clq_f6_from_int4(q4, rows, K, weights, stream=None):
    """The fp6 layout of a packed int4 buffer (weights: clq_quantize_weights,
    else clq_rotate_quant_act)."""
    nbytes = clq_weight_bytes_f6(rows, K) if weights else clq_act_bytes_f6(rows, K)
    q6 = torch.empty(nbytes, dtype=torch.uint8, device=q4.device)
    _check(_lib.clq_f6_from_int4(_ptr(q4), rows, K, 1 if weights else 0, _ptr(q6), _stream(stream)),
           "clq_f6_from_int4")
    return q6


def clq_qweight_f6(qw, stream=None):
    """An int4 QWeight (clq_quantize_weights) converted to the fp6 layout."""
    if qw.bits != 4:
        raise ValueError("qw must come from clq_quantize_weights")
    return QWeight(clq_f6_from_int4(qw.wq, qw.N, qw.K, True, stream), qw.w_scale, qw.N, qw.K, qw.block,
                   qw.perm, qw.clip_ratio, bits=6)


def _check_xq8(Xq8, x_scale, K):
    _dev(Xq8, "Xq8", torch.uint8)
    _dev(x_scale, "x_scale", torch.float32)
    M = x_scale.shape[0]
    if not Xq8.is_contiguous() or Xq8.numel() < clq_act8_bytes(M, K):
        raise ValueError("Xq8 must be the contiguous buffer clq_rotate_quant_act8 produced for "
                         "these M and K")
    return M


def clq_a8_linear(Xq8, x_scale, qw, bias=None, out=None, stream=None):
    """W4A8 (qw from clq_quantize_weights) or W8A8 (qw from
    clq_quantize_weights8) linear: fp16 [M, N]."""
    M = _check_xq8(Xq8, x_scale, qw.K)
    if bias is not None:
        _dev(bias, "bias", torch.float16)
        if bias.shape != (qw.N,) or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous fp16 [N] tensor")
    if out is None:
        out = torch.empty((M, (qw.N + 7) // 8 * 8), dtype=torch.float16, device=Xq8.device)[:, :qw.N]
    Y = out
    _dev(Y, "Y", torch.float16)
    if Y.dim() != 2 or Y.stride(1) != 1 or Y.shape != (M, qw.N):
        raise ValueError("Y must be 2-D [M, N] with unit column stride")
    _check(_lib.clq_a8_linear(_ptr(Xq8), _ptr(x_scale), _ptr(qw.wq), _ptr(qw.w_scale), qw.bits, _ptr(bias),
                              M, qw.N, qw.K, _ptr(Y), Y.stride(0), _stream(stream)), "clq_a8_linear")
    return Y


def clq_a8_accum_i32(Xq8, x_scale, qw, out=None, stream=None):
    """The exact integer sums of clq_a8_linear, int32 [M, N] (diagnostic)."""
    M = _check_xq8(Xq8, x_scale, qw.K)
    if out is None:
        out = torch.empty((M, (qw.N + 3) // 4 * 4), dtype=torch.int32, device=Xq8.device)[:, :qw.N]
    acc = out
    _dev(acc, "acc", torch.int32)
    _check(_lib.clq_a8_accum_i32(_ptr(Xq8), _ptr(qw.wq), qw.bits, M, qw.N, qw.K, _ptr(acc), acc.stride(0),
                                 _stream(stream)), "clq_a8_accum_i32")
    return acc


def clq_unswizzle_act8(Xq8, M, K, stream=None):
    """Row-major int8 codes [M, K] of an 8-bit activation buffer (diagnostic)."""
    _dev(Xq8, "Xq8", torch.uint8)
    out = torch.empty((M, K), dtype=torch.int8, device=Xq8.device)
    _check(_lib.clq_unswizzle_act8(_ptr(Xq8), M, K, _ptr(out), _stream(stream)), "clq_unswizzle_act8")
    return out


def clq_unswizzle_weights8(qw, stream=None):
    """Row-major int8 codes [N, K] of an 8-bit QWeight (diagnostic)."""
    out = torch.empty((qw.N, qw.K), dtype=torch.int8, device=qw.wq.device)
    _check(_lib.clq_unswizzle_weights8(_ptr(qw.wq), qw.N, qw.K, _ptr(out), _stream(stream)),
           "clq_unswizzle_weights8")
    return out


# ---- CLPS single-layer clip search ------------------------------------------------

def clq_clps_workspace_bytes(M, N, K):
    return int(_lib.clq_clps_workspace_bytes(M, N, K))


def clq_clps_search(X, W, Y0, block, perm=None, gamma=0.01, grid=20, workspace=None, stream=None):
    """Grid search of the weight clip ratio (W4A4) minimising ||Y0 - Yhat||_F^2
    on calibration activations X fp16 [M, K]; W fp16 [N, K]; Y0 fp32 [M, N]
    the unquantised output.  Returns device tensors (alphas fp32 [grid],
    errors fp64 [grid], best int32 [1]); nothing is synchronised."""
    _dev(X, "X", torch.float16)
    _dev(W, "W", torch.float16)
    _dev(Y0, "Y0", torch.float32)
    if X.dim() != 2 or X.stride(1) != 1 or W.dim() != 2 or not W.is_contiguous():
        raise ValueError("X must be [M, K] with unit column stride and W contiguous [N, K]")
    M, K = X.shape
    N = W.shape[0]
    if W.shape[1] != K or Y0.dim() != 2 or Y0.shape != (M, N) or Y0.stride(1) != 1:
        raise ValueError("shapes: X [M, K], W [N, K], Y0 [M, N]")
    perm = _perm(perm, K)
    need = clq_clps_workspace_bytes(M, N, K)
    if need == 0:
        raise ClqError(CLQ_ERR_SHAPE, "clq_clps_search")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=X.device)
    _dev(workspace, "workspace", torch.uint8)
    alphas = torch.empty(grid, dtype=torch.float32, device=X.device)
    errors = torch.empty(grid, dtype=torch.float64, device=X.device)
    best = torch.empty(1, dtype=torch.int32, device=X.device)
    _check(_lib.clq_clps_search(_ptr(X), X.stride(0), _ptr(W), _ptr(Y0), Y0.stride(0), _ptr(perm), M, N, K,
                                block, gamma, grid, _ptr(workspace), workspace.numel(), _ptr(alphas),
                                _ptr(errors), _ptr(best), _stream(stream)), "clq_clps_search")
    return alphas, errors, best
