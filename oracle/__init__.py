"""CLQ W4A4 linear layer: CPU oracle.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the GPU path (``paper_2509_24416_amd``) and neither imports the
other.

The arithmetic of the method lives in ``clq_oracle.c`` (plain loops, IEEE fp32
where the method's integer decisions are taken, fp64 for the dequantised
result); this module marshals numpy arrays into it and adds the fp64
references used to pin it (dense Hadamard matrix, unquantised linear, error
metric).  Paper references are to "CLQ" (arXiv 2509.24416):

  Sec. 3.1, Eq. (1)  uniform quantizer Round(Clip(.)), n = 4 bits (8 for the
                     W4A8 / W8A8 settings of Sec. 4.1); dynamic activation
                     bounds, weights quantized once.
  Sec. 3.3           OBS: G = S.H (gather vector s, block Hadamard H with
                     +-1 entries); weights absorb G offline, activations get a
                     fast Hadamard transform online.
  Sec. 4.1           per-channel weight granularity; one clip per matrix.

Every function has a pin in ``tests/test_oracle_pins.py`` that checks it
against something other than itself (closed forms, brute force, hand
examples, invariants, error bounds).  The fp16 bit pattern of the GPU output
is held only to the tolerance, not to a mirror of its rounding (parity
unpinned beyond the tolerance).
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libclq_oracle.so")
_lib = None

_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_f32 = ctypes.c_float
_p = ctypes.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b  # building the oracle is not running it
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.clqo_set_threads.argtypes = [ctypes.c_int]
    lib.clqo_get_threads.restype = ctypes.c_int
    lib.clqo_rotate.argtypes = [_p, _i64, _p, _i64, _i64, _i32, _p]
    lib.clqo_quantize.argtypes = [_p, _i64, _i64, _f32, _p, _p, _p]
    lib.clqo_quantize_q.argtypes = [_p, _i64, _i64, _f32, _f32, _p, _p, _p]
    lib.clqo_pack.argtypes = [_p, _i64, _i64, _p]
    lib.clqo_unpack.argtypes = [_p, _i64, _i64, _p]
    lib.clqo_gemm_i32.argtypes = [_p, _p, _i64, _i64, _i64, _p]
    lib.clqo_epilogue.argtypes = [_p, _p, _p, _p, _i64, _i64, _p, _p]
    for f in ("clqo_set_threads", "clqo_rotate", "clqo_quantize", "clqo_quantize_q", "clqo_pack",
              "clqo_unpack", "clqo_gemm_i32", "clqo_epilogue"):
        getattr(lib, f).restype = None
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def set_threads(n):
    _load().clqo_set_threads(int(n))


def get_threads():
    return int(_load().clqo_get_threads())


# --------------------------------------------------------------------------
# fp64 references (Sec. 3.3: the block Hadamard matrix and G = S.H)
# --------------------------------------------------------------------------

def hadamard_dense(b):
    """Sylvester-ordered, unnormalised b x b Hadamard matrix in fp64:
    H[i][j] = (-1)^popcount(i & j)."""
    i = np.arange(b)
    bits = np.bitwise_and.outer(i, i)
    pc = np.zeros_like(bits)
    while bits.any():
        pc += bits & 1
        bits >>= 1
    return np.where(pc % 2 == 0, 1.0, -1.0)


def rotation_dense(K, block, perm=None, normalised=False):
    """Dense K x K matrix G with x~ = x . G: column gather by ``perm`` followed
    by blockdiag(H_b, ..., H_b).  ``normalised`` divides by sqrt(b) so that G
    is orthogonal (G G^T = I)."""
    H = hadamard_dense(block)
    if normalised:
        H = H / np.sqrt(block)
    B = np.kron(np.eye(K // block), H)
    if perm is None:
        return B
    P = np.zeros((K, K))
    P[np.asarray(perm), np.arange(K)] = 1.0  # (x . P)[k] = x[perm[k]]
    return P @ B


# --------------------------------------------------------------------------
# the method's steps, run in the C oracle
# --------------------------------------------------------------------------

def _as_f32_rows(X):
    X = np.asarray(X)
    if X.dtype == np.float16:
        X = X.astype(np.float32)  # exact widening
    return np.ascontiguousarray(X, dtype=np.float32)


def rotate(X, block, perm=None):
    """x~ = gather(x, perm) . blockdiag(H_b) per row, in fp32 with the fixed
    ascending stage order.  X: fp16 or fp32 [rows][K]."""
    X = _as_f32_rows(X)
    rows, K = X.shape
    assert K % block == 0
    out = np.empty((rows, K), np.float32)
    pm = None if perm is None else np.ascontiguousarray(perm, dtype=np.int32)
    _load().clqo_rotate(_ptr(X), K, _ptr(pm), rows, K, int(block), _ptr(out))
    return out


def qmax(bits):
    """Largest code of the symmetric n-bit grid: 2^(n-1) - 1."""
    return (1 << (bits - 1)) - 1


def quantize(xr, alpha=1.0, bits=4):
    """Symmetric per-row quantizer of Eq. (1) with n = bits (4 or 8).
    Returns (codes int8 [rows][K] in [-qmax, qmax], scale fp32 [rows],
    nclamp int32 [rows])."""
    assert bits in (4, 8)
    xr = np.ascontiguousarray(xr, dtype=np.float32)
    rows, K = xr.shape
    codes = np.empty((rows, K), np.int8)
    scale = np.empty(rows, np.float32)
    ncl = np.empty(rows, np.int32)
    _load().clqo_quantize_q(_ptr(xr), rows, K, float(alpha), float(qmax(bits)), _ptr(codes),
                            _ptr(scale), _ptr(ncl))
    return codes, scale, ncl


def pack(codes):
    codes = np.ascontiguousarray(codes, dtype=np.int8)
    rows, K = codes.shape
    out = np.empty((rows, K // 2), np.uint8)
    _load().clqo_pack(_ptr(codes), rows, K, _ptr(out))
    return out


def unpack(packed, K):
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    rows = packed.shape[0]
    out = np.empty((rows, K), np.int8)
    _load().clqo_unpack(_ptr(packed), rows, K, _ptr(out))
    return out


def quantize_act(X, block, perm=None, bits=4):
    """Online activation path: rotate, per-token quantize (alpha = 1) and,
    for 4 bits, pack.  Returns (packed uint8 [M][K/2] for 4 bits or the int8
    codes themselves for 8, codes int8 [M][K], x_scale fp32 [M])."""
    codes, xs, _ = quantize(rotate(X, block, perm), 1.0, bits)
    return (pack(codes) if bits == 4 else codes), codes, xs


def quantize_weights(W, block, perm=None, clip_ratio=1.0, bits=4):
    """Offline weight path: W~ = W . G row-wise, per-output-channel quantizer
    with clip ratio alpha, w_scale = s / b (the Hadamard normalisation folded
    in, exact since b is a power of two).  Returns (packed canonical uint8
    [N][K/2] for 4 bits or the int8 codes for 8, codes int8 [N][K], w_scale
    fp32 [N])."""
    codes, s, _ = quantize(rotate(W, block, perm), clip_ratio, bits)
    ws = (s * np.float32(1.0 / block)).astype(np.float32)
    return (pack(codes) if bits == 4 else codes), codes, ws


def gemm_i32(qa, qw):
    """acc[m][n] = sum_k qa[m][k] * qw[n][k] in int32."""
    qa = np.ascontiguousarray(qa, dtype=np.int8)
    qw = np.ascontiguousarray(qw, dtype=np.int8)
    M, K = qa.shape
    N = qw.shape[0]
    assert qw.shape[1] == K
    acc = np.empty((M, N), np.int32)
    _load().clqo_gemm_i32(_ptr(qa), _ptr(qw), M, N, K, _ptr(acc))
    return acc


def epilogue(acc, x_scale, w_scale, bias=None):
    """Dequantised result in fp64: p64 = acc * x_scale[m] * w_scale[n] and
    y64 = p64 + bias[n].  bias: fp16/fp32 [N] or None."""
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    M, N = acc.shape
    xs = np.ascontiguousarray(x_scale, dtype=np.float32)
    ws = np.ascontiguousarray(w_scale, dtype=np.float32)
    b = None if bias is None else np.ascontiguousarray(np.asarray(bias).astype(np.float32))
    y = np.empty((M, N), np.float64)
    p = np.empty((M, N), np.float64)
    _load().clqo_epilogue(_ptr(acc), _ptr(xs), _ptr(ws), _ptr(b), M, N, _ptr(y), _ptr(p))
    return y, p


def linear(X, W, bias, block, perm=None, clip_ratio=1.0, wbits=4, abits=4):
    """The whole quantized linear on the CPU (W4A4 by default; W4A8 and W8A8
    with wbits / abits = 8).  Returns a dict with every intermediate: xq,
    xcodes, x_scale, wq, wcodes, w_scale, acc, y64, p64."""
    xq, xc, xs = quantize_act(X, block, perm, abits)
    wq, wc, ws = quantize_weights(W, block, perm, clip_ratio, wbits)
    acc = gemm_i32(xc, wc)
    y64, p64 = epilogue(acc, xs, ws, bias)
    return dict(xq=xq, xcodes=xc, x_scale=xs, wq=wq, wcodes=wc, w_scale=ws,
                acc=acc, y64=y64, p64=p64)


def linear_fp64(X, W, bias=None):
    """Unquantised reference y_fp = X W^T + bias in fp64."""
    y = np.asarray(X, np.float64) @ np.asarray(W, np.float64).T
    if bias is not None:
        y = y + np.asarray(bias, np.float64)[None, :]
    return y


def err_metric(y, y64, p64, bias=None):
    """Max over elements of |y - y64| / max(|p64| + |bias|, 2^-24): the fp16
    output's error relative to the dequantised fp64 result, normalised so
    that a bias cancelling the product does not blow up the ratio."""
    y = np.asarray(y, np.float64)
    den = np.abs(p64)
    if bias is not None:
        den = den + np.abs(np.asarray(bias, np.float64))[None, :]
    den = np.maximum(den, 2.0 ** -24)
    return float(np.max(np.abs(y - y64) / den)) if y.size else 0.0
