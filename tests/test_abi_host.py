"""Host-side checks of the C ABI (no GPU needed, no kernel is ever launched).

The library must load, export every entry point that include/clq.h declares,
and reject every precondition violation with its documented status code
before touching the GPU.  The fake device pointers used here are never
dereferenced: each call fails validation first.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "clq.h")
LIB = os.path.join(ROOT, "paper_2509_24416_amd", "libclq.so")

OK, NULL, SHAPE, BLOCK, ALIGN, ARG, HIP, WORKSPACE = range(8)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(clq_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    L = ctypes.CDLL(LIB)
    i64, i32, f32, p = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
    L.clq_status_string.restype = ctypes.c_char_p
    L.clq_status_string.argtypes = [ctypes.c_int]
    L.clq_weight_bytes.restype = ctypes.c_size_t
    L.clq_weight_bytes.argtypes = [i64, i64]
    L.clq_act_bytes.restype = ctypes.c_size_t
    L.clq_act_bytes.argtypes = [i64, i64]
    L.clq_unswizzle_act.argtypes = [p, i64, i64, p, p]
    L.clq_quantize_weights.argtypes = [p, p, i64, i64, i32, f32, p, p, p]
    L.clq_rotate_quant_act.argtypes = [p, i64, p, i64, i64, i32, p, p, p]
    L.clq_w4a4_workspace_bytes.restype = ctypes.c_size_t
    L.clq_w4a4_workspace_bytes.argtypes = []
    L.clq_w4a4_linear.argtypes = [p, p, p, p, p, i64, i64, i64, p, i64, p, ctypes.c_size_t, p]
    L.clq_w4a4_accum_i32.argtypes = [p, p, i64, i64, i64, p, i64, p, ctypes.c_size_t, p]
    L.clq_unswizzle_weights.argtypes = [p, i64, i64, p, p]
    L.clq_obs_workspace_bytes.restype = ctypes.c_size_t
    L.clq_obs_workspace_bytes.argtypes = [i64, i64, i32]
    L.clq_obs_channel_scores.argtypes = [p, i64, i64, i64, i64, i32, p, ctypes.c_size_t, p, p]
    L.clq_obs_permutation.argtypes = [p, i64, p, p]
    L.clq_act8_bytes.restype = ctypes.c_size_t
    L.clq_act8_bytes.argtypes = [i64, i64]
    L.clq_weight8_bytes.restype = ctypes.c_size_t
    L.clq_weight8_bytes.argtypes = [i64, i64]
    L.clq_rotate_quant_act8.argtypes = [p, i64, p, i64, i64, i32, p, p, p]
    L.clq_quantize_weights8.argtypes = [p, p, i64, i64, i32, f32, p, p, p]
    L.clq_a8_linear.argtypes = [p, p, p, p, i32, p, i64, i64, i64, p, i64, p]
    L.clq_a8_accum_i32.argtypes = [p, p, i32, i64, i64, i64, p, i64, p]
    L.clq_unswizzle_act8.argtypes = [p, i64, i64, p, p]
    L.clq_unswizzle_weights8.argtypes = [p, i64, i64, p, p]
    L.clq_clps_workspace_bytes.restype = ctypes.c_size_t
    L.clq_clps_workspace_bytes.argtypes = [i64, i64, i64]
    L.clq_clps_search.argtypes = [p, i64, p, p, i64, p, i64, i64, i64, i32, f32, i32, p, ctypes.c_size_t,
                                  p, p, p, p]
    L.clq_w4a4_workspace_status.argtypes = [p, ctypes.c_size_t, p, p]
    L.clq_debug_set.argtypes = [i32, i64]
    L.clq_debug_get.argtypes = [i32]
    L.clq_debug_get.restype = i64
    L.clq_w4a4_schedule.argtypes = [i64, i64, i64, i32, p]
    L.clq_w4a4_rq_linear.argtypes = [p, i64, i32, p, p, p, p, p, i64, i64, i64, p, i64, p, ctypes.c_size_t, p]
    L.clq_w4a4_rq_schedule.argtypes = [i64, i64, i64, i32, i32, p]
    L.clq_diag_mfma_probe_bytes.restype = ctypes.c_size_t
    L.clq_diag_mfma_probe.argtypes = [p, ctypes.c_size_t, i32, i32, p, p]
    L.clq_weight_bytes_f6.restype = ctypes.c_size_t
    L.clq_weight_bytes_f6.argtypes = [i64, i64]
    L.clq_act_bytes_f6.restype = ctypes.c_size_t
    L.clq_act_bytes_f6.argtypes = [i64, i64]
    L.clq_quantize_weights_f6.argtypes = [p, p, i64, i64, i32, f32, p, p, p]
    L.clq_rotate_quant_act_f6.argtypes = [p, i64, p, i64, i64, i32, p, p, p]
    L.clq_w4a4_linear_f6.argtypes = [p, p, p, p, p, i64, i64, i64, p, i64, p]
    L.clq_w4a4_accum_f6.argtypes = [p, p, i64, i64, i64, p, i64, p]
    L.clq_unswizzle_f6.argtypes = [p, i64, i64, i32, p, p]
    L.clq_f6_from_int4.argtypes = [p, i64, i64, i32, p, p]
    L.clq_diag_mfma_probe_f6.argtypes = [p, ctypes.c_size_t, i32, i32, p, p]
    L.clq_w4a4_schedule_f6.argtypes = [i64, i64, i64, p]
    return L


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) == 43, names
    for n in names:
        assert hasattr(lib, n), n


def test_binding_names_match_header():
    src = open(os.path.join(ROOT, "paper_2509_24416_amd", "__init__.py")).read()
    for n in declared_functions():
        assert re.search(rf"\bdef {n}\(", src) or f'"{n}"' in src, n


def test_version_and_strings(lib):
    assert lib.clq_version() == 8
    for code in range(8):
        s = lib.clq_status_string(code).decode()
        assert s.startswith("CLQ")
    assert b"unknown" in lib.clq_status_string(99)


def test_weight_bytes(lib):
    assert lib.clq_weight_bytes(1152, 1152) == 1152 * 576
    assert lib.clq_weight_bytes(1, 64) == 64 * 32            # rows padded to 64
    assert lib.clq_weight_bytes(3456, 1152) == 3456 * 576
    assert lib.clq_weight_bytes(100, 128) == 128 * 64
    assert lib.clq_weight_bytes(0, 64) == 0
    assert lib.clq_weight_bytes(8, 96) == 0                  # K % 64 != 0
    assert lib.clq_weight_bytes(8, 65536) == 0               # K too large
    assert lib.clq_act_bytes(8192, 1152) == 8192 * 576
    assert lib.clq_act_bytes(45, 256) == 64 * 128           # rows padded to 32
    assert lib.clq_act_bytes(0, 256) == 0


A = 0x10000          # aligned fake device address (never dereferenced)
MIS = 0x10002        # misaligned


def rq(lib, X=A, ldx=1152, perm=None, M=4, K=1152, block=64, Xq=A, xs=A):
    return lib.clq_rotate_quant_act(X, ldx, perm, M, K, block, Xq, xs, None)


def test_rotate_quant_validation(lib):
    assert rq(lib, X=None) == NULL
    assert rq(lib, Xq=None) == NULL
    assert rq(lib, xs=None) == NULL
    assert rq(lib, M=0) == SHAPE
    assert rq(lib, K=32) == SHAPE
    assert rq(lib, K=96, ldx=96) == SHAPE
    assert rq(lib, K=65536, ldx=65536) == SHAPE
    assert rq(lib, ldx=1000) == SHAPE
    assert rq(lib, ldx=1156) == SHAPE                    # not a multiple of 8
    assert rq(lib, block=16) == BLOCK
    assert rq(lib, block=256) == BLOCK
    assert rq(lib, K=192, ldx=192, block=128) == BLOCK   # K % block != 0
    assert rq(lib, X=MIS) == ALIGN
    assert rq(lib, Xq=A + 8) == ALIGN
    assert rq(lib, xs=A + 2) == ALIGN
    assert rq(lib, perm=A + 2) == ALIGN


def qw(lib, W=A, perm=None, N=8, K=1152, block=64, clip=1.0, Wq=A, ws=A):
    return lib.clq_quantize_weights(W, perm, N, K, block, clip, Wq, ws, None)


def test_quantize_weights_validation(lib):
    assert qw(lib, W=None) == NULL
    assert qw(lib, Wq=None) == NULL
    assert qw(lib, ws=None) == NULL
    assert qw(lib, N=0) == SHAPE
    assert qw(lib, K=1000) == SHAPE
    assert qw(lib, block=48) == BLOCK
    assert qw(lib, clip=0.0) == ARG
    assert qw(lib, clip=1.5) == ARG
    assert qw(lib, clip=-0.5) == ARG
    assert qw(lib, clip=float("nan")) == ARG
    assert qw(lib, W=MIS) == ALIGN
    assert qw(lib, Wq=A + 4) == ALIGN


def lin(lib, Xq=A, xs=A, Wq=A, ws=A, bias=None, M=4, N=8, K=1152, Y=A, ldy=8, wsp=None, wsb=0):
    return lib.clq_w4a4_linear(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, wsp, wsb, None)


def test_linear_validation(lib):
    assert lin(lib, Xq=None) == NULL
    assert lin(lib, xs=None) == NULL
    assert lin(lib, Wq=None) == NULL
    assert lin(lib, ws=None) == NULL
    assert lin(lib, Y=None) == NULL
    assert lin(lib, M=0) == SHAPE
    assert lin(lib, N=0) == SHAPE
    assert lin(lib, K=100) == SHAPE
    assert lin(lib, ldy=4) == SHAPE
    assert lin(lib, N=12, ldy=12) == SHAPE               # ldy % 8 != 0
    assert lin(lib, Y=A + 8) == ALIGN
    assert lin(lib, Xq=MIS) == ALIGN
    assert lin(lib, bias=A + 1) == ALIGN
    need = lib.clq_w4a4_workspace_bytes()
    assert need > 0
    assert lin(lib, wsp=A, wsb=need - 1) == WORKSPACE
    assert lin(lib, wsp=A + 8, wsb=need) == ALIGN
    assert lin(lib, Xq=None, wsp=A, wsb=need) == NULL          # checks stay in order


def test_workspace_bytes(lib):
    # one partial tile (128 x 256 int32) and four flags per workgroup, two
    # workgroups per compute unit, the grid a multiple of 8
    # 256 bytes of status words, then one partial tile (128 x 256 int32) and
    # four flags per workgroup, two workgroups per compute unit, the grid a
    # multiple of 8
    # (and 1 MiB of flags for the fused rotate+quantize items at the end)
    n = lib.clq_w4a4_workspace_bytes() - 256 - (1 << 20)
    per_wg = 128 * 256 * 4 + 4 * 4
    assert n % per_wg == 0 and (n // per_wg) % 8 == 0


def test_workspace_status_validation(lib):
    need = lib.clq_w4a4_workspace_bytes()
    assert lib.clq_w4a4_workspace_status(None, need, A, None) == NULL
    assert lib.clq_w4a4_workspace_status(A, need, None, None) == NULL
    assert lib.clq_w4a4_workspace_status(A, need - 1, A, None) == WORKSPACE
    assert lib.clq_w4a4_workspace_status(A + 8, need, A, None) == ALIGN
    assert lib.clq_w4a4_workspace_status(A, need, A + 2, None) == ALIGN


def schedule(lib, M, N, K, ws=1):
    info = (ctypes.c_int64 * 5)()
    assert lib.clq_w4a4_schedule(M, N, K, ws, ctypes.cast(info, ctypes.c_void_p)) == OK
    return list(info)


def test_schedule(lib):
    # host planning only (no device here: 256 compute units assumed, 512
    # persistent workgroups)
    info = (ctypes.c_int64 * 5)()
    assert lib.clq_w4a4_schedule(0, 8, 64, 1, ctypes.cast(info, ctypes.c_void_p)) == SHAPE
    assert lib.clq_w4a4_schedule(8, 8, 96, 1, ctypes.cast(info, ctypes.c_void_p)) == SHAPE
    assert lib.clq_w4a4_schedule(8, 8, 64, 1, None) == NULL
    # 17 x 16 tiles of 256 tokens (<= 1.25 per CU): two halves, 128-token tiles
    assert schedule(lib, 4352, 2048, 2432)[:2] == [1, 34 * 16]
    # few tiles: 64-token tiles
    assert schedule(lib, 1024, 1152, 1152)[:2] == [2, 16 * 9]
    # long k loops (K >= 2048, N < 4 K): the two-halves kernel at any tile
    # count -- the 28-block stack's fc2 at 16384 tokens, the video block's
    # fc2 (43200 tokens), the FLUX-style block's linears
    assert schedule(lib, 16384, 1152, 4608)[:2] == [1, 128 * 9]
    assert schedule(lib, 43200, 1152, 4608)[:2] == [1, 338 * 9]
    for N, K in ((9216, 3072), (3072, 3072), (3072, 12288)):
        assert schedule(lib, 4608, N, K)[:2] == [1, 36 * (N // 128)]
    # wide, shallow layers (N >= 4 K) too up to 8 tiles of 256 tokens per
    # CU (the FLUX-style fc1: 6.75), the persistent kernel beyond
    assert schedule(lib, 4608, 12288, 3072)[:2] == [1, 36 * 96]
    assert schedule(lib, 6144, 10240, 2560)[:2] == [1, 48 * 80]
    assert schedule(lib, 12288, 10240, 2560)[:2] == [0, 48 * 80]
    # 576 tiles of 30 stages: every k-stage split
    k, tiles, dp, sk, grid = schedule(lib, 16384, 1152, 1920)
    assert (k, tiles, dp, sk, grid) == (0, 576, 0, 576 * 30, 512)
    assert schedule(lib, 16384, 1152, 1920, ws=0) == [0, 576, 576, 0, 512]
    # 600 tiles of 24 stages: both rounds split, 28.1 stages per workgroup
    assert schedule(lib, 6400, 3072, 1536) == [0, 600, 0, 600 * 24, 512]
    # 1100 tiles: one whole round first, the last 588 tiles split
    assert schedule(lib, 11264, 3200, 1536) == [0, 1100, 512, 588 * 24, 512]
    # the PixArt block linears (M = 8192) and the video ones (M = 43200)
    # take whole tiles on the persistent grid
    for M, N, K in ((8192, 3456, 1152), (8192, 4608, 1152), (43200, 3456, 1152), (43200, 4608, 1152)):
        k, tiles, dp, sk, grid = schedule(lib, M, N, K)
        assert k == 0 and sk == 0 and dp == tiles


def test_mfma_probe_validation(lib):
    need = lib.clq_diag_mfma_probe_bytes()
    assert need == 1024 * 16 * 64 * 16
    assert lib.clq_diag_mfma_probe(None, need, 1, 1, A, None) == NULL
    assert lib.clq_diag_mfma_probe(A, need - 1, 1, 1, A, None) == WORKSPACE
    assert lib.clq_diag_mfma_probe(A, need, 0, 1, A, None) == ARG
    assert lib.clq_diag_mfma_probe(A, need, 1, 0, A, None) == ARG
    assert lib.clq_diag_mfma_probe(A + 8, need, 1, 1, A, None) == ALIGN


def rq_schedule(lib, M, N, K, b, ws=1):
    info = (ctypes.c_int64 * 4)()
    assert lib.clq_w4a4_rq_schedule(M, N, K, b, ws, ctypes.cast(info, ctypes.c_void_p)) == OK
    return list(info)


def test_rq_schedule(lib):
    # fused when the GEMM is the two-halves kernel, N % 16 == 0 and a
    # workspace is given; rows per item from the workgroup's lanes (one per
    # Hadamard block) and its LDS pool
    assert rq_schedule(lib, 1024, 1152, 1152, 64) == [1, 7, 147, 16 * 9]      # 64-token tiles, 128 lanes
    assert rq_schedule(lib, 1024, 3456, 1152, 64) == [1, 14, 74, 8 * 27]      # 128-token tiles, 256 lanes
    assert rq_schedule(lib, 1024, 1152, 4608, 64) == [0, 0, 0, 0]             # items of < 4 rows: two launches
    assert rq_schedule(lib, 1024, 1152, 2048, 64) == [1, 4, 256, 16 * 9]      # 32 blocks a row, 128 lanes: 4 rows
    assert rq_schedule(lib, 1024, 1152, 1152, 32) == [0, 0, 0, 0]             # 36 blocks, 128 lanes: 3 rows
    assert rq_schedule(lib, 1024, 3456, 1152, 32) == [1, 7, 147, 8 * 27]      # 256 lanes: 7 rows
    assert rq_schedule(lib, 1024, 1152, 1152, 64, ws=0)[0] == 0               # no workspace: two launches
    assert rq_schedule(lib, 43200, 3456, 1152, 64)[0] == 0                    # persistent grid: two launches
    assert rq_schedule(lib, 1024, 1000, 1152, 64)[0] == 0                     # N % 16 != 0
    info = (ctypes.c_int64 * 4)()
    assert lib.clq_w4a4_rq_schedule(1024, 1152, 1152, 48, 1, ctypes.cast(info, ctypes.c_void_p)) == BLOCK


def test_rq_linear_validation(lib):
    need = lib.clq_w4a4_workspace_bytes()
    def call(X=A, ldx=1152, b=64, Xq=A, xs=A, Wq=A, ws=A, bias=None, M=8, N=16, K=1152, Y=A, ldy=16, wsp=None, wsb=0):
        return lib.clq_w4a4_rq_linear(X, ldx, b, Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, wsp, wsb, None)
    assert call(X=None) == NULL and call(Xq=None) == NULL and call(ws=None) == NULL
    assert call(b=48) == BLOCK and call(K=96, ldx=96) == SHAPE and call(ldx=1000) == SHAPE
    assert call(X=A + 8) == ALIGN and call(ldy=12) == SHAPE
    assert call(wsp=A, wsb=need - 1) == WORKSPACE


def test_debug_knobs(lib):
    SYNC, SPIN, DROP = 0, 1, 2
    assert lib.clq_debug_get(SPIN) == 1 << 22 and lib.clq_debug_get(DROP) == 0
    assert lib.clq_debug_get(7) == -1
    assert lib.clq_debug_set(7, 0) == ARG
    assert lib.clq_debug_set(SYNC, 2) == ARG and lib.clq_debug_set(DROP, -1) == ARG
    assert lib.clq_debug_set(SPIN, -1) == ARG and lib.clq_debug_set(SPIN, (1 << 30) + 1) == ARG
    try:
        assert lib.clq_debug_set(SPIN, 5) == OK and lib.clq_debug_get(SPIN) == 5
        assert lib.clq_debug_set(DROP, 1) == OK and lib.clq_debug_get(DROP) == 1
        assert lib.clq_debug_set(SYNC, 1) == OK and lib.clq_debug_get(SYNC) == 1
    finally:
        assert lib.clq_debug_set(SPIN, 1 << 22) == OK
        assert lib.clq_debug_set(DROP, 0) == OK
        assert lib.clq_debug_set(SYNC, 0) == OK
    assert lib.clq_debug_get(SYNC) == 0


def f6_choice(lib, M, N, K):
    c = ctypes.c_int32(-1)
    assert lib.clq_w4a4_schedule_f6(M, N, K, ctypes.byref(c)) == OK
    return c.value


def test_f6_schedule_rule(lib):
    # 256 compute units (the MI355X's count, and the fallback without a GPU)
    assert f6_choice(lib, 1024, 3456, 1152) == 2     # 108 tiles of 256 tokens: two halves, 128-token tiles
    assert f6_choice(lib, 1024, 1152, 4608) == 3     # long k, 72 tiles of 128 tokens: 64-token tiles
    assert f6_choice(lib, 4096, 1152, 4608) == 2     # 144 tiles of 256 tokens
    assert f6_choice(lib, 4096, 3456, 1152) == 1     # 432 tiles: the persistent kernel
    assert f6_choice(lib, 43200, 1152, 4608) == 1    # long k, many tiles
    assert f6_choice(lib, 43200, 3456, 1152) == 1
    assert f6_choice(lib, 4608, 3072, 12288) == 1    # 432 tiles
    c = ctypes.c_int32()
    assert lib.clq_w4a4_schedule_f6(4096, 1152, 4608, None) == NULL
    assert lib.clq_w4a4_schedule_f6(4096, 1152, 64, ctypes.byref(c)) == SHAPE
    assert lib.clq_w4a4_schedule_f6(0, 1152, 1152, ctypes.byref(c)) == SHAPE
    try:
        assert lib.clq_debug_set(4, 3) == OK and f6_choice(lib, 43200, 3456, 1152) == 3
    finally:
        assert lib.clq_debug_set(4, 0) == OK


def test_f6_schedule_knob(lib):
    F6 = 4
    assert lib.clq_debug_get(F6) == 0
    assert lib.clq_debug_set(F6, -1) == ARG and lib.clq_debug_set(F6, 4) == ARG
    try:
        for v in (1, 2, 3):
            assert lib.clq_debug_set(F6, v) == OK and lib.clq_debug_get(F6) == v
    finally:
        assert lib.clq_debug_set(F6, 0) == OK
    assert lib.clq_debug_get(F6) == 0


def test_schedule_knob(lib):
    SCHED = 3
    assert lib.clq_debug_get(SCHED) == 0
    assert lib.clq_debug_set(SCHED, -1) == ARG and lib.clq_debug_set(SCHED, 5) == ARG
    try:
        # 1: persistent with its split rule; 2: persistent, whole tiles only
        assert lib.clq_debug_set(SCHED, 1) == OK and lib.clq_debug_get(SCHED) == 1
        assert schedule(lib, 1024, 1152, 1152) == [0, 36, 36, 0, 40]
        assert schedule(lib, 16384, 1152, 4608) == [0, 576, 0, 576 * 72, 512]
        assert lib.clq_debug_set(SCHED, 2) == OK
        assert schedule(lib, 16384, 1152, 4608) == [0, 576, 576, 0, 512]
        # 3 / 4: the two-halves kernel on 128- / 64-token tiles, any tile count
        assert lib.clq_debug_set(SCHED, 3) == OK
        assert schedule(lib, 43200, 3456, 1152)[:2] == [1, 338 * 27]
        assert schedule(lib, 1024, 1152, 1152)[:2] == [1, 8 * 9]
        assert lib.clq_debug_set(SCHED, 4) == OK
        assert schedule(lib, 43200, 3456, 1152)[:2] == [2, 675 * 27]
        # k loops too short to halve (K < 256) keep the automatic choice
        assert schedule(lib, 1024, 1152, 192)[0] == 0
        # the fused path follows the GEMM's schedule
        assert rq_schedule(lib, 1024, 1152, 1152, 64)[0] == 1
        assert lib.clq_debug_set(SCHED, 2) == OK
        assert rq_schedule(lib, 1024, 1152, 1152, 64)[0] == 0
    finally:
        assert lib.clq_debug_set(SCHED, 0) == OK
    assert schedule(lib, 1024, 1152, 1152)[:2] == [2, 16 * 9]


def test_accum_and_unswizzle_validation(lib):
    f = lib.clq_w4a4_accum_i32
    assert f(None, A, 4, 8, 1152, A, 8, None, 0, None) == NULL
    assert f(A, A, 4, 8, 1152, A, 6, None, 0, None) == SHAPE      # ldacc % 4 != 0
    assert f(A, A, 4, 8, 1152, A, 4, None, 0, None) == SHAPE      # ldacc < N
    assert f(A, A, 4, 8, 1152, A + 4, 8, None, 0, None) == ALIGN
    assert f(A, A, 4, 8, 1152, A, 8, A, 16, None) == WORKSPACE
    g = lib.clq_unswizzle_weights
    assert g(None, 8, 1152, A, None) == NULL
    assert g(A, 0, 1152, A, None) == SHAPE
    assert g(A, 8, 1152, A + 4, None) == ALIGN
    h = lib.clq_unswizzle_act
    assert h(None, 8, 1152, A, None) == NULL
    assert h(A, 8, 100, A, None) == SHAPE
    assert h(A, 8, 1152, A + 8, None) == ALIGN


def test_obs_workspace_bytes(lib):
    f = lib.clq_obs_workspace_bytes
    assert f(4096, 1152, 0) == 1152 * 128 and f(4096, 1152, 1) == 1152 * 128
    for m in (2, 3, 4):
        assert f(4096, 1152, m) == 4096 * 1152 * 4
    assert f(10, 8, 2) == 512                        # rounded up to 256
    assert f(0, 1152, 0) == 0 and f(16, 12, 0) == 0 and f(16, 1152, 5) == 0 and f(16, 1152, -1) == 0


def test_obs_validation(lib):
    f = lib.clq_obs_channel_scores
    need = lib.clq_obs_workspace_bytes(64, 1152, 0)

    def sc(X=A, ldx=1152, B=4, N=64, D=1152, metric=0, ws=A, wsb=need, out=A):
        return f(X, ldx, B, N, D, metric, ws, wsb, out, None)
    assert sc(X=None) == NULL
    assert sc(ws=None) == NULL
    assert sc(out=None) == NULL
    assert sc(metric=5) == ARG
    assert sc(metric=-1) == ARG
    assert sc(B=0) == SHAPE
    assert sc(N=0) == SHAPE
    assert sc(D=12, ldx=16) == SHAPE                  # D % 8 != 0
    assert sc(D=4, ldx=8) == SHAPE
    assert sc(ldx=1000) == SHAPE                      # ldx < D
    assert sc(ldx=1156) == SHAPE                      # ldx % 8 != 0
    assert sc(N=40000, metric=3, wsb=1 << 40) == SHAPE    # sort metrics: N <= 32768
    assert sc(X=A + 8) == ALIGN
    assert sc(ws=A + 8) == ALIGN
    assert sc(out=A + 2) == ALIGN
    assert sc(wsb=need - 1) == WORKSPACE
    assert sc(metric=2, wsb=need) == WORKSPACE        # the mean matrix is larger
    g = lib.clq_obs_permutation
    assert g(None, 64, A, None) == NULL
    assert g(A, 64, None, None) == NULL
    assert g(A, 63, A, None) == SHAPE
    assert g(A, 0, A, None) == SHAPE
    assert g(A, 65538, A, None) == SHAPE
    assert g(A + 2, 64, A, None) == ALIGN


def test_8bit_sizes(lib):
    assert lib.clq_act8_bytes(1, 64) == 32 * 64
    assert lib.clq_act8_bytes(8192, 1152) == 8192 * 1152
    assert lib.clq_act8_bytes(33, 1152) == 64 * 1152
    assert lib.clq_weight8_bytes(1, 64) == 64 * 64
    assert lib.clq_weight8_bytes(3456, 1152) == 3456 * 1152
    assert lib.clq_act8_bytes(0, 1152) == 0 and lib.clq_weight8_bytes(8, 100) == 0


def test_8bit_validation(lib):
    f = lib.clq_rotate_quant_act8
    assert f(None, 1152, None, 4, 1152, 64, A, A, None) == NULL
    assert f(A, 1152, None, 4, 1152, 48, A, A, None) == BLOCK
    assert f(A, 1000, None, 4, 1152, 64, A, A, None) == SHAPE
    assert f(A, 1152, None, 4, 1000, 64, A, A, None) == SHAPE
    assert f(A + 8, 1152, None, 4, 1152, 64, A, A, None) == ALIGN
    g = lib.clq_quantize_weights8
    assert g(A, None, 8, 1152, 64, 0.0, A, A, None) == ARG
    assert g(A, None, 8, 1152, 64, 1.5, A, A, None) == ARG
    assert g(A, None, 8, 1152, 64, 1.0, A + 4, A, None) == ALIGN
    h = lib.clq_a8_linear
    assert h(A, A, A, A, 4, None, 4, 8, 1152, None, 8, None) == NULL
    assert h(A, None, A, A, 4, None, 4, 8, 1152, A, 8, None) == NULL
    assert h(A, A, A, A, 5, None, 4, 8, 1152, A, 8, None) == ARG
    assert h(A, A, A, A, 8, None, 0, 8, 1152, A, 8, None) == SHAPE
    assert h(A, A, A, A, 8, None, 4, 8, 1100, A, 8, None) == SHAPE
    assert h(A, A, A, A, 8, None, 4, 12, 1152, A, 12, None) == SHAPE       # ldy % 8
    assert h(A, A, A, A, 4, None, 4, 8, 1152, A + 8, 8, None) == ALIGN
    assert h(A, A, A, A, 4, A + 1, 4, 8, 1152, A, 8, None) == ALIGN        # bias
    k = lib.clq_a8_accum_i32
    assert k(A, A, 4, 4, 8, 1152, A, 6, None) == SHAPE                     # ldacc % 4
    assert k(A, A, 0, 4, 8, 1152, A, 8, None) == ARG
    assert lib.clq_unswizzle_act8(None, 4, 1152, A, None) == NULL
    assert lib.clq_unswizzle_weights8(A, 4, 100, A, None) == SHAPE


def test_clps_validation(lib):
    need = lib.clq_clps_workspace_bytes(64, 48, 1152)
    assert need > 64 * 48 * 4
    assert lib.clq_clps_workspace_bytes(64, 48, 32768) == 0          # K <= 16384
    f = lib.clq_clps_search

    def cs(X=A, ldx=1152, W=A, Y0=A, ldy0=48, M=64, N=48, K=1152, block=64, gamma=0.01, grid=20,
           ws=A, wsb=need, al=A, er=A, best=A):
        return f(X, ldx, W, Y0, ldy0, None, M, N, K, block, gamma, grid, ws, wsb, al, er, best, None)
    assert cs(X=None) == NULL and cs(Y0=None) == NULL and cs(best=None) == NULL and cs(ws=None) == NULL
    assert cs(K=32768, ldx=32768) == SHAPE
    assert cs(block=48) == BLOCK
    assert cs(ldy0=40) == SHAPE
    assert cs(ldx=1156) == SHAPE
    assert cs(gamma=1.0) == ARG and cs(gamma=-0.1) == ARG
    assert cs(grid=0) == ARG and cs(grid=257) == ARG
    assert cs(er=A + 4) == ALIGN
    assert cs(Y0=A + 2) == ALIGN
    assert cs(wsb=need - 1) == WORKSPACE


def test_f6_sizes(lib):
    assert lib.clq_weight_bytes_f6(1152, 1152) == 1152 * 1152 * 3 // 4
    assert lib.clq_weight_bytes_f6(1, 64) == 64 * 64 * 3 // 4        # rows padded to 64
    assert lib.clq_act_bytes_f6(45, 256) == 64 * 256 * 3 // 4        # rows padded to 32
    assert lib.clq_act_bytes_f6(43200, 1152) == 43200 * 1152 * 3 // 4
    assert lib.clq_weight_bytes_f6(0, 64) == 0
    assert lib.clq_act_bytes_f6(8, 96) == 0


def test_f6_validation(lib):
    def rq6(X=A, ldx=1152, perm=None, M=4, K=1152, block=64, Xq=A, xs=A):
        return lib.clq_rotate_quant_act_f6(X, ldx, perm, M, K, block, Xq, xs, None)
    assert rq6(X=None) == NULL
    assert rq6(M=0) == SHAPE
    assert rq6(ldx=1000) == SHAPE
    assert rq6(block=16) == BLOCK
    assert rq6(Xq=A + 8) == ALIGN

    def qw6(W=A, perm=None, N=8, K=1152, block=64, clip=1.0, Wq=A, ws=A):
        return lib.clq_quantize_weights_f6(W, perm, N, K, block, clip, Wq, ws, None)
    assert qw6(ws=None) == NULL
    assert qw6(K=1000) == SHAPE
    assert qw6(block=48) == BLOCK
    assert qw6(clip=1.5) == ARG
    assert qw6(W=MIS) == ALIGN

    def lin6(Xq=A, xs=A, Wq=A, ws=A, bias=None, M=4, N=8, K=1152, Y=A, ldy=8):
        return lib.clq_w4a4_linear_f6(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, None)
    assert lin6(Xq=None) == NULL
    assert lin6(xs=None) == NULL
    assert lin6(K=64) == SHAPE          # k loops of two stages or more
    assert lin6(K=96) == SHAPE
    assert lin6(ldy=4) == SHAPE
    assert lin6(ldy=12) == SHAPE        # fp16 rows: a multiple of 8 elements
    assert lin6(Y=A + 8) == ALIGN
    assert lin6(bias=A + 1) == ALIGN

    def acc6(Xq=A, Wq=A, M=4, N=8, K=1152, acc=A, ldacc=8):
        return lib.clq_w4a4_accum_f6(Xq, Wq, M, N, K, acc, ldacc, None)
    assert acc6(acc=None) == NULL
    assert acc6(K=64) == SHAPE
    assert acc6(ldacc=10) == SHAPE      # int32 rows: a multiple of 4 elements
    assert lib.clq_unswizzle_f6(None, 4, 1152, 0, A, None) == NULL
    assert lib.clq_unswizzle_f6(A, 4, 1152, 2, A, None) == ARG
    assert lib.clq_unswizzle_f6(A, 4, 1000, 0, A, None) == SHAPE
    assert lib.clq_unswizzle_f6(A, 4, 1152, 1, A + 8, None) == ALIGN
    assert lib.clq_f6_from_int4(A, 0, 1152, 0, A, None) == SHAPE
    assert lib.clq_f6_from_int4(A, 4, 1152, 3, A, None) == ARG
    assert lib.clq_f6_from_int4(A + 4, 4, 1152, 1, A, None) == ALIGN
    nb = lib.clq_diag_mfma_probe_bytes()
    assert lib.clq_diag_mfma_probe_f6(None, nb, 1, 1, A, None) == NULL
    assert lib.clq_diag_mfma_probe_f6(A, nb - 1, 1, 1, A, None) == WORKSPACE
    assert lib.clq_diag_mfma_probe_f6(A, nb, 0, 1, A, None) == ARG
    assert lib.clq_diag_mfma_probe_f6(A, nb, 1, 1, A + 2, None) == ALIGN
