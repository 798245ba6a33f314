// C ABI of the CLQ W4A4 linear library: host-side validation and launches.
// Every entry point checks its arguments before enqueuing anything and
// returns a status code; kernels run on the caller's stream.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <atomic>

#include "../../include/clq.h"
#include "clq_internal.h"
#include "f6_codes.h"

namespace {

constexpr int kVersion = 8;
constexpr int64_t kMaxK = 32768;
constexpr int64_t kMaxRows = 2147483647;

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

clq_status check_block(int64_t K, int32_t block) {
    if (block != 32 && block != 64 && block != 128) return CLQ_ERR_BLOCK;
    if (K % block != 0) return CLQ_ERR_BLOCK;
    return CLQ_OK;
}

clq_status check_k(int64_t K) {
    if (K < 64 || K > kMaxK || K % 64 != 0) return CLQ_ERR_SHAPE;
    return CLQ_OK;
}

clq_status check_rows(int64_t R) {
    if (R < 1 || R > kMaxRows) return CLQ_ERR_SHAPE;
    return CLQ_OK;
}

// Debug knobs (process-wide host state).  CLQ_DEBUG_SYNC starts from the
// CLQ_SYNC environment variable.
std::atomic<int> debug_sync{-1};

bool sync_mode() {
    int v = debug_sync.load(std::memory_order_relaxed);
    if (v < 0) {
        const char *e = getenv("CLQ_SYNC");
        v = (e != nullptr && e[0] != '\0' && e[0] != '0') ? 1 : 0;
        int expect = -1;
        debug_sync.compare_exchange_strong(expect, v);
        v = debug_sync.load(std::memory_order_relaxed);
    }
    return v != 0;
}

// The status of an enqueued launch; in sync mode the stream is drained first,
// so that a kernel's own failure is reported by the call that launched it.
clq_status done(hipStream_t stream, hipError_t e) {
    if (e != hipSuccess) return CLQ_ERR_HIP;
    if (sync_mode()) {
        if (hipStreamSynchronize(stream) != hipSuccess) return CLQ_ERR_HIP;
        if (hipGetLastError() != hipSuccess) return CLQ_ERR_HIP;
    }
    return CLQ_OK;
}

}  // namespace

extern "C" {

int clq_version(void) { return kVersion; }

const char *clq_status_string(clq_status s) {
    switch (s) {
        case CLQ_OK: return "CLQ_OK";
        case CLQ_ERR_NULL: return "CLQ_ERR_NULL: a required pointer is NULL";
        case CLQ_ERR_SHAPE: return "CLQ_ERR_SHAPE: a size or row stride is out of range";
        case CLQ_ERR_BLOCK: return "CLQ_ERR_BLOCK: block must be 32, 64 or 128 and divide K";
        case CLQ_ERR_ALIGN: return "CLQ_ERR_ALIGN: a pointer is misaligned";
        case CLQ_ERR_ARG: return "CLQ_ERR_ARG: clip_ratio, metric, wbits, gamma or grid out of range";
        case CLQ_ERR_HIP: return "CLQ_ERR_HIP: a HIP launch failed";
        case CLQ_ERR_WORKSPACE: return "CLQ_ERR_WORKSPACE: workspace smaller than the entry point's *_workspace_bytes()";
    }
    return "CLQ: unknown status";
}

size_t clq_weight_bytes(int64_t N, int64_t K) {
    if (check_rows(N) != CLQ_OK || check_k(K) != CLQ_OK) return 0;
    return (size_t)clq::padded_rows(N) * (size_t)(K / 2);
}

size_t clq_act_bytes(int64_t M, int64_t K) {
    if (check_rows(M) != CLQ_OK || check_k(K) != CLQ_OK) return 0;
    return (size_t)clq::padded_act_rows(M) * (size_t)(K / 2);
}

clq_status clq_quantize_weights(const void *W, const int32_t *perm, int64_t N, int64_t K,
                                int32_t block, float clip_ratio, void *Wq, float *w_scale,
                                hipStream_t stream) {
    if (!W || !Wq || !w_scale) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (!(clip_ratio >= 0x1p-24f && clip_ratio <= 1.0f)) return CLQ_ERR_ARG;
    if (!aligned(W, 16) || !aligned(Wq, 16) || !aligned(w_scale, 4) || (perm && !aligned(perm, 4)))
        return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_rotate_quant(
        static_cast<const uint16_t *>(W), K, perm, N, clq::padded_rows(N), (int)K, block,
        clip_ratio, true, 1.0f / (float)block, static_cast<uint8_t *>(Wq), w_scale, stream));
}

clq_status clq_rotate_quant_act(const void *X, int64_t ldx, const int32_t *perm, int64_t M,
                                int64_t K, int32_t block, void *Xq, float *x_scale,
                                hipStream_t stream) {
    if (!X || !Xq || !x_scale) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (ldx < K || ldx % 8 != 0) return CLQ_ERR_SHAPE;
    if (!aligned(X, 16) || !aligned(Xq, 16) || !aligned(x_scale, 4) || (perm && !aligned(perm, 4)))
        return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_rotate_quant(static_cast<const uint16_t *>(X), ldx, perm, M,
                                             clq::padded_act_rows(M), (int)K, block, 1.0f, false,
                                             1.0f, static_cast<uint8_t *>(Xq), x_scale, stream));
}

static clq_status check_gemm(const void *Xq, const void *Wq, int64_t M, int64_t N, int64_t K,
                             const void *Y, int64_t ldy, int64_t ld_mult) {
    if (!Xq || !Wq || !Y) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK)
        return s;
    if (ldy < N || ldy % ld_mult != 0) return CLQ_ERR_SHAPE;
    if (!aligned(Xq, 16) || !aligned(Wq, 16) || !aligned(Y, 16)) return CLQ_ERR_ALIGN;
    return CLQ_OK;
}

static clq_status check_workspace(const void *workspace, size_t workspace_bytes) {
    if (!workspace) return CLQ_OK;
    if (workspace_bytes < clq::gemm_workspace_bytes()) return CLQ_ERR_WORKSPACE;
    if (!aligned(workspace, 16)) return CLQ_ERR_ALIGN;
    return CLQ_OK;
}

size_t clq_w4a4_workspace_bytes(void) { return clq::gemm_workspace_bytes(); }

clq_status clq_w4a4_workspace_status(const void *workspace, size_t workspace_bytes, int32_t *status,
                                     hipStream_t stream) {
    if (!workspace || !status) return CLQ_ERR_NULL;
    if (workspace_bytes < clq::gemm_workspace_bytes()) return CLQ_ERR_WORKSPACE;
    if (!aligned(workspace, 16) || !aligned(status, 4)) return CLQ_ERR_ALIGN;
    return done(stream, hipMemcpyAsync(status, workspace, 3 * sizeof(int32_t), hipMemcpyDeviceToDevice, stream));
}

clq_status clq_w4a4_schedule(int64_t M, int64_t N, int64_t K, int32_t with_workspace, int64_t *info) {
    if (!info) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    const clq::GemmPlan p = clq::plan_gemm(M, N, (int)K, with_workspace != 0);
    info[0] = p.kernel;
    info[1] = p.tiles;
    info[2] = p.dp;
    info[3] = p.sk;
    info[4] = p.grid;
    return CLQ_OK;
}

clq_status clq_w4a4_schedule_f6(int64_t M, int64_t N, int64_t K, int32_t *choice) {
    if (!choice) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (K < 128) return CLQ_ERR_SHAPE;
    *choice = clq::f6_schedule(M, N, (int)K);
    return CLQ_OK;
}

size_t clq_diag_mfma_probe_bytes(void) { return clq::mfma_probe_bytes(); }

clq_status clq_diag_mfma_probe(const void *ops, size_t ops_bytes, int32_t iters, int32_t grid, int32_t *sink,
                               hipStream_t stream) {
    if (!ops || !sink) return CLQ_ERR_NULL;
    if (ops_bytes < clq::mfma_probe_bytes()) return CLQ_ERR_WORKSPACE;
    if (iters < 1 || grid < 1 || grid > 65536) return CLQ_ERR_ARG;
    if (!aligned(ops, 16) || !aligned(sink, 4)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_mfma_probe(ops, iters, sink, grid, stream));
}

clq_status clq_diag_mfma_probe_f6(const void *ops, size_t ops_bytes, int32_t iters, int32_t grid, int32_t *sink,
                                  hipStream_t stream) {
    if (!ops || !sink) return CLQ_ERR_NULL;
    if (ops_bytes < clq::mfma_probe_bytes()) return CLQ_ERR_WORKSPACE;
    if (iters < 1 || grid < 1 || grid > 65536) return CLQ_ERR_ARG;
    if (!aligned(ops, 16) || !aligned(sink, 4)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_mfma_probe_f6(ops, iters, sink, grid, stream));
}

clq_status clq_debug_set(int32_t knob, int64_t value) {
    switch (knob) {
        case CLQ_DEBUG_SYNC:
            if (value != 0 && value != 1) return CLQ_ERR_ARG;
            debug_sync.store((int)value, std::memory_order_relaxed);
            return CLQ_OK;
        case CLQ_DEBUG_SPLIT_SPIN_LIMIT:
            if (value < 0 || value > (1 << 30)) return CLQ_ERR_ARG;
            __atomic_store_n(&clq::gemm_spin_limit, (int)value, __ATOMIC_RELAXED);
            return CLQ_OK;
        case CLQ_DEBUG_SPLIT_DROP_SIGNAL:
            if (value != 0 && value != 1) return CLQ_ERR_ARG;
            __atomic_store_n(&clq::gemm_drop_signal, (int)value, __ATOMIC_RELAXED);
            return CLQ_OK;
        case CLQ_DEBUG_GEMM_SCHEDULE:
            if (value < 0 || value > 4) return CLQ_ERR_ARG;
            __atomic_store_n(&clq::gemm_force_schedule, (int)value, __ATOMIC_RELAXED);
            return CLQ_OK;
        case CLQ_DEBUG_F6_SCHEDULE:
            if (value < 0 || value > 3) return CLQ_ERR_ARG;
            __atomic_store_n(&clq::f6_schedule_force, (int)value, __ATOMIC_RELAXED);
            return CLQ_OK;
    }
    return CLQ_ERR_ARG;
}

int64_t clq_debug_get(int32_t knob) {
    switch (knob) {
        case CLQ_DEBUG_SYNC: return sync_mode() ? 1 : 0;
        case CLQ_DEBUG_SPLIT_SPIN_LIMIT: return __atomic_load_n(&clq::gemm_spin_limit, __ATOMIC_RELAXED);
        case CLQ_DEBUG_SPLIT_DROP_SIGNAL: return __atomic_load_n(&clq::gemm_drop_signal, __ATOMIC_RELAXED);
        case CLQ_DEBUG_GEMM_SCHEDULE: return __atomic_load_n(&clq::gemm_force_schedule, __ATOMIC_RELAXED);
        case CLQ_DEBUG_F6_SCHEDULE: return __atomic_load_n(&clq::f6_schedule_force, __ATOMIC_RELAXED);
    }
    return -1;
}

clq_status clq_w4a4_linear(const void *Xq, const float *x_scale, const void *Wq,
                           const float *w_scale, const void *bias, int64_t M, int64_t N,
                           int64_t K, void *Y, int64_t ldy, void *workspace,
                           size_t workspace_bytes, hipStream_t stream) {
    if (!x_scale || !w_scale) return CLQ_ERR_NULL;
    clq_status s = check_gemm(Xq, Wq, M, N, K, Y, ldy, 8);
    if (s != CLQ_OK) return s;
    if (!aligned(x_scale, 4) || !aligned(w_scale, 4) || (bias && !aligned(bias, 2)))
        return CLQ_ERR_ALIGN;
    if ((s = check_workspace(workspace, workspace_bytes)) != CLQ_OK) return s;
    return done(stream, clq::launch_gemm(static_cast<const uint8_t *>(Xq), x_scale,
                                     static_cast<const uint8_t *>(Wq), w_scale,
                                     static_cast<const uint16_t *>(bias), M, N, (int)K, Y, ldy,
                                     false, workspace, stream));
}

clq_status clq_w4a4_linear_noalloc(const void *Xq, const float *x_scale, const void *Wq,
                                   const float *w_scale, const void *bias, int64_t M, int64_t N,
                                   int64_t K, void *Y, int64_t ldy, int32_t *status,
                                   hipStream_t stream) {
    if (!x_scale || !w_scale) return CLQ_ERR_NULL;
    clq_status s = check_gemm(Xq, Wq, M, N, K, Y, ldy, 8);
    if (s != CLQ_OK) return s;
    if (!aligned(x_scale, 4) || !aligned(w_scale, 4) || (bias && !aligned(bias, 2)) || (status && !aligned(status, 4)))
        return CLQ_ERR_ALIGN;
    if (clq::gemm_split_bytes() > clq::gemm_scratch_bytes()) return CLQ_ERR_WORKSPACE;
    return done(stream, clq::launch_gemm_noalloc(static_cast<const uint8_t *>(Xq), x_scale,
                                                 static_cast<const uint8_t *>(Wq), w_scale,
                                                 static_cast<const uint16_t *>(bias), M, N, (int)K, Y, ldy,
                                                 status, stream));
}

clq_status clq_w4a4_rq_linear(const void *X, int64_t ldx, int32_t block, void *Xq, float *x_scale,
                              const void *Wq, const float *w_scale, const void *bias, int64_t M, int64_t N,
                              int64_t K, void *Y, int64_t ldy, void *workspace, size_t workspace_bytes,
                              hipStream_t stream) {
    if (!X || !x_scale || !w_scale) return CLQ_ERR_NULL;
    clq_status s = check_gemm(Xq, Wq, M, N, K, Y, ldy, 8);
    if (s != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (ldx < K || ldx % 8 != 0) return CLQ_ERR_SHAPE;
    if (!aligned(X, 16) || !aligned(x_scale, 4) || !aligned(w_scale, 4) || (bias && !aligned(bias, 2)))
        return CLQ_ERR_ALIGN;
    if ((s = check_workspace(workspace, workspace_bytes)) != CLQ_OK) return s;
    return done(stream, clq::launch_rq_gemm(static_cast<const uint16_t *>(X), ldx, block, static_cast<uint8_t *>(Xq),
                                            x_scale, static_cast<const uint8_t *>(Wq), w_scale,
                                            static_cast<const uint16_t *>(bias), M, N, (int)K, Y, ldy, workspace,
                                            stream));
}

clq_status clq_w4a4_rq_schedule(int64_t M, int64_t N, int64_t K, int32_t block, int32_t with_workspace,
                                int64_t *info) {
    if (!info) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    const clq::RqGemmPlan p = clq::plan_rq_gemm(M, N, (int)K, block, with_workspace != 0);
    info[0] = p.fused;
    info[1] = p.rq_rows;
    info[2] = p.n_rq;
    info[3] = p.tiles;
    return CLQ_OK;
}

clq_status clq_w4a4_accum_i32(const void *Xq, const void *Wq, int64_t M, int64_t N, int64_t K,
                              int32_t *acc, int64_t ldacc, void *workspace,
                              size_t workspace_bytes, hipStream_t stream) {
    clq_status s = check_gemm(Xq, Wq, M, N, K, acc, ldacc, 4);
    if (s != CLQ_OK) return s;
    if ((s = check_workspace(workspace, workspace_bytes)) != CLQ_OK) return s;
    return done(stream, clq::launch_gemm(static_cast<const uint8_t *>(Xq), nullptr,
                                     static_cast<const uint8_t *>(Wq), nullptr, nullptr, M, N,
                                     (int)K, acc, ldacc, true, workspace, stream));
}

clq_status clq_unswizzle_weights(const void *Wq, int64_t N, int64_t K, void *Wq_canonical,
                                 hipStream_t stream) {
    if (!Wq || !Wq_canonical) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (!aligned(Wq, 16) || !aligned(Wq_canonical, 8)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_unswizzle(static_cast<const uint8_t *>(Wq), N, (int)K,
                                          static_cast<uint8_t *>(Wq_canonical), stream));
}

size_t clq_weight_bytes_f6(int64_t N, int64_t K) {
    if (check_rows(N) != CLQ_OK || check_k(K) != CLQ_OK) return 0;
    return (size_t)clq::f6_operand_bytes(clq::padded_rows(N), K);
}

size_t clq_act_bytes_f6(int64_t M, int64_t K) {
    if (check_rows(M) != CLQ_OK || check_k(K) != CLQ_OK) return 0;
    return (size_t)clq::f6_operand_bytes(clq::padded_act_rows(M), K);
}

clq_status clq_quantize_weights_f6(const void *W, const int32_t *perm, int64_t N, int64_t K,
                                   int32_t block, float clip_ratio, void *Wq, float *w_scale,
                                   hipStream_t stream) {
    if (!W || !Wq || !w_scale) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (!(clip_ratio >= 0x1p-24f && clip_ratio <= 1.0f)) return CLQ_ERR_ARG;
    if (!aligned(W, 16) || !aligned(Wq, 16) || !aligned(w_scale, 4) || (perm && !aligned(perm, 4)))
        return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_rotate_quant(
        static_cast<const uint16_t *>(W), K, perm, N, clq::padded_rows(N), (int)K, block,
        clip_ratio, true, 1.0f / (float)block, static_cast<uint8_t *>(Wq), w_scale, stream, 6));
}

clq_status clq_rotate_quant_act_f6(const void *X, int64_t ldx, const int32_t *perm, int64_t M,
                                   int64_t K, int32_t block, void *Xq, float *x_scale,
                                   hipStream_t stream) {
    if (!X || !Xq || !x_scale) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (ldx < K || ldx % 8 != 0) return CLQ_ERR_SHAPE;
    if (!aligned(X, 16) || !aligned(Xq, 16) || !aligned(x_scale, 4) || (perm && !aligned(perm, 4)))
        return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_rotate_quant(static_cast<const uint16_t *>(X), ldx, perm, M,
                                             clq::padded_act_rows(M), (int)K, block, 1.0f, false,
                                             1.0f, static_cast<uint8_t *>(Xq), x_scale, stream, 6));
}

clq_status clq_w4a4_linear_f6(const void *Xq, const float *x_scale, const void *Wq, const float *w_scale,
                              const void *bias, int64_t M, int64_t N, int64_t K, void *Y, int64_t ldy,
                              hipStream_t stream) {
    if (!x_scale || !w_scale) return CLQ_ERR_NULL;
    clq_status s = check_gemm(Xq, Wq, M, N, K, Y, ldy, 8);
    if (s != CLQ_OK) return s;
    if (K < 128) return CLQ_ERR_SHAPE;
    if (!aligned(x_scale, 4) || !aligned(w_scale, 4) || (bias && !aligned(bias, 2))) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_gemm_f6(static_cast<const uint8_t *>(Xq), x_scale, static_cast<const uint8_t *>(Wq),
                                            w_scale, static_cast<const uint16_t *>(bias), M, N, (int)K, Y, ldy, false,
                                            stream));
}

clq_status clq_w4a4_accum_f6(const void *Xq, const void *Wq, int64_t M, int64_t N, int64_t K, int32_t *acc,
                             int64_t ldacc, hipStream_t stream) {
    clq_status s = check_gemm(Xq, Wq, M, N, K, acc, ldacc, 4);
    if (s != CLQ_OK) return s;
    if (K < 128) return CLQ_ERR_SHAPE;
    return done(stream, clq::launch_gemm_f6(static_cast<const uint8_t *>(Xq), nullptr, static_cast<const uint8_t *>(Wq),
                                            nullptr, nullptr, M, N, (int)K, acc, ldacc, true, stream));
}

clq_status clq_unswizzle_f6(const void *q6, int64_t rows, int64_t K, int32_t weights, void *canonical,
                            hipStream_t stream) {
    if (!q6 || !canonical) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(rows)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (weights != 0 && weights != 1) return CLQ_ERR_ARG;
    if (!aligned(q6, 16) || !aligned(canonical, 16)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_unswizzle_f6(static_cast<const uint8_t *>(q6), rows, (int)K, weights != 0,
                                                 static_cast<uint8_t *>(canonical), stream));
}

clq_status clq_f6_from_int4(const void *q4, int64_t rows, int64_t K, int32_t weights, void *q6,
                            hipStream_t stream) {
    if (!q4 || !q6) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(rows)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (weights != 0 && weights != 1) return CLQ_ERR_ARG;
    if (!aligned(q4, 16) || !aligned(q6, 16)) return CLQ_ERR_ALIGN;
    const int64_t prows = weights ? clq::padded_rows(rows) : clq::padded_act_rows(rows);
    return done(stream, clq::launch_repack_f6(static_cast<const uint8_t *>(q4), prows / 32 * (K / 64),
                                              static_cast<uint8_t *>(q6), stream));
}

clq_status clq_unswizzle_act(const void *Xq, int64_t M, int64_t K, void *Xq_canonical,
                             hipStream_t stream) {
    if (!Xq || !Xq_canonical) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (!aligned(Xq, 16) || !aligned(Xq_canonical, 16)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_unswizzle_act(static_cast<const uint8_t *>(Xq), M, (int)K,
                                              static_cast<uint8_t *>(Xq_canonical), stream));
}

size_t clq_obs_workspace_bytes(int64_t N, int64_t D, int32_t metric) {
    if (N < 1 || N > kMaxRows || D < 8 || D > 65536 || D % 8 != 0 || metric < 0 || metric > 4) return 0;
    return clq::obs_workspace_bytes(N, D, metric);
}

clq_status clq_obs_channel_scores(const void *X, int64_t ldx, int64_t B, int64_t N, int64_t D,
                                  int32_t metric, void *workspace, size_t workspace_bytes,
                                  float *scores, hipStream_t stream) {
    if (!X || !scores || !workspace) return CLQ_ERR_NULL;
    if (metric < 0 || metric > 4) return CLQ_ERR_ARG;
    if (B < 1 || B >= (1 << 24) || N < 1 || N > kMaxRows || D < 8 || D > 65536 || D % 8 != 0)
        return CLQ_ERR_SHAPE;
    if (metric >= 2 && N > 32768) return CLQ_ERR_SHAPE;
    if (ldx < D || ldx % 8 != 0) return CLQ_ERR_SHAPE;
    if (!aligned(X, 16) || !aligned(workspace, 16) || !aligned(scores, 4)) return CLQ_ERR_ALIGN;
    if (workspace_bytes < clq::obs_workspace_bytes(N, D, metric)) return CLQ_ERR_WORKSPACE;
    return done(stream, clq::launch_obs_scores(static_cast<const uint16_t *>(X), ldx, B, N, (int)D, metric,
                                           workspace, scores, stream));
}

clq_status clq_obs_permutation(const float *scores, int64_t D, int32_t *perm, hipStream_t stream) {
    if (!scores || !perm) return CLQ_ERR_NULL;
    if (D < 2 || D > 65536 || D % 2 != 0) return CLQ_ERR_SHAPE;
    if (!aligned(scores, 4) || !aligned(perm, 4)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_obs_permutation(scores, (int)D, perm, stream));
}

/* ---- 8-bit activations (W4A8, W8A8) -------------------------------------- */

size_t clq_act8_bytes(int64_t M, int64_t K) {
    if (check_rows(M) != CLQ_OK || check_k(K) != CLQ_OK) return 0;
    return (size_t)clq::padded_act_rows(M) * (size_t)K;
}

size_t clq_weight8_bytes(int64_t N, int64_t K) {
    if (check_rows(N) != CLQ_OK || check_k(K) != CLQ_OK) return 0;
    return (size_t)clq::padded_rows(N) * (size_t)K;
}

clq_status clq_rotate_quant_act8(const void *X, int64_t ldx, const int32_t *perm, int64_t M,
                                 int64_t K, int32_t block, void *Xq8, float *x_scale,
                                 hipStream_t stream) {
    if (!X || !Xq8 || !x_scale) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (ldx < K || ldx % 8 != 0) return CLQ_ERR_SHAPE;
    if (!aligned(X, 16) || !aligned(Xq8, 16) || !aligned(x_scale, 4) || (perm && !aligned(perm, 4)))
        return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_rotate_quant(
        static_cast<const uint16_t *>(X), ldx, perm, M, clq::padded_act_rows(M), (int)K, block, 1.0f,
        false, 1.0f, static_cast<uint8_t *>(Xq8), x_scale, stream, 8));
}

clq_status clq_quantize_weights8(const void *W, const int32_t *perm, int64_t N, int64_t K,
                                 int32_t block, float clip_ratio, void *Wq8, float *w_scale,
                                 hipStream_t stream) {
    if (!W || !Wq8 || !w_scale) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (!(clip_ratio >= 0x1p-24f && clip_ratio <= 1.0f)) return CLQ_ERR_ARG;
    if (!aligned(W, 16) || !aligned(Wq8, 16) || !aligned(w_scale, 4) || (perm && !aligned(perm, 4)))
        return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_rotate_quant(
        static_cast<const uint16_t *>(W), K, perm, N, clq::padded_rows(N), (int)K, block, clip_ratio,
        true, 1.0f / (float)block, static_cast<uint8_t *>(Wq8), w_scale, stream, 8));
}

static clq_status check_a8(const void *Xq8, const void *Wq, int32_t wbits, int64_t M, int64_t N,
                           int64_t K, const void *Y, int64_t ld, int64_t ld_mult) {
    if (!Xq8 || !Wq || !Y) return CLQ_ERR_NULL;
    if (wbits != 4 && wbits != 8) return CLQ_ERR_ARG;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (ld < N || ld % ld_mult != 0) return CLQ_ERR_SHAPE;
    if (!aligned(Xq8, 16) || !aligned(Wq, 16) || !aligned(Y, 16)) return CLQ_ERR_ALIGN;
    return CLQ_OK;
}

clq_status clq_a8_linear(const void *Xq8, const float *x_scale, const void *Wq, const float *w_scale,
                         int32_t wbits, const void *bias, int64_t M, int64_t N, int64_t K, void *Y,
                         int64_t ldy, hipStream_t stream) {
    if (!x_scale || !w_scale) return CLQ_ERR_NULL;
    clq_status s = check_a8(Xq8, Wq, wbits, M, N, K, Y, ldy, 8);
    if (s != CLQ_OK) return s;
    if (!aligned(x_scale, 4) || !aligned(w_scale, 4) || (bias && !aligned(bias, 2))) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_a8_gemm(static_cast<const uint8_t *>(Xq8), x_scale,
                                        static_cast<const uint8_t *>(Wq), wbits, w_scale,
                                        static_cast<const uint16_t *>(bias), M, N, (int)K, Y, ldy, false,
                                        stream));
}

clq_status clq_a8_accum_i32(const void *Xq8, const void *Wq, int32_t wbits, int64_t M, int64_t N,
                            int64_t K, int32_t *acc, int64_t ldacc, hipStream_t stream) {
    clq_status s = check_a8(Xq8, Wq, wbits, M, N, K, acc, ldacc, 4);
    if (s != CLQ_OK) return s;
    return done(stream, clq::launch_a8_gemm(static_cast<const uint8_t *>(Xq8), nullptr,
                                        static_cast<const uint8_t *>(Wq), wbits, nullptr, nullptr, M, N,
                                        (int)K, acc, ldacc, true, stream));
}

clq_status clq_unswizzle_act8(const void *Xq8, int64_t M, int64_t K, void *codes, hipStream_t stream) {
    if (!Xq8 || !codes) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (!aligned(Xq8, 16)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_unswizzle8(static_cast<const uint8_t *>(Xq8), M, (int)K, false,
                                           static_cast<int8_t *>(codes), stream));
}

clq_status clq_unswizzle_weights8(const void *Wq8, int64_t N, int64_t K, void *codes, hipStream_t stream) {
    if (!Wq8 || !codes) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (!aligned(Wq8, 16)) return CLQ_ERR_ALIGN;
    return done(stream, clq::launch_unswizzle8(static_cast<const uint8_t *>(Wq8), N, (int)K, true,
                                           static_cast<int8_t *>(codes), stream));
}

/* ---- CLPS single-layer clip search ------------------------------------------ */

size_t clq_clps_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (check_rows(M) != CLQ_OK || check_rows(N) != CLQ_OK || check_k(K) != CLQ_OK || K > 16384) return 0;
    return clq::clps_workspace_bytes(M, N, K);
}

clq_status clq_clps_search(const void *X, int64_t ldx, const void *W, const float *Y0, int64_t ldy0,
                           const int32_t *perm, int64_t M, int64_t N, int64_t K, int32_t block,
                           float gamma, int32_t grid, void *workspace, size_t workspace_bytes,
                           float *alphas, double *errors, int32_t *best, hipStream_t stream) {
    if (!X || !W || !Y0 || !workspace || !alphas || !errors || !best) return CLQ_ERR_NULL;
    clq_status s;
    if ((s = check_rows(M)) != CLQ_OK || (s = check_rows(N)) != CLQ_OK || (s = check_k(K)) != CLQ_OK) return s;
    if (K > 16384) return CLQ_ERR_SHAPE;
    if ((s = check_block(K, block)) != CLQ_OK) return s;
    if (ldx < K || ldx % 8 != 0 || ldy0 < N) return CLQ_ERR_SHAPE;
    if (!(gamma >= 0.0f && gamma < 1.0f) || grid < 1 || grid > 256) return CLQ_ERR_ARG;
    if (!aligned(X, 16) || !aligned(W, 16) || !aligned(Y0, 4) || !aligned(workspace, 16) ||
        !aligned(alphas, 4) || !aligned(errors, 8) || !aligned(best, 4) || (perm && !aligned(perm, 4)))
        return CLQ_ERR_ALIGN;
    if (workspace_bytes < clq::clps_workspace_bytes(M, N, K)) return CLQ_ERR_WORKSPACE;
    // l = floor(gamma (K - 1)) weights above the order statistic
    const int l = (int)floor((double)gamma * (double)(K - 1));
    return done(stream, clq::launch_clps(static_cast<const uint16_t *>(X), ldx, static_cast<const uint16_t *>(W), Y0,
                                     ldy0, perm, M, N, (int)K, block, (int)(K - 1 - l), grid, workspace, alphas,
                                     errors, best, stream));
}

}  // extern "C"
