// int4 x int4 GEMM on the int8 matrix cores of gfx950, with the dequantising
// epilogue fused (CLQ, arXiv 2509.24416: the integer product of the W4A4
// codes, rescaled by the per-token activation scale and the per-channel
// weight scale of Eq. (1), plus bias).
//
// Matrix-core instruction: v_mfma_i32_32x32x32_i8 (16 int8 per lane per
// operand, 16 int32 accumulators per lane).  On gfx950 it sustains close to
// the chip's dense int8 rate, about twice what the 16x16x64 shape reaches.
//
// Operand roles.  The "row" operand is the weight (output channel n) and the
// "column" operand is the token (m).  The packed weight layout permutes rows
// inside each 32-row unit so that accumulator element v of lane l is channel
// 16*(l/32) + v of the fragment: every lane owns 16 consecutive channels of
// one token -- a 32-byte contiguous fp16 store.
//
// Data movement.  A k-stage is 64 codes deep: one 32x64 "unit" (1 KB packed,
// lane l's 16 bytes at 16*l) per 32 channels and per 32 tokens of the tile.
// Units go from global memory straight into LDS (global_load_lds_dwordx4: no
// registers, no VALU) through a ring of NS stages kept NS - 1 stages ahead of
// the matrix cores.  Each wave reads its units back with one 16-byte LDS read
// per lane and widens them to int8 in registers (packed operands halve the
// LDS traffic).  Widening keeps each nibble in the high half of its byte, so
// the int8 holds 16*q exactly; the int32 accumulator holds 256 * sum(qa*qw)
// (|.| <= 256*49*K < 2^31) and the factor 2^-8 is folded into the activation
// scale in the epilogue.  The k order inside a 32-code slice is permuted
// identically for both operands, which leaves the dot product unchanged.
//
// Synchronisation.  Every iteration issues the same number of memory
// instructions per wave, so "stage s has landed" is a fixed s_waitcnt vmcnt
// count; it is emitted together with the workgroup barrier as one asm
// statement with a memory clobber, so nothing is reordered across it.  The
// ring stages are separate LDS arrays, which lets the compiler see that a
// read of one stage does not depend on a transfer into another.
//
// Schedule: a persistent grid (one workgroup per compute unit) walks its
// tiles; the stage stream runs across tile boundaries, so the next tile's
// transfers overlap this tile's last matrix-core work and its epilogue.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "clq_internal.h"

#define CLQ_LDS __attribute__((address_space(3)))

namespace clq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// 16 int4 codes (8 packed bytes) -> 16 int8 values 16*q.  Output order:
// even codes of d0, even codes of d1, odd codes of d0, odd codes of d1.
__device__ __forceinline__ v4i widen16(uint32_t d0, uint32_t d1) {
    return v4i{(int)((d0 << 4) & 0xF0F0F0F0u), (int)((d1 << 4) & 0xF0F0F0F0u),
               (int)(d0 & 0xF0F0F0F0u), (int)(d1 & 0xF0F0F0F0u)};
}

constexpr int kStages = 5;   // ring depth
constexpr int kGroupM = 4;   // token panels per tile group (L2 reuse of channel panels)

template <int WN_, int WM_, int FN_, int FM_, int WGS_>
struct Tile {
    static constexpr int WN = WN_, WM = WM_, FN = FN_, FM = FM_;
    static constexpr int WGS = WGS_;               // workgroups per compute unit
    static constexpr int NW = WN * WM;             // waves
    static constexpr int NT = NW * 64;
    static constexpr int BN = WN * FN * 32;        // output channels per tile
    static constexpr int BM = WM * FM * 32;        // tokens per tile
    static constexpr int W_UNITS = BN / 32;        // units per stage
    static constexpr int X_UNITS = BM / 32;
    static constexpr int UNITS = W_UNITS + X_UNITS;
    static constexpr int UPW = UNITS / NW;         // units each wave moves per stage
    static constexpr int STAGE_BYTES = UNITS * 1024;
    // epilogue operand chunks of 64 values (one 4-byte transfer per lane):
    // token scales, channel scales, channel-bias pairs
    static constexpr int XS_CH = BM / 64, WS_CH = BN / 64, B_CH = BN / 128;
    static constexpr int E_CH = XS_CH + WS_CH + B_CH;
    static constexpr int EPW = (E_CH + NW - 1) / NW;   // chunks per wave per stage
    static_assert(UNITS % NW == 0, "units split evenly over waves");
};

template <class C, bool I32OUT, bool RAGGED>
__global__ void __launch_bounds__(C::NT, C::WGS)
w4a4_gemm_kernel(const uint8_t *__restrict__ Xq, const float *__restrict__ xs,
                 const uint8_t *__restrict__ Wq, const float *__restrict__ ws,
                 const uint16_t *__restrict__ bias, int M, int N, int K,
                 void *__restrict__ Y, int64_t ldy, int tiles_m, int tiles_n)
{
    constexpr int NS = kStages;
    // Ring of NS stages: operand units, then the epilogue operands of the
    // stage's tile (token scales fp32 [BM], channel scales fp32 [BN], biases
    // fp16 [BN]), so that a tile's operands have landed by its last stage.
    constexpr int E_XS = C::STAGE_BYTES, E_WS = E_XS + C::BM * 4, E_B = E_WS + C::BN * 4;
    constexpr int SLOT = I32OUT ? C::STAGE_BYTES : E_B + C::BN * 2;
    __shared__ __align__(16) uint8_t ring[NS][SLOT];

    // Persistent, XCD-aware schedule.  Workgroup b runs on XCD b % 8 (ids are
    // dealt round-robin).  Tiles are numbered in groups of kGroupM token
    // panels (within a group, consecutive numbers walk the token panels of
    // one channel panel), and the numbering is cut into 8 contiguous runs,
    // one per XCD; the gx workgroups of an XCD take turns through their run.
    // The tiles an XCD works on at any time then share few panels, which its
    // L2 serves.
    const int nks = K >> 6;
    const int ntiles = tiles_m * tiles_n;
    const int xcd = blockIdx.x & 7, jw = blockIdx.x >> 3, gx = gridDim.x >> 3;
    const int per = ntiles >> 3, rem = ntiles & 7;
    const int cnt = per + (xcd < rem ? 1 : 0);
    const int start = xcd * per + min(xcd, rem);
    const int my_tiles = jw < cnt ? (cnt - jw + gx - 1) / gx : 0;
    const int total = my_tiles * nks;   // k-stages this workgroup runs
    if (total == 0) return;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wn = wave % C::WN, wm = wave / C::WN;
    const int wunits_total = (int)(padded_rows(N) >> 5);
    const int xunits_total = (int)(padded_act_rows(M) >> 5);
    // bias == nullptr: the transfers read the (valid) channel scales instead
    // and the epilogue masks the value to zero
    const uint32_t *bsrc = reinterpret_cast<const uint32_t *>(bias ? (const void *)bias : (const void *)ws);
    const uint32_t bmask = bias ? 0xffffffffu : 0u;

    auto tile_coords = [&](int i, int &tm, int &tn) {
        const int L = start + jw + i * gx;
        const int gsz = kGroupM * tiles_n;
        const int g = L / gsz, r = L - g * gsz;
        const int m0 = g * kGroupM;
        const int gm = min(tiles_m - m0, kGroupM);
        tn = r / gm;
        tm = m0 + (r - tn * gm);
    };

    // ---- producer: one stage's transfers (the same count on every wave) -----
    // UPW operand units per wave, then (unless I32OUT) EPW chunks of 64
    // epilogue operands, 4 bytes per lane; chunk numbers past the real ones
    // re-read a channel-scale chunk into its own place (identical bytes).  The
    // ragged-edge kernel reads its biases in the epilogue instead.
    constexpr int EPW = I32OUT ? 0 : C::EPW;
    constexpr int VPI = C::UPW + EPW;   // memory instructions per wave per stage
    int p_i = 0, p_ks = 0, p_tm = 0, p_tn = 0, p_s = 0, p_q = 0;   // producer
    tile_coords(0, p_tm, p_tn);
    auto produce = [&]() {
        uint8_t *slot = &ring[p_q][0];
#pragma unroll
        for (int j = 0; j < C::UPW; ++j) {
            const int u = wave * C::UPW + j;   // wave-uniform
            const uint8_t *src;
            if (u < C::W_UNITS) {
                const int ug = min(p_tn * C::W_UNITS + u, wunits_total - 1);
                src = Wq + ((int64_t)ug * nks + p_ks) * 1024 + lane * 16;
            } else {
                const int ux = min(p_tm * C::X_UNITS + (u - C::W_UNITS), xunits_total - 1);
                src = Xq + ((int64_t)ux * nks + p_ks) * 1024 + lane * 16;
            }
            __builtin_amdgcn_global_load_lds(src, (CLQ_LDS void *)(slot + u * 1024), 16, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < EPW; ++j) {
            const int c = wave * EPW + j;      // wave-uniform chunk
            const void *src;
            int dst;
            if (c < C::XS_CH) {
                src = xs + min(p_tm * C::BM + c * 64 + lane, M - 1);
                dst = E_XS + c * 256;
            } else if (c < C::XS_CH + C::WS_CH || c >= C::E_CH || RAGGED) {
                const int w = (c - C::XS_CH) % C::WS_CH;
                src = ws + min(p_tn * C::BN + w * 64 + lane, N - 1);
                dst = E_WS + w * 256;
            } else {
                // channel pairs (2p, 2p+1) of the tile; N % 16 == 0 here
                const int b = c - C::XS_CH - C::WS_CH;
                src = bsrc + min(p_tn * (C::BN / 2) + b * 64 + lane, N / 2 - 1);
                dst = E_B + b * 256;
            }
            __builtin_amdgcn_global_load_lds(src, (CLQ_LDS void *)(slot + dst), 4, 0, 0);
        }
        // advance to the next stage (clamped at the last one)
        if (p_s < total - 1) {
            ++p_s;
            p_q = p_q == NS - 1 ? 0 : p_q + 1;
            if (++p_ks == nks) {
                p_ks = 0;
                ++p_i;
                tile_coords(p_i, p_tm, p_tn);
            }
        }
    };

    // ---- consumer ------------------------------------------------------------
    // P: packed operands of one stage (one 16-byte LDS read per unit);
    // A0/B0, A1/B1: the widened operands of its two 32-code halves.
    uint4 pa[C::FN], pb[C::FM];
    v4i a0[C::FN], b0[C::FM], a1[C::FN], b1[C::FM];
    auto read_packed = [&](int q) {
        const uint8_t *Wl = &ring[q][0];
        const uint8_t *Xl = Wl + C::W_UNITS * 1024;
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
            pa[fn] = *reinterpret_cast<const uint4 *>(Wl + (wn * C::FN + fn) * 1024 + lane * 16);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
            pb[fm] = *reinterpret_cast<const uint4 *>(Xl + (wm * C::FM + fm) * 1024 + lane * 16);
    };
    auto widen_half0 = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) a0[fn] = widen16(pa[fn].x, pa[fn].y);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) b0[fm] = widen16(pb[fm].x, pb[fm].y);
    };
    auto widen_half1 = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) a1[fn] = widen16(pa[fn].z, pa[fn].w);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) b1[fm] = widen16(pb[fm].z, pb[fm].w);
    };
    v16i acc[C::FN][C::FM];
    auto zero_acc = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = v16i{};
    };
    auto mma = [&](const v4i (&a)[C::FN], const v4i (&b)[C::FM]) {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[fn], b[fm], acc[fn][fm], 0, 0, 0);
    };
    // one matrix-core instruction, then up to `vpm` vector instructions, for
    // every instruction of a half-step: widening runs in the MFMA shadow
    constexpr int MPH = C::FN * C::FM;                         // MFMAs per half-step
    constexpr int WOPS = (C::FN + C::FM) * 6;                  // widening VALU ops per half
    constexpr int VPM = (WOPS + MPH - 1) / MPH + 1;
    auto interleave = [&](int first_plain) {
#pragma unroll
        for (int i = 0; i < MPH; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // MFMA
            if (i >= first_plain) __builtin_amdgcn_sched_group_barrier(0x002, VPM, 0);   // VALU
        }
    };

    // ---- epilogue: lane owns token m and 16 consecutive channels ----------
    const int h16 = (lane >> 5) * 16;
    auto epilogue = [&](int i, int q) {
        int tm, tn;
        tile_coords(i, tm, tn);
        const float *e_xs = reinterpret_cast<const float *>(&ring[q][E_XS]);
        const float *e_ws = reinterpret_cast<const float *>(&ring[q][E_WS]);
        const uint32_t *e_b = reinterpret_cast<const uint32_t *>(&ring[q][E_B]);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) {
            const int ml = (wm * C::FM + fm) * 32 + (lane & 31);
            const int m = tm * C::BM + ml;
            float xsm = 0.0f;
            if constexpr (!I32OUT) xsm = e_xs[ml] * (1.0f / 256.0f);
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn) {
                const int nl = (wn * C::FN + fn) * 32 + h16;
                const int n0 = tn * C::BN + nl;
                const v16i &a = acc[fn][fm];
                if constexpr (I32OUT) {
                    int32_t *dst = reinterpret_cast<int32_t *>(Y) + (int64_t)m * ldy + n0;
                    if (m < M && n0 < N) {
                        if (!RAGGED || n0 + 16 <= N) {
#pragma unroll
                            for (int q4 = 0; q4 < 4; ++q4)
                                reinterpret_cast<int4 *>(dst)[q4] =
                                    make_int4(a[4 * q4] >> 8, a[4 * q4 + 1] >> 8, a[4 * q4 + 2] >> 8, a[4 * q4 + 3] >> 8);
                        } else {
#pragma unroll
                            for (int v = 0; v < 16; ++v)
                                if (n0 + v < N) dst[v] = a[v] >> 8;
                        }
                    }
                } else {
                    float wsv[16];
                    uint32_t bw[8];
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const float4 w4 = reinterpret_cast<const float4 *>(e_ws + nl)[q4];
                        wsv[4 * q4] = w4.x; wsv[4 * q4 + 1] = w4.y; wsv[4 * q4 + 2] = w4.z; wsv[4 * q4 + 3] = w4.w;
                    }
                    if constexpr (RAGGED) {
#pragma unroll
                        for (int v = 0; v < 16; v += 2) {
                            const int na = min(n0 + v, N - 1), nb = min(n0 + v + 1, N - 1);
                            bw[v / 2] = bias ? ((uint32_t)bias[na] | ((uint32_t)bias[nb] << 16)) : 0u;
                        }
                    } else {
#pragma unroll
                        for (int q2 = 0; q2 < 2; ++q2) {
                            const uint4 b4 = reinterpret_cast<const uint4 *>(e_b + nl / 2)[q2];
                            bw[4 * q2] = b4.x & bmask; bw[4 * q2 + 1] = b4.y & bmask;
                            bw[4 * q2 + 2] = b4.z & bmask; bw[4 * q2 + 3] = b4.w & bmask;
                        }
                    }
                    uint32_t hv[8];
#pragma unroll
                    for (int v = 0; v < 16; v += 2) {
                        float y2[2];
#pragma unroll
                        for (int d = 0; d < 2; ++d) {
                            const float p = (float)a[v + d] * xsm;
                            const uint16_t bb = (uint16_t)(bw[v / 2] >> (16 * d));
                            y2[d] = __builtin_fmaf(p, wsv[v + d], __half2float(__ushort_as_half(bb)));
                        }
                        hv[v / 2] = (uint32_t)__half_as_ushort(__float2half_rn(y2[0])) |
                                    ((uint32_t)__half_as_ushort(__float2half_rn(y2[1])) << 16);
                    }
                    uint16_t *dst = reinterpret_cast<uint16_t *>(Y) + (int64_t)m * ldy + n0;
                    if (m < M && n0 < N) {
                        if (!RAGGED || n0 + 16 <= N) {
                            reinterpret_cast<uint4 *>(dst)[0] = make_uint4(hv[0], hv[1], hv[2], hv[3]);
                            reinterpret_cast<uint4 *>(dst)[1] = make_uint4(hv[4], hv[5], hv[6], hv[7]);
                        } else {
#pragma unroll
                            for (int v = 0; v < 16; ++v)
                                if (n0 + v < N) dst[v] = (uint16_t)(hv[v >> 1] >> (16 * (v & 1)));
                        }
                    }
                }
            }
        }
    };

    // ---- pipeline ------------------------------------------------------------
    // Stage s lives in ring stage s % NS.  Prologue: stages 0 .. NS-2 in
    // flight; once stages 0 and 1 have landed, read stage 0 and widen its
    // first half.  Iteration s (packed stage s in P, its first half in A0/B0):
    //   wait until stage s+1 has landed -- its transfers are older than the
    //   (NS-3) * VPI memory instructions this wave issued since -- and for
    //   this wave's LDS reads; barrier.  Every wave is then done with ring
    //   stage (s - 1) % NS, which receives stage s + NS - 1.
    //   MFMAs on half 0 of stage s, widening half 1 of stage s in their shadow;
    //   read stage s+1 into P;
    //   MFMAs on half 1 of stage s, widening half 0 of stage s+1 in their
    //   shadow (the first few MFMAs cover the LDS read latency);
    //   after a tile's last stage, the epilogue (its scales and biases
    //   travelled with the stage).
    for (int k = 0; k < NS - 1; ++k) produce();
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((NS - 3) * VPI) : "memory");
    read_packed(0);
    widen_half0();
    zero_acc();

    int c_ks = 0, c_i = 0, c_q = 0;   // consumer position: k-stage, tile, ring stage
    for (int s = 0; s < total; ++s) {
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"((NS - 3) * VPI) : "memory");
        produce();
        __builtin_amdgcn_sched_barrier(0);
        widen_half1();
        mma(a0, b0);
        interleave(0);
        __builtin_amdgcn_sched_barrier(0);
        const int nq = c_q == NS - 1 ? 0 : c_q + 1;
        read_packed(nq);
        __builtin_amdgcn_sched_barrier(0);
        widen_half0();
        mma(a1, b1);
        interleave(2);
        __builtin_amdgcn_sched_barrier(0);
        if (c_ks == nks - 1) {
            epilogue(c_i, c_q);
            zero_acc();
            c_ks = 0;
            ++c_i;
        } else {
            ++c_ks;
        }
        c_q = nq;
    }
    // drain: no transfer may still be writing LDS when the workgroup exits
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Workgroups for the persistent schedule: a multiple of 8 (one share per
// XCD), at most `per_cu` per compute unit.
int persistent_grid(int ntiles, int per_cu) {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
    }
    const int g = min(ntiles, cus * per_cu);
    return max(8, (g + 7) / 8 * 8);
}

template <class C, bool I32OUT, bool RAGGED>
hipError_t launch_cfg(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                      const uint16_t *bias, int64_t M, int64_t N, int K, void *Y,
                      int64_t ldy, hipStream_t stream) {
    const int tiles_m = (int)((M + C::BM - 1) / C::BM);
    const int tiles_n = (int)((N + C::BN - 1) / C::BN);
    const int grid = persistent_grid(tiles_m * tiles_n, C::WGS);
    hipLaunchKernelGGL((w4a4_gemm_kernel<C, I32OUT, RAGGED>), dim3((unsigned)grid), dim3(C::NT),
                       0, stream, Xq, xs, Wq, ws, bias, (int)M, (int)N, K, Y, ldy, tiles_m,
                       tiles_n);
    return hipGetLastError();
}

// 8 waves of 128 channels x 64 tokens; one workgroup per compute unit
using T256x256 = Tile<2, 4, 4, 2, 1>;

template <bool I32OUT>
hipError_t launch_shape(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                        const uint16_t *bias, int64_t M, int64_t N, int K, void *Y, int64_t ldy,
                        hipStream_t stream) {
    if (N % 16 != 0)  // a ragged channel edge needs element-wise stores
        return launch_cfg<T256x256, I32OUT, true>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream);
    return launch_cfg<T256x256, I32OUT, false>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream);
}

}  // namespace

hipError_t launch_gemm(const uint8_t *Xq, const float *xs, const uint8_t *Wq,
                       const float *ws, const uint16_t *bias, int64_t M, int64_t N,
                       int K, void *Y, int64_t ldy, bool i32out, hipStream_t stream) {
    return i32out ? launch_shape<true>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream)
                  : launch_shape<false>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream);
}

}  // namespace clq
