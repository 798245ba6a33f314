// W4A8 and W8A8 GEMM with the CLQ epilogue (arXiv 2509.24416, Sec. 4.1: the
// method is run at the bit settings W8A8, W4A8 and W4A4; Sec. 3.1 Eq. (1)
// with n = 8 for the activations, and for the weights of W8A8).
//
// Activations arrive as int8 codes in the int8 layout (clq_internal.h), one
// fp32 scale per token; weights as int4 (the packed weight layout of the W4A4
// path) or int8 codes (the int8 layout, fragment rows in the int4 weights'
// order), one fp32 scale per output channel with 1/b folded in.  Both feed
// v_mfma_i32_32x32x32_i8 directly, except that int4 weights are widened to
// int8 holding 16 q (so the int32 accumulator holds 16 * sum for W4A8).
//
// Tiles: 128 channels x 128 tokens per workgroup of two waves (each wave 128
// channels x 64 tokens: 4 x 2 fragments, 128 accumulator registers), four
// (W4A8) or three (W8A8) workgroups per compute unit.  A k-stage is 64 codes:
// 4 weight units (1 KB int4 / 2 KB int8) and 4 token units (2 KB) that go
// global -> LDS with global_load_lds_dwordx4 through a ring of 3 stages kept
// 2 ahead.  LDS reads are asm (the compiler would otherwise wait for every
// transfer in flight before them, as in the W4A4 kernel), and the wait for a
// stage is an explicit vmcnt count fused with the barrier.  The grid has one
// workgroup per tile, tiles handed to XCDs in contiguous runs.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "clq_internal.h"

#define CLQ_LDS __attribute__((address_space(3)))

namespace clq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef _Float16 h2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)reinterpret_cast<size_t>((CLQ_LDS const void *)p);
}
template <int OFF>
__device__ __forceinline__ v4u lds_read16(uint32_t addr) {
    v4u v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
}
template <int I, int N, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, N>(f);
    }
}
// 16 int4 codes (two dwords) -> 16 int8 holding 16 q: even codes, then odd
__device__ __forceinline__ v4i widen16(uint32_t d0, uint32_t d1) {
    return v4i{(int)((d0 << 4) & 0xF0F0F0F0u), (int)((d1 << 4) & 0xF0F0F0F0u),
               (int)(d0 & 0xF0F0F0F0u), (int)(d1 & 0xF0F0F0F0u)};
}

constexpr int kBN = 128, kBM = 128;      // channels, tokens per tile
constexpr int kFN = 4, kFM = 2;          // fragments per wave
constexpr int kWaves = 2;
constexpr int kNS = 3;                   // ring depth

template <int WB>
struct A8Cfg {
    static constexpr int W_UNIT = WB == 4 ? 1024 : 2048;       // bytes per 32 rows x 64 codes
    static constexpr int W_BYTES = 4 * W_UNIT;
    static constexpr int X_BYTES = 4 * 2048;
    static constexpr int STAGE = W_BYTES + X_BYTES;
    static constexpr int PIECES = STAGE / 1024;                 // 1 KB transfers per stage
    static constexpr int PPW = PIECES / kWaves;                 // per wave
    static constexpr int WGS = WB == 4 ? 4 : 3;                 // workgroups per CU (LDS)
    static_assert(PIECES % kWaves == 0, "pieces split evenly");
};

struct A8Args {
    const uint8_t *Xq;
    const float *xs;
    const uint8_t *Wq;
    const float *ws;
    const uint16_t *bias;
    void *Y;
    int64_t ldy;
    int M, N, K, tiles_m, tiles_n, per_xcd;
};

template <int WB, bool I32OUT, bool BIAS>
__global__ void __launch_bounds__(kWaves * 64, 2) a8_gemm_kernel(A8Args a)
{
    using C = A8Cfg<WB>;
    __shared__ __align__(16) uint8_t ring[kNS][C::STAGE];

    // tile: XCD b % 8 takes a contiguous run of tiles, grouped 8 token panels
    // at a time so that a weight panel serves consecutive tiles
    const int b = blockIdx.x;
    const int L = (b & 7) * a.per_xcd + (b >> 3);
    if (L >= a.tiles_m * a.tiles_n) return;
    const int gsz = 8 * a.tiles_n;
    const int g = L / gsz, rr = L - g * gsz;
    const int m0 = g * 8, gm = min(a.tiles_m - m0, 8);
    const int tn = rr / gm, tm = m0 + (rr - tn * gm);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nks = a.K >> 6;
    const int wunits = (int)(padded_rows(a.N) >> 5), xunits = (int)(padded_act_rows(a.M) >> 5);

    // this wave's transfers of a stage: piece p of the stage (1 KB each);
    // weight pieces first, then token pieces.  Source = base + k * step.
    const uint8_t *src[C::PPW];
    int step[C::PPW];
#pragma unroll
    for (int i = 0; i < C::PPW; ++i) {
        const int p = wave * C::PPW + i;
        if (p < C::W_BYTES / 1024) {
            const int per = C::W_UNIT / 1024;                 // pieces per weight unit
            const int u = min(tn * 4 + p / per, wunits - 1);
            src[i] = a.Wq + (int64_t)u * nks * C::W_UNIT + (p % per) * 1024 + lane * 16;
            step[i] = C::W_UNIT;
        } else {
            const int px = p - C::W_BYTES / 1024;
            const int u = min(tm * 4 + px / 2, xunits - 1);
            src[i] = a.Xq + (int64_t)u * nks * 2048 + (px & 1) * 1024 + lane * 16;
            step[i] = 2048;
        }
    }
    auto produce = [&](int k, int slot) {
        uint8_t *dst = &ring[slot][0];
#pragma unroll
        for (int i = 0; i < C::PPW; ++i) {
            const uint8_t *sp = src[i] + (int64_t)k * step[i];
            __builtin_amdgcn_global_load_lds(sp, (CLQ_LDS void *)(dst + (wave * C::PPW + i) * 1024), 16, 0, 0);
        }
    };
    // stage k has landed once at most `later` stages' transfers (issued after
    // it) are outstanding; then every wave's transfers are in after the barrier
    auto landed = [&](int later) {
        if (later >= 1)
            asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(C::PPW) : "memory");
        else
            asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    };
    static_assert(kNS == 3, "at most one stage in flight behind the one waited for");

    v16i acc[kFN][kFM];
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
        for (int fm = 0; fm < kFM; ++fm) acc[fn][fm] = v16i{};

    produce(0, 0);
    if (nks > 1) produce(1, 1);
    const uint32_t base0 = lds_addr(&ring[0][0]);
    for (int k = 0; k < nks; ++k) {
        landed(min(1, nks - 1 - k));
        if (k + 2 < nks) produce(k + 2, (k + 2) % kNS);
        // operands of stage k
        uint32_t ad = base0 + (uint32_t)((k % kNS) * C::STAGE) + (uint32_t)lane * 16;
        asm volatile("" : "+v"(ad));
        v4u pw[kFN][WB == 4 ? 1 : 2], px[kFM][2];
        static_for<0, kFN>([&](auto fc) {
            constexpr int fn = decltype(fc)::value;
            pw[fn][0] = lds_read16<fn * C::W_UNIT>(ad);
            if constexpr (WB == 8) pw[fn][WB == 4 ? 0 : 1] = lds_read16<fn * C::W_UNIT + 1024>(ad);
        });
        static_for<0, kFM>([&](auto fc) {
            constexpr int fm = decltype(fc)::value;
            constexpr int off = C::W_BYTES + fm * 2048;   // this wave's unit is 2*wave + fm
            px[fm][0] = lds_read16<off>(ad + (uint32_t)(wave * 2 * 2048));
            px[fm][1] = lds_read16<off + 1024>(ad + (uint32_t)(wave * 2 * 2048));
        });
        // the wait names every read result, so no use can be scheduled above it
        if constexpr (WB == 4)
            asm volatile("s_waitcnt lgkmcnt(0)"
                         : "+v"(pw[0][0]), "+v"(pw[1][0]), "+v"(pw[2][0]), "+v"(pw[3][0]),
                           "+v"(px[0][0]), "+v"(px[0][1]), "+v"(px[1][0]), "+v"(px[1][1]));
        else
            asm volatile("s_waitcnt lgkmcnt(0)"
                         : "+v"(pw[0][0]), "+v"(pw[1][0]), "+v"(pw[2][0]), "+v"(pw[3][0]),
                           "+v"(pw[0][WB == 4 ? 0 : 1]), "+v"(pw[1][WB == 4 ? 0 : 1]),
                           "+v"(pw[2][WB == 4 ? 0 : 1]), "+v"(pw[3][WB == 4 ? 0 : 1]),
                           "+v"(px[0][0]), "+v"(px[0][1]), "+v"(px[1][0]), "+v"(px[1][1]));
        v4i a0[kFN], a1[kFN], b0[kFM], b1[kFM];
#pragma unroll
        for (int fn = 0; fn < kFN; ++fn) {
            if constexpr (WB == 4) {
                a0[fn] = widen16(pw[fn][0][0], pw[fn][0][1]);
                a1[fn] = widen16(pw[fn][0][2], pw[fn][0][3]);
            } else {
                a0[fn] = __builtin_bit_cast(v4i, pw[fn][0]);
                a1[fn] = __builtin_bit_cast(v4i, pw[fn][WB == 4 ? 0 : 1]);
            }
        }
#pragma unroll
        for (int fm = 0; fm < kFM; ++fm) {
            b0[fm] = __builtin_bit_cast(v4i, px[fm][0]);
            b1[fm] = __builtin_bit_cast(v4i, px[fm][1]);
        }
#pragma unroll
        for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0[fn], b0[fm], acc[fn][fm], 0, 0, 0);
#pragma unroll
        for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a1[fn], b1[fm], acc[fn][fm], 0, 0, 0);
    }

    // ---- epilogue: lane owns token m and 16 consecutive channels ------------
    // channel operands outer (loaded once per fragment column), tokens inner
    const int M = a.M, N = a.N;
    const int h16 = (lane >> 5) * 16;
    float xsc[kFM];
    int mrow[kFM];
#pragma unroll
    for (int fm = 0; fm < kFM; ++fm) {
        mrow[fm] = tm * kBM + wave * 64 + fm * 32 + (lane & 31);
        // accumulators hold 16 * sum for int4 weights
        xsc[fm] = I32OUT ? 0.0f : a.xs[min(mrow[fm], M - 1)] * (WB == 4 ? 0.0625f : 1.0f);
    }
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
        const int n0 = tn * kBN + fn * 32 + h16;
        if (n0 >= N) continue;
        const bool full = n0 + 16 <= N;
        float wsv[16], bv[16];
        if constexpr (!I32OUT) {
            if (full) {
                const float4 *w4 = reinterpret_cast<const float4 *>(a.ws + n0);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float4 w = w4[q];
                    wsv[4 * q] = w.x;
                    wsv[4 * q + 1] = w.y;
                    wsv[4 * q + 2] = w.z;
                    wsv[4 * q + 3] = w.w;
                }
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) wsv[v] = a.ws[min(n0 + v, N - 1)];
            }
#pragma unroll
            for (int v = 0; v < 16; ++v)
                bv[v] = BIAS ? (float)reinterpret_cast<const _Float16 *>(a.bias)[min(n0 + v, N - 1)] : 0.0f;
        }
#pragma unroll
        for (int fm = 0; fm < kFM; ++fm) {
            const int m = mrow[fm];
            if (m >= M) continue;
            const v16i &x = acc[fn][fm];
            if constexpr (I32OUT) {
                int32_t *dst = reinterpret_cast<int32_t *>(a.Y) + (int64_t)m * a.ldy + n0;
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (full || n0 + v < N) dst[v] = WB == 4 ? (x[v] >> 4) : x[v];
            } else {
                uint32_t hv[8];
#pragma unroll
                for (int v = 0; v < 16; v += 2) {
                    const float p0 = (float)x[v] * xsc[fm], p1 = (float)x[v + 1] * xsc[fm];
                    h2v h;
                    h[0] = (_Float16)__builtin_fmaf(p0, wsv[v], bv[v]);
                    h[1] = (_Float16)__builtin_fmaf(p1, wsv[v + 1], bv[v + 1]);
                    hv[v / 2] = __builtin_bit_cast(uint32_t, h);
                }
                uint16_t *dst = reinterpret_cast<uint16_t *>(a.Y) + (int64_t)m * a.ldy + n0;
                if (full) {
                    reinterpret_cast<v4u *>(dst)[0] = v4u{hv[0], hv[1], hv[2], hv[3]};
                    reinterpret_cast<v4u *>(dst)[1] = v4u{hv[4], hv[5], hv[6], hv[7]};
                } else {
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        if (n0 + v < N) dst[v] = (uint16_t)(hv[v >> 1] >> (16 * (v & 1)));
                }
            }
        }
    }
}

template <int WB, bool I32OUT, bool BIAS>
hipError_t launch_cfg(const A8Args &g, hipStream_t stream) {
    const int tiles = g.tiles_m * g.tiles_n;
    A8Args a = g;
    a.per_xcd = (tiles + 7) / 8;
    hipLaunchKernelGGL((a8_gemm_kernel<WB, I32OUT, BIAS>), dim3((unsigned)(a.per_xcd * 8)),
                       dim3(kWaves * 64), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_a8_gemm(const uint8_t *Xq8, const float *xs, const uint8_t *Wq, int wbits,
                          const float *ws, const uint16_t *bias, int64_t M, int64_t N, int K,
                          void *Y, int64_t ldy, bool i32out, hipStream_t stream) {
    A8Args g{};
    g.Xq = Xq8;
    g.xs = xs;
    g.Wq = Wq;
    g.ws = ws;
    g.bias = bias;
    g.Y = Y;
    g.ldy = ldy;
    g.M = (int)M;
    g.N = (int)N;
    g.K = K;
    g.tiles_m = (int)((M + kBM - 1) / kBM);
    g.tiles_n = (int)((N + kBN - 1) / kBN);
    if (wbits == 4) {
        if (i32out) return launch_cfg<4, true, false>(g, stream);
        return bias ? launch_cfg<4, false, true>(g, stream) : launch_cfg<4, false, false>(g, stream);
    }
    if (wbits == 8) {
        if (i32out) return launch_cfg<8, true, false>(g, stream);
        return bias ? launch_cfg<8, false, true>(g, stream) : launch_cfg<8, false, false>(g, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace clq
