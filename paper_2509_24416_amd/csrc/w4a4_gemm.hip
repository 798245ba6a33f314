// int4 x int4 GEMM on the int8 matrix cores of gfx950, with the dequantising
// epilogue fused (CLQ, arXiv 2509.24416: the integer product of the W4A4
// codes, rescaled by the per-token activation scale and the per-channel
// weight scale of Eq. (1), plus bias).
//
// Operand roles.  The matrix-core "row" operand is the weight (n) and the
// "column" operand is the token (m), so each lane's 16x16 accumulator tile
// holds one token and four output channels; the packed weight layout permutes
// rows inside each group of 64 so that, over the four fragments of a group, a
// lane owns 16 consecutive channels -- a 32-byte contiguous fp16 store.
//
// Data flow per k-step of KT codes: packed int4 tiles are loaded from global
// memory into registers (one k-step ahead), widened to int8 and written to a
// double-buffered LDS stage, then read back as 16-byte matrix-core fragments
// (one contiguous 1 KB run per 16x64 fragment).  Widening keeps each nibble
// in the high half of its byte: the int8 holds 16*q, exactly, so the int32
// accumulator holds 256 * sum(qa*qw) (|.| <= 256*49*K < 2^31) and the factor
// 2^-8 is folded into the activation scale in the epilogue.  The k order
// inside a 16-code group is permuted identically for both operands, which
// leaves the dot product unchanged.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "clq_internal.h"

namespace clq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

// 16 int4 codes (8 packed bytes) -> 16 int8 values 16*q.  Output order:
// even codes of d0, even codes of d1, odd codes of d0, odd codes of d1.
__device__ __forceinline__ uint4 widen16(uint32_t d0, uint32_t d1) {
    return make_uint4((d0 << 4) & 0xF0F0F0F0u, (d1 << 4) & 0xF0F0F0F0u,
                      d0 & 0xF0F0F0F0u, d1 & 0xF0F0F0F0u);
}

template <int WN_, int WM_, int FN_, int FM_, int KT_>
struct Tile {
    static constexpr int WN = WN_, WM = WM_, FN = FN_, FM = FM_, KT = KT_;
    static constexpr int NT = WN * WM * 64;
    static constexpr int BN = WN * FN * 16;   // output channels per tile
    static constexpr int BM = WM * FM * 16;   // tokens per tile
    static constexpr int KU = KT / 64;        // 64-code fragment units per k-step
    static constexpr int W_UNITS = BN / 16 * KU;
    static constexpr int X_UNITS = BM / 16 * KU;
    static constexpr int STAGE_BYTES = (W_UNITS + X_UNITS) * 1024;
    static constexpr int W_CHUNKS = W_UNITS * 32;   // 16-byte packed chunks
    static constexpr int X_CHUNKS = BM * KT / 32;
    static constexpr int WPT = W_CHUNKS / NT;
    static constexpr int XPT = X_CHUNKS / NT;
    static constexpr int CPR = KT / 32;             // packed chunks per token row
    static_assert(FN % 4 == 0, "a wave owns whole groups of 64 channels");
    static_assert(W_CHUNKS % NT == 0 && X_CHUNKS % NT == 0, "even load split");
};

template <class C, bool I32OUT>
__global__ void __launch_bounds__(C::NT)
w4a4_gemm_kernel(const uint8_t *__restrict__ Xq, const float *__restrict__ xs,
                 const uint8_t *__restrict__ Wq, const float *__restrict__ ws,
                 const uint16_t *__restrict__ bias, int M, int N, int K,
                 void *__restrict__ Y, int64_t ldy, int tiles_m, int tiles_n)
{
    extern __shared__ __align__(16) uint8_t smem[];

    // XCD-aware tile order: workgroup ids are dealt round-robin to the 8 XCDs;
    // give each XCD a contiguous run of logical tiles, which walk the channel
    // tiles of one token panel before moving to the next panel.
    const int ntiles = tiles_m * tiles_n;
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int per = ntiles >> 3, rem = ntiles & 7;
    const int L = xcd * per + min(xcd, rem) + slot;
    const int tm = L / tiles_n, tn = L - tm * tiles_n;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wn = wave % C::WN, wm = wave / C::WN;
    const int kunits = K >> 6;
    const int wunits_total = (int)(padded_rows(N) >> 4);

    // global sources of this thread's chunks
    const uint8_t *wsrc[C::WPT];
#pragma unroll
    for (int it = 0; it < C::WPT; ++it) {
        const int c = it * C::NT + tid;
        const int ul = c / (C::KU * 32), within = c % (C::KU * 32);
        const int ug = min(tn * (C::BN / 16) + ul, wunits_total - 1);
        wsrc[it] = Wq + ((int64_t)ug * kunits) * 512 + within * 16;
    }
    const uint8_t *xsrc[C::XPT];
    int xdst[C::XPT];
#pragma unroll
    for (int it = 0; it < C::XPT; ++it) {
        const int c = it * C::NT + tid;
        const int ml = (c & 15) + 16 * (c / (16 * C::CPR));
        const int cc = (c >> 4) % C::CPR;
        const int64_t row = min(tm * C::BM + ml, M - 1);
        xsrc[it] = Xq + row * (K >> 1) + cc * 16;
        xdst[it] = C::W_UNITS * 1024 + ((ml >> 4) * C::KU + (cc >> 1)) * 1024 +
                   ((2 * (cc & 1)) * 16 + (ml & 15)) * 16;
    }

    uint4 wreg[C::WPT], xreg[C::XPT];
    auto load_stage = [&](int ks) {
#pragma unroll
        for (int it = 0; it < C::WPT; ++it)
            wreg[it] = *reinterpret_cast<const uint4 *>(wsrc[it] + (int64_t)ks * C::KU * 512);
#pragma unroll
        for (int it = 0; it < C::XPT; ++it)
            xreg[it] = *reinterpret_cast<const uint4 *>(xsrc[it] + (int64_t)ks * (C::KT / 2));
    };
    auto store_stage = [&](int buf) {
        uint8_t *base = smem + buf * C::STAGE_BYTES;
#pragma unroll
        for (int it = 0; it < C::WPT; ++it) {
            const int c = it * C::NT + tid;
            uint4 *d = reinterpret_cast<uint4 *>(base + c * 32);
            d[0] = widen16(wreg[it].x, wreg[it].y);
            d[1] = widen16(wreg[it].z, wreg[it].w);
        }
#pragma unroll
        for (int it = 0; it < C::XPT; ++it) {
            uint4 *d = reinterpret_cast<uint4 *>(base + xdst[it]);
            d[0] = widen16(xreg[it].x, xreg[it].y);
            d[16] = widen16(xreg[it].z, xreg[it].w);
        }
    };

    v4i acc[C::FN][C::FM];
#pragma unroll
    for (int a = 0; a < C::FN; ++a)
#pragma unroll
        for (int b = 0; b < C::FM; ++b) acc[a][b] = v4i{0, 0, 0, 0};

    const int nks = K / C::KT;
    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int ks = 0; ks < nks; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < nks) load_stage(ks + 1);
        const uint8_t *Wl = smem + cur * C::STAGE_BYTES;
        const uint8_t *Xl = Wl + C::W_UNITS * 1024;
#pragma unroll
        for (int ku = 0; ku < C::KU; ++ku) {
            v4i a[C::FN], b[C::FM];
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
                a[fn] = *reinterpret_cast<const v4i *>(Wl + ((wn * C::FN + fn) * C::KU + ku) * 1024 + lane * 16);
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                b[fm] = *reinterpret_cast<const v4i *>(Xl + ((wm * C::FM + fm) * C::KU + ku) * 1024 + lane * 16);
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
                for (int fm = 0; fm < C::FM; ++fm)
                    acc[fn][fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[fn], b[fm], acc[fn][fm], 0, 0, 0);
        }
        if (ks + 1 < nks) store_stage(cur ^ 1);
        __syncthreads();
    }

    // epilogue: lane owns token m and channels n0 .. n0+15 of each 64-group
    const int q4 = lane >> 4;
#pragma unroll
    for (int fm = 0; fm < C::FM; ++fm) {
        const int64_t m = (int64_t)tm * C::BM + (wm * C::FM + fm) * 16 + (lane & 15);
        if (m >= M) continue;
        float xsm = 0.0f;
        if constexpr (!I32OUT) xsm = xs[m] * (1.0f / 256.0f);
#pragma unroll
        for (int G = 0; G < C::FN / 4; ++G) {
            const int64_t n0 = (int64_t)tn * C::BN + (wn * (C::FN / 4) + G) * 64 + q4 * 16;
            if (n0 >= N) continue;
            const bool full = n0 + 16 <= N;
            if constexpr (I32OUT) {
                int32_t *dst = reinterpret_cast<int32_t *>(Y) + m * ldy + n0;
                int32_t v[16];
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[4 * j + i] = acc[4 * G + j][fm][i] >> 8;
                if (full) {
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        reinterpret_cast<int4 *>(dst)[c] = make_int4(v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]);
                } else {
                    for (int e = 0; e < 16 && n0 + e < N; ++e) dst[e] = v[e];
                }
            } else {
                uint16_t *dst = reinterpret_cast<uint16_t *>(Y) + m * ldy + n0;
                uint32_t h[8];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
#pragma unroll
                    for (int i = 0; i < 4; i += 2) {
                        float y2[2];
#pragma unroll
                        for (int d = 0; d < 2; ++d) {
                            const int64_t n = min(n0 + 4 * j + i + d, (int64_t)N - 1);
                            const float bv = bias ? __half2float(__ushort_as_half(bias[n])) : 0.0f;
                            const float p = (float)acc[4 * G + j][fm][i + d] * xsm;
                            y2[d] = __builtin_fmaf(p, ws[n], bv);
                        }
                        const uint32_t lo = __half_as_ushort(__float2half_rn(y2[0]));
                        const uint32_t hi = __half_as_ushort(__float2half_rn(y2[1]));
                        h[2 * j + i / 2] = lo | (hi << 16);
                    }
                }
                if (full) {
                    reinterpret_cast<uint4 *>(dst)[0] = make_uint4(h[0], h[1], h[2], h[3]);
                    reinterpret_cast<uint4 *>(dst)[1] = make_uint4(h[4], h[5], h[6], h[7]);
                } else {
                    for (int e = 0; e < 16 && n0 + e < N; ++e)
                        dst[e] = (uint16_t)(h[e >> 1] >> (16 * (e & 1)));
                }
            }
        }
    }
}

template <class C, bool I32OUT>
hipError_t launch_cfg(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                      const uint16_t *bias, int64_t M, int64_t N, int K, void *Y,
                      int64_t ldy, hipStream_t stream) {
    static bool attr_set = false;
    const size_t lds = 2 * (size_t)C::STAGE_BYTES;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)w4a4_gemm_kernel<C, I32OUT>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int tiles_m = (int)((M + C::BM - 1) / C::BM);
    const int tiles_n = (int)((N + C::BN - 1) / C::BN);
    const int64_t grid = (int64_t)tiles_m * tiles_n;
    hipLaunchKernelGGL((w4a4_gemm_kernel<C, I32OUT>), dim3((unsigned)grid), dim3(C::NT), lds,
                       stream, Xq, xs, Wq, ws, bias, (int)M, (int)N, K, Y, ldy, tiles_m, tiles_n);
    return hipGetLastError();
}

using T128x128k128 = Tile<2, 2, 4, 4, 128>;
using T128x128k64 = Tile<2, 2, 4, 4, 64>;

}  // namespace

hipError_t launch_gemm(const uint8_t *Xq, const float *xs, const uint8_t *Wq,
                       const float *ws, const uint16_t *bias, int64_t M, int64_t N,
                       int K, void *Y, int64_t ldy, bool i32out, hipStream_t stream) {
    if (K % 128 == 0) {
        return i32out ? launch_cfg<T128x128k128, true>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream)
                      : launch_cfg<T128x128k128, false>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream);
    }
    return i32out ? launch_cfg<T128x128k64, true>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream)
                  : launch_cfg<T128x128k64, false>(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, stream);
}

}  // namespace clq
