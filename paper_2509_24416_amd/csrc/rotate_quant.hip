// Fused online rotation + per-row int4 quantization (gfx950).
//
// Paper (CLQ, arXiv 2509.24416): Sec. 3.3 applies G = S.H to the activations
// at inference time with a fast Hadamard transform (S a column swap given as a
// gather vector, H block-diagonal with +-1 entries) and absorbs the same G
// into the weights offline; Sec. 3.1 Eq. (1) quantizes with Round(Clip(.)),
// n = 4, dynamically per token for activations and once per output channel
// for weights.
//
// Weights (offline) use a one-shot kernel; activations use a persistent,
// software-pipelined variant of the same per-block arithmetic (below).
//
// One workgroup handles R whole rows.  The rows are first copied into LDS
// with coalesced 16-byte loads (each 16-byte chunk of a Hadamard block lands
// in an XOR-swizzled slot so that the later per-lane block reads hit distinct
// banks).  Each lane then owns one Hadamard block of b elements in registers
// and runs every butterfly stage there in fp32, stage order h = 1, 2, ...,
// b/2 (the first stage is fused with the fp16 -> fp32 widening).  Block
// abs-maxima meet in an LDS max per row; every lane derives the row's scale
// and reciprocal with correctly rounded divisions, then quantizes with one
// fma per element:
//     fma(x, r, 1.5 * 2^23 + 8)
// rounds the exact product x * r to the nearest integer, ties to even (the
// sum lands in the binade where the float spacing is 1), and leaves q + 8 in
// the low nibble of the result's bit pattern with bits 4..21 clear, which
// makes packing a few shifts and one byte permute.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "clq_internal.h"
#include "rq_device.h"
#include "f6_codes.h"

namespace clq {
namespace {

// Activation kernel lane order: for b >= 64 lane t owns block j = t / R of
// row r = t % R (rows fastest), so that the code stores of consecutive lanes
// land side by side in the tiled code layout; the eight lanes reading chunk
// i together then differ in j * R + r, which picks the XOR key.  For b = 32
// lanes stay blocks-fastest with the shared slot rule.
template <int B>
constexpr bool rows_fastest() { return B >= 64; }

template <int B>
__device__ __forceinline__ int act_slot(int i, int j, int r, int R) {
    if constexpr (rows_fastest<B>()) return i ^ ((j * R + r) & 7);
    else return chunk_slot<B>(i, j);
}

// Sixteen quantized words (code + 128 in bits 0..7, bits 8..21 clear) into
// one 16-byte int8 operand piece: codes 0, 2, ..., 14 in bytes 0..7, codes 1,
// 3, ..., 15 in bytes 8..15 (the order of the widened 4-bit operands), two's
// complement.
__device__ __forceinline__ uint4 pack16_q8(const uint32_t *w) {
    auto four = [](uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
        const uint32_t ab = __builtin_amdgcn_perm(b, a, 0x0c0c0400u);
        const uint32_t cd = __builtin_amdgcn_perm(d, c, 0x0c0c0400u);
        return __builtin_amdgcn_perm(cd, ab, 0x05040100u) ^ 0x80808080u;
    };
    return make_uint4(four(w[0], w[2], w[4], w[6]), four(w[8], w[10], w[12], w[14]),
                      four(w[1], w[3], w[5], w[7]), four(w[9], w[11], w[13], w[15]));
}

// The int8 codes of one lane's b-element block (codes 32c .. of the row's
// 32-code chunks j * b/32 + c): two 16-byte operand pieces per chunk.
template <int B, bool WEIGHT>
__device__ __forceinline__ void store_q8(const float *x, float rc, int64_t grow, int j, int K,
                                         uint8_t *__restrict__ out) {
    constexpr float M = Grid<8>::magic, Q = Grid<8>::qmax;
    const int64_t u = grow >> 5;
    const int rho = WEIGHT ? wq_rho((int)(grow & 31)) : (int)(grow & 31);
#pragma unroll
    for (int c = 0; c < B / 32; ++c) {
        const int64_t c32 = (int64_t)j * (B / 32) + c;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            uint32_t w[16];
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                float v = __builtin_fmaf(x[32 * c + 16 * q + t], rc, M);
                if constexpr (WEIGHT) v = __builtin_amdgcn_fmed3f(v, M - Q, M + Q);
                w[t] = __float_as_uint(v);
            }
            *reinterpret_cast<uint4 *>(out + q8_piece_offset(u, rho, c32, q, K)) = pack16_q8(w);
        }
    }
}

// Lanes per workgroup never exceed 512 for b >= 64 (at most 512 blocks per
// row, and rows are only batched up to 512 lanes), which lets the compiler
// keep a 128-element block in registers.
template <int B>
constexpr int rq_max_threads() { return B == 32 ? 1024 : 512; }

template <int B, bool WEIGHT, int QB>
__global__ void __launch_bounds__(rq_max_threads<B>())
rotate_quant_kernel(const uint16_t *__restrict__ X, int64_t ldx,
                    const int32_t *__restrict__ perm, int64_t rows_valid,
                    int64_t rows_alloc, int K, int R, float alpha, const float *__restrict__ alpha_dev,
                    float post_scale, uint8_t *__restrict__ out, float *__restrict__ scale_out,
                    int64_t out_stride, int64_t scale_stride)
{
    extern __shared__ __align__(16) unsigned char smem[];
    // blockIdx.y selects one of several quantizations of the same rows
    // (clip ratio alpha_dev[y], outputs at y * stride)
    out += (int64_t)blockIdx.y * out_stride;
    scale_out += (int64_t)blockIdx.y * scale_stride;
    if (alpha_dev != nullptr) alpha_dev += blockIdx.y;
    constexpr int CPB = B / 8;            // 16-byte chunks per block
    const int cpr = K >> 3;               // chunks per row
    const int nb = K / B;                 // blocks per row
    uint4 *tile = reinterpret_cast<uint4 *>(smem);
    unsigned *rowmax = reinterpret_cast<unsigned *>(smem + (size_t)R * K * 2);

    const int t = threadIdx.x;
    const int T = blockDim.x;
    const int64_t row0 = (int64_t)blockIdx.x * R;
    const int rows = (int)min((int64_t)R, rows_alloc - row0);

    if (t < R) rowmax[t] = 0u;

    // 1. coalesced copy of the rows into LDS (rows past rows_valid are zeros)
    {
        int r = t / cpr, cc = t - r * cpr;
        const int dr = T / cpr, dc = T - dr * cpr;
        while (r < rows) {
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            const int64_t grow = row0 + r;
            if (grow < rows_valid)
                v = *reinterpret_cast<const uint4 *>(X + grow * ldx + (int64_t)cc * 8);
            const int j = cc / CPB, i = cc % CPB;
            tile[r * cpr + j * CPB + chunk_slot<B>(i, j)] = v;
            cc += dc;
            r += dr;
            if (cc >= cpr) { cc -= cpr; ++r; }
        }
    }
    __syncthreads();

    // 2. one Hadamard block per lane
    const int r = t / nb, j = t - r * nb;
    const bool active = r < rows;
    float x[B];
    float bmax = 0.0f;
    if (active) {
        if (perm == nullptr) {
            const uint4 *src = tile + r * cpr + j * CPB;
#pragma unroll
            for (int i = 0; i < CPB; ++i) {
                const uint4 v = src[chunk_slot<B>(i, j)];
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    stage1_packed(w[e], x[8 * i + 2 * e], x[8 * i + 2 * e + 1]);   // stage h = 1
                }
            }
        } else {
            const uint16_t *rowh = reinterpret_cast<const uint16_t *>(tile + r * cpr);
            const int32_t *p = perm + j * B;
#pragma unroll
            for (int e = 0; e < B; e += 2) {
                const int k0 = p[e], k1 = p[e + 1];
                const int c0 = k0 >> 3, c1 = k1 >> 3;
                const int s0 = (c0 / CPB) * CPB + chunk_slot<B>(c0 % CPB, c0 / CPB);
                const int s1 = (c1 / CPB) * CPB + chunk_slot<B>(c1 % CPB, c1 / CPB);
                stage1_pair(rowh[s0 * 8 + (k0 & 7)], rowh[s1 * 8 + (k1 & 7)], x[e], x[e + 1]);
            }
        }
#pragma unroll
        for (int h = 2; h < B; h <<= 1) {
#pragma unroll
            for (int i = 0; i < B; ++i) {
                if ((i & h) == 0) {
                    const float u = x[i], v = x[i + h];
                    x[i] = u + v;
                    x[i + h] = u - v;
                }
            }
        }
        bmax = block_absmax<B>(x);
        atomicMax(&rowmax[r], __float_as_uint(bmax));
    }
    __syncthreads();
    if (!active) return;

    // 3. per-row scale and codes
    const float a = __uint_as_float(rowmax[r]);
    // the clip ratio: a launch argument, or read from device memory (a
    // search that picks it on the GPU)
    const float al = alpha_dev != nullptr ? *alpha_dev : alpha;
    const float ac = WEIGHT ? al * a : a;
    const float rc = (ac == 0.0f) ? 0.0f : Grid<QB>::qmax / ac;
    const int64_t grow = row0 + r;
    if (j == 0 && grow < rows_valid) scale_out[grow] = (ac / Grid<QB>::qmax) * post_scale;
    if constexpr (QB == 8) {
        store_q8<B, WEIGHT>(x, rc, grow, j, K, out);
        return;
    }

    if constexpr (QB == 6) {
        // fp6 layout: the codes as exact floats, six dwords per 32 codes
        const int rho = WEIGHT ? wq_rho((int)(grow & 31)) : (int)(grow & 31);
#pragma unroll
        for (int i = 0; i < B; ++i) {
            float v = __builtin_fmaf(x[i], rc, kMagic);
            if constexpr (WEIGHT) v = __builtin_amdgcn_fmed3f(v, kMagic - 7.0f, kMagic + 7.0f);
            x[i] = v - kMagic;
        }
#pragma unroll
        for (int c = 0; c < B / 32; ++c) {
            const int64_t c32 = (int64_t)j * (B / 32) + c;
            uint32_t w6[6];
            f6_from_codes(&x[32 * c], w6);
            f6_store(out + f6_unit_offset(grow >> 5, c32, K), f6_lane(c32, rho), w6);
        }
        return;
    }
    uint32_t words[B / 8];
#pragma unroll
    for (int g = 0; g < B / 8; ++g) {
        uint32_t w[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float v = __builtin_fmaf(x[8 * g + e], rc, kMagic);
            if constexpr (WEIGHT) v = __builtin_amdgcn_fmed3f(v, kMagic - 7.0f, kMagic + 7.0f);
            w[e] = __float_as_uint(v);
        }
        words[g] = pack8(w);
    }

    if constexpr (!WEIGHT) {
        // packed activation layout: one 16-byte chunk per 32 codes
#pragma unroll
        for (int c = 0; c < B / 32; ++c) {
            const int64_t c32 = (int64_t)j * (B / 32) + c;
            *reinterpret_cast<uint4 *>(out + xq_chunk_offset(grow, c32, K)) =
                make_uint4(words[4 * c], words[4 * c + 1], words[4 * c + 2], words[4 * c + 3]);
        }
    } else {
        // packed weight layout: one 8-byte piece per k-group of 16 codes
#pragma unroll
        for (int g = 0; g < B / 16; ++g) {
            const int64_t kg = (int64_t)j * (B / 16) + g;
            uint2 *dst = reinterpret_cast<uint2 *>(out + wq_piece_offset(grow, kg, K));
            *dst = make_uint2(words[2 * g], words[2 * g + 1]);
        }
    }
}

// Activation path: persistent, software-pipelined over batches of R rows.
// Batch i's rows are converted and transformed from one LDS buffer while
// batch i+1 (already in registers) is written to the other buffer and batch
// i+2's loads are in flight, so HBM never waits for the arithmetic.  One
// barrier per batch: before it, block maxima meet in rowmax[i % 3]; after it,
// codes are formed and stored.  The third rowmax buffer is cleared one batch
// after its use, when no lane can still be reading it.
// GATHER: perm is set (a separate instance, so that the loads of the
// permutation leave no pending-load state in the ungathered loop)
template <int B, int QB, bool GATHER>
__global__ void __launch_bounds__(256)
rq_act_kernel(const uint16_t *__restrict__ X, int64_t ldx, const int32_t *__restrict__ perm,
              int64_t rows_valid, int64_t rows_alloc, int64_t nbatch, int K, int R,
              uint8_t *__restrict__ out, float *__restrict__ scale_out)
{
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int CPB = B / 8;
    constexpr int LPT = CPB;   // chunks each lane loads per batch (T >= R * nb lanes)
    const int cpr = K >> 3;
    const int nb = K / B;
    const int chunks = R * cpr;
    uint4 *tile0 = reinterpret_cast<uint4 *>(smem);
    uint4 *tile1 = tile0 + chunks;
    unsigned *rowmax = reinterpret_cast<unsigned *>(tile1 + chunks);   // [3][R]

    const int t = threadIdx.x, T = blockDim.x;
    const int64_t G = gridDim.x;

    // this lane's load chunks (the same for every batch): row, source
    // offset within the batch, swizzled LDS slot
    int lrow[LPT], lsrc[LPT], lslot[LPT];
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
        const int c = t + k * T;
        const int r = c / cpr, cc = c - r * cpr;
        lrow[k] = c < chunks ? r : -1;
        lsrc[k] = r * (int)ldx + cc * 8;
        const int jj = cc / CPB, ii = cc - jj * CPB;
        lslot[k] = r * cpr + jj * CPB + act_slot<B>(ii, jj, r, R);
    }
    uint4 ld[LPT];
    auto load = [&](int64_t batch) {
        const int64_t row0 = batch * R;
        const uint16_t *base = X + row0 * ldx;
#pragma unroll
        for (int k = 0; k < LPT; ++k) {
            ld[k] = make_uint4(0u, 0u, 0u, 0u);
            if (lrow[k] >= 0 && row0 + lrow[k] < rows_valid)
                ld[k] = *reinterpret_cast<const uint4 *>(base + lsrc[k]);
        }
    };
    auto stash = [&](uint4 *tile) {
#pragma unroll
        for (int k = 0; k < LPT; ++k)
            if (lrow[k] >= 0) tile[lslot[k]] = ld[k];
    };

    int r, j;
    if constexpr (rows_fastest<B>()) {
        j = t / R;
        r = t - j * R;
    } else {
        r = t / nb;
        j = t - r * nb;
    }
    const bool active = rows_fastest<B>() ? j < nb : r < R;
    int64_t b = blockIdx.x;
    if (b >= nbatch) return;
    for (int q = t; q < 3 * R; q += T) rowmax[q] = 0u;
    load(b);
    stash(tile0);
    if (b + G < nbatch) load(b + G);
    __syncthreads();

    for (int i = 0; b < nbatch; ++i, b += G) {
        const uint4 *tcur = (i & 1) ? tile1 : tile0;
        uint4 *tnxt = (i & 1) ? tile0 : tile1;
        unsigned *rm = rowmax + (i % 3) * R;

        // 1. one Hadamard block per lane, fp32, stage order h = 1, 2, ..., b/2
        float x[B];
        if (active) {
            float bmax = 0.0f;
            if constexpr (!GATHER) {
                const uint4 *src = tcur + r * cpr + j * CPB;
#pragma unroll
                for (int ii = 0; ii < CPB; ++ii) {
                    const uint4 v = src[act_slot<B>(ii, j, r, R)];
                    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        stage1_packed(w[e], x[8 * ii + 2 * e], x[8 * ii + 2 * e + 1]);   // stage h = 1
                    }
                }
            } else {
                const uint16_t *rowh = reinterpret_cast<const uint16_t *>(tcur + r * cpr);
                const int32_t *p = perm + j * B;
#pragma unroll
                for (int e = 0; e < B; e += 2) {
                    const int k0 = p[e], k1 = p[e + 1];
                    const int c0 = k0 >> 3, c1 = k1 >> 3;
                    const int s0 = (c0 / CPB) * CPB + act_slot<B>(c0 % CPB, c0 / CPB, r, R);
                    const int s1 = (c1 / CPB) * CPB + act_slot<B>(c1 % CPB, c1 / CPB, r, R);
                    stage1_pair(rowh[s0 * 8 + (k0 & 7)], rowh[s1 * 8 + (k1 & 7)], x[e], x[e + 1]);
                }
            }
#pragma unroll
            for (int h = 2; h < B; h <<= 1) {
#pragma unroll
                for (int ii = 0; ii < B; ++ii) {
                    if ((ii & h) == 0) {
                        const float u = x[ii], v = x[ii + h];
                        x[ii] = u + v;
                        x[ii + h] = u - v;
                    }
                }
            }
            bmax = block_absmax<B>(x);
            atomicMax(&rm[r], __float_as_uint(bmax));
        }
        // 2. the next batch into the other buffer, the one after into registers
        if (b + G < nbatch) stash(tnxt);
        if (b + 2 * G < nbatch) load(b + 2 * G);
        __syncthreads();
        // 3. codes of this batch; the rowmax buffer of the previous batch is free
        if (t < R) rowmax[((i + 2) % 3) * R + t] = 0u;
        if (!active) continue;
        const float a = __uint_as_float(rm[r]);
        const float rc = (a == 0.0f) ? 0.0f : Grid<QB>::qmax / a;
        const int64_t grow = b * R + r;
        if (grow >= rows_alloc) continue;   // past the padded rows
        if (j == 0 && grow < rows_valid) scale_out[grow] = a / Grid<QB>::qmax;
        if constexpr (QB == 8) {
            store_q8<B, false>(x, rc, grow, j, K, out);
            continue;
        }
        if constexpr (QB == 6) {
            // the codes as exact floats, in place (x is dead after this)
#pragma unroll
            for (int e = 0; e < B; ++e) x[e] = __builtin_fmaf(x[e], rc, kMagic) - kMagic;
#pragma unroll
            for (int c = 0; c < B / 32; ++c) {
                const int64_t c32 = (int64_t)j * (B / 32) + c;
                uint32_t w6[6];
                f6_from_codes(&x[32 * c], w6);
                f6_store(out + f6_unit_offset(grow >> 5, c32, K), f6_lane(c32, (int)(grow & 31)), w6);
            }
            continue;
        }
        uint32_t words[B / 8];
#pragma unroll
        for (int g = 0; g < B / 8; ++g) {
            uint32_t w[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = __float_as_uint(__builtin_fmaf(x[8 * g + e], rc, kMagic));
            words[g] = pack8(w);
        }
#pragma unroll
        for (int c = 0; c < B / 32; ++c) {
            const int64_t c32 = (int64_t)j * (B / 32) + c;
            *reinterpret_cast<uint4 *>(out + xq_chunk_offset(grow, c32, K)) =
                make_uint4(words[4 * c], words[4 * c + 1], words[4 * c + 2], words[4 * c + 3]);
        }
    }
}

// Activations with long rows (K >= 2048): batches of exactly 8 token rows,
// aligned to 8, so that with the rows-fastest lane order every 128-byte line
// of the code layout (8 rows x 16 bytes, or 8 rows x 16 bytes of an int8
// operand piece) is written whole by one store instruction -- partial lines
// written by several batches cost long-row launches about 40% at full HBM
// rate.  One workgroup per CU with one LDS buffer of 8 rows; the next batch
// waits in registers.  Two barriers per batch: after the block reads (the
// buffer may be refilled, and the previous maxima have been read) and after
// the block maxima (codes may be formed).  Codes of batch i are formed at the
// top of iteration i+1, from the registers that still hold its rotated
// blocks.  The buffer is refilled after the butterflies: the wait for the
// next batch's loads then also finds the previous codes' stores complete,
// instead of stalling on them right after they were issued.
// at most 8 x 80 lanes (b = 64, K <= 5120)
template <int B>
constexpr int rows8_threads() { return 640; }

template <int B, int QB, bool GATHER>
__global__ void __launch_bounds__(rows8_threads<B>())
rq_rows8_kernel(const uint16_t *__restrict__ X, int64_t ldx, const int32_t *__restrict__ perm,
                int64_t rows_valid, int64_t rows_alloc, int64_t nbatch, int K,
                uint8_t *__restrict__ out, float *__restrict__ scale_out)
{
    constexpr int R = 8;
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int CPB = B / 8;
    constexpr int LPT = CPB;
    const int cpr = K >> 3;
    const int nb = K / B;
    const int chunks = R * cpr;
    uint4 *tile = reinterpret_cast<uint4 *>(smem);
    unsigned *rowmax = reinterpret_cast<unsigned *>(tile + chunks);   // [2][R]

    const int t = threadIdx.x, T = blockDim.x;
    const int64_t G = gridDim.x;

    // this lane's chunks: source offset, and LDS slot | row << 16 | valid << 19
    // in one register (slots < 8 * 640)
    int lsrc[LPT], lmeta[LPT];
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
        const int c = t + k * T;
        const int r = c / cpr, cc = c - r * cpr;
        lsrc[k] = r * (int)ldx + cc * 8;
        const int jj = cc / CPB, ii = cc - jj * CPB;
        const int slot = r * cpr + jj * CPB + (ii ^ r);   // key (jj * 8 + r) & 7 = r
        lmeta[k] = c < chunks ? slot | (r << 16) | (1 << 19) : 0;
    }
    uint4 ld[LPT];
    auto load = [&](int64_t batch) {
        const int64_t row0 = batch * R;
        const uint16_t *base = X + row0 * ldx;
#pragma unroll
        for (int k = 0; k < LPT; ++k) {
            ld[k] = make_uint4(0u, 0u, 0u, 0u);
            if ((lmeta[k] >> 19) && row0 + ((lmeta[k] >> 16) & 7) < rows_valid)
                ld[k] = *reinterpret_cast<const uint4 *>(base + lsrc[k]);
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int k = 0; k < LPT; ++k)
            if (lmeta[k] >> 19) tile[lmeta[k] & 0xFFFF] = ld[k];
    };

    const int j = t >> 3, r = t & 7;   // rows fastest
    const bool active = j < nb;
    int64_t b = blockIdx.x;
    if (b >= nbatch) return;
    if (t < 2 * R) rowmax[t] = 0u;
    load(b);
    stash();
    if (b + G < nbatch) load(b + G);
    __syncthreads();

    float x[B];
#pragma unroll
    for (int e = 0; e < B; ++e) x[e] = 0.0f;
    int64_t prev = -1;   // batch whose rotated blocks x holds, codes pending
    int i = 0;
    auto codes = [&](int64_t pb, int pi) {
        const float a = __uint_as_float(rowmax[(pi & 1) * R + r]);
        const float rc = (a == 0.0f) ? 0.0f : Grid<QB>::qmax / a;
        const int64_t grow = pb * R + r;
        if (!active || grow >= rows_alloc) return;
        if (j == 0 && grow < rows_valid) scale_out[grow] = a / Grid<QB>::qmax;
        if constexpr (QB == 8) {
            store_q8<B, false>(x, rc, grow, j, K, out);
        } else {
            if constexpr (QB == 6) {
                // the codes as exact floats, in place (x is reloaded after this)
#pragma unroll
                for (int e = 0; e < B; ++e) x[e] = __builtin_fmaf(x[e], rc, kMagic) - kMagic;
#pragma unroll
                for (int c = 0; c < B / 32; ++c) {
                    const int64_t c32 = (int64_t)j * (B / 32) + c;
                    uint32_t w6[6];
                    f6_from_codes(&x[32 * c], w6);
                    f6_store(out + f6_unit_offset(grow >> 5, c32, K), f6_lane(c32, (int)(grow & 31)), w6);
                }
                return;
            }
            uint32_t words[B / 8];
#pragma unroll
            for (int g = 0; g < B / 8; ++g) {
                uint32_t w[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) w[e] = __float_as_uint(__builtin_fmaf(x[8 * g + e], rc, kMagic));
                words[g] = pack8(w);
            }
#pragma unroll
            for (int c = 0; c < B / 32; ++c) {
                const int64_t c32 = (int64_t)j * (B / 32) + c;
                *reinterpret_cast<uint4 *>(out + xq_chunk_offset(grow, c32, K)) =
                    make_uint4(words[4 * c], words[4 * c + 1], words[4 * c + 2], words[4 * c + 3]);
            }
        }
    };

    for (; b < nbatch; ++i, b += G) {
        // codes of the previous batch (its maxima are complete), then this
        // batch's blocks into registers
        if (prev >= 0) codes(prev, i - 1);
        if (active) {
            if constexpr (!GATHER) {
                const uint4 *src = tile + r * cpr + j * CPB;
#pragma unroll
                for (int ii = 0; ii < CPB; ++ii) {
                    const uint4 v = src[ii ^ r];
                    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        stage1_packed(w[e], x[8 * ii + 2 * e], x[8 * ii + 2 * e + 1]);   // stage h = 1
                    }
                }
            } else {
                const uint16_t *rowh = reinterpret_cast<const uint16_t *>(tile + r * cpr);
                const int32_t *p = perm + j * B;
#pragma unroll
                for (int e = 0; e < B; e += 2) {
                    const int k0 = p[e], k1 = p[e + 1];
                    const int c0 = k0 >> 3, c1 = k1 >> 3;
                    const int s0 = (c0 / CPB) * CPB + ((c0 % CPB) ^ r);
                    const int s1 = (c1 / CPB) * CPB + ((c1 % CPB) ^ r);
                    stage1_pair(rowh[s0 * 8 + (k0 & 7)], rowh[s1 * 8 + (k1 & 7)], x[e], x[e + 1]);
                }
            }
        }
        __syncthreads();   // every block read and every read of the previous maxima done
        if (t < R) rowmax[((i + 1) & 1) * R + t] = 0u;   // batch i+1's buffer, read last by codes(i-1)
        if (active) {
#pragma unroll
            for (int h = 2; h < B; h <<= 1) {
#pragma unroll
                for (int ii = 0; ii < B; ++ii) {
                    if ((ii & h) == 0) {
                        const float u = x[ii], v = x[ii + h];
                        x[ii] = u + v;
                        x[ii + h] = u - v;
                    }
                }
            }
            atomicMax(&rowmax[(i & 1) * R + r], __float_as_uint(block_absmax<B>(x)));
        }
        if (b + G < nbatch) stash();
        if (b + 2 * G < nbatch) load(b + 2 * G);
        __syncthreads();   // maxima complete, next batch staged
        prev = b;
    }
    if (prev >= 0) codes(prev, i - 1);
}

// Long rows (b = 64, 2048 <= K <= 5120: one buffer of 8 rows within 80 KB,
// at most 640 lanes) take the 8-row kernel.
template <int B>
bool use_rows8(int K) {
    return B == 64 && K >= 2048 && K <= 5120;
}

// Rows per workgroup: the largest lane utilisation R*nb / roundup(R*nb, 64)
// with at most 512 lanes (unless one row alone needs more) and at most 64 KB
// of staged fp16 rows.
int pick_rows(int K, int block) {
    const int nb = K / block;
    int best = 1;
    double best_u = -1.0;
    for (int R = 1; R * nb <= 1024; ++R) {
        if (R > 1 && (R * nb > 512 || (size_t)R * K * 2 > 65536)) break;
        const int T = (R * nb + 63) / 64 * 64;
        const double u = (double)(R * nb) / T;
        if (u > best_u + 1e-9) { best_u = u; best = R; }
    }
    return best;
}

template <int B, bool WEIGHT, int QB>
hipError_t launch_rq(const uint16_t *X, int64_t ldx, const int32_t *perm,
                     int64_t rows_valid, int64_t rows_alloc, int K, float alpha,
                     float post_scale, uint8_t *out, float *scale, hipStream_t stream,
                     const float *alpha_dev = nullptr, int batch = 1, int64_t out_stride = 0,
                     int64_t scale_stride = 0) {
    const int R = pick_rows(K, B);
    const int nb = K / B;
    const int T = (R * nb + 63) / 64 * 64;
    if (T > rq_max_threads<B>()) return hipErrorInvalidConfiguration;
    const size_t lds = (size_t)R * K * 2 + (size_t)R * 4;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)rotate_quant_kernel<B, WEIGHT, QB>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 65536 + 4096);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int64_t grid = (rows_alloc + R - 1) / R;
    hipLaunchKernelGGL((rotate_quant_kernel<B, WEIGHT, QB>), dim3((unsigned)grid, (unsigned)batch), dim3(T), lds,
                       stream, X, ldx, perm, rows_valid, rows_alloc, K, R, alpha, alpha_dev, post_scale,
                       out, scale, out_stride, scale_stride);
    return hipGetLastError();
}

// Activation batches: the largest lane utilisation R*nb / roundup(R*nb, 64)
// with at most 256 lanes and two staged batches within 64 KB of LDS.
int pick_act_rows(int K, int block) {
    const int nb = K / block;
    int best = 1;
    double best_u = -1.0;
    for (int R = 1; R * nb <= 256; ++R) {
        if ((size_t)2 * R * K * 2 > 65536) break;
        const int T = (R * nb + 63) / 64 * 64;
        const double u = (double)(R * nb) / T;
        if (u > best_u + 1e-9) { best_u = u; best = R; }
    }
    return best;
}

template <int B, int QB, bool GATHER>
hipError_t launch_rq_act_g(const uint16_t *X, int64_t ldx, const int32_t *perm, int64_t rows_valid,
                           int64_t rows_alloc, int K, uint8_t *out, float *scale, hipStream_t stream) {
    const int R = pick_act_rows(K, B);
    const int nb = K / B;
    const int T = (R * nb + 63) / 64 * 64;
    const size_t lds = (size_t)2 * R * K * 2 + (size_t)3 * R * 4;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)rq_act_kernel<B, QB, GATHER>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, 65536 + 4096);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
    }
    // The one-shot kernel (up to 1024 lanes and 64 KB of staged row) takes
    // what this kernel's launch cannot: very wide strides (32-bit in-batch
    // offsets), rows of more than 256 blocks (b = 32, K > 8192) and rows
    // whose two staged copies exceed the LDS limit (K > 16384).
    if ((int64_t)R * ldx > INT32_MAX || R * nb > 256 || lds > 65536 + 4096)
        return launch_rq<B, false, QB>(X, ldx, perm, rows_valid, rows_alloc, K, 1.0f, 1.0f, out, scale, stream);
    if constexpr (B == 64) if (use_rows8<B>(K) && (int64_t)8 * ldx <= INT32_MAX) {
        static bool attr8 = false;
        if (!attr8) {
            hipError_t e = hipFuncSetAttribute((const void *)rq_rows8_kernel<B, QB, GATHER>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, 80 * 1024 + 64);
            if (e != hipSuccess) return e;
            attr8 = true;
        }
        const int T8 = (8 * (K / B) + 63) / 64 * 64;
        const size_t lds8 = (size_t)8 * K * 2 + 2 * 8 * 4;
        const int64_t nb8 = (rows_alloc + 7) / 8;
        const int64_t grid8 = std::min<int64_t>(nb8, (int64_t)cus);
        hipLaunchKernelGGL((rq_rows8_kernel<B, QB, GATHER>), dim3((unsigned)grid8), dim3(T8), lds8, stream, X, ldx, perm,
                           rows_valid, rows_alloc, nb8, K, out, scale);
        return hipGetLastError();
    }
    const int64_t nbatch = (rows_alloc + R - 1) / R;
    const int per_cu = (int)std::min<size_t>(4, (160 * 1024) / lds);
    const int64_t grid = std::min<int64_t>(nbatch, (int64_t)cus * per_cu);
    hipLaunchKernelGGL((rq_act_kernel<B, QB, GATHER>), dim3((unsigned)grid), dim3(T), lds, stream, X, ldx, perm,
                       rows_valid, rows_alloc, nbatch, K, R, out, scale);
    return hipGetLastError();
}

template <int B, int QB>
hipError_t launch_rq_act(const uint16_t *X, int64_t ldx, const int32_t *perm, int64_t rows_valid,
                         int64_t rows_alloc, int K, uint8_t *out, float *scale, hipStream_t stream) {
    if (perm != nullptr) return launch_rq_act_g<B, QB, true>(X, ldx, perm, rows_valid, rows_alloc, K, out, scale, stream);
    return launch_rq_act_g<B, QB, false>(X, ldx, perm, rows_valid, rows_alloc, K, out, scale, stream);
}

__global__ void unswizzle_kernel(const uint8_t *__restrict__ Wq, int64_t N, int K,
                                 uint8_t *__restrict__ out) {
    const int64_t kgs = K / 16;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= N * kgs) return;
    const int64_t n = idx / kgs, kg = idx - n * kgs;
    const uint2 v = *reinterpret_cast<const uint2 *>(Wq + wq_piece_offset(n, kg, K));
    *reinterpret_cast<uint2 *>(out + n * (K / 2) + kg * 8) = v;
}

__global__ void unswizzle_act_kernel(const uint8_t *__restrict__ Xq, int64_t M, int K,
                                     uint8_t *__restrict__ out) {
    const int64_t cpr = K / 32;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= M * cpr) return;
    const int64_t r = idx / cpr, c = idx - r * cpr;
    const uint4 v = *reinterpret_cast<const uint4 *>(Xq + xq_chunk_offset(r, c, K));
    *reinterpret_cast<uint4 *>(out + r * (K / 2) + c * 16) = v;
}

// one 16-byte operand piece per thread, scattered back to canonical codes
__global__ void unswizzle8_kernel(const uint8_t *__restrict__ q8, int64_t rows, int K, bool weights,
                                  int8_t *__restrict__ out) {
    const int64_t cpr = K / 32;   // 32-code chunks per row
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= rows * cpr * 2) return;
    const int q = (int)(idx & 1);
    const int64_t rc = idx >> 1, r = rc / cpr, c = rc - r * cpr;
    const int rho = weights ? wq_rho((int)(r & 31)) : (int)(r & 31);
    const uint4 v = *reinterpret_cast<const uint4 *>(q8 + q8_piece_offset(r >> 5, rho, c, q, K));
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    int8_t *dst = out + r * K + c * 32 + q * 16;
#pragma unroll
    for (int t = 0; t < 16; ++t) {
        const int byte = (t & 1) * 8 + (t >> 1);
        dst[t] = (int8_t)(w[byte >> 2] >> (8 * (byte & 3)));
    }
}

}  // namespace

hipError_t launch_unswizzle8(const uint8_t *q8, int64_t rows, int K, bool weights, int8_t *out,
                             hipStream_t stream) {
    const int64_t total = rows * (K / 32) * 2;
    hipLaunchKernelGGL(unswizzle8_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                       q8, rows, K, weights, out);
    return hipGetLastError();
}

template <int QB>
hipError_t launch_rq_bits(const uint16_t *X, int64_t ldx, const int32_t *perm,
                          int64_t rows, int64_t rows_alloc, int K, int block,
                          float alpha, bool weight_mode, float post_scale,
                          uint8_t *out, float *scale, hipStream_t stream, const float *alpha_dev, int batch,
                          int64_t out_stride, int64_t scale_stride) {
    if (weight_mode) {
        switch (block) {
            case 32: return launch_rq<32, true, QB>(X, ldx, perm, rows, rows_alloc, K, alpha, post_scale, out, scale, stream, alpha_dev, batch, out_stride, scale_stride);
            case 64: return launch_rq<64, true, QB>(X, ldx, perm, rows, rows_alloc, K, alpha, post_scale, out, scale, stream, alpha_dev, batch, out_stride, scale_stride);
            case 128: return launch_rq<128, true, QB>(X, ldx, perm, rows, rows_alloc, K, alpha, post_scale, out, scale, stream, alpha_dev, batch, out_stride, scale_stride);
        }
    } else {
        switch (block) {
            case 32: return launch_rq_act<32, QB>(X, ldx, perm, rows, rows_alloc, K, out, scale, stream);
            case 64: return launch_rq_act<64, QB>(X, ldx, perm, rows, rows_alloc, K, out, scale, stream);
            case 128: return launch_rq_act<128, QB>(X, ldx, perm, rows, rows_alloc, K, out, scale, stream);
        }
    }
    return hipErrorInvalidValue;
}

hipError_t launch_rotate_quant(const uint16_t *X, int64_t ldx, const int32_t *perm,
                               int64_t rows, int64_t rows_alloc, int K, int block,
                               float alpha, bool weight_mode, float post_scale,
                               uint8_t *out, float *scale, hipStream_t stream, int bits,
                               const float *alpha_dev, int batch, int64_t out_stride, int64_t scale_stride) {
    if (batch > 1 && (!weight_mode || alpha_dev == nullptr)) return hipErrorInvalidValue;
    if (bits == 8)
        return launch_rq_bits<8>(X, ldx, perm, rows, rows_alloc, K, block, alpha, weight_mode, post_scale,
                                 out, scale, stream, alpha_dev, batch, out_stride, scale_stride);
    if (bits == 4)
        return launch_rq_bits<4>(X, ldx, perm, rows, rows_alloc, K, block, alpha, weight_mode, post_scale,
                                 out, scale, stream, alpha_dev, batch, out_stride, scale_stride);
    if (bits == 6)
        return launch_rq_bits<6>(X, ldx, perm, rows, rows_alloc, K, block, alpha, weight_mode, post_scale,
                                 out, scale, stream, alpha_dev, batch, out_stride, scale_stride);
    return hipErrorInvalidValue;
}

namespace {

// canonical packed int4 codes [rows][K/2] of an fp6 operand (weights: the
// fragment-row order undone): one thread per 32-code chunk
__global__ void unswizzle_f6_kernel(const uint8_t *__restrict__ q6, int64_t rows, int K, bool weights,
                                    uint8_t *__restrict__ out) {
    const int64_t cpr = K / 32;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= rows * cpr) return;
    const int64_t r = idx / cpr, c32 = idx - r * cpr;
    const int rho = weights ? wq_rho((int)(r & 31)) : (int)(r & 31);
    const uint8_t *unit = q6 + f6_unit_offset(r >> 5, c32, K);
    const int l = f6_lane(c32, rho);
    const uint4 a = *reinterpret_cast<const uint4 *>(unit + l * 16);
    const uint2 b = *reinterpret_cast<const uint2 *>(unit + f6_tail_offset(l));
    const uint32_t w[6] = {a.x, a.y, a.z, a.w, b.x, b.y};
    uint32_t d[4];
    nibbles_from_f6(w, d);
    *reinterpret_cast<uint4 *>(out + r * (K / 2) + c32 * 16) = make_uint4(d[0], d[1], d[2], d[3]);
}

}  // namespace

hipError_t launch_unswizzle_f6(const uint8_t *q6, int64_t rows, int K, bool weights, uint8_t *out,
                               hipStream_t stream) {
    const int64_t total = rows * (K / 32);
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(unswizzle_f6_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, q6, rows, K,
                       weights, out);
    return hipGetLastError();
}

hipError_t launch_unswizzle(const uint8_t *Wq, int64_t N, int K, uint8_t *out,
                            hipStream_t stream) {
    const int64_t total = N * (K / 16);
    const int64_t grid = (total + 255) / 256;
    hipLaunchKernelGGL(unswizzle_kernel, dim3((unsigned)grid), dim3(256), 0, stream, Wq, N, K, out);
    return hipGetLastError();
}

hipError_t launch_unswizzle_act(const uint8_t *Xq, int64_t M, int K, uint8_t *out,
                                hipStream_t stream) {
    const int64_t total = M * (K / 32);
    const int64_t grid = (total + 255) / 256;
    hipLaunchKernelGGL(unswizzle_act_kernel, dim3((unsigned)grid), dim3(256), 0, stream, Xq, M, K, out);
    return hipGetLastError();
}

}  // namespace clq
