// fp6 (e2m3) code layout of the W4A4 operands: 4-bit codes carried in the
// format of gfx950's fp6 matrix instructions (CLQ, arXiv 2509.24416, Sec. 3.1
// Eq. (1): the integer grid -7..7 of the 4-bit quantizer).
//
// e2m3: sign bit 5, exponent bits 4..3 (bias 1), mantissa bits 2..0.  The
// integers 0..7 are 000000, 001000, 010000, 010100, 011000, 011010, 011100,
// 011110; a negative code sets bit 5.  Every code of the grid is exact.
//
// Layout: units of 32 rows x 64 codes, the unit and lane map of the packed
// int4 layouts (lane l = 32h + rho holds codes 32h .. 32h+31 of the unit's
// row rho: the token row itself for activations, the fragment-row order
// wq_rho for weights).  A lane's 32 codes take 192 bits, six dwords w0..w5,
// code i of the 32 at bits 6i .. 6i+5 of the concatenation (w0 lowest).  A
// unit is 1536 bytes: lane l's w0..w3 at 16 l, and its w4, w5 at
// 1024 + 16 rho + 8 h, so that the 16 bytes of both halves of a row sit
// together and eight consecutive rows fill whole 128-byte lines in both
// parts.  Units are stored [row unit][k unit].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace clq {

constexpr int kF6Unit = 1536;

// bytes of an fp6 operand with rows_padded rows (a multiple of 32) and K codes
__host__ __device__ inline int64_t f6_operand_bytes(int64_t rows_padded, int64_t K) {
    return rows_padded / 32 * (K / 64) * kF6Unit;
}

// byte offset of the unit holding 32-code chunk c32 of row unit u
__host__ __device__ inline int64_t f6_unit_offset(int64_t u, int64_t c32, int64_t K) {
    return (u * (K >> 6) + (c32 >> 1)) * kF6Unit;
}
// the lane of chunk c32 of unit row rho
__host__ __device__ inline int f6_lane(int64_t c32, int rho) { return 32 * (int)(c32 & 1) + rho; }

// e2m3 of four codes held one per byte as t = code + 8 (1..15): two 8-entry
// byte tables (t < 8: negative codes; t >= 8: 0..7) and a byte select on
// bit 3 of t
__device__ __forceinline__ uint32_t f6_of_tbytes(uint32_t x) {
    const uint32_t sel = x & 0x07070707u;
    const uint32_t neg = __builtin_amdgcn_perm(0x28303438u, 0x3A3C3E00u, sel);   // t = 0..7: t - 8
    const uint32_t pos = __builtin_amdgcn_perm(0x1E1C1A18u, 0x14100800u, sel);   // t = 8..15: t - 8
    return __builtin_amdgcn_perm(pos, neg, 0x03020100u | ((x >> 1) & 0x04040404u));
}
// four 6-bit values held one per byte -> 24 bits, byte i at bits 6i
__device__ __forceinline__ uint32_t f6_compress4(uint32_t b) {
    const uint32_t t = (b & 0x003F003Fu) | ((b >> 2) & 0x0FC00FC0u);
    return (t & 0xFFFu) | ((t >> 4) & 0xFFF000u);
}
// byte 0 of four dwords -> one dword (the low byte of a quantizer's magic
// word holds t = code + 8)
__device__ __forceinline__ uint32_t f6_gather4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
    const uint32_t ab = __builtin_amdgcn_perm(b, a, 0x0c0c0400u);
    const uint32_t cd = __builtin_amdgcn_perm(d, c, 0x0c0c0400u);
    return __builtin_amdgcn_perm(cd, ab, 0x05040100u);
}

// 32 codes as eight dwords of t-bytes (code 4k + i in byte i of t[k]) -> the
// lane's six fp6 dwords
__device__ __forceinline__ void f6_from_tbytes(const uint32_t t[8], uint32_t w[6]) {
    uint32_t g[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) g[k] = f6_compress4(f6_of_tbytes(t[k]));
    // 24-bit groups concatenated: three bytes of each
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        w[3 * h] = __builtin_amdgcn_perm(g[4 * h + 1], g[4 * h], 0x04020100u);
        w[3 * h + 1] = __builtin_amdgcn_perm(g[4 * h + 2], g[4 * h + 1], 0x05040201u);
        w[3 * h + 2] = __builtin_amdgcn_perm(g[4 * h + 3], g[4 * h + 2], 0x06050402u);
    }
}

// 32 codes as four dwords of two's-complement nibbles (code 8k + i at bits
// 4i of d[k]) -> the lane's six fp6 dwords
__device__ __forceinline__ void f6_from_nibbles(const uint32_t d[4], uint32_t w[6]) {
    uint32_t t[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t lo = d[k] & 0x0F0F0F0Fu, hi = (d[k] >> 4) & 0x0F0F0F0Fu;   // codes 0,2,4,6 / 1,3,5,7
        // natural order, and t = n ^ 8 = code + 8 for a two's-complement nibble n
        t[2 * k] = __builtin_amdgcn_perm(hi, lo, 0x05010400u) ^ 0x08080808u;
        t[2 * k + 1] = __builtin_amdgcn_perm(hi, lo, 0x07030602u) ^ 0x08080808u;
    }
    f6_from_tbytes(t, w);
}

// 32 codes held as exact floats (-7..7) -> the lane's six fp6 dwords: the
// matrix-operand conversion instruction (round to nearest even, exact on the
// grid; scale 1), which writes element i of its first source to field 2i and
// element i of its second to field 2i + 1
typedef float f6_v16f __attribute__((ext_vector_type(16)));
__device__ __forceinline__ void f6_from_codes(const float *q, uint32_t w[6]) {
    f6_v16f a, b;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        a[i] = q[2 * i];
        b[i] = q[2 * i + 1];
    }
    const auto r = __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(a, b, 1.0f);
#pragma unroll
    for (int i = 0; i < 6; ++i) w[i] = (uint32_t)r[i];
}

// the inverse: six fp6 dwords -> four dwords of nibbles
__device__ __forceinline__ void nibbles_from_f6(const uint32_t w[6], uint32_t d[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) d[k] = 0u;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
        const int bit = 6 * i, q = bit >> 5, o = bit & 31;
        uint32_t v = w[q] >> o;
        if (o > 26) v |= w[q + 1] << (32 - o);
        v &= 0x3Fu;
        const uint32_t e = (v >> 3) & 3u, m = v & 7u;
        const int mag = e == 0 ? 0 : (int)(((8u + m) << e) >> 4);
        const int c = (v & 0x20u) ? -mag : mag;
        d[i >> 3] |= ((uint32_t)c & 15u) << (4 * (i & 7));
    }
}

// byte offset, inside its unit, of the last 8 bytes of lane l
__host__ __device__ inline int f6_tail_offset(int lane) { return 1024 + 16 * (lane & 31) + 8 * (lane >> 5); }

// store a lane's six fp6 dwords
__device__ __forceinline__ void f6_store(uint8_t *unit, int lane, const uint32_t w[6]) {
    *reinterpret_cast<uint4 *>(unit + lane * 16) = make_uint4(w[0], w[1], w[2], w[3]);
    *reinterpret_cast<uint2 *>(unit + f6_tail_offset(lane)) = make_uint2(w[4], w[5]);
}

}  // namespace clq
