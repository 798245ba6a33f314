/*
 * CLQ W4A4 linear layer: plain CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * reference that the GPU path is checked against.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load it; the product
 * library never links or calls it, and it shares no code with the GPU path.
 *
 * What is computed (paper: "CLQ", arXiv 2509.24416):
 *   - Sec. 3.3 (Orthogonal Smoothing, Overhead Analysis): G = S.H, a column
 *     swap S (stored as a gather vector s) followed by a block-diagonal
 *     Hadamard matrix H with +-1 entries, applied to activation rows online
 *     with a fast Hadamard transform and absorbed into the weights offline
 *     (W~ = W.G row-wise for a weight stored [N][K]).
 *   - Sec. 3.1 Eq. (1): uniform quantizer Round(Clip(.)) with n = 4 bits,
 *     in its symmetric per-row form: codes in [-7, 7], scale = a_c / 7.
 *   - Sec. 3.1: activations are quantized dynamically (scale from the live
 *     row); weights are quantized once, one scale per output channel
 *     (Sec. 4.1 "per-channel"), with one clip ratio per matrix (Sec. 4.1).
 *   - Sec. 3.2: the layer computes Y = X W; here Y = X W^T + bias with W
 *     stored [N][K] (the same linear map).
 *
 * Fixed readings (where the paper is silent):
 *   - Hadamard: Sylvester order, unnormalised, H[i][j] = (-1)^popcount(i&j).
 *     The fast transform runs stages h = 1, 2, 4, ..., b/2 in ascending order,
 *     each butterfly (u, v) -> (u + v, u - v) in IEEE fp32.  The whole 1/b
 *     normalisation is folded into the weight scale (exact: power of two).
 *   - Quantizer: a = max|x~| over the row; a_c = fl32(alpha * a);
 *     s = fl32(a_c / 7), r = fl32(7 / a_c) (correctly rounded divisions);
 *     q = clamp(rne(x~ * r), -7, 7) where the product x~ * r is taken exactly
 *     (computed in fp64, where a product of two fp32 values is exact) and
 *     rne rounds half to even.  a_c == 0 gives s = 0 and all codes 0.
 *   - Pack: byte j = (q[2j] & 0xF) | ((q[2j+1] & 0xF) << 4), two's complement.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (no fast-math, no
 * intrinsics).  OpenMP parallelises over independent rows only.
 */
#include <stdint.h>
#include <stddef.h>
#include <math.h>
#include <omp.h>

/* ---- threads ------------------------------------------------------------ */

void clqo_set_threads(int n) { if (n > 0) omp_set_num_threads(n); }
int clqo_get_threads(void) { return omp_get_max_threads(); }

/* ---- Sec. 3.3: gather by s, then block fast Hadamard transform ---------- */

/* One Hadamard block of length b, in place, fp32.  Stage h pairs element i
 * with i + h for every i whose bit h is clear; stages run h = 1, 2, ..., b/2.
 * In exact arithmetic the result is x . H_b with Sylvester-ordered H_b. */
static void fwht_block_f32(float *x, int b)
{
    for (int h = 1; h < b; h <<= 1) {
        for (int i = 0; i < b; ++i) {
            if ((i & h) == 0) {
                float u = x[i];
                float v = x[i + h];
                x[i] = u + v;
                x[i + h] = u - v;
            }
        }
    }
}

/* out[r][k] = FWHT_b( x[r][perm[k]] ) block by block.
 * x: fp32 rows (exact copies of fp16 inputs) with row stride ldx elements.
 * perm: gather vector of length K, or NULL for the identity.
 * out: [rows][K] fp32, row stride K. */
void clqo_rotate(const float *x, int64_t ldx, const int32_t *perm,
                 int64_t rows, int64_t K, int32_t block, float *out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const float *src = x + r * ldx;
        float *dst = out + r * K;
        for (int64_t k = 0; k < K; ++k)
            dst[k] = perm ? src[perm[k]] : src[k];
        for (int64_t k0 = 0; k0 < K; k0 += block)
            fwht_block_f32(dst + k0, block);
    }
}

/* ---- Sec. 3.1 Eq. (1): symmetric per-row quantizer, n = 4 or 8 bits ------ */

/* codes[r][k] in [-qmax, qmax] with qmax = 2^(n-1) - 1 (7 for n = 4 bits,
 * 127 for n = 8); scale[r] = fl32(a_c / qmax), a_c = fl32(alpha * max|x|).
 * The number of clamped elements per row is written to nclamp[r] if
 * non-NULL. */
void clqo_quantize_q(const float *xr, int64_t rows, int64_t K, float alpha, float qmax,
                     int8_t *codes, float *scale, int32_t *nclamp)
{
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const float *x = xr + r * K;
        int8_t *q = codes + r * K;
        float a = 0.0f;
        for (int64_t k = 0; k < K; ++k) {
            float m = fabsf(x[k]);
            if (m > a) a = m;
        }
        float ac = alpha * a;
        int32_t nc = 0;
        if (ac == 0.0f) {
            scale[r] = 0.0f;
            for (int64_t k = 0; k < K; ++k) q[k] = 0;
        } else {
            float s = ac / qmax;
            float rc = qmax / ac;
            scale[r] = s;
            for (int64_t k = 0; k < K; ++k) {
                double t = rint((double)x[k] * (double)rc); /* exact product, RNE */
                if (t > qmax) { t = qmax; ++nc; }
                if (t < -qmax) { t = -qmax; ++nc; }
                q[k] = (int8_t)t;
            }
        }
        if (nclamp) nclamp[r] = nc;
    }
}

/* The 4-bit quantizer of the W4A4 path: qmax = 7. */
void clqo_quantize(const float *xr, int64_t rows, int64_t K, float alpha,
                   int8_t *codes, float *scale, int32_t *nclamp)
{
    clqo_quantize_q(xr, rows, K, alpha, 7.0f, codes, scale, nclamp);
}

void clqo_pack(const int8_t *codes, int64_t rows, int64_t K, uint8_t *out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t j = 0; j < K / 2; ++j) {
            uint8_t lo = (uint8_t)codes[r * K + 2 * j] & 0xFu;
            uint8_t hi = (uint8_t)codes[r * K + 2 * j + 1] & 0xFu;
            out[r * (K / 2) + j] = (uint8_t)(lo | (hi << 4));
        }
}

void clqo_unpack(const uint8_t *packed, int64_t rows, int64_t K, int8_t *codes)
{
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t j = 0; j < K / 2; ++j) {
            uint8_t byte = packed[r * (K / 2) + j];
            int lo = byte & 0xF, hi = byte >> 4;
            codes[r * K + 2 * j] = (int8_t)(lo >= 8 ? lo - 16 : lo);
            codes[r * K + 2 * j + 1] = (int8_t)(hi >= 8 ? hi - 16 : hi);
        }
}

/* ---- integer GEMM: acc[m][n] = sum_k qa[m][k] * qw[n][k] ---------------- */

void clqo_gemm_i32(const int8_t *qa, const int8_t *qw, int64_t M, int64_t N,
                   int64_t K, int32_t *acc)
{
    #pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n) {
            int32_t s = 0;
            for (int64_t k = 0; k < K; ++k)
                s += (int32_t)qa[m * K + k] * (int32_t)qw[n * K + k];
            acc[m * N + n] = s;
        }
}

/* ---- dequantising epilogue in fp64 --------------------------------------
 * p64 = acc * x_scale[m] * w_scale[n]; y64 = p64 + bias[n] (bias may be
 * NULL).  Either output pointer may be NULL. */
void clqo_epilogue(const int32_t *acc, const float *xs, const float *ws,
                   const float *bias, int64_t M, int64_t N,
                   double *y64, double *p64)
{
    #pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n) {
            double p = (double)acc[m * N + n] * (double)xs[m] * (double)ws[n];
            if (p64) p64[m * N + n] = p;
            if (y64) y64[m * N + n] = p + (bias ? (double)bias[n] : 0.0);
        }
}
