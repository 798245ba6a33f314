// Exact order statistics of 32-bit keys in LDS, for one workgroup (the
// device side of the OBS ablation scores and of the CLPS clip bounds).
// Keys compare as unsigned integers: the bit patterns of non-negative
// floats, or an order-preserving encoding of signed ones.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace clq {

// The rank-th smallest (0-based) of the n keys in LDS, by four passes over
// 8-bit digits from the top: a histogram of the keys that match the digits
// chosen so far, then a scan of the 256 bins for the one holding the rank.
// Called by every thread of a workgroup of NT >= 256 threads (the scan
// runs on the first four waves); returns the key.  hist[256], wsum[4] and
// pick[2] are LDS scratch; the keys are not modified.
template <int NT>
__device__ uint32_t radix_select(const uint32_t *keys, int n, int rank, uint32_t *hist, uint32_t *wsum,
                                 uint32_t *pick)
{
    static_assert(NT >= 256 && NT % 64 == 0, "four scan waves");
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    uint32_t prefix = 0u, mask = 0u;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = t; i < 256; i += NT) hist[i] = 0u;
        __syncthreads();
        for (int i = t; i < n; i += NT) {
            const uint32_t k = keys[i];
            if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
        }
        __syncthreads();
        // inclusive scan of the 256 counts (threads 0-255: four waves)
        uint32_t c = 0u, inc = 0u;
        if (t < 256) {
            c = hist[t];
            inc = c;
            for (int off = 1; off < 64; off <<= 1) {
                const uint32_t o = __shfl_up(inc, off);
                if (lane >= off) inc += o;
            }
            if (lane == 63) wsum[wv] = inc;
        }
        __syncthreads();
        if (t < 256) {
            for (int w = 0; w < wv; ++w) inc += wsum[w];
            const uint32_t exc = inc - c;
            if (exc <= (uint32_t)rank && (uint32_t)rank < inc) {   // exactly one bin
                pick[0] = (uint32_t)t;
                pick[1] = exc;
            }
        }
        __syncthreads();
        prefix |= pick[0] << shift;
        mask |= 255u << shift;
        rank -= (int)pick[1];
        __syncthreads();   // pick and hist are rewritten by the next pass
    }
    return prefix;
}

}  // namespace clq
