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
// registers, no VALU) through a ring of kStages stages kept kStages - 1 ahead
// of the matrix cores; the epilogue operands of a tile (scales, biases) go
// once per tile, with its first stage, into a small ring of their own.  Each wave reads its units back with one 16-byte LDS
// read per lane and widens them to int8 in registers.  Widening keeps each
// nibble in the high half of its byte, so the int8 holds 16*q exactly; the
// int32 accumulator holds 256 * sum(qa*qw) (|.| <= 256*49*K < 2^31) and the
// factor 2^-8 is folded into the activation scale in the epilogue.  The k
// order inside a 32-code slice is permuted identically for both operands,
// which leaves the dot product unchanged.
//
// Synchronisation.  Vector-memory operations complete in issue order, so
// "stage s has landed" is an s_waitcnt vmcnt count of the transfers issued
// after it (one of three immediates, depending on whether the last two
// productions carried epilogue operands), emitted with the workgroup barrier
// as one asm statement.  The ring
// stages are separate LDS arrays and the loop is unrolled over them, so each
// stage index is a compile-time constant; the LDS reads of operands and
// epilogue values are asm too, each followed by an explicit lgkmcnt wait,
// because the compiler would otherwise wait for every transfer in flight
// before any LDS read it cannot prove independent.
//
// Schedule.  Two workgroups of four waves (one wave per SIMD each) share a
// compute unit; a persistent grid of that many workgroups walks the tiles,
// and the stage stream runs across tile boundaries, so the next tile's
// transfers overlap this tile's last matrix-core work and its epilogue.
// When the tile count leaves the last round badly filled and a workspace is
// given, the tiles of the last one or two rounds are split along k into
// equal shares of stages for every workgroup (integer sums are exact in any
// order); the workgroup that computes a split tile's first stages owns it
// and adds the others' partial accumulators before its epilogue.
//
// With at most 1.25 such tiles per compute unit a second kernel runs instead
// (w4a4_gemm_halves_kernel, below): tiles of 128 or 64 tokens, each split
// into two halves of the k loop run by two groups of waves and summed in LDS,
// two workgroups per compute unit.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "clq_internal.h"
#include "rq_device.h"

#define CLQ_LDS __attribute__((address_space(3)))

namespace clq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
template <int Q> using IC = std::integral_constant<int, Q>;

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

__device__ __forceinline__ v4i widen16(uint32_t d0, uint32_t d1) {
    return v4i{(int)((d0 << 4) & 0xF0F0F0F0u), (int)((d1 << 4) & 0xF0F0F0F0u),
               (int)(d0 & 0xF0F0F0F0u), (int)(d1 & 0xF0F0F0F0u)};
}

// two fp16 outputs fma(p, w, bias) rounded once from fp32 operands and a
// packed fp16 bias pair (low half: first output), no separate conversions
__device__ __forceinline__ uint32_t fma_mix2(float p0, float w0, float p1, float w1, uint32_t b) {
    uint32_t r;
    asm("v_fma_mixlo_f16 %0, %1, %2, %3 op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixhi_f16 %0, %4, %5, %3 op_sel:[0,0,1] op_sel_hi:[0,0,1]"
        : "=&v"(r)
        : "v"(p0), "v"(w0), "v"(b), "v"(p1), "v"(w1));
    return r;
}

// the same with fp32 bias operands (each exactly an fp16 value), so that
// every kernel's outputs are rounded by the same instruction
__device__ __forceinline__ uint32_t fma_mix2f(float p0, float w0, float b0, float p1, float w1, float b1) {
    uint32_t r;
    asm("v_fma_mixlo_f16 %0, %1, %2, %3\n\t"
        "v_fma_mixhi_f16 %0, %4, %5, %6"
        : "=&v"(r)
        : "v"(p0), "v"(w0), "v"(b0), "v"(p1), "v"(w1), "v"(b1));
    return r;
}

constexpr int kStages = 5;   // ring depth
constexpr int kGroupM = 4;          // token panels per tile group (L2 reuse of channel panels)
constexpr int kSpinLimit = 1 << 22;  // bound on a split-tile wait (about a second)
// Split-k status words at the head of the workspace: [0] the number of waves
// whose wait for a contributor's partial gave up, [1] the first such tile,
// [2] its contributor's rank (see launch_gemm)
constexpr int kStatusBytes = 256;

template <int WN_, int WM_, int FN_, int FM_, int WGS_>
struct Tile {
    static constexpr int WN = WN_, WM = WM_, FN = FN_, FM = FM_;
    static constexpr int WGS = WGS_;
    static constexpr int NW = WN * WM;
    static constexpr int NT = NW * 64;
    static constexpr int BN = WN * FN * 32;
    static constexpr int BM = WM * FM * 32;
    static constexpr int W_UNITS = BN / 32;
    static constexpr int X_UNITS = BM / 32;
    static constexpr int UNITS = W_UNITS + X_UNITS;
    static constexpr int UPW = UNITS / NW;
    static constexpr int STAGE_BYTES = UNITS * 1024;
    static constexpr int XS_CH = BM / 64, WS_CH = BN / 64, B_CH = BN / 128;
    static constexpr int PART_INTS = NT * FN * FM * 16;   // one partial tile
    static_assert(UNITS % NW == 0, "units split evenly over waves");
};

// A run of k-stages [kb, ke) of tile L; j counts the runs of a workgroup.
struct Seg {
    int j, L, kb, ke, k;
};

struct GemmArgs {
    const uint8_t *Xq;
    const float *xs;
    const uint8_t *Wq;
    const float *ws;
    const uint16_t *bias;
    void *Y;
    int64_t ldy;
    int M, N, K, tiles_m, tiles_n;
    int dp;        // tiles computed whole (the first dp in tile order)
    int sk;        // k-stages of the remaining tiles, split evenly over the grid
    int32_t *part; // partial accumulators, one tile per workgroup
    int *flags;    // one per wave of every workgroup
    int *status;   // split-k status words (kStatusBytes at the workspace head)
    int spin_limit;   // bound on a wait for a contributor's flag (sleeps)
    int drop_signal;  // test only: contributors never raise their flags
    int full_grid;    // two workgroups on every compute unit (the uneven deal applies only then)
    // fused rotate+quantize (the two-halves kernel with FB != 0): fp16
    // activations fx (row stride ldfx) quantized into Xq / xs by the first
    // n_rq work items (rq_rows rows each), the GEMM tiles after them; qhdr:
    // queue, finished and epoch words; qflags: one per rotate+quantize item
    const uint16_t *fx;
    int64_t ldfx;
    int rq_rows, n_rq;
    int *qhdr;
    int *qflags;
    // squared-error mode: target Y0 fp32 [M][ldy0]; one fp64 partial per
    // wave of every tile, at errp[tile * waves + wave]
    const float *y0;
    int64_t ldy0;
    double *errp;
};

// ERR: instead of storing Y, the epilogue sums (Y0 - sum * x_scale * w_scale)^2
// over the tile in fp64 (the integer sum exact, the products in the order
// written) and stores one partial per wave.
template <class C, bool I32OUT, bool RAGGED, bool BIAS, bool ERR>
__global__ void __launch_bounds__(C::NT, C::WGS) w4a4_gemm_kernel(GemmArgs a)
{
    static_assert(!ERR || (!I32OUT && !BIAS), "the error mode has no output and no bias");
    constexpr int NS = kStages;
    constexpr bool BIAS_CH = BIAS && !RAGGED && !I32OUT;
    constexpr int E_CH = I32OUT ? 0 : C::XS_CH + C::WS_CH + (BIAS_CH ? C::B_CH : 0);
    constexpr int EPW = (E_CH + C::NW - 1) / C::NW;
    // epilogue operands of a segment (token scales fp32 [BM], channel scales
    // fp32 [BN], bias fp16 [BN]) travel once per segment into their own ring
    // of NS entries indexed by segment number: the producer runs at most
    // NS - 1 stages, hence NS - 1 segments, ahead of the consumer
    constexpr int E_XS = 0, E_WS = E_XS + C::BM * 4, E_B = E_WS + C::BN * 4;
    constexpr int E_BYTES = I32OUT ? 16 : E_B + (BIAS_CH ? C::BN * 2 : 0);
    constexpr int SLOT = C::STAGE_BYTES;
    static_assert(NS == 5 || NS == 6, "ring arrays below");
    __shared__ __align__(16) uint8_t ring0[SLOT], ring1[SLOT], ring2[SLOT], ring3[SLOT], ring4[SLOT];
    __shared__ __align__(16) uint8_t ring5[NS == 6 ? SLOT : 16];
    __shared__ __align__(16) uint8_t ebuf[NS][E_BYTES];
    auto slot = [&](auto qc) -> uint8_t * {
        constexpr int q = decltype(qc)::value;
        if constexpr (q == 0) return ring0;
        else if constexpr (q == 1) return ring1;
        else if constexpr (q == 2) return ring2;
        else if constexpr (q == 3) return ring3;
        else if constexpr (q == 4) return ring4;
        else return ring5;
    };

    const int M = a.M, N = a.N, nks = a.K >> 6;
    const int G = gridDim.x, gx = G >> 3, xcd = blockIdx.x & 7, jw = blockIdx.x >> 3;
    const int rank = xcd * gx + jw;
    const int dp = a.dp, S = a.sk;
    const int per = dp >> 3, rem = dp & 7;
    const int cnt = per + (xcd < rem ? 1 : 0);
    const int dstart = xcd * per + min(xcd, rem);
    // Uneven deal on a full grid of whole tiles (several rounds): the two
    // workgroups on a compute unit do not progress at the same rate (the one
    // placed first, jw < gx / 2 in dispatch order, wins the issue arbitration
    // and finishes a tile in about two thirds of the other's time), so the
    // later one gets about 40% of the unit's tiles: nb rounds for every
    // workgroup, the remaining rr tiles for the first half only.
    const int H = gx >> 1;
    const bool asym = S == 0 && G == a.full_grid && cnt >= 4 * gx;
    int nb = 0, rr = 0;
    if (asym) {
        nb = min(cnt / gx, (cnt * 2 * 40 + gx * 50) / (gx * 100));
        rr = cnt - nb * gx;
    }
    const int my_dp = !asym ? (jw < cnt ? (cnt - jw + gx - 1) / gx : 0)
                            : nb + (jw < H && jw < rr ? (rr - jw + H - 1) / H : 0);
    const int sk_a = rank * S / G, sk_b = (rank + 1) * S / G;
    const int total = my_dp * nks + (sk_b - sk_a);
    if (total == 0) return;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wn = wave % C::WN, wm = wave / C::WN;
    const int wunits_total = (int)(padded_rows(N) >> 5);
    const int xunits_total = (int)(padded_act_rows(M) >> 5);

    auto coords = [&](int L, int &tm, int &tn) {
        const int gsz = kGroupM * a.tiles_n;
        const int g = L / gsz, r = L - g * gsz;
        const int m0 = g * kGroupM;
        const int gm = min(a.tiles_m - m0, kGroupM);
        tn = r / gm;
        tm = m0 + (r - tn * gm);
    };
    // A segment: k-stages [kb, ke) of tile L.  Whole tiles first, then this
    // workgroup's share of the split region.
    auto next_seg = [&](Seg &c) {
        ++c.j;
        if (c.j < my_dp) {
            c.L = !asym || c.j < nb ? dstart + jw + c.j * gx : dstart + nb * gx + jw + (c.j - nb) * H;
            c.kb = 0;
            c.ke = nks;
        } else {
            const int g = c.j == my_dp ? sk_a : (c.L - dp + 1) * nks;
            const int u = g / nks;
            c.L = dp + u;
            c.kb = g - u * nks;
            c.ke = min(nks, c.kb + (sk_b - g));
        }
        c.k = c.kb;
    };

    // ---- producer -------------------------------------------------------------
    Seg pc{-1, 0, 0, 0, 0};
    next_seg(pc);
    int p_s = 0;
    const uint8_t *usrc[C::UPW];
    const uint8_t *esrc[EPW > 0 ? EPW : 1];
    int edst[EPW > 0 ? EPW : 1];
    auto p_setup = [&]() {
        int tm, tn;
        coords(pc.L, tm, tn);
#pragma unroll
        for (int j = 0; j < C::UPW; ++j) {
            const int u = wave * C::UPW + j;
            if (u < C::W_UNITS) {
                const int ug = min(tn * C::W_UNITS + u, wunits_total - 1);
                usrc[j] = a.Wq + (int64_t)ug * nks * 1024;
            } else {
                const int ux = min(tm * C::X_UNITS + (u - C::W_UNITS), xunits_total - 1);
                usrc[j] = a.Xq + (int64_t)ux * nks * 1024;
            }
        }
#pragma unroll
        for (int j = 0; j < EPW; ++j) {
            const int c = wave * EPW + j;
            if (c < C::XS_CH) {
                esrc[j] = reinterpret_cast<const uint8_t *>(a.xs + min(tm * C::BM + c * 64 + lane, M - 1));
                edst[j] = E_XS + c * 256;
            } else if (c < C::XS_CH + C::WS_CH || c >= E_CH) {
                const int w = (c - C::XS_CH) % C::WS_CH;
                esrc[j] = reinterpret_cast<const uint8_t *>(a.ws + min(tn * C::BN + w * 64 + lane, N - 1));
                edst[j] = E_WS + w * 256;
            } else {
                const int b = c - C::XS_CH - C::WS_CH;
                esrc[j] = reinterpret_cast<const uint8_t *>(reinterpret_cast<const uint32_t *>(a.bias) + min(tn * (C::BN / 2) + b * 64 + lane, N / 2 - 1));
                edst[j] = E_B + b * 256;
            }
        }
    };
    p_setup();
    int e_next = 0;          // stage whose production carries the next segment's operands
    unsigned phist = 0;      // 1 bit per production call: epilogue operands issued
    auto produce = [&](auto qc) {
        // the segment's epilogue operands go out with its first stage,
        // ahead of the units (the wait counts below rely on that order)
        int e_now = 0;
        if (EPW > 0 && pc.k == pc.kb && p_s == e_next) {
            uint8_t *ed = &ebuf[pc.j % NS][0];
#pragma unroll
            for (int j = 0; j < EPW; ++j)
                __builtin_amdgcn_global_load_lds(esrc[j], (CLQ_LDS void *)(ed + edst[j]), 4, 0, 0);
            e_now = 1;
            e_next = -1;
        }
        phist = (phist << 1) | e_now;
        uint8_t *dst = slot(qc);
        const uint32_t voff = (uint32_t)(pc.k * 1024 + lane * 16);
#pragma unroll
        for (int j = 0; j < C::UPW; ++j)
        {
            const uint8_t *sp = usrc[j] + voff;
            __builtin_amdgcn_global_load_lds(sp, (CLQ_LDS void *)(dst + (wave * C::UPW + j) * 1024), 16, 0, 0);
        }
        if (p_s < total - 1) {
            ++p_s;
            if (++pc.k == pc.ke) {
                next_seg(pc);
                p_setup();
                e_next = p_s;
            }
        }
    };

    // ---- consumer -------------------------------------------------------------
    v4u pa[C::FN], pb[C::FM];
    v4i a0[C::FN], b0[C::FM], a1[C::FN], b1[C::FM];
    const uint32_t wl0 = (uint32_t)(wn * C::FN * 1024 + lane * 16);
    const uint32_t xl0 = (uint32_t)((C::W_UNITS + wm * C::FM) * 1024 + lane * 16);
    auto read_packed = [&](auto qc) {
        // the lane offsets pass through an empty asm so that the per-stage
        // addresses are formed here, not hoisted into 30 live registers
        uint32_t wl = wl0, xl = xl0;
        asm volatile("" : "+v"(wl), "+v"(xl));
        wl += lds_addr(slot(qc));
        xl += lds_addr(slot(qc));
        static_for<0, C::FN>([&](auto f) { pa[f] = lds_read16<decltype(f)::value * 1024>(wl); });
        static_for<0, C::FM>([&](auto f) { pb[f] = lds_read16<decltype(f)::value * 1024>(xl); });
    };
    auto operands_ready = [&]() {
        static_assert(C::FN == 4 && C::FM == 2, "operand list below");
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(pa[0]), "+v"(pa[1]), "+v"(pa[2]), "+v"(pa[3]), "+v"(pb[0]), "+v"(pb[1]));
    };
    auto widen_half0 = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) a0[fn] = widen16(pa[fn][0], pa[fn][1]);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) b0[fm] = widen16(pb[fm][0], pb[fm][1]);
    };
    auto widen_half1 = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) a1[fn] = widen16(pa[fn][2], pa[fn][3]);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) b1[fm] = widen16(pb[fm][2], pb[fm][3]);
    };
    v16i acc[C::FN][C::FM];
    auto zero_acc = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = v16i{};
    };
    auto mma = [&](const v4i (&x)[C::FN], const v4i (&y)[C::FM]) {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(x[fn], y[fm], acc[fn][fm], 0, 0, 0);
    };
    constexpr int MPH = C::FN * C::FM;
    constexpr int WOPS = (C::FN + C::FM) * 6;
    constexpr int GA = 4, GB = 2;
    auto interleave = [&](auto fpc, auto vpmc, auto dsc) {
        constexpr int first_plain = decltype(fpc)::value, vpm = decltype(vpmc)::value;
        constexpr int ds_after = decltype(dsc)::value;
#pragma unroll
        for (int i = 0; i < MPH; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (i >= first_plain) __builtin_amdgcn_sched_group_barrier(0x002, vpm, 0);
            if (i == ds_after) __builtin_amdgcn_sched_group_barrier(0x100, C::FN + C::FM, 0);
        }
    };

    // ---- split tiles: partial accumulators through global memory ---------------
    // The workgroup that computes a split tile's first stages owns it; every
    // other workgroup that computes some of its stages starts its own range
    // there, stores its accumulators and raises its flags; the owner adds them
    // before its epilogue.  Waves pair one to one (same wave, same lane).
    constexpr int WPART = C::FN * C::FM * 16 * 64;   // ints per wave
    // Partial tiles cross XCDs, whose L2 caches are not coherent with each
    // other: they are written through to memory and read back past the L2
    // (device-scope cache policy), and the flags are relaxed device-scope
    // atomics.  Each wave orders its own data before its flag with a wait.
    auto contribute = [&]() {
        uint32_t lo = (uint32_t)lane * 16;
        asm volatile("" : "+v"(lo));   // addresses formed here, not hoisted out of the loop
        uint8_t *base = reinterpret_cast<uint8_t *>(a.part + (size_t)rank * C::PART_INTS + wave * WPART) + lo;
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) {
                const v16i x = acc[fn][fm];
                uint8_t *p = base + (fn * C::FM + fm) * 4096;
                asm volatile(
                    "global_store_dwordx4 %0, %1, off sc1\n\t"
                    "global_store_dwordx4 %0, %2, off offset:1024 sc1\n\t"
                    "global_store_dwordx4 %0, %3, off offset:2048 sc1\n\t"
                    "global_store_dwordx4 %0, %4, off offset:3072 sc1"
                    ::"v"(p), "v"(__builtin_shufflevector(x, x, 0, 1, 2, 3)),
                    "v"(__builtin_shufflevector(x, x, 4, 5, 6, 7)), "v"(__builtin_shufflevector(x, x, 8, 9, 10, 11)),
                    "v"(__builtin_shufflevector(x, x, 12, 13, 14, 15))
                    : "memory");
            }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        if (!a.drop_signal)
            __hip_atomic_store(a.flags + rank * C::NW + wave, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    // Partials are read two contributors at a time (16 loads in flight per
    // wave), so a tile split many ways pays half as many memory round trips.
    // The wait is bounded: all workgroups of the grid are meant to be
    // resident at once, but nothing stops other kernels from holding compute
    // units.  A wait that gives up leaves that contributor's partial out of
    // the sum (its flag may still rise later and is not cleared), and records
    // the failure in the status words for the host: the call's output is then
    // invalid and the workspace must be zero-filled again before reuse.
    auto wait_flag = [&](int L, int r2) -> bool {
        int *fl = a.flags + r2 * C::NW + wave;
        for (int spin = 0; spin < a.spin_limit; ++spin) {
            if (__hip_atomic_load(fl, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) return true;
            __builtin_amdgcn_s_sleep(8);
        }
        if (__hip_atomic_load(fl, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) return true;
        if (lane == 0) {
            const int old = __hip_atomic_fetch_add(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (old == 0) {
                __hip_atomic_store(a.status + 1, L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(a.status + 2, r2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        return false;
    };
    auto part_base = [&](int r2) -> const uint8_t * {
        uint32_t lo = (uint32_t)lane * 16;
        asm volatile("" : "+v"(lo));
        return reinterpret_cast<const uint8_t *>(a.part + (size_t)r2 * C::PART_INTS + wave * WPART) + lo;
    };
    auto add8 = [&](int fn, v4i q0, v4i q1, v4i q2, v4i q3, v4i q4, v4i q5, v4i q6, v4i q7) {
        acc[fn][0] += __builtin_shufflevector(__builtin_shufflevector(q0, q1, 0, 1, 2, 3, 4, 5, 6, 7),
                                              __builtin_shufflevector(q2, q3, 0, 1, 2, 3, 4, 5, 6, 7),
                                              0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
        acc[fn][1] += __builtin_shufflevector(__builtin_shufflevector(q4, q5, 0, 1, 2, 3, 4, 5, 6, 7),
                                              __builtin_shufflevector(q6, q7, 0, 1, 2, 3, 4, 5, 6, 7),
                                              0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
    };
    auto add_one = [&](int r2) {
        const uint8_t *base = part_base(r2);
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) {
            const uint8_t *p0 = base + (fn * C::FM) * 4096, *p1 = p0 + 4096;
            v4i q0, q1, q2, q3, q4, q5, q6, q7;
            asm volatile(
                "global_load_dwordx4 %0, %8, off sc1\n\t"
                "global_load_dwordx4 %1, %8, off offset:1024 sc1\n\t"
                "global_load_dwordx4 %2, %8, off offset:2048 sc1\n\t"
                "global_load_dwordx4 %3, %8, off offset:3072 sc1\n\t"
                "global_load_dwordx4 %4, %9, off sc1\n\t"
                "global_load_dwordx4 %5, %9, off offset:1024 sc1\n\t"
                "global_load_dwordx4 %6, %9, off offset:2048 sc1\n\t"
                "global_load_dwordx4 %7, %9, off offset:3072 sc1\n\t"
                "s_waitcnt vmcnt(0)"
                : "=&v"(q0), "=&v"(q1), "=&v"(q2), "=&v"(q3), "=&v"(q4), "=&v"(q5), "=&v"(q6), "=&v"(q7)
                : "v"(p0), "v"(p1)
                : "memory");
            add8(fn, q0, q1, q2, q3, q4, q5, q6, q7);
        }
    };
    auto add_two = [&](int r2, int r3) {
        const uint8_t *base = part_base(r2), *bas2 = part_base(r3);
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) {
            const uint8_t *p0 = base + (fn * C::FM) * 4096, *p1 = p0 + 4096;
            const uint8_t *p2 = bas2 + (fn * C::FM) * 4096, *p3 = p2 + 4096;
            v4i q0, q1, q2, q3, q4, q5, q6, q7, t0, t1, t2, t3, t4, t5, t6, t7;
            asm volatile(
                "global_load_dwordx4 %0, %16, off sc1\n\t"
                "global_load_dwordx4 %1, %16, off offset:1024 sc1\n\t"
                "global_load_dwordx4 %2, %16, off offset:2048 sc1\n\t"
                "global_load_dwordx4 %3, %16, off offset:3072 sc1\n\t"
                "global_load_dwordx4 %4, %17, off sc1\n\t"
                "global_load_dwordx4 %5, %17, off offset:1024 sc1\n\t"
                "global_load_dwordx4 %6, %17, off offset:2048 sc1\n\t"
                "global_load_dwordx4 %7, %17, off offset:3072 sc1\n\t"
                "global_load_dwordx4 %8, %18, off sc1\n\t"
                "global_load_dwordx4 %9, %18, off offset:1024 sc1\n\t"
                "global_load_dwordx4 %10, %18, off offset:2048 sc1\n\t"
                "global_load_dwordx4 %11, %18, off offset:3072 sc1\n\t"
                "global_load_dwordx4 %12, %19, off sc1\n\t"
                "global_load_dwordx4 %13, %19, off offset:1024 sc1\n\t"
                "global_load_dwordx4 %14, %19, off offset:2048 sc1\n\t"
                "global_load_dwordx4 %15, %19, off offset:3072 sc1\n\t"
                "s_waitcnt vmcnt(0)"
                : "=&v"(q0), "=&v"(q1), "=&v"(q2), "=&v"(q3), "=&v"(q4), "=&v"(q5), "=&v"(q6), "=&v"(q7),
                  "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3), "=&v"(t4), "=&v"(t5), "=&v"(t6), "=&v"(t7)
                : "v"(p0), "v"(p1), "v"(p2), "v"(p3)
                : "memory");
            add8(fn, q0, q1, q2, q3, q4, q5, q6, q7);
            add8(fn, t0, t1, t2, t3, t4, t5, t6, t7);
        }
    };
    auto fixup = [&](int L) {
        static_assert(C::FM == 2, "two token fragments per load group");
        const int u = L - dp;
        const int beg = u * nks, end = beg + nks;
        int pending = -1;
        for (int r2 = rank + 1; r2 < G; ++r2) {
            const int st = r2 * S / G;
            if (st >= end) break;
            const int en = (r2 + 1) * S / G;
            if (en <= st || st <= beg) continue;
            if (!wait_flag(L, r2)) continue;   // not added; its flag is left as it is
            if (pending < 0) {
                pending = r2;
                continue;
            }
            add_two(pending, r2);
            __hip_atomic_store(a.flags + pending * C::NW + wave, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.flags + r2 * C::NW + wave, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            pending = -1;
        }
        if (pending >= 0) {
            add_one(pending);
            __hip_atomic_store(a.flags + pending * C::NW + wave, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    };

    // ---- epilogue: lane owns token m and 16 consecutive channels ----------------
    const int h16 = (lane >> 5) * 16;
    // The epilogue operands are read with asm too (same reason as the
    // operand units); one explicit wait per channel fragment orders their use.
    auto epilogue = [&](int L, int sj, auto qc) {
        int tm, tn;
        coords(L, tm, tn);
        uint32_t lx = (uint32_t)((wm * C::FM * 32 + (lane & 31)) * 4);
        uint32_t lw = (uint32_t)((wn * C::FN * 32 + h16) * 4);
        asm volatile("" : "+v"(lx), "+v"(lw));
        const uint32_t sb = lds_addr(&ebuf[0][0]) + (uint32_t)((sj % NS) * E_BYTES);
        const uint32_t axs = sb + E_XS + lx, aws = sb + E_WS + lw, ab = sb + E_B + lw / 2;
        float xsm[C::FM];
        int mrow[C::FM];
        double esum = 0.0;
        if constexpr (!I32OUT) {
            static_assert(C::FM == 2, "two token scales per lane");
            asm volatile("ds_read_b32 %0, %2\n\tds_read_b32 %1, %2 offset:128\n\ts_waitcnt lgkmcnt(0)"
                         : "=&v"(xsm[0]), "=&v"(xsm[1]) : "v"(axs));
        }
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) mrow[fm] = tm * C::BM + (wm * C::FM + fm) * 32 + (lane & 31);
        // fp16 output: the lane's row pointers at its first channel, formed
        // once per tile (a fragment's channels are a constant offset on them)
        const int nl = tn * C::BN + wn * C::FN * 32 + h16;
        uint16_t *rowp[C::FM];
        float xsc[C::FM];
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) {
            rowp[fm] = reinterpret_cast<uint16_t *>(a.Y) + (int64_t)mrow[fm] * a.ldy + nl;
            xsc[fm] = xsm[fm] * (1.0f / 256.0f);   // accumulators hold 256 * sum
        }
        // channel operands outer, tokens inner: each channel scale and bias
        // is loaded once and dies after its fragments
        static_for<0, C::FN>([&](auto fc) {
            constexpr int fn = decltype(fc)::value;
            const int n0 = nl + fn * 32;
            v4f w4[4];
            v4u b8[2];
            if constexpr (!I32OUT) {
                // one asm block: the reads and their wait, so no use can be
                // scheduled between them
                asm volatile(
                    "ds_read_b128 %0, %4 offset:%6\n\t"
                    "ds_read_b128 %1, %4 offset:%7\n\t"
                    "ds_read_b128 %2, %4 offset:%8\n\t"
                    "ds_read_b128 %3, %4 offset:%9\n\t"
                    "s_waitcnt lgkmcnt(0)"
                    : "=&v"(w4[0]), "=&v"(w4[1]), "=&v"(w4[2]), "=&v"(w4[3])
                    : "v"(aws), "v"(ab), "n"(fn * 128), "n"(fn * 128 + 16), "n"(fn * 128 + 32), "n"(fn * 128 + 48));
                if constexpr (BIAS_CH)
                    asm volatile(
                        "ds_read_b128 %0, %2 offset:%3\n\t"
                        "ds_read_b128 %1, %2 offset:%4\n\t"
                        "s_waitcnt lgkmcnt(0)"
                        : "=&v"(b8[0]), "=&v"(b8[1])
                        : "v"(ab), "n"(fn * 64), "n"(fn * 64 + 16));
            }
            // (element reads of the asm results stay typed: no bit casts of
            // vector elements, which this compiler mis-vectorizes)
            float wsv[16];
            uint32_t bw[8];   // bias pairs, packed fp16 (low half: even channel)
            if constexpr (!I32OUT) {
#pragma unroll
                for (int v = 0; v < 16; ++v) wsv[v] = w4[v / 4][v % 4];
            }
            if constexpr (!BIAS || I32OUT) {
#pragma unroll
                for (int v = 0; v < 8; ++v) bw[v] = 0u;
            } else if constexpr (RAGGED) {
#pragma unroll
                for (int v = 0; v < 16; v += 2) {
                    const int na = min(n0 + v, N - 1), nb = min(n0 + v + 1, N - 1);
                    const uint16_t *bh = a.bias;
                    bw[v / 2] = (uint32_t)bh[na] | ((uint32_t)bh[nb] << 16);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 8; ++v) bw[v] = b8[v / 4][v % 4];
            }
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) {
                const int m = mrow[fm];
                const v16i &x = acc[fn][fm];
                if constexpr (I32OUT) {
                    int32_t *dst = reinterpret_cast<int32_t *>(a.Y) + (int64_t)m * a.ldy + n0;
                    if (m < M && n0 < N) {
                        if (!RAGGED || n0 + 16 <= N) {
#pragma unroll
                            for (int q4 = 0; q4 < 4; ++q4)
                                reinterpret_cast<v4i *>(dst)[q4] =
                                    v4i{x[4 * q4] >> 8, x[4 * q4 + 1] >> 8, x[4 * q4 + 2] >> 8, x[4 * q4 + 3] >> 8};
                        } else {
#pragma unroll
                            for (int v = 0; v < 16; ++v)
                                if (n0 + v < N) dst[v] = x[v] >> 8;
                        }
                    }
                } else if constexpr (ERR) {
                    // the exact integer sum is x >> 8; d = Y0 - ((sum * x_scale) * w_scale)
                    if (m < M && n0 < N) {
                        const float *yr = a.y0 + (int64_t)m * a.ldy0 + n0;
                        float yv[16];
                        if constexpr (!RAGGED) {   // 16-byte aligned rows of whole 16-channel pieces
#pragma unroll
                            for (int q4 = 0; q4 < 4; ++q4) {
                                const v4f t = reinterpret_cast<const v4f *>(yr)[q4];
                                yv[4 * q4] = t[0];
                                yv[4 * q4 + 1] = t[1];
                                yv[4 * q4 + 2] = t[2];
                                yv[4 * q4 + 3] = t[3];
                            }
                        } else {
#pragma unroll
                            for (int v = 0; v < 16; ++v) yv[v] = n0 + v < N ? yr[v] : 0.0f;
                        }
                        const double xm = (double)xsm[fm];
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            if (RAGGED && n0 + v >= N) continue;
                            const double d = (double)yv[v] - (double)(x[v] >> 8) * xm * (double)wsv[v];
                            esum += d * d;
                        }
                    }
                } else {
                    uint32_t hv[8];
#pragma unroll
                    for (int v = 0; v < 16; v += 2)
                        hv[v / 2] = fma_mix2((float)x[v] * xsc[fm], wsv[v], (float)x[v + 1] * xsc[fm], wsv[v + 1], bw[v / 2]);
                    uint16_t *dst = rowp[fm] + fn * 32;
                    if (m < M && n0 < N) {
                        if (!RAGGED || n0 + 16 <= N) {
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
            __builtin_amdgcn_sched_barrier(0);
        });
        if constexpr (ERR) {
            // fixed butterfly over the wave; lane 0 holds the wave's partial
            for (int off = 32; off > 0; off >>= 1) esum += __shfl_xor(esum, off);
            if (lane == 0) a.errp[(int64_t)L * C::NW + wave] = esum;
        }
    };

    // Stage s+1 has landed once at most the VMEM instructions issued after
    // its last transfer are outstanding (completion is in issue order): the
    // NS-3 later productions, with their epilogue operand transfers if any
    // (operands precede a production's units, so only the last NS-3 calls
    // count).  Epilogue stores are not counted, which only makes the wait
    // stricter.
    static_assert(NS == 5, "two-call history below");
    constexpr int W0 = (NS - 3) * C::UPW;
    auto landed_wait = [&]() {
        switch (__builtin_popcount(phist & 3u)) {
            case 0: asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(W0) : "memory"); break;
            case 1: asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(W0 + EPW) : "memory"); break;
            default: asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(W0 + 2 * EPW) : "memory"); break;
        }
    };

    // ---- pipeline ---------------------------------------------------------------
    produce(IC<0>{});
    produce(IC<1>{});
    produce(IC<2>{});
    produce(IC<3>{});
    if constexpr (NS == 6) produce(IC<4>{});
    landed_wait();
    read_packed(IC<0>{});
    operands_ready();
    widen_half0();
    zero_acc();

    Seg cc{-1, 0, 0, 0, 0};
    next_seg(cc);
    int s = 0;
    constexpr int VH1 = (WOPS + GA - 1) / GA;
    constexpr int VH2 = (WOPS + (MPH - GB) - 1) / (MPH - GB);
    auto iter = [&](auto qc) -> bool {
        constexpr int q = decltype(qc)::value;
        constexpr IC<(q + 1) % NS> nqc{};
        constexpr IC<(q + NS - 1) % NS> pqc{};
        landed_wait();
        produce(pqc);
        __builtin_amdgcn_sched_barrier(0);
        widen_half1();
        mma(a0, b0);
        read_packed(nqc);
        interleave(IC<0>{}, IC<VH1>{}, IC<GA - 1>{});
        __builtin_amdgcn_sched_barrier(0);
        operands_ready();
        widen_half0();
        mma(a1, b1);
        interleave(IC<GB>{}, IC<VH2>{}, IC<-1>{});
        __builtin_amdgcn_sched_barrier(0);
        if (cc.k == cc.ke - 1) {
            if constexpr (ERR) {   // launched with whole tiles only: no split code
                epilogue(cc.L, cc.j, qc);
            } else if (cc.kb != 0) {
                contribute();
            } else {
                if (cc.ke != nks) fixup(cc.L);
                epilogue(cc.L, cc.j, qc);
            }
            zero_acc();
            if (s + 1 < total) next_seg(cc);
        } else {
            ++cc.k;
        }
        ++s;
        return s < total;
    };
    auto iter5 = [&]() -> bool {
        if constexpr (NS == 6) return iter(IC<5>{});
        else return true;
    };
    while (iter(IC<0>{}) && iter(IC<1>{}) && iter(IC<2>{}) && iter(IC<3>{}) && iter(IC<4>{}) && iter5()) {
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// the tiles of the two-halves kernel: 128 channels x 128 tokens, a half of
// two waves (a four-wave workgroup, two per compute unit), or x 64 tokens,
// a half of one wave, when the 128-token tiles would fill at most half the
// compute units
using TileHalf128 = Tile<1, 2, 4, 2, 2>;
using TileHalf64 = Tile<1, 1, 4, 2, 2>;

// ---- few tiles: the k loop in two halves ---------------------------------------
// With about one 256-token tile per compute unit, a lone workgroup's k loop
// is bound by the instruction stream of its one wave per SIMD (matrix-core
// work and the ~180 other instructions of a stage run mostly in series).
// This kernel gives each smaller tile two halves of C::NW waves: the first
// half runs the first half of the k-stages and the second half the rest, each
// half through its own LDS ring, in lockstep on the workgroup barrier, with
// two workgroups per compute unit.  The halves swap integer sums in LDS
// (exact) and each runs the epilogue of two channel fragments with the same
// arithmetic as the persistent kernel.
constexpr int kHalfStages = 4;   // ring depth per half

// FB != 0: the fused variant (rotate+quantize of the activations folded in,
// Hadamard block FB).  Work items come from an atomic counter in order: the
// first n_rq items rotate and quantize rq_rows activation rows each and
// publish them; the rest are the GEMM tiles, each of which first waits for
// the items covering its token rows.  A tile only ever waits for items taken
// before its own, by workgroups that are already running and never wait, so
// the grid cannot deadlock whatever part of it is resident.
template <class C, bool I32OUT, bool RAGGED, bool BIAS, int FB = 0>
__global__ void __launch_bounds__(2 * C::NT, 2) w4a4_gemm_halves_kernel(GemmArgs a)
{
    static_assert(!(I32OUT && BIAS), "no bias on the integer output");
    static_assert(C::WN == 1 && C::FN == 4 && C::FM == 2, "one channel panel, 4 x 2 fragments per wave");
    constexpr int NS = kHalfStages;
    constexpr int SLOT = C::STAGE_BYTES;
    // the two rings (96 or 64 KB), reused at the end for the exchange of the
    // halves' sums (16 KB per wave each way)
    constexpr int kExch = C::NW * 16384;
    __shared__ __align__(16) uint8_t pool[2 * NS * SLOT > 2 * kExch ? 2 * NS * SLOT : 2 * kExch];
    auto ring = reinterpret_cast<uint8_t (*)[NS][SLOT]>(pool);
    // the tile's epilogue operands, staged at the start as floats: channel
    // scales, biases (fp16 widened, exact), token scales
    constexpr int EPN = 2 * C::BN + C::BM;
    __shared__ float ep[EPN];
    const float *ep_ws = ep, *ep_b = ep + C::BN, *ep_xs = ep + 2 * C::BN;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w8 = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = w8 / C::NW, wm = w8 % C::NW;   // one channel panel per tile: wn = 0
    const int M = a.M, N = a.N, nks = a.K >> 6;
    // tile order: workgroups are dealt to the 8 XCDs round-robin; each XCD
    // takes a contiguous run of tiles (in the grouped order below), so the
    // operand panels a run shares stay in that XCD's L2
    int L;
    {
        const int G = gridDim.x, x = blockIdx.x & 7, j = blockIdx.x >> 3;
        const int per = G >> 3, rem = G & 7;
        L = x * per + min(x, rem) + j;
    }
    int e1 = 0;   // fused: this call's epoch + 1, the value of a published item's flag
    if constexpr (FB != 0) {
        static_assert(!I32OUT, "the fused variant writes fp16");
        __shared__ int s_item, s_epoch;
        if (tid == 0) {
            s_epoch = __hip_atomic_load(a.qhdr + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_item = __hip_atomic_fetch_add(a.qhdr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();
        const int item = s_item;
        e1 = s_epoch + 1;
        auto finish = [&]() {
            // the last workgroup to finish resets the queue for the next call
            if (tid == 0) {
                const int done = __hip_atomic_fetch_add(a.qhdr + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (done == (int)gridDim.x - 1) {
                    __hip_atomic_store(a.qhdr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(a.qhdr + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(a.qhdr + 2, e1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        };
        if (item < a.n_rq) {
            const int64_t row0 = (int64_t)item * a.rq_rows;
            const int rows = (int)min((int64_t)a.rq_rows, padded_act_rows(M) - row0);
            rq_rows_coherent<FB>(a.fx, a.ldfx, M, row0, rows, a.K, const_cast<uint8_t *>(a.Xq),
                                 const_cast<float *>(a.xs), pool);
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's codes and scales written through
            __syncthreads();
            if (tid == 0) __hip_atomic_store(a.qflags + item, e1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            finish();
            return;
        }
        L = item - a.n_rq;
        // defer the finish count to the end of the tile (below)
    }
    int tm, tn;
    {
        const int gsz = kGroupM * a.tiles_n;
        const int g = L / gsz, r = L - g * gsz;
        const int m0 = g * kGroupM;
        const int gm = min(a.tiles_m - m0, kGroupM);
        tn = r / gm;
        tm = m0 + (r - tn * gm);
    }
    const int h0 = (nks + 1) >> 1;
    const int kb = half ? h0 : 0, len = half ? nks - h0 : h0;   // len >= 1 (nks >= 2)
    const int wunits_total = (int)(padded_rows(N) >> 5);
    const int xunits_total = (int)(padded_act_rows(M) >> 5);
    const uint8_t *usrc[C::UPW];
#pragma unroll
    for (int j = 0; j < C::UPW; ++j) {
        const int u = wm * C::UPW + j;
        if (u < C::W_UNITS) {
            const int ug = min(tn * C::W_UNITS + u, wunits_total - 1);
            usrc[j] = a.Wq + ((int64_t)ug * nks + kb) * 1024;
        } else {
            const int ux = min(tm * C::X_UNITS + (u - C::W_UNITS), xunits_total - 1);
            usrc[j] = a.Xq + ((int64_t)ux * nks + kb) * 1024;
        }
    }
    // stage k of this half into slot q; past the end the last stage is
    // loaded again (into a free slot, never read), so every wave issues the
    // same transfers and the wait counts stay fixed
    // (fused: the activation units were written in this launch, possibly on
    // another XCD, so they are read device-coherent, past this XCD's L2)
    auto produce = [&](int q, int k) {
        const uint32_t voff = (uint32_t)(min(k, len - 1) * 1024 + lane * 16);
        uint8_t *dst = &ring[half][q][0];
#pragma unroll
        for (int j = 0; j < C::UPW; ++j) {
            const uint8_t *sp = usrc[j] + voff;
            CLQ_LDS void *dp = (CLQ_LDS void *)(dst + (wm * C::UPW + j) * 1024);
            if (FB != 0 && wm * C::UPW + j >= C::W_UNITS)
                __builtin_amdgcn_global_load_lds(sp, dp, 16, 0, 16);
            else
                __builtin_amdgcn_global_load_lds(sp, dp, 16, 0, 0);
        }
    };
    v4u pa[C::FN], pb[C::FM];
    v4i a0[C::FN], b0[C::FM], a1[C::FN], b1[C::FM];
    const uint32_t wl0 = (uint32_t)(lane * 16);
    const uint32_t xl0 = (uint32_t)((C::W_UNITS + wm * C::FM) * 1024 + lane * 16);
    auto read_packed = [&](int q) {
        uint32_t wl = wl0, xl = xl0;
        asm volatile("" : "+v"(wl), "+v"(xl));
        wl += lds_addr(&ring[half][q][0]);
        xl += lds_addr(&ring[half][q][0]);
        static_for<0, C::FN>([&](auto f) { pa[f] = lds_read16<decltype(f)::value * 1024>(wl); });
        static_for<0, C::FM>([&](auto f) { pb[f] = lds_read16<decltype(f)::value * 1024>(xl); });
    };
    auto operands_ready = [&]() {
        static_assert(C::FN == 4 && C::FM == 2, "operand list below");
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(pa[0]), "+v"(pa[1]), "+v"(pa[2]), "+v"(pa[3]), "+v"(pb[0]), "+v"(pb[1]));
    };
    auto widen_half0 = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) a0[fn] = widen16(pa[fn][0], pa[fn][1]);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) b0[fm] = widen16(pb[fm][0], pb[fm][1]);
    };
    auto widen_half1 = [&]() {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn) a1[fn] = widen16(pa[fn][2], pa[fn][3]);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) b1[fm] = widen16(pb[fm][2], pb[fm][3]);
    };
    v16i acc[C::FN][C::FM];
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = v16i{};
    auto mma = [&](const v4i (&x)[C::FN], const v4i (&y)[C::FM]) {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(x[fn], y[fm], acc[fn][fm], 0, 0, 0);
    };
    // stage i+1 has landed once only the transfers of stage i+2 (NS - 3
    // later productions of UPW each) may be outstanding
    static_assert(NS == 4, "wait count below");
    auto landed_wait = [&]() {
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"((NS - 3) * C::UPW) : "memory");
    };

    // epilogue operands: loaded first (EPR per thread at clamped indices,
    // branch-free, ahead of the transfers), held in registers through the k
    // loop and written to LDS after it, when no transfer into LDS is in
    // flight (an LDS store during the transfers would wait for all of them)
    if constexpr (FB != 0) {
        // wait until the items holding this tile's token rows are published
        if (tid == 0) {
            const int64_t r0 = (int64_t)tm * C::BM;
            const int64_t r1 = min(r0 + C::BM, padded_act_rows(M)) - 1;
            const int i1 = (int)min(r1 / a.rq_rows, (int64_t)a.n_rq - 1);
            for (int i = (int)(r0 / a.rq_rows); i <= i1; ++i) {
                int spin = 0;
                while (__hip_atomic_load(a.qflags + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != e1) {
                    if (++spin > a.spin_limit) {   // reported, never expected (see above)
                        const int old = __hip_atomic_fetch_add(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if (old == 0) {
                            __hip_atomic_store(a.status + 1, L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            __hip_atomic_store(a.status + 2, i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        }
                        break;
                    }
                    __builtin_amdgcn_s_sleep(2);
                }
            }
        }
        __syncthreads();
    }
    constexpr int EPR = (EPN + 2 * C::NT - 1) / (2 * C::NT);
    float epv[EPR];
    _Float16 epb[EPR];
#pragma unroll
    for (int r = 0; r < EPR; ++r) {
        const int e = min(tid + r * 2 * C::NT, EPN - 1);
        const int ec = e & (C::BN - 1), er = max(e - 2 * C::BN, 0);
        const float *esrc = e < 2 * C::BN ? a.ws + min(tn * C::BN + ec, N - 1) : a.xs + min(tm * C::BM + er, M - 1);
        if constexpr (FB != 0)   // token scales written in this launch, possibly on another XCD
            epv[r] = __hip_atomic_load(esrc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else
            epv[r] = *esrc;
        epb[r] = (_Float16)0.0f;
        if constexpr (BIAS) epb[r] = reinterpret_cast<const _Float16 *>(a.bias)[min(tn * C::BN + ec, N - 1)];
    }
    __builtin_amdgcn_sched_barrier(0);
    for (int q = 0; q < NS - 1; ++q) produce(q, q);
    landed_wait();
    read_packed(0);
    operands_ready();
    widen_half0();
    // both halves take h0 steps; a second half one stage shorter idles on
    // its last step (wave-uniform)
    int i = 0;
    auto iter = [&](auto qc) -> bool {
        constexpr int q = decltype(qc)::value;
        constexpr int nq = (q + 1) % NS, pq = (q + NS - 1) % NS;
        const bool active = i < len;
        landed_wait();
        produce(pq, i + NS - 1);
        __builtin_amdgcn_sched_barrier(0);
        widen_half1();
        if (active) mma(a0, b0);
        read_packed(nq);
        __builtin_amdgcn_sched_barrier(0);
        operands_ready();
        widen_half0();
        if (active) mma(a1, b1);
        __builtin_amdgcn_sched_barrier(0);
        return ++i < h0;
    };
    while (iter(IC<0>{}) && iter(IC<1>{}) && iter(IC<2>{}) && iter(IC<3>{})) {
    }
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

    // the epilogue operands into LDS (a thread past the end writes the last
    // value again); the barrier after the sends below publishes them
#pragma unroll
    for (int r = 0; r < EPR; ++r) {
        const int e = min(tid + r * 2 * C::NT, EPN - 1);
        ep[e] = e >= C::BN && e < 2 * C::BN ? (float)epb[r] : epv[r];
    }

    // the halves swap sums through the idle rings: half 0 finishes channel
    // fragments 0-1 and half 1 fragments 2-3, each adding the other's
    // partial (16 KB per wave each way, 16-byte pieces with lanes consecutive)
    auto send = [&](auto f0c) {
        constexpr int f0 = decltype(f0c)::value;
        v4i *out = reinterpret_cast<v4i *>(pool + half * kExch);
        static_for<0, 2>([&](auto fc) {
            constexpr int f = decltype(fc)::value;
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const v16i &x = acc[f0 + f][fm];
                    out[(((wm * 2 + f) * C::FM + fm) * 4 + c) * 64 + lane] =
                        v4i{x[4 * c], x[4 * c + 1], x[4 * c + 2], x[4 * c + 3]};
                }
        });
    };
    auto receive = [&](auto f0c) {
        constexpr int f0 = decltype(f0c)::value;
        const v4i *in = reinterpret_cast<const v4i *>(pool + (1 - half) * kExch);
        static_for<0, 2>([&](auto fc) {
            constexpr int f = decltype(fc)::value;
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const v4i t = in[(((wm * 2 + f) * C::FM + fm) * 4 + c) * 64 + lane];
                    acc[f0 + f][fm][4 * c] += t[0];
                    acc[f0 + f][fm][4 * c + 1] += t[1];
                    acc[f0 + f][fm][4 * c + 2] += t[2];
                    acc[f0 + f][fm][4 * c + 3] += t[3];
                }
        });
    };
    if (half == 0) send(IC<2>{});
    else send(IC<0>{});
    __syncthreads();
    if (half == 0) receive(IC<0>{});
    else receive(IC<2>{});

    // epilogue: lane owns token m and 16 consecutive channels; each half
    // its two channel fragments
    const int h16 = (lane >> 5) * 16;
    auto epilogue = [&](auto f0c) {
    static_for<0, 2>([&](auto fc) {
        constexpr int fn = decltype(f0c)::value + decltype(fc)::value;
        const int c0 = fn * 32 + h16, n0 = tn * C::BN + c0;
        float wsv[16], bw[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            wsv[v] = ep_ws[c0 + v];
            bw[v] = BIAS ? ep_b[c0 + v] : 0.0f;
        }
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) {
            const int r0 = (wm * C::FM + fm) * 32 + (lane & 31), m = tm * C::BM + r0;
            const v16i &x = acc[fn][fm];
            if constexpr (I32OUT) {   // the exact integer sums
                int32_t *dst = reinterpret_cast<int32_t *>(a.Y) + (int64_t)m * a.ldy + n0;
                if (m < M && n0 < N) {
                    if (!RAGGED || n0 + 16 <= N) {
#pragma unroll
                        for (int q4 = 0; q4 < 4; ++q4)
                            reinterpret_cast<v4i *>(dst)[q4] =
                                v4i{x[4 * q4] >> 8, x[4 * q4 + 1] >> 8, x[4 * q4 + 2] >> 8, x[4 * q4 + 3] >> 8};
                    } else {
#pragma unroll
                        for (int v = 0; v < 16; ++v)
                            if (n0 + v < N) dst[v] = x[v] >> 8;
                    }
                }
                continue;
            }
            uint32_t hv[8];
            const float xsc = ep_xs[r0] * (1.0f / 256.0f);   // accumulators hold 256 * sum
#pragma unroll
            for (int v = 0; v < 16; v += 2) {
                const float p0 = (float)x[v] * xsc, p1 = (float)x[v + 1] * xsc;
                hv[v / 2] = fma_mix2f(p0, wsv[v], bw[v], p1, wsv[v + 1], bw[v + 1]);
            }
            uint16_t *dst = reinterpret_cast<uint16_t *>(a.Y) + (int64_t)m * a.ldy + n0;
            if (m < M && n0 < N) {
                if (!RAGGED || n0 + 16 <= N) {
                    reinterpret_cast<v4u *>(dst)[0] = v4u{hv[0], hv[1], hv[2], hv[3]};
                    reinterpret_cast<v4u *>(dst)[1] = v4u{hv[4], hv[5], hv[6], hv[7]};
                } else {
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        if (n0 + v < N) dst[v] = (uint16_t)(hv[v >> 1] >> (16 * (v & 1)));
                }
            }
        }
    });
    };
    if (half == 0) epilogue(IC<0>{});
    else epilogue(IC<2>{});
    if constexpr (FB != 0) {
        if (tid == 0) {
            const int done = __hip_atomic_fetch_add(a.qhdr + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (done == (int)gridDim.x - 1) {
                __hip_atomic_store(a.qhdr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(a.qhdr + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(a.qhdr + 2, e1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
}

// four waves of 128 channels x 64 tokens: 128 channels x 256 tokens per
// workgroup, two workgroups per compute unit
using TCfg = Tile<1, 4, 4, 2, 2>;
// the schedule counts channel tiles once for every kernel
static_assert(TCfg::BN == TileHalf128::BN && TCfg::BN == TileHalf64::BN, "one channel-tile width");

int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
    }
    return cus;
}

// Persistent grid: the workgroups that fit on the chip at once, a multiple of
// 8 (one equal share per XCD).
int full_grid() { return (device_cus() * TCfg::WGS + 7) / 8 * 8; }

// Splitting the last rounds along k costs each split tile a partial write and
// read per contributing workgroup (a few microseconds of latency on the
// critical path), so it is used only when it saves more than that: at least
// kSplitMinSaved k-stages per workgroup and a sixth of the whole-tile
// schedule, with shares of at least kSplitMinShare stages (a tile is then
// summed from at most nks / kSplitMinShare + 1 pieces).
constexpr int kSplitMinSaved = 16;
constexpr int kSplitMinShare = 8;
constexpr int kHalvesMinStages = 4;   // k-stages for the two-halves kernel

template <class C>
hipError_t launch_halves(const GemmArgs &g, bool i32out, bool bias, bool rag, hipStream_t stream) {
    const dim3 grid((unsigned)(g.tiles_m * g.tiles_n)), block(2 * C::NT);
    if (i32out && rag)
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, true, true, false>), grid, block, 0, stream, g);
    else if (i32out)
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, true, false, false>), grid, block, 0, stream, g);
    else if (bias && rag)
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, false, true, true>), grid, block, 0, stream, g);
    else if (bias)
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, false, false, true>), grid, block, 0, stream, g);
    else if (rag)
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, false, true, false>), grid, block, 0, stream, g);
    else
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, false, false, false>), grid, block, 0, stream, g);
    return hipGetLastError();
}

// The persistent kernel's schedule: whole tiles for all but the last one or
// two rounds; when that fills the chip badly (and a workspace is given) the
// rest is spread over every workgroup in k-stage units (1 to 2 tiles each).
void plan_persistent(int ntiles, int nks, bool may_split, int &dp, int &sk, int &grid) {
    grid = full_grid();
    dp = ntiles;
    sk = 0;
    if (may_split && ntiles % grid != 0) {
        const int d = max(0, ntiles / grid - 1) * grid;
        const int64_t whole = (int64_t)((ntiles + grid - 1) / grid) * nks;
        const int64_t split = (int64_t)(d / grid) * nks + ((int64_t)(ntiles - d) * nks + grid - 1) / grid;
        const bool share_ok = (int64_t)(ntiles - d) * nks >= (int64_t)kSplitMinShare * grid;
        if (share_ok && whole - split > kSplitMinSaved && 6 * (whole - split) > whole) {
            dp = d;
            sk = (ntiles - d) * nks;
        }
    }
    if (sk == 0) grid = max(8, (min(ntiles, grid) + 7) / 8 * 8);
}

template <class C, bool I32OUT, bool RAGGED, bool BIAS, bool ERR = false>
hipError_t launch_cfg(GemmArgs g, bool may_split, hipStream_t stream) {
    int grid;
    plan_persistent(g.tiles_m * g.tiles_n, g.K >> 6, may_split, g.dp, g.sk, grid);
    g.full_grid = full_grid();
    hipLaunchKernelGGL((w4a4_gemm_kernel<C, I32OUT, RAGGED, BIAS, ERR>), dim3((unsigned)grid), dim3(C::NT), 0, stream, g);
    return hipGetLastError();
}

}  // namespace

int gemm_schedule_knob() { return __atomic_load_n(&gemm_force_schedule, __ATOMIC_RELAXED); }

GemmPlan plan_gemm(int64_t M, int64_t N, int K, bool may_split) { return plan_gemm(M, N, K, may_split, gemm_schedule_knob()); }

// force: 0 automatic, 1 persistent, 2 persistent whole tiles, 3 / 4 the
// two-halves kernel on 128- / 64-token tiles (the debug knob)
GemmPlan plan_gemm(int64_t M, int64_t N, int K, bool may_split, int force) {
    GemmPlan p{};
    const int tiles_n = (int)((N + TCfg::BN - 1) / TCfg::BN);
    const int ntiles = (int)((M + TCfg::BM - 1) / TCfg::BM) * tiles_n;
    const bool halves_ok = (K >> 6) >= kHalvesMinStages;
    // the two-halves kernel: at most 1.25 256-token tiles per compute unit
    // (just past one tile per CU the persistent kernel doubles up on a few
    // CUs while the rest idle; the two-halves kernel fills one round of two
    // workgroups per CU and runs a short second round on the remaining
    // quarter at most), or long k loops (K >= 2048).  On such loops its
    // 128-token tiles with the k range split between two halves of the
    // workgroup beat the persistent kernel at every tile count measured,
    // 2-16% (the schedule sweep over 36 shapes from 512 to 24576 tokens),
    // except on layers more than four times wider than deep at more than 8
    // tiles per compute unit, where the persistent kernel's grouped weight
    // reuse wins.
    const bool deep = K >= 2048 && (N < 4 * (int64_t)K || ntiles <= 8 * device_cus());
    const bool halves = halves_ok && (force >= 3 || (force == 0 && (4 * ntiles <= 5 * device_cus() || deep)));
    if (halves) {
        // 128-token tiles (two four-wave workgroups per compute unit), or 64
        // while those would fill at most half the compute units
        const int tm128 = (int)((M + TileHalf128::BM - 1) / TileHalf128::BM);
        if (force == 4 || (force != 3 && 2 * tm128 * tiles_n <= device_cus())) {
            p.kernel = 2;
            p.tiles_m = (int)((M + TileHalf64::BM - 1) / TileHalf64::BM);
        } else {
            p.kernel = 1;
            p.tiles_m = tm128;
        }
        p.tiles = p.tiles_m * tiles_n;
        p.dp = p.tiles;
        p.grid = p.tiles;
        return p;
    }
    p.kernel = 0;
    p.tiles_m = (int)((M + TCfg::BM - 1) / TCfg::BM);
    p.tiles = ntiles;
    p.may_split = may_split && force != 2;
    plan_persistent(ntiles, K >> 6, p.may_split, p.dp, p.sk, p.grid);
    return p;
}

// Workspace: status words (the first three for the split-k report, words
// 4..6 the fused variant's queue, finished count and epoch) | one flag per
// wave of every persistent workgroup | one partial tile per workgroup | one
// flag per rotate+quantize item of the fused variant.
constexpr int kRqFlagInts = 1 << 18;
constexpr int kFusedMinRows = 4;   // rows per rotate+quantize item of the fused variant

size_t gemm_split_bytes() {
    const size_t G = (size_t)full_grid();
    return kStatusBytes + G * TCfg::NW * sizeof(int) + G * TCfg::PART_INTS * sizeof(int32_t);
}

size_t gemm_workspace_bytes() { return gemm_split_bytes() + (size_t)kRqFlagInts * sizeof(int); }

int gemm_spin_limit = kSpinLimit;
int gemm_force_schedule = 0;
int gemm_drop_signal = 0;

// ---- the allocation-free GEMM entry point's scratch ---------------------------
// The workspace of the split schedule (status words, flags, one partial tile
// per workgroup) for grids of up to kScratchGrid workgroups (256 compute
// units), held by the library: each device the library runs on keeps its own
// copy for the life of the process.  Host code reaches it only through the
// address hipGetSymbolAddress returns for the current device.
constexpr int kScratchGrid = 512;
constexpr size_t kScratchBytes =
    kStatusBytes + (size_t)kScratchGrid * TCfg::NW * sizeof(int) + (size_t)kScratchGrid * TCfg::PART_INTS * sizeof(int32_t);
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
void *scratch_ptr[kMaxDevices];   // per device, set once
std::mutex scratch_mu;

// clears the status words and flags before a split launch (a fill kernel,
// not a memset: callers may capture the call in a graph)
__global__ void clear_words_kernel(int *p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// the call's status words (zeros when the call did not split)
__global__ void status_copy_kernel(const int *hdr, int *out, int split) {
    const int i = threadIdx.x;
    if (i < 3) out[i] = split ? hdr[i] : 0;
}

hipError_t device_scratch(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

size_t gemm_scratch_bytes() { return kScratchBytes; }

hipError_t launch_gemm_noalloc(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                               const uint16_t *bias, int64_t M, int64_t N, int K, void *Y, int64_t ldy,
                               int32_t *status, hipStream_t stream) {
    if (gemm_split_bytes() > kScratchBytes) return hipErrorInvalidValue;   // more CUs than the scratch serves
    void *sp = nullptr;
    hipError_t e = device_scratch(&sp);
    if (e != hipSuccess) return e;
    const int force = gemm_schedule_knob();
    const GemmPlan pl = plan_gemm(M, N, K, true, force);
    const int split = pl.sk > 0;
    if (split) {
        // status words and flags start at zero on every split call
        const int nwords = (int)((kStatusBytes + (size_t)full_grid() * TCfg::NW * sizeof(int)) / sizeof(int));
        hipLaunchKernelGGL(clear_words_kernel, dim3((nwords + 255) / 256), dim3(256), 0, stream,
                           reinterpret_cast<int *>(sp), nwords);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    e = launch_gemm(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, false, sp, stream, force);
    if (e != hipSuccess || status == nullptr) return e;
    hipLaunchKernelGGL(status_copy_kernel, dim3(1), dim3(64), 0, stream, reinterpret_cast<const int *>(sp), status,
                       split);
    return hipGetLastError();
}

hipError_t launch_gemm(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                       const uint16_t *bias, int64_t M, int64_t N, int K, void *Y, int64_t ldy,
                       bool i32out, void *workspace, hipStream_t stream) {
    return launch_gemm(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, i32out, workspace, stream, gemm_schedule_knob());
}

hipError_t launch_gemm(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                       const uint16_t *bias, int64_t M, int64_t N, int K, void *Y, int64_t ldy,
                       bool i32out, void *workspace, hipStream_t stream, int force) {
    GemmArgs g{};
    g.Xq = Xq;
    g.xs = xs;
    g.Wq = Wq;
    g.ws = ws;
    g.bias = bias;
    g.Y = Y;
    g.ldy = ldy;
    g.M = (int)M;
    g.N = (int)N;
    g.K = K;
    g.tiles_m = (int)((M + TCfg::BM - 1) / TCfg::BM);
    g.tiles_n = (int)((N + TCfg::BN - 1) / TCfg::BN);
    const size_t G = (size_t)full_grid();
    // workspace: status words | one flag per wave of every workgroup | one
    // partial tile per workgroup
    uint8_t *wsb = reinterpret_cast<uint8_t *>(workspace);
    g.status = workspace ? reinterpret_cast<int *>(wsb) : nullptr;
    g.flags = workspace ? reinterpret_cast<int *>(wsb + kStatusBytes) : nullptr;
    g.part = workspace ? reinterpret_cast<int32_t *>(wsb + kStatusBytes + G * TCfg::NW * sizeof(int)) : nullptr;
    g.spin_limit = __atomic_load_n(&gemm_spin_limit, __ATOMIC_RELAXED);
    g.drop_signal = __atomic_load_n(&gemm_drop_signal, __ATOMIC_RELAXED);
    const GemmPlan pl = plan_gemm(M, N, K, workspace != nullptr, force);
    const bool may_split = pl.may_split;
    if (pl.kernel == 2) {
        g.tiles_m = pl.tiles_m;
        return launch_halves<TileHalf64>(g, i32out, bias != nullptr, N % 16 != 0, stream);
    }
    if (pl.kernel == 1) {
        g.tiles_m = pl.tiles_m;
        return launch_halves<TileHalf128>(g, i32out, bias != nullptr, N % 16 != 0, stream);
    }
    // ragged channel edges, and biases not 4-byte aligned (the fast path
    // moves them in channel pairs), use element-wise epilogue accesses
    const bool ragged = N % 16 != 0 || (bias && reinterpret_cast<uintptr_t>(bias) % 4 != 0);
    if (i32out)
        return ragged ? launch_cfg<TCfg, true, true, false>(g, may_split, stream)
                      : launch_cfg<TCfg, true, false, false>(g, may_split, stream);
    if (ragged)
        return bias ? launch_cfg<TCfg, false, true, true>(g, may_split, stream)
                    : launch_cfg<TCfg, false, true, false>(g, may_split, stream);
    return bias ? launch_cfg<TCfg, false, false, true>(g, may_split, stream)
                : launch_cfg<TCfg, false, false, false>(g, may_split, stream);
}

namespace {

template <class C, int FB>
hipError_t launch_fused(const GemmArgs &g, bool bias, hipStream_t stream) {
    const dim3 grid((unsigned)(g.n_rq + g.tiles_m * g.tiles_n)), block(2 * C::NT);
    if (bias)
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, false, false, true, FB>), grid, block, 0, stream, g);
    else
        hipLaunchKernelGGL((w4a4_gemm_halves_kernel<C, false, false, false, FB>), grid, block, 0, stream, g);
    return hipGetLastError();
}

template <class C>
hipError_t launch_fused_b(const GemmArgs &g, int block, bool bias, hipStream_t stream) {
    switch (block) {
        case 32: return launch_fused<C, 32>(g, bias, stream);
        case 64: return launch_fused<C, 64>(g, bias, stream);
        case 128: return launch_fused<C, 128>(g, bias, stream);
    }
    return hipErrorInvalidValue;
}

// LDS bytes of the two-halves kernel's ring pool (the fused items stage
// their fp16 rows there)
template <class C>
constexpr int halves_pool_bytes() {
    return 2 * kHalfStages * C::STAGE_BYTES > 2 * C::NW * 16384 ? 2 * kHalfStages * C::STAGE_BYTES
                                                                 : 2 * C::NW * 16384;
}

}  // namespace

RqGemmPlan plan_rq_gemm(int64_t M, int64_t N, int K, int block, bool have_workspace) {
    RqGemmPlan p{};
    const GemmPlan g = plan_gemm(M, N, K, false);
    if (!have_workspace || (g.kernel != 1 && g.kernel != 2) || N % 16 != 0) return p;
    const int T = g.kernel == 2 ? 2 * TileHalf64::NT : 2 * TileHalf128::NT;
    const int pool = g.kernel == 2 ? halves_pool_bytes<TileHalf64>() : halves_pool_bytes<TileHalf128>();
    const int nb = K / block;
    int R = min(T / nb, pool / (K * 2 + 4));
    // items of fewer rows leave most of a workgroup idle on a latency-bound
    // load: long rows take the two launches
    if (R < kFusedMinRows) return p;
    const int64_t mpad = padded_act_rows(M);
    const int64_t n_rq = (mpad + R - 1) / R;
    if (n_rq > kRqFlagInts) return p;
    p.fused = 1;
    p.kernel = g.kernel;
    p.tiles = g.tiles;
    p.rq_rows = R;
    p.n_rq = (int)n_rq;
    return p;
}

hipError_t launch_rq_gemm(const uint16_t *X, int64_t ldx, int block, uint8_t *Xq, float *xs, const uint8_t *Wq,
                          const float *ws, const uint16_t *bias, int64_t M, int64_t N, int K, void *Y,
                          int64_t ldy, void *workspace, hipStream_t stream) {
    const RqGemmPlan p = plan_rq_gemm(M, N, K, block, workspace != nullptr);
    if (!p.fused) {   // two launches: rotate+quantize, then the linear
        hipError_t e = launch_rotate_quant(X, ldx, nullptr, M, padded_act_rows(M), K, block, 1.0f, false, 1.0f,
                                           Xq, xs, stream);
        if (e != hipSuccess) return e;
        return launch_gemm(Xq, xs, Wq, ws, bias, M, N, K, Y, ldy, false, workspace, stream);
    }
    GemmArgs g{};
    g.Xq = Xq;
    g.xs = xs;
    g.Wq = Wq;
    g.ws = ws;
    g.bias = bias;
    g.Y = Y;
    g.ldy = ldy;
    g.M = (int)M;
    g.N = (int)N;
    g.K = K;
    g.tiles_n = (int)((N + TCfg::BN - 1) / TCfg::BN);
    g.tiles_m = p.tiles / g.tiles_n;
    uint8_t *wsb = reinterpret_cast<uint8_t *>(workspace);
    g.status = reinterpret_cast<int *>(wsb);
    g.qhdr = reinterpret_cast<int *>(wsb) + 4;
    g.qflags = reinterpret_cast<int *>(wsb + gemm_split_bytes());
    g.spin_limit = __atomic_load_n(&gemm_spin_limit, __ATOMIC_RELAXED);
    g.fx = X;
    g.ldfx = ldx;
    g.rq_rows = p.rq_rows;
    g.n_rq = p.n_rq;
    if (p.kernel == 2) return launch_fused_b<TileHalf64>(g, block, bias != nullptr, stream);
    return launch_fused_b<TileHalf128>(g, block, bias != nullptr, stream);
}

int64_t gemm_err_partials(int64_t M, int64_t N) {
    return ((M + TCfg::BM - 1) / TCfg::BM) * ((N + TCfg::BN - 1) / TCfg::BN) * TCfg::NW;
}

hipError_t launch_gemm_err(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                           int64_t M, int64_t N, int K, const float *Y0, int64_t ldy0, double *partials,
                           hipStream_t stream) {
    GemmArgs g{};
    g.Xq = Xq;
    g.xs = xs;
    g.Wq = Wq;
    g.ws = ws;
    g.M = (int)M;
    g.N = (int)N;
    g.K = K;
    g.tiles_m = (int)((M + TCfg::BM - 1) / TCfg::BM);
    g.tiles_n = (int)((N + TCfg::BN - 1) / TCfg::BN);
    g.y0 = Y0;
    g.ldy0 = ldy0;
    g.errp = partials;
    // whole tiles (no workspace): each tile's partials come from its one epilogue
    const bool ragged = N % 16 != 0 || ldy0 % 4 != 0 || reinterpret_cast<uintptr_t>(Y0) % 16 != 0;
    return ragged ? launch_cfg<TCfg, false, true, false, true>(g, false, stream)
                  : launch_cfg<TCfg, false, false, false, true>(g, false, stream);
}

}  // namespace clq
