// W4A4 GEMM on the fp6 matrix cores of gfx950, with the dequantising
// epilogue fused (CLQ, arXiv 2509.24416: the integer product of the W4A4
// codes, rescaled by the per-token activation scale and the per-channel
// weight scale of Eq. (1), plus bias).
//
// Codes carried as fp6.  gfx950 has no 4-bit integer matrix instruction.  Its
// fp6 format e2m3 (1 sign, 2 exponent, 3 mantissa bits, bias 1) holds every
// code of the 4-bit grid, -7..7, exactly, and v_mfma_f32_32x32x64_f8f6f4 on
// two fp6 operands multiplies them at twice the int8 instruction's rate.
// Each product of two codes is an integer of magnitude at most 49, and every
// partial sum of a k loop shorter than 2^24 / 49 codes is an integer below
// 2^24, which fp32 holds exactly: the accumulators are the exact integers
// sum_k qa * qw, whatever the order of the additions.
//
// fp6 code layout (weights and activations): the unit and lane map of the
// packed int4 layouts (32 rows x 64 codes per unit, lane l = 32h + rho
// holding codes 32h .. 32h+31 of fragment row rho; weights with their
// fragment-row order, so that accumulator element v of lane l is channel
// 16 (l / 32) + v of the fragment), 24 bytes per lane: code i of the lane's
// 32 at bits 6i .. 6i+5 of its 192 bits (f6_codes.h).  A unit is 1536
// bytes: lane l's first 16 bytes at 16 l, its last 8 after the first 1 KB
// (aligned LDS reads of 16 and 8 bytes; the transfer into LDS is one 16-byte
// load per lane for the first 1 KB and one 16-byte load on 32 lanes for the
// rest).  Units are stored [row unit][k unit].
//
// The kernel is the persistent W4A4 kernel's pipeline (see w4a4_gemm.hip)
// with 1536-byte units, one matrix instruction per fragment and k-stage of
// 64 codes, no operand widening, and a 4-slot ring: the slot of stage s is
// refilled with stage s + 4 in iteration s, its contents having been read
// into registers in iteration s - 1 (the workgroup barrier of iteration s
// orders those reads before the transfer).  Whole tiles only: 128 channels by
// 256 tokens, or by 128 tokens where the larger tiles would leave compute
// units without a tile.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "clq_internal.h"
#include "f6_codes.h"

#define CLQ_LDS __attribute__((address_space(3)))

namespace clq {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
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
template <int OFF>
__device__ __forceinline__ v2u lds_read8(uint32_t addr) {
    v2u v;
    asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
}
template <int I, int N, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, N>(f);
    }
}

// two fp16 outputs fma(p, w, bias) rounded once from fp32 operands and a
// packed fp16 bias pair (low half: first output)
__device__ __forceinline__ uint32_t fma_mix2(float p0, float w0, float p1, float w1, uint32_t b) {
    uint32_t r;
    asm("v_fma_mixlo_f16 %0, %1, %2, %3 op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixhi_f16 %0, %4, %5, %3 op_sel:[0,0,1] op_sel_hi:[0,0,1]"
        : "=&v"(r)
        : "v"(p0), "v"(w0), "v"(b), "v"(p1), "v"(w1));
    return r;
}

constexpr int kUnit = kF6Unit;  // bytes of a 32 x 64 fp6 unit
constexpr int kNS = 4;          // ring slots
constexpr int kGroupM = 8;      // token panels per tile group (L2 reuse of channel panels)

// Tile shape of the persistent kernel: four waves, each 128 channels (4
// fragments of 32) by FM fragments of 32 tokens; two workgroups per compute
// unit.
template <int FM_>
struct F6Tile {
    static constexpr int WN = 1, WM = 4, FN = 4, FM = FM_;
    static constexpr int NW = WN * WM, NT = NW * 64;
    static constexpr int BN = WN * FN * 32, BM = WM * FM * 32;
    static constexpr int WUnits = BN / 32, XUnits = BM / 32, Units = WUnits + XUnits;
    static constexpr int UPW = Units / NW;   // units per wave and stage
    static constexpr int VPW = 2 * UPW;      // transfers per wave and stage
    static constexpr int Slot = Units * kUnit;
    static_assert(Units % NW == 0, "units split evenly over waves");
};
using F6Tile256 = F6Tile<2>;   // 128 channels x 256 tokens

// global -> LDS transfers of 16 and 4 bytes per lane (plain functions, so that
// the builtin's operands never depend on a template parameter, which the
// host compilation pass does not accept)
__device__ __forceinline__ void dma_lds16(const uint8_t *src, uint8_t *dst) {
    __builtin_amdgcn_global_load_lds(src, (CLQ_LDS void *)dst, 16, 0, 0);
}
__device__ __forceinline__ void dma_lds4(const uint8_t *src, uint8_t *dst) {
    __builtin_amdgcn_global_load_lds(src, (CLQ_LDS void *)dst, 4, 0, 0);
}

// waits for all but N outstanding transfers (and the LDS reads), then the
// workgroup barrier
template <int N>
__device__ __forceinline__ void wait_landed_barrier() {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

struct F6Args {
    const uint8_t *Xq;
    const float *xs;
    const uint8_t *Wq;
    const float *ws;
    const uint16_t *bias;
    void *Y;
    int64_t ldy;
    int M, N, K, tiles_m, tiles_n;
};

struct Seg {
    int j, L, k;
};

// The LDS reads of one stage's operands have landed: one wait that names
// every destination register, so that no use is scheduled before it.
template <int FM>
__device__ __forceinline__ void wait_operands(v4u (&ra)[4], v4u (&rb)[FM], v2u (&sa)[4], v2u (&sb)[FM]) {
    static_assert(FM == 1 || FM == 2, "operand lists below");
    if constexpr (FM == 2)
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(ra[0]), "+v"(ra[1]), "+v"(ra[2]), "+v"(ra[3]), "+v"(rb[0]), "+v"(rb[1]),
                       "+v"(sa[0]), "+v"(sa[1]), "+v"(sa[2]), "+v"(sa[3]), "+v"(sb[0]), "+v"(sb[1]));
    else
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(ra[0]), "+v"(ra[1]), "+v"(ra[2]), "+v"(ra[3]), "+v"(rb[0]),
                       "+v"(sa[0]), "+v"(sa[1]), "+v"(sa[2]), "+v"(sa[3]), "+v"(sb[0]));
}

template <class C, bool I32OUT, bool RAGGED, bool BIAS>
__global__ void __launch_bounds__(C::NT, 2) f6_gemm_kernel(F6Args a)
{
    constexpr int NS = kNS;
    constexpr int kFN = C::FN, kFM = C::FM, kNW = C::NW, kBN = C::BN, kBM = C::BM;
    constexpr int kWUnits = C::WUnits, kXUnits = C::XUnits, kUPW = C::UPW, kVPW = C::VPW, kSlot = C::Slot;
    constexpr bool BIAS_CH = BIAS && !RAGGED && !I32OUT;
    constexpr int XS_CH = kBM / 64, WS_CH = kBN / 64, B_CH = kBN / 128;
    constexpr int E_CH = I32OUT ? 0 : XS_CH + WS_CH + (BIAS_CH ? B_CH : 0);
    constexpr int EPW = (E_CH + kNW - 1) / kNW;
    constexpr int E_XS = 0, E_WS = E_XS + kBM * 4, E_B = E_WS + kBN * 4;
    constexpr int E_BYTES = I32OUT ? 16 : E_B + (BIAS_CH ? kBN * 2 : 0);
    __shared__ __align__(16) uint8_t ring0[kSlot], ring1[kSlot], ring2[kSlot], ring3[kSlot];
    __shared__ __align__(16) uint8_t ebuf[NS][E_BYTES];
    auto slot = [&](auto qc) -> uint8_t * {
        constexpr int q = decltype(qc)::value;
        if constexpr (q == 0) return ring0;
        else if constexpr (q == 1) return ring1;
        else if constexpr (q == 2) return ring2;
        else return ring3;
    };

    const int M = a.M, N = a.N, nks = a.K >> 6;
    const int G = gridDim.x, gx = G >> 3, xcd = blockIdx.x & 7, jw = blockIdx.x >> 3;
    const int ntiles = a.tiles_m * a.tiles_n;
    const int per = ntiles >> 3, rem = ntiles & 7;
    const int cnt = per + (xcd < rem ? 1 : 0);
    const int dstart = xcd * per + min(xcd, rem);
    const int my_tiles = jw < cnt ? (cnt - jw + gx - 1) / gx : 0;
    const int total = my_tiles * nks;
    if (total == 0) return;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave;   // one channel panel per tile
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
    auto next_seg = [&](Seg &c) {
        ++c.j;
        c.L = dstart + jw + c.j * gx;
        c.k = 0;
    };

    // ---- producer -------------------------------------------------------------
    Seg pc{-1, 0, 0};
    next_seg(pc);
    int p_s = 0;
    const uint8_t *usrc[C::UPW];
    const uint8_t *esrc[EPW > 0 ? EPW : 1];
    int edst[EPW > 0 ? EPW : 1];
    auto p_setup = [&]() {
        int tm, tn;
        coords(pc.L, tm, tn);
#pragma unroll
        for (int j = 0; j < kUPW; ++j) {
            const int u = wave * kUPW + j;
            if (u < kWUnits) {
                const int ug = min(tn * kWUnits + u, wunits_total - 1);
                usrc[j] = a.Wq + (int64_t)ug * nks * kUnit;
            } else {
                const int ux = min(tm * kXUnits + (u - kWUnits), xunits_total - 1);
                usrc[j] = a.Xq + (int64_t)ux * nks * kUnit;
            }
        }
#pragma unroll
        for (int j = 0; j < EPW; ++j) {
            const int c = wave * EPW + j;
            if (c < XS_CH) {
                esrc[j] = reinterpret_cast<const uint8_t *>(a.xs + min(tm * kBM + c * 64 + lane, M - 1));
                edst[j] = E_XS + c * 256;
            } else if (c < XS_CH + WS_CH || c >= E_CH) {
                const int w = (c - XS_CH) % WS_CH;
                esrc[j] = reinterpret_cast<const uint8_t *>(a.ws + min(tn * kBN + w * 64 + lane, N - 1));
                edst[j] = E_WS + w * 256;
            } else {
                const int b = c - XS_CH - WS_CH;
                esrc[j] = reinterpret_cast<const uint8_t *>(reinterpret_cast<const uint32_t *>(a.bias) +
                                                            min(tn * (kBN / 2) + b * 64 + lane, N / 2 - 1));
                edst[j] = E_B + b * 256;
            }
        }
    };
    p_setup();
    int e_next = 0;        // stage whose production carries the next tile's epilogue operands
    unsigned phist = 0;    // 1 bit per production call: epilogue operands issued
    auto produce = [&](auto qc) {
        // the tile's epilogue operands go out with its first stage, ahead of
        // the units (the wait counts below rely on that order)
        int e_now = 0;
        if (EPW > 0 && pc.k == 0 && p_s == e_next) {
            uint8_t *ed = &ebuf[pc.j % NS][0];
#pragma unroll
            for (int j = 0; j < EPW; ++j)
                dma_lds4(esrc[j], ed + edst[j]);
            e_now = 1;
            e_next = -1;
        }
        phist = (phist << 1) | e_now;
        uint8_t *dst = slot(qc);
        const uint32_t voff = (uint32_t)(pc.k * kUnit + lane * 16);
#pragma unroll
        for (int j = 0; j < kUPW; ++j)
            dma_lds16(usrc[j] + voff, dst + (wave * kUPW + j) * kUnit);
        // the units' last 512 bytes: 16 bytes on each of lanes 0..31
        if (lane < 32) {
#pragma unroll
            for (int j = 0; j < kUPW; ++j)
                dma_lds16(usrc[j] + voff + 1024, dst + (wave * kUPW + j) * kUnit + 1024);
        }
        if (p_s < total - 1) {
            ++p_s;
            if (++pc.k == nks) {
                next_seg(pc);
                p_setup();
                e_next = p_s;
            }
        }
    };

    // ---- consumer -------------------------------------------------------------
    // operands of one stage: 16 + 8 bytes of each of the wave's 4 channel and
    // 2 token units, in two register sets used by alternate stages (stage s
    // in set s & 1), so that the next stage's reads land while the matrix
    // instructions read the other set, with no copies between them.  The
    // ragged-shape instances, whose epilogue needs more registers, read into
    // set 1 and copy it to set 0 at the start of each iteration instead.
    constexpr bool kAlt = !RAGGED;
    v4u ra[2][kFN], rb[2][kFM];
    v2u sa[2][kFN], sb[2][kFM];
    const uint32_t wl0 = (uint32_t)(lane * 16), wl1 = (uint32_t)f6_tail_offset(lane);
    auto read_stage = [&](auto qc, auto pc) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        uint32_t b16 = wl0, b8 = wl1;
        asm volatile("" : "+v"(b16), "+v"(b8));
        b16 += lds_addr(slot(qc));
        b8 += lds_addr(slot(qc));
        // this wave's token units: the offset exceeds the 16-bit immediate
        // range for the later waves, so it goes into the address
        const uint32_t xo = (uint32_t)((kWUnits + wm * kFM) * kUnit);
        const uint32_t bx16 = b16 + xo, bx8 = b8 + xo;
        static_for<0, kFN>([&](auto f) {
            constexpr int o = decltype(f)::value * kUnit;
            ra[P][f] = lds_read16<o>(b16);
            sa[P][f] = lds_read8<o>(b8);
        });
        static_for<0, kFM>([&](auto f) {
            constexpr int o = decltype(f)::value * kUnit;
            rb[P][f] = lds_read16<o>(bx16);
            sb[P][f] = lds_read8<o>(bx8);
        });
    };
    auto stage_ready = [&](auto pc) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        wait_operands(ra[P], rb[P], sa[P], sb[P]);
    };
    v16f acc[kFN][kFM];
    auto zero_acc = [&]() {
#pragma unroll
        for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm) acc[fn][fm] = v16f{};
    };
    // format codes 2, 2: both operands fp6 e2m3; no block scales
    auto mma = [&](auto pc) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        v8i opa[kFN], opb[kFM];
#pragma unroll
        for (int f = 0; f < kFN; ++f)
            opa[f] = v8i{(int)ra[P][f][0], (int)ra[P][f][1], (int)ra[P][f][2], (int)ra[P][f][3],
                         (int)sa[P][f][0], (int)sa[P][f][1], 0, 0};
#pragma unroll
        for (int f = 0; f < kFM; ++f)
            opb[f] = v8i{(int)rb[P][f][0], (int)rb[P][f][1], (int)rb[P][f][2], (int)rb[P][f][3],
                         (int)sb[P][f][0], (int)sb[P][f][1], 0, 0};
#pragma unroll
        for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opa[fn], opb[fm], acc[fn][fm], 2, 2, 0, 0, 0, 0);
    };

    // ---- epilogue: lane owns token m and 16 consecutive channels ----------------
    const int h16 = (lane >> 5) * 16;
    // always inlined: an outlined epilogue takes the accumulators by reference
    // (through memory) and the ragged-shape instances then spill
    auto epilogue = [&](int L, int sj) __attribute__((always_inline)) {
        int tm, tn;
        coords(L, tm, tn);
        uint32_t lx = (uint32_t)((wm * kFM * 32 + (lane & 31)) * 4);
        uint32_t lw = (uint32_t)(h16 * 4);
        asm volatile("" : "+v"(lx), "+v"(lw));
        const uint32_t sbase = lds_addr(&ebuf[0][0]) + (uint32_t)((sj % NS) * E_BYTES);
        const uint32_t axs = sbase + E_XS + lx, aws = sbase + E_WS + lw, ab = sbase + E_B + lw / 2;
        float xsm[kFM];
        int mrow[kFM];
        if constexpr (!I32OUT) {
            if constexpr (kFM == 2)
                asm volatile("ds_read_b32 %0, %2\n\tds_read_b32 %1, %2 offset:128\n\ts_waitcnt lgkmcnt(0)"
                             : "=&v"(xsm[0]), "=&v"(xsm[1]) : "v"(axs));
            else
                asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=&v"(xsm[0]) : "v"(axs));
        }
#pragma unroll
        for (int fm = 0; fm < kFM; ++fm) mrow[fm] = tm * kBM + (wm * kFM + fm) * 32 + (lane & 31);
        const int nl = tn * kBN + h16;
        uint16_t *rowp[kFM];
#pragma unroll
        for (int fm = 0; fm < kFM; ++fm) rowp[fm] = reinterpret_cast<uint16_t *>(a.Y) + (int64_t)mrow[fm] * a.ldy + nl;
        static_for<0, kFN>([&](auto fc) {
            constexpr int fn = decltype(fc)::value;
            const int n0 = nl + fn * 32;
            v4f w4[4];
            v4u b8[2];
            if constexpr (!I32OUT) {
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
            float wsv[16];
            uint32_t bw[8];
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
                    bw[v / 2] = (uint32_t)a.bias[na] | ((uint32_t)a.bias[nb] << 16);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 8; ++v) bw[v] = b8[v / 4][v % 4];
            }
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm) {
                const int m = mrow[fm];
                const v16f &x = acc[fn][fm];
                if constexpr (I32OUT) {
                    int32_t *dst = reinterpret_cast<int32_t *>(a.Y) + (int64_t)m * a.ldy + n0;
                    if (m < M && n0 < N) {
                        if (!RAGGED || n0 + 16 <= N) {
#pragma unroll
                            for (int q4 = 0; q4 < 4; ++q4)
                                reinterpret_cast<v4i *>(dst)[q4] =
                                    v4i{(int)x[4 * q4], (int)x[4 * q4 + 1], (int)x[4 * q4 + 2], (int)x[4 * q4 + 3]};
                        } else {
#pragma unroll
                            for (int v = 0; v < 16; ++v)
                                if (n0 + v < N) dst[v] = (int)x[v];
                        }
                    }
                } else {
                    uint32_t hv[8];
#pragma unroll
                    for (int v = 0; v < 16; v += 2)
                        hv[v / 2] = fma_mix2(x[v] * xsm[fm], wsv[v], x[v + 1] * xsm[fm], wsv[v + 1], bw[v / 2]);
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
    };

    // Stage s+1 has landed once at most the VMEM instructions issued after
    // its last transfer are outstanding (completion is in issue order): the
    // two later productions, with their epilogue operand transfers if any.
    // Epilogue stores are not counted, which only makes the wait stricter.
    constexpr int W0 = 2 * kVPW;
    auto landed_wait = [&]() {
        switch (__builtin_popcount(phist & 3u)) {
            case 0: asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(W0) : "memory"); break;
            case 1: asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(W0 + EPW) : "memory"); break;
            default: asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(W0 + 2 * EPW) : "memory"); break;
        }
    };

    // ---- pipeline ---------------------------------------------------------------
    // prologue: stages 0..3 in flight, stage 0 read into registers
    produce(IC<0>{});
    produce(IC<1>{});
    produce(IC<2>{});
    produce(IC<3>{});
    // stage 0 landed: the three later productions may be outstanding
    switch (__builtin_popcount(phist & 7u)) {
        case 0: asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(3 * kVPW) : "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(3 * kVPW + EPW) : "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(3 * kVPW + 2 * EPW) : "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(3 * kVPW + 3 * EPW) : "memory"); break;
    }
    read_stage(IC<0>{}, IC<kAlt ? 0 : 1>{});
    stage_ready(IC<kAlt ? 0 : 1>{});
    zero_acc();

    Seg cc{-1, 0, 0};
    next_seg(cc);
    int s = 0;
    auto iter = [&](auto qc) __attribute__((always_inline)) -> bool {
        constexpr int q = decltype(qc)::value;
        constexpr IC<(q + 1) % NS> nqc{};
        constexpr IC<kAlt ? (q & 1) : 0> cur{};
        constexpr IC<kAlt ? ((q + 1) & 1) : 1> nxt{};
        static_assert(NS % 2 == 0, "stage s uses register set s & 1 across the ring's wrap");
        if constexpr (!kAlt) {
#pragma unroll
            for (int f = 0; f < kFN; ++f) {
                ra[0][f] = ra[1][f];
                sa[0][f] = sa[1][f];
            }
#pragma unroll
            for (int f = 0; f < kFM; ++f) {
                rb[0][f] = rb[1][f];
                sb[0][f] = sb[1][f];
            }
        }
        landed_wait();
        // slot q held stage s, read into registers last iteration: refill it
        // with stage s + 4 (the producer's next)
        if (s + 1 < total) read_stage(nqc, nxt);
        produce(qc);
        __builtin_amdgcn_sched_barrier(0);
        mma(cur);
        __builtin_amdgcn_sched_barrier(0);
        stage_ready(nxt);
        if (cc.k == nks - 1) {
            epilogue(cc.L, cc.j);
            zero_acc();
            if (s + 1 < total) next_seg(cc);
        } else {
            ++cc.k;
        }
        ++s;
        return s < total;
    };
    while (iter(IC<0>{}) && iter(IC<1>{}) && iter(IC<2>{}) && iter(IC<3>{})) {
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ---- few tiles with long k loops: the k loop in two halves ---------------------
// The two-halves scheme of the int4 GEMM on fp6 operands.  Each tile (128
// channels x BM tokens) gets two halves of NWH waves: half 0 runs the first
// half of the k-stages and half 1 the rest, each through its own NS-slot LDS
// ring (the fp6 kernel's ring protocol), in lockstep on the workgroup
// barrier; a second half one stage shorter idles on its last step.  At the
// end the halves swap their fp32 sums (exact integers, so exact sums) through
// the idle rings and each finishes two of the four channel fragments with
// the epilogue arithmetic of the kernel above.  One tile per workgroup, two
// workgroups per compute unit.
template <int NWH_, int NS_>
struct F6HalfTile {
    static constexpr int NWH = NWH_, NS = NS_, FN = 4, FM = 2;
    static constexpr int NT = 2 * NWH * 64;
    static constexpr int BN = FN * 32, BM = NWH * FM * 32;
    static constexpr int WUnits = BN / 32, XUnits = BM / 32, Units = WUnits + XUnits;
    static constexpr int UPW = Units / NWH;   // units per wave and stage, within a half
    static constexpr int VPW = 2 * UPW;       // transfers per wave and stage
    static constexpr int Slot = Units * kUnit;
    static constexpr int Exch = NWH * 16384;  // one half's outgoing sums: 2 fragments x 2 x 16 floats x 64 lanes per wave
    static constexpr int Pool = 2 * NS * Slot > 2 * Exch ? 2 * NS * Slot : 2 * Exch;
    static_assert(Units % NWH == 0, "units split evenly over a half's waves");
};
using F6Half128 = F6HalfTile<2, 3>;   // 128 x 128 tiles, 72 KB of rings
using F6Half64 = F6HalfTile<1, 4>;    // 128 x 64 tiles, 72 KB of rings

// the mixed fma of fma_mix2 with fp32 bias operands (each exactly an fp16 value)
__device__ __forceinline__ uint32_t fma_mix2f(float p0, float w0, float b0, float p1, float w1, float b1) {
    uint32_t r;
    asm("v_fma_mixlo_f16 %0, %1, %2, %3\n\t"
        "v_fma_mixhi_f16 %0, %4, %5, %6"
        : "=&v"(r)
        : "v"(p0), "v"(w0), "v"(b0), "v"(p1), "v"(w1), "v"(b1));
    return r;
}

template <class C, bool I32OUT, bool RAGGED, bool BIAS>
__global__ void __launch_bounds__(C::NT, C::NWH == 1 ? 1 : 2) f6_gemm_halves_kernel(F6Args a)
{
    static_assert(!(I32OUT && BIAS), "no bias on the integer output");
    constexpr int NS = C::NS, kFN = C::FN, kFM = C::FM, kUPW = C::UPW, kVPW = C::VPW, kSlot = C::Slot;
    __shared__ __align__(16) uint8_t pool[C::Pool];
    // the tile's epilogue operands, staged after the k loop as floats:
    // channel scales, biases (fp16 widened, exact), token scales
    constexpr int EPN = 2 * C::BN + C::BM;
    __shared__ float ep[EPN];
    const float *ep_ws = ep, *ep_b = ep + C::BN, *ep_xs = ep + 2 * C::BN;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w8 = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = w8 / C::NWH, wm = w8 % C::NWH;
    const int M = a.M, N = a.N, nks = a.K >> 6;
    // one tile per workgroup: workgroups are dealt to the 8 XCDs
    // round-robin, and each XCD takes a contiguous run of the grouped order
    int L;
    {
        const int G = gridDim.x, x = blockIdx.x & 7, j = blockIdx.x >> 3;
        const int per = G >> 3, rem = G & 7;
        L = x * per + min(x, rem) + j;
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
    uint8_t *ring = pool + half * NS * kSlot;
    const uint8_t *usrc[C::UPW];
#pragma unroll
    for (int j = 0; j < kUPW; ++j) {
        const int u = wm * kUPW + j;
        if (u < C::WUnits) {
            const int ug = min(tn * C::WUnits + u, wunits_total - 1);
            usrc[j] = a.Wq + ((int64_t)ug * nks + kb) * kUnit;
        } else {
            const int ux = min(tm * C::XUnits + (u - C::WUnits), xunits_total - 1);
            usrc[j] = a.Xq + ((int64_t)ux * nks + kb) * kUnit;
        }
    }
    // stage k of this half into slot q; past the end the last stage is
    // loaded again (into a slot whose contents are never read), so every wave
    // issues the same transfers and the wait counts stay fixed
    auto produce = [&](int q, int k) {
        const uint32_t voff = (uint32_t)(min(k, len - 1) * kUnit + lane * 16);
        uint8_t *dst = ring + q * kSlot;
#pragma unroll
        for (int j = 0; j < kUPW; ++j) dma_lds16(usrc[j] + voff, dst + (wm * kUPW + j) * kUnit);
        if (lane < 32) {
#pragma unroll
            for (int j = 0; j < kUPW; ++j) dma_lds16(usrc[j] + voff + 1024, dst + (wm * kUPW + j) * kUnit + 1024);
        }
    };
    // two operand register sets used by alternate stages (the persistent
    // kernel's scheme; the ragged instances read into set 1 and copy it)
    constexpr bool kAlt = !RAGGED;
    v4u ra[2][kFN], rb[2][kFM];
    v2u sa[2][kFN], sb[2][kFM];
    const uint32_t wl0 = (uint32_t)(lane * 16), wl1 = (uint32_t)f6_tail_offset(lane);
    const uint32_t xo = (uint32_t)((C::WUnits + wm * kFM) * kUnit);
    auto read_stage = [&](int q, auto pc) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        uint32_t b16 = wl0, b8 = wl1;
        asm volatile("" : "+v"(b16), "+v"(b8));
        const uint32_t base = lds_addr(ring + q * kSlot);
        b16 += base;
        b8 += base;
        const uint32_t bx16 = b16 + xo, bx8 = b8 + xo;
        static_for<0, kFN>([&](auto f) {
            constexpr int o = decltype(f)::value * kUnit;
            ra[P][f] = lds_read16<o>(b16);
            sa[P][f] = lds_read8<o>(b8);
        });
        static_for<0, kFM>([&](auto f) {
            constexpr int o = decltype(f)::value * kUnit;
            rb[P][f] = lds_read16<o>(bx16);
            sb[P][f] = lds_read8<o>(bx8);
        });
    };
    auto stage_ready = [&](auto pc) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        wait_operands(ra[P], rb[P], sa[P], sb[P]);
    };
    v16f acc[kFN][kFM];
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
        for (int fm = 0; fm < kFM; ++fm) acc[fn][fm] = v16f{};
    auto mma = [&](auto pc) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        v8i opa[kFN], opb[kFM];
#pragma unroll
        for (int f = 0; f < kFN; ++f)
            opa[f] = v8i{(int)ra[P][f][0], (int)ra[P][f][1], (int)ra[P][f][2], (int)ra[P][f][3],
                         (int)sa[P][f][0], (int)sa[P][f][1], 0, 0};
#pragma unroll
        for (int f = 0; f < kFM; ++f)
            opb[f] = v8i{(int)rb[P][f][0], (int)rb[P][f][1], (int)rb[P][f][2], (int)rb[P][f][3],
                         (int)sb[P][f][0], (int)sb[P][f][1], 0, 0};
#pragma unroll
        for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm)
                acc[fn][fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(opa[fn], opb[fm], acc[fn][fm], 2, 2, 0, 0, 0, 0);
    };

    // epilogue operands: loaded first (EPR per thread at clamped indices,
    // ahead of the transfers), held in registers through the k loop and
    // written to LDS after it, when no transfer into LDS is in flight
    constexpr int EPR = (EPN + C::NT - 1) / C::NT;
    float epv[EPR];
    _Float16 epb[EPR];
#pragma unroll
    for (int r = 0; r < EPR; ++r) {
        const int e = min(tid + r * C::NT, EPN - 1);
        const int ec = e & (C::BN - 1), er = max(e - 2 * C::BN, 0);
        const float *esrc = e < 2 * C::BN ? a.ws + min(tn * C::BN + ec, N - 1) : a.xs + min(tm * C::BM + er, M - 1);
        epv[r] = I32OUT ? 0.0f : *esrc;
        epb[r] = (_Float16)0.0f;
        if constexpr (BIAS) epb[r] = reinterpret_cast<const _Float16 *>(a.bias)[min(tn * C::BN + ec, N - 1)];
    }
    __builtin_amdgcn_sched_barrier(0);

    // stage s+1 has landed once at most the NS - 2 later productions are
    // outstanding (completion is in issue order)
    // prologue: stages 0..NS-1 in flight, stage 0 read into registers
    for (int q = 0; q < NS; ++q) produce(q, q);
    wait_vm_barrier<(NS - 1) * kVPW>();
    read_stage(0, IC<kAlt ? 0 : 1>{});
    stage_ready(IC<kAlt ? 0 : 1>{});
    // both halves take h0 steps; stage s in register set s & 1
    int q = 0, s = 0;
    auto step = [&](auto pc) __attribute__((always_inline)) -> bool {
        constexpr IC<kAlt ? decltype(pc)::value : 0> cur{};
        constexpr IC<kAlt ? 1 - decltype(pc)::value : 1> nxt{};
        const int nq = q + 1 == NS ? 0 : q + 1;
        const bool active = s < len;
        if constexpr (!kAlt) {
#pragma unroll
            for (int f = 0; f < kFN; ++f) {
                ra[0][f] = ra[1][f];
                sa[0][f] = sa[1][f];
            }
#pragma unroll
            for (int f = 0; f < kFM; ++f) {
                rb[0][f] = rb[1][f];
                sb[0][f] = sb[1][f];
            }
        }
        wait_landed_barrier<(NS - 2) * kVPW>();
        read_stage(nq, nxt);
        produce(q, s + NS);
        __builtin_amdgcn_sched_barrier(0);
        if (active) mma(cur);
        __builtin_amdgcn_sched_barrier(0);
        stage_ready(nxt);
        q = nq;
        ++s;
        return s < h0;
    };
    if (h0 > 0)
        while (step(IC<0>{}) && step(IC<1>{})) {
        }
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");

    // the epilogue operands into LDS (a thread past the end writes the last
    // value again); the barrier after the sends below publishes them
#pragma unroll
    for (int r = 0; r < EPR; ++r) {
        const int e = min(tid + r * C::NT, EPN - 1);
        ep[e] = e >= C::BN && e < 2 * C::BN ? (float)epb[r] : epv[r];
    }

    // the halves swap sums through the idle rings: half 0 finishes channel
    // fragments 0-1 and half 1 fragments 2-3, each adding the other's
    auto send = [&](auto f0c) {
        constexpr int f0 = decltype(f0c)::value;
        v4f *out = reinterpret_cast<v4f *>(pool + half * C::Exch + wm * 16384);
        static_for<0, 2>([&](auto fc) {
            constexpr int fn = f0 + decltype(fc)::value;
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const v16f &x = acc[fn][fm];
                    out[((decltype(fc)::value * kFM + fm) * 4 + q4) * 64 + lane] =
                        v4f{x[4 * q4], x[4 * q4 + 1], x[4 * q4 + 2], x[4 * q4 + 3]};
                }
        });
    };
    auto receive = [&](auto f0c) {
        constexpr int f0 = decltype(f0c)::value;
        const v4f *in = reinterpret_cast<const v4f *>(pool + (1 - half) * C::Exch + wm * 16384);
        static_for<0, 2>([&](auto fc) {
            constexpr int fn = f0 + decltype(fc)::value;
#pragma unroll
            for (int fm = 0; fm < kFM; ++fm)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const v4f y = in[((decltype(fc)::value * kFM + fm) * 4 + q4) * 64 + lane];
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[fn][fm][4 * q4 + e] += y[e];
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
            for (int fm = 0; fm < kFM; ++fm) {
                const int r0 = (wm * kFM + fm) * 32 + (lane & 31), m = tm * C::BM + r0;
                const v16f &x = acc[fn][fm];
                if constexpr (I32OUT) {   // the exact integer sums
                    int32_t *dst = reinterpret_cast<int32_t *>(a.Y) + (int64_t)m * a.ldy + n0;
                    if (m < M && n0 < N) {
                        if (!RAGGED || n0 + 16 <= N) {
#pragma unroll
                            for (int q4 = 0; q4 < 4; ++q4)
                                reinterpret_cast<v4i *>(dst)[q4] =
                                    v4i{(int)x[4 * q4], (int)x[4 * q4 + 1], (int)x[4 * q4 + 2], (int)x[4 * q4 + 3]};
                        } else {
#pragma unroll
                            for (int v = 0; v < 16; ++v)
                                if (n0 + v < N) dst[v] = (int)x[v];
                        }
                    }
                    continue;
                }
                uint32_t hv[8];
                const float xsc = ep_xs[r0];
#pragma unroll
                for (int v = 0; v < 16; v += 2)
                    hv[v / 2] = fma_mix2f(x[v] * xsc, wsv[v], bw[v], x[v + 1] * xsc, wsv[v + 1], bw[v + 1]);
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
}

// ---- format conversion: packed int4 units -> fp6 units ---------------------------
// One thread per lane slot: its 16 bytes (32 nibbles) become its six fp6
// dwords (the code order of f6_codes.h).
__global__ void repack_f6_kernel(const uint8_t *__restrict__ in, uint8_t *__restrict__ out, int64_t slots) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= slots) return;
    const int64_t unit = t >> 6;
    const int l = (int)(t & 63);
    const v4u src = *reinterpret_cast<const v4u *>(in + unit * 1024 + l * 16);
    const uint32_t d[4] = {src[0], src[1], src[2], src[3]};
    uint32_t w[6];
    f6_from_nibbles(d, w);
    f6_store(out + unit * kF6Unit, l, w);
}

int f6_device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
    }
    return cus;
}

}  // namespace

hipError_t launch_repack_f6(const uint8_t *in, int64_t units, uint8_t *out, hipStream_t stream) {
    const int64_t slots = units * 64;
    if (slots == 0) return hipSuccess;
    hipLaunchKernelGGL(repack_f6_kernel, dim3((unsigned)((slots + 255) / 256)), dim3(256), 0, stream, in, out, slots);
    return hipGetLastError();
}

namespace {

template <class C>
hipError_t launch_gemm_f6_tile(F6Args g, bool i32out, bool ragged, hipStream_t stream) {
    g.tiles_m = (g.M + C::BM - 1) / C::BM;
    g.tiles_n = (g.N + C::BN - 1) / C::BN;
    const int ntiles = g.tiles_m * g.tiles_n;
    const int full = (f6_device_cus() * 2 + 7) / 8 * 8;
    const int grid = std::max(8, (std::min(ntiles, full) + 7) / 8 * 8);
    const dim3 gd((unsigned)grid), bd(C::NT);
    if (i32out) {
        if (ragged) hipLaunchKernelGGL((f6_gemm_kernel<C, true, true, false>), gd, bd, 0, stream, g);
        else hipLaunchKernelGGL((f6_gemm_kernel<C, true, false, false>), gd, bd, 0, stream, g);
    } else if (ragged) {
        if (g.bias) hipLaunchKernelGGL((f6_gemm_kernel<C, false, true, true>), gd, bd, 0, stream, g);
        else hipLaunchKernelGGL((f6_gemm_kernel<C, false, true, false>), gd, bd, 0, stream, g);
    } else {
        if (g.bias) hipLaunchKernelGGL((f6_gemm_kernel<C, false, false, true>), gd, bd, 0, stream, g);
        else hipLaunchKernelGGL((f6_gemm_kernel<C, false, false, false>), gd, bd, 0, stream, g);
    }
    return hipGetLastError();
}

template <class C>
hipError_t launch_gemm_f6_halves(F6Args g, bool i32out, bool ragged, hipStream_t stream) {
    g.tiles_m = (g.M + C::BM - 1) / C::BM;
    g.tiles_n = (g.N + C::BN - 1) / C::BN;
    const dim3 gd((unsigned)(g.tiles_m * g.tiles_n)), bd(C::NT);   // one tile per workgroup
    if (i32out) {
        if (ragged) hipLaunchKernelGGL((f6_gemm_halves_kernel<C, true, true, false>), gd, bd, 0, stream, g);
        else hipLaunchKernelGGL((f6_gemm_halves_kernel<C, true, false, false>), gd, bd, 0, stream, g);
    } else if (ragged) {
        if (g.bias) hipLaunchKernelGGL((f6_gemm_halves_kernel<C, false, true, true>), gd, bd, 0, stream, g);
        else hipLaunchKernelGGL((f6_gemm_halves_kernel<C, false, true, false>), gd, bd, 0, stream, g);
    } else {
        if (g.bias) hipLaunchKernelGGL((f6_gemm_halves_kernel<C, false, false, true>), gd, bd, 0, stream, g);
        else hipLaunchKernelGGL((f6_gemm_halves_kernel<C, false, false, false>), gd, bd, 0, stream, g);
    }
    return hipGetLastError();
}

}  // namespace

int f6_schedule_force = 0;

// The fp6 GEMM schedule for an M x N x K product: 1 the persistent kernel,
// 2 the two-halves kernel on 128-token tiles, 3 on 64-token tiles.  The two
// halves while the 256-token tiles would not give every compute unit a tile,
// on 64-token tiles for long k loops (K >= 2048) whose 128-token tiles would
// fill at most half the compute units.  With more tiles the persistent
// kernel wins inside a block's chain of launches, long k loops included
// (its operands then come from HBM, and the one-tile-per-workgroup halves
// read them more often), although the halves win those shapes when timed
// alone with their operands cache-resident.
int f6_schedule(int64_t M, int64_t N, int K) {
    const int force = __atomic_load_n(&f6_schedule_force, __ATOMIC_RELAXED);
    if (force >= 1 && force <= 3) return force;
    const int cus = f6_device_cus();
    const int64_t tn = (N + 127) / 128;
    const int64_t t256 = (M + 255) / 256 * tn, t128 = (M + 127) / 128 * tn;
    if (t256 > cus) return 1;
    return K >= 2048 && 2 * t128 <= cus ? 3 : 2;
}

hipError_t launch_gemm_f6(const uint8_t *Xq, const float *xs, const uint8_t *Wq, const float *ws,
                          const uint16_t *bias, int64_t M, int64_t N, int K, void *Y, int64_t ldy, bool i32out,
                          hipStream_t stream) {
    F6Args g{};
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
    const bool ragged = N % 16 != 0 || (bias && reinterpret_cast<uintptr_t>(bias) % 4 != 0);
    switch (f6_schedule(M, N, K)) {
        case 2: return launch_gemm_f6_halves<F6Half128>(g, i32out, ragged, stream);
        case 3: return launch_gemm_f6_halves<F6Half64>(g, i32out, ragged, stream);
        default: return launch_gemm_f6_tile<F6Tile256>(g, i32out, ragged, stream);
    }
}

}  // namespace clq
