// High-deviation token selection (Section 3 Insight 1, Section 4.2): the
// n_sel positions of largest deviation, ties to the lower position, emitted
// in ascending order.
//
// One 1024-thread workgroup; thread t owns the contiguous positions
// [t E, t E + E), E = ceil(n / 1024), held in registers when E <= 8 (read
// once, through LDS so the global reads are coalesced) and read again from
// global memory otherwise.  For non-negative floats the bit pattern orders
// like the value, so a 4-pass, 8-bit-digit radix select over the bits finds
// the threshold value T with count(> T) < n_sel <= count(>= T); each pass
// finds its digit by a block-wide scan of the 256 counts.  The counts are
// aggregated per wave before they reach the LDS histogram (the lanes sharing
// the first pending lane's digit add once, twice over, then the rest one by
// one): deviations share their exponent, and 64 lanes adding to one LDS
// word would otherwise take turns.  The output is one block-wide scan of
// each thread's (> T, == T) counts: with G and E the counts before a
// position, a position > T goes to G + min(E, need) and a position == T with
// E < need to G + E, where need is the number of copies of T taken; this
// yields the ascending output directly.  With a candidate map the values
// belong to candidates map[0 .. n) (ascending positions, e.g. the tokens the
// previous layer recomputed) and the selected candidates' positions are
// written instead of their indices.
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kT = 1024;
constexpr int kWaves = kT / 64;

__device__ __forceinline__ uint32_t key_of(float f) {
    return f == 0.0f ? 0u : __float_as_uint(f);  // -0 sorts with +0
}

// Exclusive block-wide prefix sum of two counters at once; returns totals.
__device__ __forceinline__ void block_scan2(uint32_t a, uint32_t b, uint32_t& ea, uint32_t& eb,
                                            uint32_t& ta, uint32_t& tb, uint32_t (*sw)[2]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t ia = a, ib = b;  // inclusive wave scan
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t na = __shfl_up(ia, o), nb = __shfl_up(ib, o);
        if (lane >= o) { ia += na; ib += nb; }
    }
    if (lane == 63) { sw[wave][0] = ia; sw[wave][1] = ib; }
    __syncthreads();
    uint32_t pa = 0, pb = 0, sa = 0, sb = 0;
    for (int w = 0; w < kWaves; ++w) {
        const uint32_t xa = sw[w][0], xb = sw[w][1];
        if (w < wave) { pa += xa; pb += xb; }
        sa += xa;
        sb += xb;
    }
    ea = pa + ia - a;
    eb = pb + ib - b;
    ta = sa;
    tb = sb;
    __syncthreads();
}

constexpr int kReg = 8;  // positions per thread held in registers (n <= 8192)

// Adds one count for digit d of every lane with act set, aggregated per wave
// (all lanes of the wave call it together).
__device__ __forceinline__ void add_digit(uint32_t* hist, uint32_t d, bool act) {
    const int lane = threadIdx.x & 63;
    bool pend = act;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const uint64_t live = __ballot(pend);
        if (live == 0) return;
        const int lead = __ffsll((unsigned long long)live) - 1;
        const uint32_t dl = __shfl(d, lead);
        const bool mine = pend && d == dl;
        const uint64_t same = __ballot(mine);
        if (lane == lead) atomicAdd(&hist[dl], (uint32_t)__popcll(same));
        if (mine) pend = false;
    }
    if (pend) atomicAdd(&hist[d], 1u);
}

template <bool kInRegs>
__global__ __launch_bounds__(kT) void select_kernel(const float* __restrict__ sigma, int32_t n_tok,
                                                    int32_t n_sel, const int32_t* __restrict__ map,
                                                    int32_t* __restrict__ out) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_digit, s_need;
    __shared__ uint32_t sw[kWaves][2];
    __shared__ uint32_t s_keys[kInRegs ? kT * kReg : 1];
    const int tid = threadIdx.x;
    const int32_t per = (n_tok + kT - 1) / kT;  // positions per thread (the same for every thread)
    const int32_t i0 = tid * per;
    const int32_t cnt = n_tok - i0 < 0 ? 0 : (n_tok - i0 < per ? n_tok - i0 : per);

    uint32_t key[kInRegs ? kReg : 1];
    if constexpr (kInRegs) {
        for (int32_t i = tid; i < n_tok; i += kT) s_keys[i] = key_of(sigma[i]);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kReg; ++j) key[j] = j < cnt ? s_keys[i0 + j] : 0u;
    }
    auto key_at = [&](int j) -> uint32_t {
        if constexpr (kInRegs) return key[j];
        else return key_of(sigma[i0 + j]);
    };

    uint32_t prefix = 0, hi_mask = 0, need = (uint32_t)n_sel;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += kT) hist[i] = 0;
        if (tid == 0) {  // overwritten below by the thread whose digit crosses `need` (1 <= need)
            s_digit = 0;
            s_need = need;
        }
        __syncthreads();
        if constexpr (kInRegs) {
#pragma unroll
            for (int j = 0; j < kReg; ++j)
                if (j < per) {  // uniform: every lane of the wave calls add_digit together
                    const uint32_t u = key[j];
                    add_digit(hist, (u >> shift) & 255u, j < cnt && (u & hi_mask) == prefix);
                }
        } else {
            for (int32_t j = 0; j < per; ++j) {
                const uint32_t u = j < cnt ? key_at(j) : 0u;
                add_digit(hist, (u >> shift) & 255u, j < cnt && (u & hi_mask) == prefix);
            }
        }
        __syncthreads();
        // the digit: counts of the higher digits summed from the top, the one
        // thread whose digit crosses `need` publishes it (a block-wide scan,
        // not a serial walk over the 256 bins)
        {
            const uint32_t h = tid < 256 ? hist[255 - tid] : 0u;
            uint32_t above, d1, tot, d2;
            block_scan2(h, 0u, above, d1, tot, d2, sw);
            if (tid < 256 && above < need && above + h >= need) {
                s_digit = 255u - (uint32_t)tid;
                s_need = need - above;
            }
        }
        __syncthreads();
        prefix |= s_digit << shift;
        hi_mask |= 255u << shift;
        need = s_need;
        __syncthreads();
    }
    const uint32_t thr = prefix;  // the n_sel-th largest key; `need` of its copies are taken

    uint32_t ngt = 0, neq = 0;
    if constexpr (kInRegs) {
#pragma unroll
        for (int j = 0; j < kReg; ++j)
            if (j < cnt) {
                ngt += key[j] > thr;
                neq += key[j] == thr;
            }
    } else {
        for (int32_t j = 0; j < cnt; ++j) {
            const uint32_t u = key_at(j);
            ngt += u > thr;
            neq += u == thr;
        }
    }
    uint32_t g, e, tg, te;
    block_scan2(ngt, neq, g, e, tg, te, sw);
    auto emit = [&](int j, uint32_t u) {
        const int32_t i = i0 + j;
        if (u > thr) {
            out[g + (e < need ? e : need)] = map ? map[i] : i;
            ++g;
        } else if (u == thr) {
            if (e < need) out[g + e] = map ? map[i] : i;
            ++e;
        }
    };
    if constexpr (kInRegs) {
#pragma unroll
        for (int j = 0; j < kReg; ++j)
            if (j < cnt) emit(j, key[j]);
    } else {
        for (int32_t j = 0; j < cnt; ++j) emit(j, key_at(j));
    }
}

}  // namespace

hipError_t launch_select_recompute(const float* sigma, int64_t n_tok, int64_t n_sel,
                                   int32_t* sel_pos, hipStream_t s, const int32_t* map) {
    if (n_tok <= (int64_t)kT * kReg)
        hipLaunchKernelGGL(select_kernel<true>, dim3(1), dim3(kT), 0, s, sigma, (int32_t)n_tok, (int32_t)n_sel, map,
                           sel_pos);
    else
        hipLaunchKernelGGL(select_kernel<false>, dim3(1), dim3(kT), 0, s, sigma, (int32_t)n_tok, (int32_t)n_sel,
                           map, sel_pos);
    return hipGetLastError();
}

}  // namespace semshare
