// High-deviation token selection (Section 3 Insight 1, Section 4.2): the
// n_sel positions of largest deviation, ties to the lower position, emitted
// in ascending order.
//
// One 1024-thread workgroup.  For non-negative floats the bit pattern orders
// like the value, so a 4-pass, 8-bit-digit radix select over the bits finds
// the threshold value T with count(> T) < n_sel <= count(>= T); each pass
// finds its digit by a block-wide scan of the 256 counts.  A final pass
// walks the positions in order and keeps every value > T plus the first
// (n_sel - count(> T)) values == T, compacting with block-wide prefix sums,
// which yields the ascending output directly.  With a candidate map the
// values belong to candidates map[0 .. n) (ascending positions, e.g. the
// tokens the previous layer recomputed) and the selected candidates'
// positions are written instead of their indices.
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

__global__ __launch_bounds__(kT) void select_kernel(const float* __restrict__ sigma, int32_t n_tok,
                                                    int32_t n_sel, const int32_t* __restrict__ map,
                                                    int32_t* __restrict__ out) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_digit, s_need;
    __shared__ uint32_t sw[kWaves][2];
    const int tid = threadIdx.x;

    uint32_t prefix = 0, hi_mask = 0, need = (uint32_t)n_sel;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += kT) hist[i] = 0;
        if (tid == 0) {  // overwritten below by the thread whose digit crosses `need` (1 <= need)
            s_digit = 0;
            s_need = need;
        }
        __syncthreads();
        for (int32_t i = tid; i < n_tok; i += kT) {
            const uint32_t u = key_of(sigma[i]);
            if ((u & hi_mask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1u);
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

    uint32_t base = 0, eq_taken = 0;
    for (int32_t c0 = 0; c0 < n_tok; c0 += kT) {
        const int32_t i = c0 + tid;
        const uint32_t u = i < n_tok ? key_of(sigma[i]) : 0u;
        const uint32_t gt = i < n_tok && u > thr;
        const uint32_t eq = i < n_tok && u == thr;
        uint32_t e_eq, e_dummy, t_eq, t_dummy;
        block_scan2(eq, 0u, e_eq, e_dummy, t_eq, t_dummy, sw);
        const uint32_t take = gt || (eq && eq_taken + e_eq < need);
        uint32_t e_take, e_d2, t_take, t_d2;
        block_scan2(take, 0u, e_take, e_d2, t_take, t_d2, sw);
        if (take) out[base + e_take] = map ? map[i] : i;
        base += t_take;
        eq_taken += t_eq;
    }
}

}  // namespace

hipError_t launch_select_recompute(const float* sigma, int64_t n_tok, int64_t n_sel,
                                   int32_t* sel_pos, hipStream_t s, const int32_t* map) {
    hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kT), 0, s, sigma, (int32_t)n_tok, (int32_t)n_sel, map,
                       sel_pos);
    return hipGetLastError();
}

}  // namespace semshare
