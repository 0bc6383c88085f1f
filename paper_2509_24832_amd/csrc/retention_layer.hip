// Retention on a later layer (Section 4.3.4; Appendix A.6, Retain[i] =
// T prod alpha_retain[j]): the tokens the first layer's ranking places below
// n_retain, plus the tokens this layer recomputes (never evicted), kept in
// position order.  The compacted cache of the layer holds exactly these rows,
// so the layer's recomputed tokens attend over it through their rows in it
// (their causal limit is their own row: every kept token before them sits at
// a lower row, every later one at a higher).
//
// One 1024-thread workgroup.  The kept set is a bitmask in LDS (one bit per
// position, n_tok <= 2^20), built one position per lane from coalesced reads
// of the ranking (a wave's ballot gives two words at once); every thread then
// owns a contiguous run of words, counts its kept positions, and after a
// block-wide scan writes them (and the reference row each one copies) in
// ascending order.  The row of a recomputed token is the number of kept
// positions before it, counted in LDS from its word's owner's offset.
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kT = 1024;
constexpr int kMaxWords = kMaxRetainTok / 32;

// Exclusive block-wide prefix sum; *total gets the sum of all.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* total, uint32_t* sw) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint32_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t y = __shfl_up(x, d);
        if (lane >= d) x += y;
    }
    if (lane == 63) sw[w] = x;
    __syncthreads();
    uint32_t pre = 0, tot = 0;
    for (int i = 0; i < kT / 64; ++i) {
        const uint32_t c = sw[i];
        pre += i < w ? c : 0u;
        tot += c;
    }
    *total = tot;
    __syncthreads();
    return pre + x - v;
}

__global__ __launch_bounds__(kT) void retention_layer_kernel(const int32_t* __restrict__ rank, int32_t n_tok,
                                                             int32_t n_retain, const int32_t* __restrict__ sel_pos,
                                                             int32_t n_sel, const int32_t* __restrict__ idx,
                                                             int32_t* __restrict__ kept_pos,
                                                             int32_t* __restrict__ src_idx,
                                                             int32_t* __restrict__ sel_rows,
                                                             int32_t* __restrict__ n_kept) {
    __shared__ uint32_t bits[kMaxWords];
    __shared__ uint32_t sw[kT / 64];
    __shared__ uint32_t s_off[kT];  // each thread's first row in the kept list
    const int tid = threadIdx.x, lane = tid & 63;
    const int32_t n_words = (n_tok + 31) / 32;
    // the positions ranked below n_retain: a wave covers 64 consecutive
    // positions, two words (the trip count is the same in every lane)
    for (int32_t base = 0; base < 32 * n_words; base += kT) {
        const int32_t p = base + tid;
        const bool keep = p < n_tok && rank[p] >= 0 && rank[p] < n_retain;
        const uint64_t m = __ballot(keep);
        const int32_t w = (base + (tid & ~63)) >> 5;
        if (lane == 0 && w < n_words) bits[w] = (uint32_t)m;
        if (lane == 0 && w + 1 < n_words) bits[w + 1] = (uint32_t)(m >> 32);
    }
    __syncthreads();
    for (int32_t i = tid; i < n_sel; i += kT) {  // recomputed tokens are never evicted
        const int32_t p = sel_pos[i];
        if (p >= 0 && p < n_tok) atomicOr(&bits[p >> 5], 1u << (p & 31));
    }
    __syncthreads();
    // thread t owns words [t * per, (t + 1) * per)
    const int32_t per = n_words > 0 ? (n_words + kT - 1) / kT : 1;
    const int32_t w0 = tid * per, w1 = min(w0 + per, n_words);
    uint32_t cnt = 0;
    for (int32_t w = w0; w < w1; ++w) cnt += __popc(bits[w]);
    uint32_t total;
    uint32_t o = block_excl_scan(cnt, &total, sw);
    s_off[tid] = o;
    for (int32_t w = w0; w < w1; ++w) {
        uint32_t m = bits[w];
        while (m) {
            const int b = __ffs(m) - 1;
            m &= m - 1;
            const int32_t p = 32 * w + b;
            kept_pos[o] = p;
            if (src_idx) src_idx[o] = idx[p];
            ++o;
        }
    }
    if (tid == 0) *n_kept = (int32_t)total;
    __syncthreads();
    // the row of every recomputed token in the compacted cache: the kept
    // positions before it (its word's owner's first row, the owner's words
    // before its word, the lower bits of its word)
    for (int32_t i = tid; i < n_sel; i += kT) {
        const int32_t p = sel_pos[i];
        int32_t row = -1;
        if (p >= 0 && p < n_tok) {
            const int32_t w = p >> 5, b = p & 31;
            const int32_t t = w / per;
            uint32_t r = s_off[t];
            for (int32_t v = t * per; v < w; ++v) r += __popc(bits[v]);
            r += __popc(bits[w] & ((1u << b) - 1u));
            if ((bits[w] >> b) & 1u) row = (int32_t)r;
        }
        sel_rows[i] = row;
    }
}

}  // namespace

hipError_t launch_retention_layer(const int32_t* rank, int32_t n_tok, int32_t n_retain, const int32_t* sel_pos,
                                  int32_t n_sel, const int32_t* idx, int32_t* kept_pos, int32_t* src_idx,
                                  int32_t* sel_rows, int32_t* n_kept, hipStream_t s) {
    hipLaunchKernelGGL(retention_layer_kernel, dim3(1), dim3(kT), 0, s, rank, n_tok, n_retain, sel_pos, n_sel, idx,
                       kept_pos, src_idx, sel_rows, n_kept);
    return hipGetLastError();
}

}  // namespace semshare
