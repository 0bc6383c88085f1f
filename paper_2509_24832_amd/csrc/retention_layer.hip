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
// of the ranking (a wave's ballot gives two words at once); then, one block
// of 1024 positions at a time, a block-wide scan of the kept flags places
// every kept position (and the reference row it copies) in ascending order.
// The row of a recomputed token is the number of kept positions before it,
// counted in LDS from its block's first row.
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
    __shared__ uint32_t s_blk[kMaxRetainTok / kT];  // each block of kT positions' first row in the kept list
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
    // the kept positions in ascending order: each block of kT positions is
    // compacted in parallel (one position per thread, a block-wide scan of
    // the kept flags), with coalesced reads of the match index; s_blk holds
    // each block's first row for the rows of the recomputed tokens below
    uint32_t base_out = 0;
    for (int32_t base = 0; base < 32 * n_words; base += kT) {  // the same trip count in every thread
        const int32_t p = base + tid;
        const uint32_t keep = p < n_tok ? (bits[p >> 5] >> (p & 31)) & 1u : 0u;
        uint32_t total;
        const uint32_t o = base_out + block_excl_scan(keep, &total, sw);
        if (tid == 0) s_blk[base / kT] = base_out;
        if (keep) {
            kept_pos[o] = p;
            if (src_idx) src_idx[o] = idx[p];
        }
        base_out += total;
    }
    if (tid == 0) *n_kept = (int32_t)base_out;
    __syncthreads();
    // the row of every recomputed token in the compacted cache: the kept
    // positions before it (its block's first row, the block's words before
    // its word, the lower bits of its word)
    for (int32_t i = tid; i < n_sel; i += kT) {
        const int32_t p = sel_pos[i];
        int32_t row = -1;
        if (p >= 0 && p < n_tok) {
            const int32_t w = p >> 5, b = p & 31, blk = p / kT;
            uint32_t r = s_blk[blk];
            for (int32_t v = blk * (kT / 32); v < w; ++v) r += __popc(bits[v]);
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
