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
// of 1024 positions at a time, a block-wide count of the kept flags (ballot
// populations) places every kept position (and the reference row it copies)
// in ascending order.  The row of a recomputed token is the number of kept
// positions before it: the count before its 256-position group, kept in LDS,
// plus at most eight word populations.  The kernel is latency-bound, so its
// global reads for up to 8192 positions (ranks, match indices, selected
// positions) are all requested at its start (10.8 -> 7.2 us per call at 5120
// tokens with the ballot counts, of which about 2.5 us is the launch).
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kT = 1024;
constexpr int kMaxWords = kMaxRetainTok / 32;

// Exclusive block-wide count of the set flags before this thread; *total
// gets the count of all.  Within a wave the count is the population of the
// ballot below the lane (mbcnt), across waves a sum of the wave totals.
__device__ __forceinline__ uint32_t block_excl_count(bool flag, uint32_t* total, uint32_t* sw) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t bal = __ballot(flag);
    const uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
    if (lane == 0) sw[w] = (uint32_t)__popcll(bal);
    __syncthreads();
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kT / 64; ++i) {
        const uint32_t c = sw[i];
        pre += i < w ? c : 0u;
        tot += c;
    }
    *total = tot;
    __syncthreads();
    return pre + below;
}

// Positions (and selected entries) per thread in one batch: the global reads
// of a batch are all issued before any is used, so a phase waits for memory
// once per batch instead of once per 1024 positions.
constexpr int kU = 8;

__global__ __launch_bounds__(kT) void retention_layer_kernel(const int32_t* __restrict__ rank, int32_t n_tok,
                                                             int32_t n_retain, const int32_t* __restrict__ sel_pos,
                                                             int32_t n_sel, const int32_t* __restrict__ idx,
                                                             int32_t* __restrict__ kept_pos,
                                                             int32_t* __restrict__ src_idx,
                                                             int32_t* __restrict__ sel_rows,
                                                             int32_t* __restrict__ n_kept) {
    __shared__ uint32_t bits[kMaxWords];
    __shared__ uint32_t sw[kT / 64];
    // the kept positions before each group of 256 positions (8 words)
    __shared__ uint32_t s_pre[kMaxRetainTok / 256];
    const int tid = threadIdx.x, lane = tid & 63;
    const int32_t n_words = (n_tok + 31) / 32;
    const int32_t n_pos = 32 * n_words;  // positions covered, a multiple of 32
    constexpr int32_t kBatch = kT * kU;
    // the first batch of every input, requested together: the ranks and match
    // indices of positions tid + kT u, the selected positions tid + kT u
    int32_t rk[kU], ix[kU], sp[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int32_t p = tid + kT * u;
        rk[u] = p < n_tok ? rank[p] : -1;
        ix[u] = src_idx && p < n_tok ? idx[p] : 0;
        sp[u] = p < n_sel ? sel_pos[p] : -1;
    }
    // the positions ranked below n_retain: a wave covers 64 consecutive
    // positions, two words (the trip counts are the same in every lane)
    for (int32_t b0 = 0; b0 < n_pos; b0 += kBatch) {
        if (b0 > 0) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int32_t p = b0 + tid + kT * u;
                rk[u] = p < n_tok ? rank[p] : -1;
            }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int32_t base = b0 + kT * u;
            const uint64_t m = __ballot(rk[u] >= 0 && rk[u] < n_retain);
            const int32_t w = (base + (tid & ~63)) >> 5;
            if (lane == 0 && w < n_words) bits[w] = (uint32_t)m;
            if (lane == 0 && w + 1 < n_words) bits[w + 1] = (uint32_t)(m >> 32);
        }
    }
    __syncthreads();
    // recomputed tokens are never evicted
    for (int32_t i0 = 0; i0 < n_sel; i0 += kBatch) {
        int32_t q[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int32_t i = i0 + tid + kT * u;
            q[u] = i0 == 0 ? sp[u] : (i < n_sel ? sel_pos[i] : -1);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
            if (q[u] >= 0 && q[u] < n_tok) atomicOr(&bits[q[u] >> 5], 1u << (q[u] & 31));
    }
    __syncthreads();
    // the kept positions in ascending order: each block of kT positions is
    // compacted in parallel (one position per thread, a block-wide count of
    // the kept flags before it), with the match indices read a batch ahead;
    // s_pre keeps the count before every 256-position group for the rows of
    // the recomputed tokens below
    uint32_t base_out = 0;
    for (int32_t b0 = 0; b0 < n_pos; b0 += kBatch) {  // the same trip counts in every thread
        if (b0 > 0 && src_idx) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int32_t p = b0 + tid + kT * u;
                ix[u] = p < n_tok ? idx[p] : 0;
            }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int32_t base = b0 + kT * u;
            if (base >= n_pos) break;
            const int32_t p = base + tid;
            const bool keep = p < n_tok && ((bits[p >> 5] >> (p & 31)) & 1u);
            uint32_t total;
            const uint32_t o = base_out + block_excl_count(keep, &total, sw);
            if ((p & 255) == 0) s_pre[p >> 8] = o;
            if (keep) {
                kept_pos[o] = p;
                if (src_idx) src_idx[o] = ix[u];
            }
            base_out += total;
        }
    }
    if (tid == 0) *n_kept = (int32_t)base_out;
    __syncthreads();
    // the row of every recomputed token in the compacted cache: the kept
    // positions before it (those before its 256-position group, the group's
    // words before its word, the lower bits of its word)
    for (int32_t i0 = 0; i0 < n_sel; i0 += kBatch) {
        int32_t q[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int32_t i = i0 + tid + kT * u;
            q[u] = i0 == 0 ? sp[u] : (i < n_sel ? sel_pos[i] : -1);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int32_t i = i0 + tid + kT * u;
            if (i >= n_sel) break;
            const int32_t p = q[u];
            int32_t row = -1;
            if (p >= 0 && p < n_tok) {
                const int32_t w = p >> 5, b = p & 31;
                uint32_t r = s_pre[p >> 8];
                for (int32_t v = w & ~7; v < w; ++v) r += __popc(bits[v]);
                r += __popc(bits[w] & ((1u << b) - 1u));
                if ((bits[w] >> b) & 1u) row = (int32_t)r;
            }
            sel_rows[i] = row;
        }
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
