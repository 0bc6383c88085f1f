// The dynamic recompute set (Section 4.3.3 with the Attention Recovery
// equation of Section 3) and the first-layer retention ranking (Section
// 4.3.4) for prompts longer than the one-workgroup sort of attention_mass.hip
// takes (8192 < n_tok <= 65536), with the same keys and therefore the same
// results.
//
// Ranks are counted rather than sorted: the rank of a token is the number of
// keys smaller than its own (keys are unique: the position sits in the low
// bits), and every workgroup counts for 256 tokens while all keys stream
// through LDS in tiles; n^2 comparisons spread over n / 256 workgroups.  The
// pass that ranks the masses also sums, per token, the 2^-40 fixed-point
// masses of every key up to its own (its inclusive prefix in mass order), so
// AR is the smallest rank + 1 whose prefix reaches thres of the total (an
// atomic min).  The hot set is then every key up to the key of rank AR - 1,
// which a small pass finds; the deviation ranking within the hot and cold
// groups and the retention ranking recompute the hot flags from that key.
// The output buffers serve as the scratch of the intermediate steps: sel_pos
// holds the mass ranks, then the selection flags; counts[1..2] and
// kept_pos[0..1] hold the key of rank AR - 1.  A last one-workgroup pass
// compacts the chosen positions in ascending order.
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kRB = 256;       // tokens ranked per workgroup
constexpr int kTile = 2048;    // keys per LDS tile
constexpr int kCT = 1024;      // threads of the compaction workgroup
constexpr int kMaxWords = kMaxDynTokLarge / 32;

__device__ __forceinline__ float clamp01(float m) { return m > 0.0f ? (m < 1.0f ? m : 1.0f) : 0.0f; }

// mass order: larger mass first, lower position first on ties
__device__ __forceinline__ uint64_t mass_key(float m, int32_t i) {
    return ((uint64_t)(0xFFFFFFFFu - __float_as_uint(clamp01(m))) << 32) | (uint32_t)i;
}

__device__ __forceinline__ int64_t mass_fixed(float m) {
    return (int64_t)floor((double)clamp01(m) * 1099511627776.0);  // 2^40
}

// group (0 first), then larger value first, then lower position
__device__ __forceinline__ uint64_t group_key(uint32_t group, float v, int32_t i) {
    const uint32_t b = __float_as_uint(v > 0.0f ? v : 0.0f) & 0x7FFFFFFFu;
    return ((uint64_t)group << 62) | ((uint64_t)(0x7FFFFFFFu - b) << 20) | (uint32_t)i;
}

__device__ __forceinline__ uint64_t kstar_of(const int32_t* p) {
    return ((uint64_t)(uint32_t)p[1] << 32) | (uint32_t)p[0];
}

__global__ void set_kernel(int32_t* p, int32_t v) { *p = v; }

// rank_out[i] = number of mass keys below token i's; with ar != null, AR as an
// atomic min over the tokens whose inclusive fixed-point prefix reaches thres
// of the total.
__global__ __launch_bounds__(kRB) void mass_rank_kernel(const float* __restrict__ mass, int32_t n, double thres,
                                                        int32_t* __restrict__ rank_out, int32_t* __restrict__ ar) {
    __shared__ uint64_t s_key[kTile];
    __shared__ int64_t s_fx[kTile];
    const int32_t i = blockIdx.x * kRB + threadIdx.x;
    const bool live = i < n;
    const uint64_t ki = live ? mass_key(mass[i], i) : ~0ull;
    uint32_t cnt = 0;
    int64_t below = 0, total = 0;
    for (int32_t t0 = 0; t0 < n; t0 += kTile) {
        const int32_t m = min(kTile, n - t0);
        for (int32_t j = threadIdx.x; j < m; j += kRB) {
            const float v = mass[t0 + j];
            s_key[j] = mass_key(v, t0 + j);
            s_fx[j] = mass_fixed(v);
        }
        __syncthreads();
        for (int32_t j = 0; j < m; ++j) {
            const uint64_t kj = s_key[j];
            const int64_t f = s_fx[j];
            cnt += kj < ki ? 1u : 0u;
            below += kj <= ki ? f : 0;
            total += f;
        }
        __syncthreads();
    }
    if (!live) return;
    rank_out[i] = (int32_t)cnt;
    if (ar && (double)below >= thres * (double)total) atomicMin(ar, (int32_t)cnt + 1);
}

// the mass key of rank *ar - 1 (the last hot token), as two int32 halves at out
__global__ void kstar_kernel(const float* __restrict__ mass, const int32_t* __restrict__ rank, int32_t n,
                             const int32_t* __restrict__ ar, int32_t* __restrict__ out) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n && rank[i] == *ar - 1) {
        const uint64_t k = mass_key(mass[i], i);
        out[0] = (int32_t)(uint32_t)k;
        out[1] = (int32_t)(uint32_t)(k >> 32);
    }
}

// chosen_out[i] = 1 if token i is recomputed: hot tokens by deviation among
// the hot (the first n_hot), cold tokens likewise among the cold.
__global__ __launch_bounds__(kRB) void group_select_kernel(const float* __restrict__ mass,
                                                           const float* __restrict__ sigma, int32_t n,
                                                           const int32_t* __restrict__ counts, double w_hot,
                                                           double w_cold, int32_t* __restrict__ chosen_out) {
    __shared__ uint64_t s_key[kTile];
    const uint64_t kstar = kstar_of(counts + 1);
    const int32_t ar = counts[0];
    const int32_t i = blockIdx.x * kRB + threadIdx.x;
    const bool live = i < n;
    const uint64_t ki = live ? group_key(mass_key(mass[i], i) <= kstar ? 0u : 1u, sigma[i], i) : ~0ull;
    uint32_t cnt = 0;
    for (int32_t t0 = 0; t0 < n; t0 += kTile) {
        const int32_t m = min(kTile, n - t0);
        for (int32_t j = threadIdx.x; j < m; j += kRB) {
            const int32_t p = t0 + j;
            s_key[j] = group_key(mass_key(mass[p], p) <= kstar ? 0u : 1u, sigma[p], p);
        }
        __syncthreads();
        for (int32_t j = 0; j < m; ++j) cnt += s_key[j] < ki ? 1u : 0u;
        __syncthreads();
    }
    if (!live) return;
    const int32_t n_hot = (int32_t)floor(w_hot * (double)ar + 0.5);
    const int32_t n_cold = (int32_t)floor(w_cold * (double)(n - ar) + 0.5);
    const bool hot = (ki >> 62) == 0;
    chosen_out[i] = hot ? ((int32_t)cnt < n_hot) : ((int32_t)cnt - ar < n_cold);
}

// rank[i] of the retention ranking: never-evicted tokens (hot or recomputed)
// first in position order, then the others by score, larger first.
__global__ __launch_bounds__(kRB) void retention_rank_kernel(const float* __restrict__ mass,
                                                             const float* __restrict__ score, int32_t n,
                                                             const int32_t* __restrict__ sel_pos,
                                                             const int32_t* __restrict__ counts,
                                                             const int32_t* __restrict__ kstar_p,
                                                             int32_t* __restrict__ rank) {
    __shared__ uint64_t s_key[kTile];
    __shared__ uint32_t s_sel[kMaxWords];
    const uint64_t kstar = kstar_of(kstar_p);
    const int32_t n_sel = counts[1] < n ? counts[1] : n;
    const int32_t n_words = (n + 31) / 32;
    for (int32_t w = threadIdx.x; w < n_words; w += kRB) s_sel[w] = 0;
    __syncthreads();
    for (int32_t s = threadIdx.x; s < n_sel; s += kRB) {
        const int32_t p = sel_pos[s];
        if (p >= 0 && p < n) atomicOr(&s_sel[p >> 5], 1u << (p & 31));
    }
    __syncthreads();
    auto key = [&](int32_t p) -> uint64_t {
        const bool forced = mass_key(mass[p], p) <= kstar || ((s_sel[p >> 5] >> (p & 31)) & 1u);
        return forced ? (uint64_t)(uint32_t)p : group_key(1u, score[p], p);
    };
    const int32_t i = blockIdx.x * kRB + threadIdx.x;
    const bool live = i < n;
    const uint64_t ki = live ? key(i) : ~0ull;
    uint32_t cnt = 0;
    for (int32_t t0 = 0; t0 < n; t0 += kTile) {
        const int32_t m = min(kTile, n - t0);
        for (int32_t j = threadIdx.x; j < m; j += kRB) s_key[j] = key(t0 + j);
        __syncthreads();
        for (int32_t j = 0; j < m; ++j) cnt += s_key[j] < ki ? 1u : 0u;
        __syncthreads();
    }
    if (live) rank[i] = (int32_t)cnt;
}

// Exclusive block-wide prefix sum over kCT threads; *total gets the sum.
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
    for (int k = 0; k < kCT / 64; ++k) {
        const uint32_t c = sw[k];
        pre += k < w ? c : 0u;
        tot += c;
    }
    *total = tot;
    __syncthreads();
    return pre + x - v;
}

// Positions whose bit is set, ascending, to out; returns the count (every thread).
__device__ __forceinline__ uint32_t compact_bits(const uint32_t* bits, int32_t n, int32_t* out, uint32_t* sw) {
    const int32_t n_words = (n + 31) / 32;
    const int32_t per = (n_words + kCT - 1) / kCT;
    const int32_t w0 = threadIdx.x * per, w1 = min(w0 + per, n_words);
    uint32_t cnt = 0;
    for (int32_t w = w0; w < w1; ++w) cnt += __popc(bits[w]);
    uint32_t total;
    uint32_t o = block_excl_scan(cnt, &total, sw);
    for (int32_t w = w0; w < w1; ++w) {
        uint32_t m = bits[w];
        while (m) {
            const int b = __ffs(m) - 1;
            m &= m - 1;
            out[o++] = 32 * w + b;
        }
    }
    return total;
}

// sel_pos holds 0/1 flags on entry and the chosen positions (ascending) on exit.
__global__ __launch_bounds__(kCT) void dyn_compact_kernel(int32_t* __restrict__ sel_pos, int32_t n,
                                                          int32_t* __restrict__ counts, double w_hot) {
    __shared__ uint32_t bits[kMaxWords];
    __shared__ uint32_t sw[kCT / 64];
    const int32_t n_words = (n + 31) / 32;
    for (int32_t w = threadIdx.x; w < n_words; w += kCT) {
        uint32_t m = 0;
        for (int b = 0; b < 32; ++b)
            if (32 * w + b < n && sel_pos[32 * w + b]) m |= 1u << b;
        bits[w] = m;
    }
    const int32_t ar = counts[0];
    __syncthreads();
    const uint32_t total = compact_bits(bits, n, sel_pos, sw);
    if (threadIdx.x == 0) {
        counts[1] = (int32_t)total;
        counts[2] = (int32_t)floor(w_hot * (double)ar + 0.5);
    }
}

// kept = the first R of the ranking, R = max(floor(max(min_keep, AR/T) T + 1/2), never-evicted count).
__global__ __launch_bounds__(kCT) void retention_compact_kernel(const float* __restrict__ mass,
                                                                const int32_t* __restrict__ rank, int32_t n,
                                                                const int32_t* __restrict__ sel_pos,
                                                                const int32_t* __restrict__ counts, double min_keep,
                                                                int32_t* __restrict__ kept_pos,
                                                                int32_t* __restrict__ n_kept) {
    __shared__ uint32_t bits[kMaxWords];
    __shared__ uint32_t sw[kCT / 64];
    const uint64_t kstar = kstar_of(kept_pos);  // read before kept_pos is written
    const int32_t ar = counts[0] < n ? counts[0] : n;
    const int32_t n_sel = counts[1] < n ? counts[1] : n;
    const int32_t n_words = (n + 31) / 32;
    for (int32_t w = threadIdx.x; w < n_words; w += kCT) bits[w] = 0;
    __syncthreads();
    for (int32_t s = threadIdx.x; s < n_sel; s += kCT) {
        const int32_t p = sel_pos[s];
        if (p >= 0 && p < n) atomicOr(&bits[p >> 5], 1u << (p & 31));
    }
    __syncthreads();
    uint32_t f = 0;
    for (int32_t p = threadIdx.x; p < n; p += kCT)
        f += (mass_key(mass[p], p) <= kstar || ((bits[p >> 5] >> (p & 31)) & 1u)) ? 1u : 0u;
    uint32_t n_forced;
    (void)block_excl_scan(f, &n_forced, sw);
    const double ratio = n > 0 && (double)ar / (double)n > min_keep ? (double)ar / (double)n : min_keep;
    int32_t keep = (int32_t)floor(ratio * (double)n + 0.5);
    if (keep < (int32_t)n_forced) keep = (int32_t)n_forced;
    if (keep > n) keep = n;
    __syncthreads();
    for (int32_t w = threadIdx.x; w < n_words; w += kCT) {
        uint32_t m = 0;
        for (int b = 0; b < 32; ++b)
            if (32 * w + b < n && rank[32 * w + b] < keep) m |= 1u << b;
        bits[w] = m;
    }
    __syncthreads();
    const uint32_t total = compact_bits(bits, n, kept_pos, sw);
    if (threadIdx.x == 0) *n_kept = (int32_t)total;
}

}  // namespace

hipError_t launch_dynamic_recompute_large(const float* mass, const float* sigma, int32_t n, double thres,
                                          double w_hot, double w_cold, int32_t* sel_pos, int32_t* counts,
                                          hipStream_t s) {
    const unsigned grid = (unsigned)((n + kRB - 1) / kRB);
    hipLaunchKernelGGL(set_kernel, dim3(1), dim3(1), 0, s, counts, n);
    hipLaunchKernelGGL(mass_rank_kernel, dim3(grid), dim3(kRB), 0, s, mass, n, thres, sel_pos, counts);
    hipLaunchKernelGGL(kstar_kernel, dim3(grid), dim3(kRB), 0, s, mass, sel_pos, n, counts, counts + 1);
    hipLaunchKernelGGL(group_select_kernel, dim3(grid), dim3(kRB), 0, s, mass, sigma, n, counts, w_hot, w_cold,
                       sel_pos);
    hipLaunchKernelGGL(dyn_compact_kernel, dim3(1), dim3(kCT), 0, s, sel_pos, n, counts, w_hot);
    return hipGetLastError();
}

hipError_t launch_retention_large(const float* mass, const float* score, int32_t n, const int32_t* sel_pos,
                                  const int32_t* counts, double min_keep, int32_t* rank, int32_t* kept_pos,
                                  int32_t* n_kept, hipStream_t s) {
    const unsigned grid = (unsigned)((n + kRB - 1) / kRB);
    hipLaunchKernelGGL(mass_rank_kernel, dim3(grid), dim3(kRB), 0, s, mass, n, 0.0, rank, nullptr);
    hipLaunchKernelGGL(kstar_kernel, dim3(grid), dim3(kRB), 0, s, mass, rank, n, counts, kept_pos);
    hipLaunchKernelGGL(retention_rank_kernel, dim3(grid), dim3(kRB), 0, s, mass, score, n, sel_pos, counts, kept_pos,
                       rank);
    hipLaunchKernelGGL(retention_compact_kernel, dim3(1), dim3(kCT), 0, s, mass, rank, n, sel_pos, counts, min_keep,
                       kept_pos, n_kept);
    return hipGetLastError();
}

}  // namespace semshare
