// KV rearrangement (Section 4.3; keys kept post-RoPE, Section 4.3.2):
// out[l][t] = ref[l][idx[t]] for every layer, one row = all kv heads of a
// token.  A pure HBM copy: each wave owns 4 rows, decodes them once
// (wave-uniform scalar math: tensor, layer, target token, source row) and
// moves them with 16-byte loads and non-temporal stores, keeping up to 8
// vector loads in flight per lane before the first store.  The loads go
// through the caches: a source row the index repeats is then read from them
// (32 layers x 5120 rows with a uniformly random index, 63% distinct: 185 us
// against 230 us with non-temporal loads; the same time with no repeats).  Rows whose index
// lies outside [0, n_ref) are written as zeros and never read.  The variant
// with an exception list leaves the listed target rows untouched (the rows a
// partial prefill recomputes and overwrites anyway).
#include "semshare_internal.h"

namespace semshare {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowsPerWave = 4;
constexpr int kColBlock = 128;  // 16-byte chunks per row handled per pass (2 per lane)

__global__ __launch_bounds__(256) void gather_rows_kernel(const u32x4* __restrict__ src_a,
                                                          const u32x4* __restrict__ src_b,
                                                          const int32_t* __restrict__ idx,
                                                          uint32_t n_tgt, uint32_t n_ref,
                                                          u32x4* __restrict__ dst_a,
                                                          u32x4* __restrict__ dst_b,
                                                          uint32_t rows_per_tensor,
                                                          uint32_t rows_total, uint32_t cpr,
                                                          const int32_t* __restrict__ except_pos,
                                                          uint32_t n_except) {
    const int lane = threadIdx.x & 63;
    const uint32_t wave = blockIdx.x * 4u + (threadIdx.x >> 6);
    const uint32_t row0 = wave * kRowsPerWave;
    if (row0 >= rows_total) return;

    const u32x4* src[kRowsPerWave];
    u32x4* dst[kRowsPerWave];
    bool live[kRowsPerWave], readable[kRowsPerWave];
#pragma unroll
    for (int u = 0; u < kRowsPerWave; ++u) {
        const uint32_t row = row0 + u;
        live[u] = row < rows_total;
        const uint32_t r = live[u] ? row : row0;
        const bool second = r >= rows_per_tensor;
        const uint32_t rem = second ? r - rows_per_tensor : r;
        const uint32_t l = rem / n_tgt, t = rem - l * n_tgt;
        const int32_t j = idx[t];
        if (n_except) {  // target rows listed (ascending) in except_pos are left as they are
            uint32_t lo = 0, hi = n_except;
            while (lo < hi) {
                const uint32_t mid = (lo + hi) >> 1;
                if ((uint32_t)except_pos[mid] < t) lo = mid + 1; else hi = mid;
            }
            if (lo < n_except && (uint32_t)except_pos[lo] == t) live[u] = false;
        }
        readable[u] = j >= 0 && (uint32_t)j < n_ref;
        const uint32_t jj = readable[u] ? (uint32_t)j : 0u;
        src[u] = (second ? src_b : src_a) + ((size_t)l * n_ref + jj) * cpr;
        dst[u] = (second ? dst_b : dst_a) + ((size_t)l * n_tgt + t) * cpr;
    }
    for (uint32_t cb = 0; cb < cpr; cb += kColBlock) {
        u32x4 v[kRowsPerWave][2];
#pragma unroll
        for (int u = 0; u < kRowsPerWave; ++u) {
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const uint32_t c = cb + lane + 64 * k;
                v[u][k] = u32x4{0u, 0u, 0u, 0u};
                if (live[u] && readable[u] && c < cpr) v[u][k] = src[u][c];
            }
        }
#pragma unroll
        for (int u = 0; u < kRowsPerWave; ++u) {
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const uint32_t c = cb + lane + 64 * k;
                if (live[u] && c < cpr) __builtin_nontemporal_store(v[u][k], dst[u] + c);
            }
        }
    }
}

}  // namespace

hipError_t launch_gather_rows(const void* src_a, const void* src_b, const int32_t* idx,
                              int64_t n_tgt, int64_t n_ref, void* dst_a, void* dst_b,
                              int32_t n_layers, int64_t row_bytes, hipStream_t s,
                              const int32_t* except_pos, int64_t n_except) {
    const int64_t rows_per_tensor = (int64_t)n_layers * n_tgt;
    const int64_t rows_total = rows_per_tensor * (src_b ? 2 : 1);
    const int64_t waves = (rows_total + kRowsPerWave - 1) / kRowsPerWave;
    const int64_t blocks = (waves + 3) / 4;
    hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                       static_cast<const u32x4*>(src_a), static_cast<const u32x4*>(src_b), idx,
                       (uint32_t)n_tgt, (uint32_t)n_ref, static_cast<u32x4*>(dst_a),
                       static_cast<u32x4*>(dst_b), (uint32_t)rows_per_tensor, (uint32_t)rows_total,
                       (uint32_t)(row_bytes / 16), except_pos, (uint32_t)n_except);
    return hipGetLastError();
}

}  // namespace semshare
