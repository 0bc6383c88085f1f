// KV rearrangement (Section 4.3; keys kept post-RoPE, Section 4.3.2):
// out[l][t] = ref[l][idx[t]] for every layer, one row = all kv heads of a
// token.  A pure HBM copy.  A wave owns R consecutive target rows of one
// tensor across a group of NL layers: it decodes them once (the source index
// of each row and, with an exception list, whether the row is listed: one
// binary search for the first row, then a short forward scan) and then copies
// them, up to two layers at a time, with 16-byte non-temporal loads and
// stores (R x min(NL, 2) x C vector loads in flight per lane before the first
// store, C = 2 chunks per lane and pass; rows of 8 KB or more, such as hidden
// states, go one per wave with C = 8, so a few thousand rows still keep
// every CU busy and all their bytes in flight).  Measured at 32 layers x 5120 rows of 2 KiB (K and V): every row,
// 8 rows x 1 layer per wave, 222 us (6.0 TB/s); 31 layers without 1280 listed
// rows, 2 rows x 2 layers, 174 us (5.6 TB/s): wider groups leave more lanes
// idle on listed rows, longer layer groups lengthen the tail.  Non-temporal
// loads were 14% faster than cached ones on the second shape.  Rows whose
// index lies outside [0, n_ref) are written as zeros and never read.  Listed
// rows (the rows a partial prefill recomputes and overwrites anyway) are left
// untouched.
#include "semshare_internal.h"

namespace semshare {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Grid: one wave per (tensor, layer group, block of R target rows), in that
// order from slowest to fastest.  A pass covers 64 * kChunks 16-byte chunks
// of each row (kChunks per lane).
template <int kRowsPerWave, int kLayersPerWave, int kChunks>
__global__ __launch_bounds__(256) void gather_rows_kernel(const u32x4* __restrict__ src_a,
                                                          const u32x4* __restrict__ src_b,
                                                          const int32_t* __restrict__ idx,
                                                          uint32_t n_tgt, uint32_t n_ref, uint32_t n_layers,
                                                          u32x4* __restrict__ dst_a,
                                                          u32x4* __restrict__ dst_b,
                                                          uint32_t row_blocks, uint32_t layer_groups,
                                                          uint32_t waves_per_tensor, uint32_t waves_total,
                                                          uint32_t cpr,
                                                          const int32_t* __restrict__ except_pos,
                                                          uint32_t n_except) {
    const int lane = threadIdx.x & 63;
    const uint32_t wave = blockIdx.x * 4u + (threadIdx.x >> 6);
    if (wave >= waves_total) return;
    const bool second = wave >= waves_per_tensor;
    const uint32_t w = second ? wave - waves_per_tensor : wave;
    const uint32_t lg = w / row_blocks, rb = w - lg * row_blocks;
    const uint32_t t0 = rb * kRowsPerWave;
    const uint32_t l0 = lg * kLayersPerWave;
    const uint32_t l1 = l0 + kLayersPerWave < n_layers ? l0 + kLayersPerWave : n_layers;

    // listed rows among t0 .. t0 + R - 1: the first entry >= t0, then a forward scan
    uint32_t first = n_except;
    if (n_except) {
        uint32_t lo = 0, hi = n_except;
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if ((uint32_t)except_pos[mid] < t0) lo = mid + 1; else hi = mid;
        }
        first = lo;
    }
    bool live[kRowsPerWave], readable[kRowsPerWave];
    uint32_t srow[kRowsPerWave], trow[kRowsPerWave];
    uint32_t e = first;
#pragma unroll
    for (int u = 0; u < kRowsPerWave; ++u) {
        const uint32_t t = t0 + u;
        live[u] = t < n_tgt;
        const uint32_t tt = live[u] ? t : t0;
        while (e < n_except && (uint32_t)except_pos[e] < t) ++e;
        if (e < n_except && (uint32_t)except_pos[e] == t) live[u] = false;
        const int32_t j = idx[tt];
        readable[u] = j >= 0 && (uint32_t)j < n_ref;
        srow[u] = readable[u] ? (uint32_t)j : 0u;
        trow[u] = tt;
    }
    const u32x4* src = second ? src_b : src_a;
    u32x4* dst = second ? dst_b : dst_a;

    constexpr uint32_t kColBlock = 64 * kChunks;
    for (uint32_t l = l0; l < l1; l += 2) {
        const bool two = kLayersPerWave > 1 && l + 1 < l1;
        for (uint32_t cb = 0; cb < cpr; cb += kColBlock) {
            u32x4 v[2][kRowsPerWave][kChunks];
#pragma unroll
            for (int ll = 0; ll < 2; ++ll) {
                const size_t lay = (size_t)(l + ll);
#pragma unroll
                for (int u = 0; u < kRowsPerWave; ++u) {
                    const u32x4* s = src + (lay * n_ref + srow[u]) * cpr;
#pragma unroll
                    for (int k = 0; k < kChunks; ++k) {
                        const uint32_t c = cb + lane + 64 * k;
                        v[ll][u][k] = u32x4{0u, 0u, 0u, 0u};
                        if ((ll == 0 || two) && live[u] && readable[u] && c < cpr) v[ll][u][k] = __builtin_nontemporal_load(s + c);
                    }
                }
            }
#pragma unroll
            for (int ll = 0; ll < 2; ++ll) {
                const size_t lay = (size_t)(l + ll);
#pragma unroll
                for (int u = 0; u < kRowsPerWave; ++u) {
                    u32x4* d = dst + (lay * n_tgt + trow[u]) * cpr;
#pragma unroll
                    for (int k = 0; k < kChunks; ++k) {
                        const uint32_t c = cb + lane + 64 * k;
                        if ((ll == 0 || two) && live[u] && c < cpr) __builtin_nontemporal_store(v[ll][u][k], d + c);
                    }
                }
            }
        }
    }
}

}  // namespace

namespace {
template <int R, int NL, int CH>
void launch_shape(const void* src_a, const void* src_b, const int32_t* idx, int64_t n_tgt, int64_t n_ref,
                  void* dst_a, void* dst_b, int32_t n_layers, int64_t row_bytes, hipStream_t s,
                  const int32_t* except_pos, int64_t n_except) {
    const int64_t row_blocks = (n_tgt + R - 1) / R;
    const int64_t layer_groups = (n_layers + NL - 1) / NL;
    const int64_t waves_per_tensor = row_blocks * layer_groups;
    const int64_t waves_total = waves_per_tensor * (src_b ? 2 : 1);
    const int64_t blocks = (waves_total + 3) / 4;
    hipLaunchKernelGGL((gather_rows_kernel<R, NL, CH>), dim3((unsigned)blocks), dim3(256), 0, s,
                       static_cast<const u32x4*>(src_a), static_cast<const u32x4*>(src_b), idx,
                       (uint32_t)n_tgt, (uint32_t)n_ref, (uint32_t)n_layers, static_cast<u32x4*>(dst_a),
                       static_cast<u32x4*>(dst_b), (uint32_t)row_blocks, (uint32_t)layer_groups,
                       (uint32_t)waves_per_tensor, (uint32_t)waves_total, (uint32_t)(row_bytes / 16), except_pos,
                       (uint32_t)n_except);
}
}  // namespace

hipError_t launch_gather_rows(const void* src_a, const void* src_b, const int32_t* idx,
                              int64_t n_tgt, int64_t n_ref, void* dst_a, void* dst_b,
                              int32_t n_layers, int64_t row_bytes, hipStream_t s,
                              const int32_t* except_pos, int64_t n_except) {
    if (n_except > 0)
        launch_shape<2, 2, 2>(src_a, src_b, idx, n_tgt, n_ref, dst_a, dst_b, n_layers, row_bytes, s, except_pos,
                              n_except);
    else if (row_bytes >= 8192)  // wide rows: one row per wave, 8 KB of it per pass
        launch_shape<1, 1, 8>(src_a, src_b, idx, n_tgt, n_ref, dst_a, dst_b, n_layers, row_bytes, s, nullptr, 0);
    else if ((n_tgt + 7) / 8 * n_layers * (src_b ? 2 : 1) < 2048)  // few rows: 2 per wave, so all CUs get some
        launch_shape<2, 1, 2>(src_a, src_b, idx, n_tgt, n_ref, dst_a, dst_b, n_layers, row_bytes, s, nullptr, 0);
    else
        launch_shape<8, 1, 2>(src_a, src_b, idx, n_tgt, n_ref, dst_a, dst_b, n_layers, row_bytes, s, nullptr, 0);
    return hipGetLastError();
}

}  // namespace semshare
