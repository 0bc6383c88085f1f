// Fuzzy token matching (Sections 4.2, 4.3): top-1 Hamming nearest reference
// token for every target token, lowest reference index on ties.
//
// Integer VALU kernel.  A workgroup owns 64*R target codes (R per lane, held
// in VGPRs) and one split of the reference range.  Reference codes are staged
// through LDS in chunks; every lane of a wave reads the same LDS address
// (broadcast) and the four waves take interleaved reference rows.  Per pair
// the work is 2W XORs, 2W accumulating popcounts (v_bcnt_u32_b32), one
// shift-or that forms the key (dist << 23 | ref_index) and one v_min_u32:
// comparing packed keys orders by distance first and index second, so the
// lowest index wins ties with no extra compare.  Waves reduce through LDS;
// with several reference splits the workgroups combine through a 32-bit
// atomicMin on the key, held temporarily in the idx output itself, and a
// finalize pass unpacks (idx, dist).
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kIdxBits = 23;
constexpr uint32_t kIdxMask = (1u << kIdxBits) - 1;
constexpr int kStage = 512;  // reference codes per LDS stage
constexpr int kR = 2;        // target codes per lane

template <int W>
__global__ __launch_bounds__(256) void match_kernel(const uint64_t* __restrict__ tgt, int64_t n_tgt,
                                                    const uint64_t* __restrict__ ref, int64_t n_ref,
                                                    int64_t refs_per_split, uint32_t* __restrict__ keys,
                                                    int32_t* __restrict__ dist, int direct) {
    __shared__ uint64_t sref[kStage * W];
    __shared__ uint32_t sred[4][64 * kR];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t t_base = (int64_t)blockIdx.x * 64 * kR;

    uint32_t tc[kR][2 * W];
#pragma unroll
    for (int r = 0; r < kR; ++r) {
        int64_t t = t_base + lane + 64 * r;
        if (t > n_tgt - 1) t = n_tgt - 1;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const uint64_t c = tgt[t * W + w];
            tc[r][2 * w] = (uint32_t)c;
            tc[r][2 * w + 1] = (uint32_t)(c >> 32);
        }
    }
    uint32_t best[kR];
#pragma unroll
    for (int r = 0; r < kR; ++r) best[r] = 0xFFFFFFFFu;

    const int64_t j_begin = (int64_t)blockIdx.y * refs_per_split;
    const int64_t j_end = j_begin + refs_per_split < n_ref ? j_begin + refs_per_split : n_ref;
    for (int64_t s0 = j_begin; s0 < j_end; s0 += kStage) {
        const int cnt = (int)(j_end - s0 < kStage ? j_end - s0 : kStage);
        __syncthreads();
        for (int i = threadIdx.x; i < cnt * W; i += 256) sref[i] = ref[s0 * W + i];
        __syncthreads();
        for (int jj = wave; jj < cnt; jj += 4) {
            uint32_t rc[2 * W];
#pragma unroll
            for (int w = 0; w < W; ++w) {
                const uint64_t c = sref[jj * W + w];
                rc[2 * w] = (uint32_t)c;
                rc[2 * w + 1] = (uint32_t)(c >> 32);
            }
            const uint32_t jglob = (uint32_t)(s0 + jj);
#pragma unroll
            for (int r = 0; r < kR; ++r) {
                uint32_t d = 0;
#pragma unroll
                for (int w = 0; w < 2 * W; ++w) d += __popc(tc[r][w] ^ rc[w]);
                const uint32_t key = (d << kIdxBits) | jglob;
                best[r] = best[r] < key ? best[r] : key;
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kR; ++r) sred[wave][lane + 64 * r] = best[r];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int r = 0; r < kR; ++r) {
            uint32_t m = sred[0][lane + 64 * r];
#pragma unroll
            for (int w = 1; w < 4; ++w) {
                const uint32_t o = sred[w][lane + 64 * r];
                m = m < o ? m : o;
            }
            const int64_t t = t_base + lane + 64 * r;
            if (t < n_tgt) {
                if (direct) {
                    keys[t] = m & kIdxMask;
                    if (dist) dist[t] = (int32_t)(m >> kIdxBits);
                } else {
                    atomicMin(&keys[t], m);
                }
            }
        }
    }
}

__global__ void fill_u32_kernel(uint32_t* p, int64_t n, uint32_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void finalize_kernel(uint32_t* keys, int32_t* dist, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t k = keys[i];
    keys[i] = k & kIdxMask;
    if (dist) dist[i] = (int32_t)(k >> kIdxBits);
}

}  // namespace

hipError_t launch_match(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                        int32_t n_words, int32_t* idx, int32_t* dist, hipStream_t s) {
    const int64_t n_tiles = (n_tgt + 64 * kR - 1) / (64 * kR);
    // enough workgroups to cover the chip (~8 per CU), each split >= 256 references
    int64_t splits = (2048 + n_tiles - 1) / n_tiles;
    const int64_t max_splits = (n_ref + 255) / 256;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    if (splits > 65535) splits = 65535;
    const int64_t per_split = (n_ref + splits - 1) / splits;
    splits = (n_ref + per_split - 1) / per_split;
    auto* keys = reinterpret_cast<uint32_t*>(idx);
    const int direct = splits == 1;
    if (!direct)
        hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((n_tgt + 255) / 256)), dim3(256), 0, s, keys,
                           n_tgt, 0xFFFFFFFFu);
    const dim3 grid((unsigned)n_tiles, (unsigned)splits);
    switch (n_words) {
    case 1: hipLaunchKernelGGL(match_kernel<1>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    case 2: hipLaunchKernelGGL(match_kernel<2>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    case 3: hipLaunchKernelGGL(match_kernel<3>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    default: hipLaunchKernelGGL(match_kernel<4>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    }
    if (!direct)
        hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)((n_tgt + 255) / 256)), dim3(256), 0, s, keys,
                           dist, n_tgt);
    return hipGetLastError();
}

}  // namespace semshare
