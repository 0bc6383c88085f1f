// Top-1 Hamming match on the matrix cores (Sections 4.2, 4.3; the same
// contract as semshare_match: lowest reference index on ties).
//
// Read the reference bits a as 0/1 and the target bits t as -1/+1 scaled by
// 64: sum_k a_k * 64 (2 t_k - 1) = 64 (2 |a & t| - |a|) = 64 (|t| - H), with
// H the Hamming distance, so for a fixed target the nearest reference is the
// one with the largest product and an int8 GEMM (v_mfma_i32_32x32x32_i8)
// followed by an arg-max finds it.  The accumulator starts at 63 - r for the
// reference at row r of its 64-row pair of blocks, so one signed max over a
// pair's outputs picks the largest product and, among equal ones, the lowest
// row; H = |t| - (key >> 6).
//
// A workgroup owns 256 target codes (wave w: 64 of them, two 32-column MFMA
// groups, expanded once into registers) and one split of the reference range,
// which it walks in chunks of 128 references: the chunk's bits are expanded
// to 0/1 bytes in LDS (double-buffered; the next chunk's words are loaded
// while the current one is multiplied) and each wave multiplies both its
// column groups with every row block of the chunk, so one LDS read feeds two
// MFMAs.  A lane keeps, per column group and half, the best key and the pair
// it came from (a strictly larger product replaces it, so an earlier pair
// keeps a tie); the two halves meet at the end.  With several splits the
// workgroups combine through a 32-bit atomicMin on (H << 23 | index), held in
// the idx output until a finalize pass unpacks it.
#include "semshare_internal.h"

namespace semshare {
namespace {

typedef int32_t i32x16_t __attribute__((ext_vector_type(16)));
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));

constexpr int kIdxBits = 23;
constexpr uint32_t kIdxMask = (1u << kIdxBits) - 1;
constexpr int kChunk = 128;  // references per LDS chunk (two 64-row pairs of blocks)
constexpr int kTgt = 256;    // targets per workgroup (64 per wave)
// accumulator start of a row past the end: far below any real key (|key| <=
// 64 * 256 + 63) and far above INT32_MIN, the "nothing seen" key
constexpr int32_t kDead = INT32_MIN + (1 << 20);

// max(max(a, b), c): one v_max3_i32
__device__ __forceinline__ int32_t max3i(int32_t a, int32_t b, int32_t c) { return max(max(a, b), c); }

// bits 4q .. 4q+3 of x -> 4 bytes of 0 or 1
__device__ __forceinline__ uint32_t spread4(uint32_t x, int q) {
    return (__builtin_amdgcn_ubfe(x, 4 * q, 4) * 0x00204081u) & 0x01010101u;  // bit i -> bit 8i
}

template <int W>  // 64-bit words per code
__global__ __launch_bounds__(256) void match_mfma_kernel(const uint64_t* __restrict__ tgt, int64_t n_tgt,
                                                         const uint64_t* __restrict__ ref, int64_t n_ref,
                                                         int64_t refs_per_split, uint32_t* __restrict__ keys,
                                                         int32_t* __restrict__ dist, int direct) {
    constexpr int kBits = 64 * W;
    constexpr int kSteps = kBits / 32;  // MFMA k-steps (32 int8 each) per code
    constexpr int kRow = kBits + 16;    // LDS bytes per expanded reference (padded)
    __shared__ __attribute__((aligned(16))) unsigned char sA[2][kChunk * kRow];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, l32 = lane & 31;

    // B operands: target column l32 of group c, bits [32 ks + 16 half, +16) as
    // +64 (set) or -64 (clear); |t| per column
    int64_t tc[2];
    bool t_ok[2];
    int32_t pop_t[2];
    i32x4_t bop[2][kSteps];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        int64_t t = (int64_t)blockIdx.x * kTgt + 64 * wave + 32 * c + l32;
        t_ok[c] = t < n_tgt;
        if (!t_ok[c]) t = n_tgt - 1;  // computed, never written
        tc[c] = t;
        int32_t pc = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) pc += __popcll(tgt[t * W + w]);
        pop_t[c] = pc;
#pragma unroll
        for (int ks = 0; ks < kSteps; ++ks) {
            const uint32_t bits = (uint32_t)(tgt[t * W + ks / 2] >> (32 * (ks & 1) + 16 * half)) & 0xFFFFu;
#pragma unroll
            for (int q = 0; q < 4; ++q) bop[c][ks][q] = (int32_t)((spread4(bits, q) * 0x80u) ^ 0xC0C0C0C0u);
        }
    }
    // accumulator start: 63 - r, r = row within the 64-row pair (output v of a
    // 32-row block sits at row 8 (v / 4) + 4 half + v % 4)
    i32x16_t bias0, bias1;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        bias0[v] = 63 - (8 * (v >> 2) + 4 * half + (v & 3));
        bias1[v] = bias0[v] - 32;
    }

    const int64_t j_begin = (int64_t)blockIdx.y * refs_per_split;
    const int64_t j_end = j_begin + refs_per_split < n_ref ? j_begin + refs_per_split : n_ref;
    // staging of a chunk (references [c0, c0 + 128)): thread k loads 64-bit
    // words k, k + 256, ... of the chunk into registers, and later expands
    // each into 64 bytes of its reference's LDS row (rows past the end: zeros)
    constexpr int kWords = kChunk * W, kPer = (kWords + 255) / 256;
    uint64_t raw[kPer];
    auto load = [&](int64_t c0) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int p = tid + 256 * i;
            const int64_t j = c0 + p / W;
            raw[i] = (p < kWords && j < j_end) ? __builtin_nontemporal_load(&ref[j * W + p % W]) : 0;
        }
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int p = tid + 256 * i;
            if (p >= kWords) continue;
            unsigned char* dst = &sA[buf][(p / W) * kRow + 64 * (p % W)];
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const uint32_t x = (uint32_t)(raw[i] >> (16 * h));
                *reinterpret_cast<i32x4_t*>(dst + 16 * h) =
                    i32x4_t{(int32_t)spread4(x, 0), (int32_t)spread4(x, 1), (int32_t)spread4(x, 2),
                            (int32_t)spread4(x, 3)};
            }
        }
    };

    int32_t best_key[2] = {INT32_MIN, INT32_MIN};
    int32_t best_pair[2] = {0, 0};
    int buf = 0;
    if (j_begin < j_end) {
        load(j_begin);  // words past j_end load as 0: zero rows, masked below
        store(0);
    }
    for (int64_t c0 = j_begin; c0 < j_end; c0 += kChunk) {
        __syncthreads();  // chunk c0 is in sA[buf]; nobody reads sA[buf ^ 1] any more
        const bool more = c0 + kChunk < j_end;
        if (more) load(c0 + kChunk);  // in flight during this chunk's products
        const int cnt = (int)(j_end - c0 < kChunk ? j_end - c0 : kChunk);
        const int pair0 = (int)((c0 - j_begin) / 64);
#pragma unroll 1
        for (int pr = 0; pr < kChunk / 64; ++pr) {
            if (64 * pr >= cnt) break;
            i32x16_t acc[2][2];  // [column group][block of the pair]
#pragma unroll
            for (int ks = 0; ks < kSteps; ++ks) {
#pragma unroll
                for (int hb = 0; hb < 2; ++hb) {
                    // A operand: row l32 of block 2 pr + hb, bytes [32 ks + 16 half, +16)
                    const i32x4_t a = *reinterpret_cast<const i32x4_t*>(
                        &sA[buf][(64 * pr + 32 * hb + l32) * kRow + 32 * ks + 16 * half]);
#pragma unroll
                    for (int c = 0; c < 2; ++c)
                        acc[c][hb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
                            a, bop[c][ks], ks ? acc[c][hb] : (hb ? bias1 : bias0), 0, 0, 0);
                }
            }
            if (64 * pr + 64 > cnt) {  // the last, partial pair: rows past the end never win
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int r = 64 * pr + 8 * (v >> 2) + 4 * half + (v & 3);
#pragma unroll
                    for (int c = 0; c < 2; ++c) {
                        if (r >= cnt) acc[c][0][v] = kDead;
                        if (r + 32 >= cnt) acc[c][1][v] = kDead;
                    }
                }
            }
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                int32_t m = max3i(acc[c][0][0], acc[c][1][0], acc[c][0][1]);
#pragma unroll
                for (int v = 1; v < 16; ++v) m = max3i(m, acc[c][1][v], v < 15 ? acc[c][0][v + 1] : acc[c][1][v]);
                if ((m >> 6) > (best_key[c] >> 6)) {  // a larger product only: an earlier pair keeps a tie
                    best_key[c] = m;
                    best_pair[c] = pair0 + pr;
                }
            }
        }
        if (more) store(buf ^ 1);
        buf ^= 1;
    }

#pragma unroll
    for (int c = 0; c < 2; ++c) {
        // this lane's candidate: distance and global index; the two halves of a column meet
        const int32_t key = best_key[c];
        const int32_t hd = pop_t[c] - (key >> 6);
        const int64_t gi = j_begin + 64 * (int64_t)best_pair[c] + (63 - (key & 63));
        const int32_t okey = __shfl_xor(key, 32);
        const int32_t opair = __shfl_xor(best_pair[c], 32);
        const int32_t ohd = pop_t[c] - (okey >> 6);
        const int64_t ogi = j_begin + 64 * (int64_t)opair + (63 - (okey & 63));
        const bool has = key > kDead / 2, ohas = okey > kDead / 2;  // a real reference was seen
        // the better of the two: smaller distance, then lower index
        const bool take_other = ohas && (!has || ohd < hd || (ohd == hd && ogi < gi));
        const int32_t h_best = take_other ? ohd : hd;
        const int64_t i_best = take_other ? ogi : gi;
        if (half == 0 && t_ok[c] && (has || ohas)) {
            if (direct) {
                keys[tc[c]] = (uint32_t)i_best;
                if (dist) dist[tc[c]] = h_best;
            } else {
                atomicMin(&keys[tc[c]], ((uint32_t)h_best << kIdxBits) | (uint32_t)i_best);
            }
        }
    }
}

__global__ void mm_fill_kernel(uint32_t* p, int64_t n, uint32_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void mm_finalize_kernel(uint32_t* keys, int32_t* dist, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t k = keys[i];
    keys[i] = k & kIdxMask;
    if (dist) dist[i] = (int32_t)(k >> kIdxBits);
}

}  // namespace

hipError_t launch_match_mfma(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                             int32_t n_words, int32_t* idx, int32_t* dist, hipStream_t s) {
    const int64_t n_tiles = (n_tgt + kTgt - 1) / kTgt;
    // about 2048 workgroups, each split of at least 256 references (2 chunks)
    int64_t splits = (2048 + n_tiles - 1) / n_tiles;
    const int64_t max_splits = (n_ref + 255) / 256;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    if (splits > 65535) splits = 65535;
    int64_t per_split = (n_ref + splits - 1) / splits;
    per_split = (per_split + kChunk - 1) / kChunk * kChunk;  // whole chunks
    splits = (n_ref + per_split - 1) / per_split;
    auto* keys = reinterpret_cast<uint32_t*>(idx);
    const int direct = splits == 1;
    if (!direct)
        hipLaunchKernelGGL(mm_fill_kernel, dim3((unsigned)((n_tgt + 255) / 256)), dim3(256), 0, s, keys, n_tgt,
                           0xFFFFFFFFu);
    const dim3 grid((unsigned)n_tiles, (unsigned)splits);
    switch (n_words) {
    case 1: hipLaunchKernelGGL(match_mfma_kernel<1>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    case 2: hipLaunchKernelGGL(match_mfma_kernel<2>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    case 3: hipLaunchKernelGGL(match_mfma_kernel<3>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    default: hipLaunchKernelGGL(match_mfma_kernel<4>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, per_split, keys, dist, direct); break;
    }
    if (!direct)
        hipLaunchKernelGGL(mm_finalize_kernel, dim3((unsigned)((n_tgt + 255) / 256)), dim3(256), 0, s, keys, dist,
                           n_tgt);
    return hipGetLastError();
}

}  // namespace semshare
