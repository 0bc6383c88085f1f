// Reference retrieval over a bank of prompts (Appendix A.3 score, Section 5
// gate): for each reference prompt b (codes [offsets[b], offsets[b+1]) of the
// bank) the sum over the target tokens of their top-1 Hamming distance within
// that prompt, and the similarity clip(1 - (mean - dmin) / (dmax - dmin), 0, 1)
// of the mean.  A prompt with no tokens counts every target token at the
// largest distance, 64 * n_words.
//
// Integer VALU kernel on the match kernel's scheme: a workgroup owns 128
// target codes (two per lane, in VGPRs) and one prompt, whose codes are staged
// through LDS and read by every lane of a wave at the same address
// (broadcast), the four waves taking interleaved codes.  Per pair: 2W XORs
// and 2W accumulating popcounts and one min.  The workgroup's 128 minima are
// summed to one partial per (target tile, prompt); a second kernel, one wave
// per prompt, adds a prompt's partials (integers: the result does not depend
// on the order) and forms the score in fp64.
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kStage = 512;  // reference codes per LDS stage
constexpr int kR = 2;        // target codes per lane
constexpr int kTile = 64 * kR;

template <int W>
__global__ __launch_bounds__(256) void bank_dist_kernel(const uint64_t* __restrict__ tgt, int64_t n_tgt,
                                                        const uint64_t* __restrict__ ref, int64_t n_ref,
                                                        const int64_t* __restrict__ offsets, int32_t n_prompts,
                                                        int64_t* __restrict__ partial) {
    __shared__ uint64_t sref[kStage * W];
    __shared__ uint32_t sred[4][kTile];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t t_base = (int64_t)blockIdx.x * kTile;
    const int b = blockIdx.y;

    uint32_t tc[kR][2 * W];
#pragma unroll
    for (int r = 0; r < kR; ++r) {
        int64_t t = t_base + lane + 64 * r;
        if (t > n_tgt - 1) t = n_tgt - 1;  // past the end: computed, not counted
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const uint64_t c = tgt[t * W + w];
            tc[r][2 * w] = (uint32_t)c;
            tc[r][2 * w + 1] = (uint32_t)(c >> 32);
        }
    }
    // the prompt's codes, clamped to the bank (offsets are the caller's contract)
    int64_t lo = offsets[b], hi = offsets[b + 1];
    lo = lo < 0 ? 0 : (lo > n_ref ? n_ref : lo);
    hi = hi < lo ? lo : (hi > n_ref ? n_ref : hi);
    uint32_t best[kR];
#pragma unroll
    for (int r = 0; r < kR; ++r) best[r] = 64u * W;  // the distance to an empty prompt

    for (int64_t s0 = lo; s0 < hi; s0 += kStage) {
        const int cnt = (int)(hi - s0 < kStage ? hi - s0 : kStage);
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
#pragma unroll
            for (int r = 0; r < kR; ++r) {
                uint32_t d = 0;
#pragma unroll
                for (int w = 0; w < 2 * W; ++w) d += __popc(tc[r][w] ^ rc[w]);
                best[r] = best[r] < d ? best[r] : d;
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kR; ++r) sred[wave][lane + 64 * r] = best[r];
    __syncthreads();
    if (wave == 0) {
        uint32_t sum = 0;  // at most 128 * 256: no overflow
#pragma unroll
        for (int r = 0; r < kR; ++r) {
            uint32_t m = sred[0][lane + 64 * r];
#pragma unroll
            for (int w = 1; w < 4; ++w) {
                const uint32_t o = sred[w][lane + 64 * r];
                m = m < o ? m : o;
            }
            if (t_base + lane + 64 * r < n_tgt) sum += m;
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
        if (lane == 0) partial[blockIdx.x * (int64_t)n_prompts + b] = (int64_t)sum;
    }
}

// One wave per prompt: the lanes add strided tile partials, then the wave
// adds the lanes (integer sums: the order does not change the result).
__global__ __launch_bounds__(64) void bank_final_kernel(const int64_t* __restrict__ partial, int64_t n_tiles,
                                                        int32_t n_prompts, int64_t n_tgt, double dmin, double dmax,
                                                        int64_t* __restrict__ dist_sum,
                                                        double* __restrict__ similarity) {
    const int b = blockIdx.x, lane = threadIdx.x;
    int64_t s = 0;
    for (int64_t k = lane; k < n_tiles; k += 64) s += partial[k * n_prompts + b];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
    if (lane != 0) return;
    dist_sum[b] = s;
    double sim = 0.0;
    if (n_tgt > 0) {
        const double mean = (double)s / (double)n_tgt;
        sim = 1.0 - (mean - dmin) / (dmax - dmin);
        sim = sim < 0.0 ? 0.0 : (sim > 1.0 ? 1.0 : sim);
    }
    similarity[b] = sim;
}

}  // namespace

size_t bank_similarity_workspace(int64_t n_tgt, int32_t n_prompts) {
    const int64_t n_tiles = (n_tgt + kTile - 1) / kTile;
    return (size_t)n_tiles * (size_t)(n_prompts > 0 ? n_prompts : 0) * sizeof(int64_t);
}

hipError_t launch_bank_similarity(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                                  const int64_t* offsets, int32_t n_prompts, int32_t n_words, double dmin,
                                  double dmax, int64_t* dist_sum, double* similarity, void* workspace,
                                  hipStream_t s) {
    const int64_t n_tiles = (n_tgt + kTile - 1) / kTile;
    auto* partial = static_cast<int64_t*>(workspace);
    if (n_tiles > 0) {
        const dim3 grid((unsigned)n_tiles, (unsigned)n_prompts);
        switch (n_words) {
        case 1: hipLaunchKernelGGL(bank_dist_kernel<1>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, offsets, n_prompts, partial); break;
        case 2: hipLaunchKernelGGL(bank_dist_kernel<2>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, offsets, n_prompts, partial); break;
        case 3: hipLaunchKernelGGL(bank_dist_kernel<3>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, offsets, n_prompts, partial); break;
        default: hipLaunchKernelGGL(bank_dist_kernel<4>, grid, dim3(256), 0, s, tgt, n_tgt, ref, n_ref, offsets, n_prompts, partial); break;
        }
    }
    hipLaunchKernelGGL(bank_final_kernel, dim3((unsigned)n_prompts), dim3(64), 0, s, partial, n_tiles, n_prompts, n_tgt,
                       dmin, dmax, dist_sum, similarity);
    return hipGetLastError();
}

}  // namespace semshare
