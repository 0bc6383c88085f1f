// RoPE injected into token embeddings (Section 4.3.1, Appendix A.1 Eq. 1,
// read as the standard rotary embedding with angle m * theta_k).
//
// HBM-bound elementwise pass: each thread owns VEC consecutive (even, odd)
// pairs of a row segment and walks several rows, so theta_k (an fp64 power)
// is formed once per thread and reused.  Angles are formed and reduced in
// fp64, rotated in fp32.  Loads/stores are 16-byte vectors when the width
// allows it.
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kThreads = 256;

template <int VEC>
struct PairsBF16 {
    uint32_t w[VEC];  // each word = one (even, odd) pair
};

template <int DT, int VEC>
__global__ __launch_bounds__(kThreads) void rope_embed_kernel(const void* x, void* y,
                                                              int64_t n_tok,
                                                              int32_t dim, int64_t pos0,
                                                              double log2_base,
                                                              int64_t rows_per_block) {
    const int32_t half = dim / 2;
    const int64_t pair0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * VEC;
    if (pair0 >= half) return;
    double theta[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v)
        theta[v] = exp2(-(2.0 * (double)(pair0 + v) / (double)dim) * log2_base);

    const int64_t r0 = (int64_t)blockIdx.y * rows_per_block;
    const int64_t r1 = r0 + rows_per_block < n_tok ? r0 + rows_per_block : n_tok;
    for (int64_t r = r0; r < r1; ++r) {
        const double m = (double)(pos0 + r);
        const int64_t off = r * (int64_t)half + pair0;  // in pairs
        float x0[VEC], x1[VEC];
        if constexpr (DT == SEMSHARE_BF16) {
            const uint32_t* src = reinterpret_cast<const uint32_t*>(x) + off;
            PairsBF16<VEC> in;
            if constexpr (VEC == 4) {
                *reinterpret_cast<uint4*>(in.w) = *reinterpret_cast<const uint4*>(src);
            } else {
#pragma unroll
                for (int v = 0; v < VEC; ++v) in.w[v] = src[v];
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v) { x0[v] = bf16_lo(in.w[v]); x1[v] = bf16_hi(in.w[v]); }
        } else {
            const float* src = reinterpret_cast<const float*>(x) + 2 * off;
#pragma unroll
            for (int v = 0; v < VEC; ++v) { x0[v] = src[2 * v]; x1[v] = src[2 * v + 1]; }
        }
        float y0[VEC], y1[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            float s, c;
            rope_sincos(m, theta[v], &s, &c);
            y0[v] = c * x0[v] - s * x1[v];
            y1[v] = s * x0[v] + c * x1[v];
        }
        if constexpr (DT == SEMSHARE_BF16) {
            uint32_t* dst = reinterpret_cast<uint32_t*>(y) + off;
            PairsBF16<VEC> outw;
#pragma unroll
            for (int v = 0; v < VEC; ++v) outw.w[v] = pack_bf16x2(y0[v], y1[v]);
            if constexpr (VEC == 4) {
                *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(outw.w);
            } else {
#pragma unroll
                for (int v = 0; v < VEC; ++v) dst[v] = outw.w[v];
            }
        } else {
            float* dst = reinterpret_cast<float*>(y) + 2 * off;
#pragma unroll
            for (int v = 0; v < VEC; ++v) { dst[2 * v] = y0[v]; dst[2 * v + 1] = y1[v]; }
        }
    }
}

template <int DT, int VEC>
hipError_t launch(const void* x, void* y, int64_t n_tok, int32_t dim, int64_t pos0, double base,
                  hipStream_t s) {
    const int64_t half = dim / 2;
    const int64_t col_blocks = (half + (int64_t)kThreads * VEC - 1) / ((int64_t)kThreads * VEC);
    // about 4 rows per block, fewer blocks along y if the grid limit requires it
    int64_t gy = (n_tok + 3) / 4;
    if (gy > 65535) gy = 65535;
    const int64_t rows_per_block = (n_tok + gy - 1) / gy;
    gy = (n_tok + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL((rope_embed_kernel<DT, VEC>), dim3((unsigned)col_blocks, (unsigned)gy),
                       dim3(kThreads), 0, s, x, y, n_tok, dim, pos0, log2(base), rows_per_block);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_rope_embed(const void* x, void* y, int64_t n_tok, int32_t dim, int64_t pos0,
                             double base, int dtype, hipStream_t s) {
    const bool vec = (dim % 8) == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(y) % 16 == 0;
    if (dtype == SEMSHARE_BF16)
        return vec ? launch<SEMSHARE_BF16, 4>(x, y, n_tok, dim, pos0, base, s)
                   : launch<SEMSHARE_BF16, 1>(x, y, n_tok, dim, pos0, base, s);
    return vec ? launch<SEMSHARE_FP32, 4>(x, y, n_tok, dim, pos0, base, s)
               : launch<SEMSHARE_FP32, 1>(x, y, n_tok, dim, pos0, base, s);
}

}  // namespace semshare
