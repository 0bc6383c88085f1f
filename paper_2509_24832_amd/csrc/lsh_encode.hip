// Random-hyperplane LSH encode (Section 4.3, Appendix A.2): bit j of row t is
// [<x_t, r_j> > 0], packed LSB-first into 64-bit words.
//
// bf16: a [T, d] x [n_bits, d]^T GEMM on v_mfma_f32_32x32x16_bf16.  A
// workgroup owns 32 rows and all n_bits columns; wave w owns columns
// [32w, 32w + 32).  Each lane streams 64 contiguous bytes of its row (and of
// its hyperplane) per 64-wide K chunk; the K order inside the chunk is
// permuted identically for both operands, which leaves the dot products
// unchanged.  The epilogue never materialises the projections: a wave ballot
// of (acc > 0) over one accumulator register yields 32 code bits of two rows
// at once, written as 32-bit halves of the code words.
//
// fp32: projections on the VALU (one lane per hyperplane, four partial sums),
// packed by a ballot over the 64 lanes of a wave.
#include "semshare_internal.h"

namespace semshare {
namespace {

// Loads 32 bf16 (64 B) starting at p into four 8-element MFMA operands.
__device__ __forceinline__ void load_chunk(const uint16_t* p, bf16x8_t (&v)[4]) {
    const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint4 w = q[i];
        v[i] = __builtin_bit_cast(bf16x8_t, w);
    }
}

template <int NB>  // n_bits / 32 = waves per workgroup
__global__ __launch_bounds__(64 * NB) void lsh_encode_bf16_kernel(const uint16_t* __restrict__ x,
                                                                   const uint16_t* __restrict__ planes,
                                                                   uint32_t* __restrict__ codes32,
                                                                   int64_t n_tok, int32_t dim) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int half = lane >> 5;
    const int64_t row0 = (int64_t)blockIdx.x * 32;
    int64_t row = row0 + (lane & 31);
    if (row > n_tok - 1) row = n_tok - 1;  // rows past the end compute garbage, never stored
    const uint16_t* xa = x + row * (int64_t)dim + 32 * half;
    const uint16_t* pb = planes + (int64_t)(32 * wave + (lane & 31)) * dim + 32 * half;

    f32x16_t acc = {};
    bf16x8_t a[4], b[4], an[4], bn[4];
    load_chunk(xa, a);
    load_chunk(pb, b);
    for (int32_t k0 = 64; k0 <= dim; k0 += 64) {
        const bool more = k0 < dim;
        if (more) {
            load_chunk(xa + k0, an);
            load_chunk(pb + k0, bn);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], b[s], acc, 0, 0, 0);
        if (more) {
#pragma unroll
            for (int s = 0; s < 4; ++s) { a[s] = an[s]; b[s] = bn[s]; }
        }
    }

    // acc[v] holds C[row = 8*(v/4) + 4*half + (v%4)][col = 32*wave + (lane%32)]
    constexpr int words32 = NB;  // 32-bit halves per code row
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const uint64_t bits = __ballot(acc[v] > 0.0f);
        const int r_lo = 8 * (v / 4) + (v % 4);
        const int64_t t_lo = row0 + r_lo, t_hi = t_lo + 4;
        if (lane == 0 && t_lo < n_tok) codes32[t_lo * words32 + wave] = (uint32_t)bits;
        if (lane == 1 && t_hi < n_tok) codes32[t_hi * words32 + wave] = (uint32_t)(bits >> 32);
    }
}

__global__ __launch_bounds__(256) void lsh_encode_f32_kernel(const float* __restrict__ x,
                                                             const float* __restrict__ planes,
                                                             uint64_t* __restrict__ codes,
                                                             int64_t n_tok, int32_t dim,
                                                             int32_t n_words) {
    const int lane = threadIdx.x & 63;
    const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (row, word)
    if (item >= n_tok * n_words) return;
    const int64_t t = item / n_words;
    const int w = (int)(item % n_words);
    const float4* xr = reinterpret_cast<const float4*>(x + t * (int64_t)dim);
    const float4* rr = reinterpret_cast<const float4*>(planes + (int64_t)(64 * w + lane) * dim);
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    for (int32_t i = 0; i < dim / 4; ++i) {
        const float4 a = xr[i], b = rr[i];
        s0 = fmaf(a.x, b.x, s0);
        s1 = fmaf(a.y, b.y, s1);
        s2 = fmaf(a.z, b.z, s2);
        s3 = fmaf(a.w, b.w, s3);
    }
    const float p = (s0 + s1) + (s2 + s3);
    const uint64_t bits = __ballot(p > 0.0f);
    if (lane == 0) codes[t * n_words + w] = bits;
}

}  // namespace

hipError_t launch_lsh_encode(const void* x, const void* planes, uint64_t* codes, int64_t n_tok,
                             int32_t dim, int32_t n_bits, int dtype, hipStream_t s) {
    if (dtype == SEMSHARE_BF16) {
        const dim3 grid((unsigned)((n_tok + 31) / 32));
        const auto* xp = static_cast<const uint16_t*>(x);
        const auto* pp = static_cast<const uint16_t*>(planes);
        auto* cp = reinterpret_cast<uint32_t*>(codes);
        switch (n_bits) {
        case 64: hipLaunchKernelGGL(lsh_encode_bf16_kernel<2>, grid, dim3(128), 0, s, xp, pp, cp, n_tok, dim); break;
        case 128: hipLaunchKernelGGL(lsh_encode_bf16_kernel<4>, grid, dim3(256), 0, s, xp, pp, cp, n_tok, dim); break;
        default: hipLaunchKernelGGL(lsh_encode_bf16_kernel<8>, grid, dim3(512), 0, s, xp, pp, cp, n_tok, dim); break;
        }
        return hipGetLastError();
    }
    const int32_t n_words = n_bits / 64;
    const int64_t items = n_tok * n_words;
    hipLaunchKernelGGL(lsh_encode_f32_kernel, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, s,
                       static_cast<const float*>(x), static_cast<const float*>(planes), codes, n_tok,
                       dim, n_words);
    return hipGetLastError();
}

}  // namespace semshare
