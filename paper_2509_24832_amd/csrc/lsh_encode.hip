// Random-hyperplane LSH encode (Section 4.3, Appendix A.2): bit j of row t is
// [<x_t, r_j> > 0], packed LSB-first into 64-bit words.
//
// bf16: a [T, d] x [n_bits, d]^T GEMM on v_mfma_f32_32x32x16_bf16.  A
// workgroup owns 32 rows and all n_bits columns; wave w owns columns
// [32w, 32w + 32).  The hyperplanes (n_bits x d, L2-resident) are re-read by
// every workgroup, so the kernel is bound by how many bytes each CU keeps in
// flight: 64-wide K chunks of both operands stream through a ring of up to 7
// LDS stages filled by direct-to-LDS loads (6 chunks, 120 KB, in flight at
// 128 bits), with 128-byte rows whose 16-byte chunks are XOR-swizzled by
// (row / 2) mod 8.  Inside a chunk each lane half consumes its own 16-byte
// chunks (the K order is permuted identically for both operands, which leaves
// the dot products unchanged).  The epilogue never materialises the
// projections: a wave ballot of (acc > 0) over one accumulator register
// yields 32 code bits of two rows at once, written as 32-bit halves of the
// code words.  256-bit codes use a simpler variant that streams both operands
// through registers one chunk ahead.
//
// fp32: projections on the VALU (one lane per hyperplane, four partial sums),
// packed by a ballot over the 64 lanes of a wave.
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kCUs = 256;  // compute units of the chip

// Loads 32 bf16 (64 B) starting at p into four 8-element MFMA operands.
__device__ __forceinline__ void load_chunk(const uint16_t* p, bf16x8_t (&v)[4]) {
    const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint4 w = q[i];
        v[i] = __builtin_bit_cast(bf16x8_t, w);
    }
}

typedef __attribute__((address_space(3))) const bf16x8_t lds_bf16x8_t;

template <int NB>
struct LshCfg {
    static constexpr int kRows = 32 + 32 * NB;                // rows of a stage: 32 of x, then 32*NB planes
    static constexpr int kStage = kRows * 128;                 // bytes: 64 bf16 per row
    static constexpr int kStages = (144 * 1024) / kStage < 7 ? (144 * 1024) / kStage : 7;
    static constexpr int kLoads = kRows / 8;                   // 1-KB direct loads per stage (8 rows each)
    static constexpr int kLoadsPerWave = kLoads / NB;
    static_assert(kLoads % NB == 0, "loads divide over the waves");
    static_assert((kStages - 1) * kLoadsPerWave < 64, "vmcnt range");
};

template <int NB>  // n_bits / 32 = waves per workgroup (2 or 4)
__global__ __launch_bounds__(64 * NB) void lsh_encode_ring_kernel(const uint16_t* __restrict__ x,
                                                                  const uint16_t* __restrict__ planes,
                                                                  uint32_t* __restrict__ codes32,
                                                                  int64_t n_tok, int32_t dim) {
    using C = LshCfg<NB>;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[C::kStages * C::kStage];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int half = lane >> 5, l32 = lane & 31;
    const int64_t row0 = (int64_t)blockIdx.x * 32;
    const uint32_t smem_base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)smem;

    // direct-load sources: load i of a stage fills stage rows [8i, 8i + 8);
    // lane -> (row 8i + lane/8, physical chunk lane%8), fetching the logical
    // chunk the swizzle stores there.  Rows < 32 are rows of x (clamped to
    // the last token: computed, never stored), the rest hyperplanes.
    uint32_t off[C::kLoadsPerWave];
    bool is_x[C::kLoadsPerWave];
#pragma unroll
    for (int j = 0; j < C::kLoadsPerWave; ++j) {
        const int i = wave * C::kLoadsPerWave + j;
        const int r = 8 * i + (lane >> 3);
        const uint32_t chunk = (uint32_t)((lane & 7) ^ ((r >> 1) & 7));
        is_x[j] = r < 32;  // uniform per load: 8 rows never straddle row 32
        if (r < 32) {
            const int64_t t = row0 + r < n_tok ? r : n_tok - 1 - row0;
            off[j] = (uint32_t)(t * dim + 8 * chunk) * 2u;
        } else {
            off[j] = (uint32_t)((r - 32) * dim + 8 * chunk) * 2u;
        }
    }
    const uint16_t* xb = x + row0 * (int64_t)dim;
    auto issue = [&](int kt, int st) {
#pragma unroll
        for (int j = 0; j < C::kLoadsPerWave; ++j) {
            const int i = wave * C::kLoadsPerWave + j;
            g2lds(is_x[j] ? (const void*)(xb + (int64_t)kt * 64) : (const void*)(planes + (int64_t)kt * 64), off[j],
                  smem_base + st * C::kStage + i * 1024);
        }
    };
    const int nk = dim / 64;
    // workgroups walk the K chunks from staggered starts, so that they do not
    // all fetch the same hyperplane chunk (the same L2 channels) at once; the
    // ring always holds kStages - 1 chunks in flight, and past the last chunk
    // the last one is fetched again into a stage nobody reads any more
    const int k0 = (int)((blockIdx.x * 5u) % (unsigned)nk);
    auto chunk_of = [&](int i) { const int c = k0 + (i < nk ? i : nk - 1); return c < nk ? c : c - nk; };
#pragma unroll
    for (int c = 0; c < C::kStages - 1; ++c) issue(chunk_of(c), c);

    // read offsets: A rows l32, B rows 32 + 32 wave + l32; step s of a chunk
    // reads 16-byte chunk 4 half + s, at its swizzled place
    const uint32_t a_ro = l32 * 128, b_ro = (32 + 32 * wave + l32) * 128;
    uint32_t koff[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) koff[s] = (uint32_t)(((4 * half + s) ^ ((l32 >> 1) & 7)) << 4);

    f32x16_t acc = {};
    int st = 0;
    for (int kt = 0; kt < nk; ++kt) {
        wait_vmcnt<(C::kStages - 2) * C::kLoadsPerWave>();  // chunk kt has landed
        ring_barrier();  // ... for every wave, and every wave is done with chunk kt - 1
        issue(chunk_of(kt + C::kStages - 1), st == 0 ? C::kStages - 1 : st - 1);  // into chunk kt - 1's stage
        const uint32_t sb = smem_base + st * C::kStage;
        bf16x8_t a[4], b[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            a[s] = *(lds_bf16x8_t*)(uintptr_t)(sb + a_ro + koff[s]);
            b[s] = *(lds_bf16x8_t*)(uintptr_t)(sb + b_ro + koff[s]);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], b[s], acc, 0, 0, 0);
        st = st + 1 == C::kStages ? 0 : st + 1;
    }
    wait_vmcnt<0>();  // the repeated loads past the last chunk have landed before the workgroup ends

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

// RoPE fused into the encode (Section 4.3: the codes are taken of the
// RoPE-embedded rows): the same ring, but each workgroup owns R <= 32 rows
// (R chosen so that the rows spread over every CU) and rotates the x rows of
// a chunk in LDS once it has landed, one chunk ahead of the products.
// The workgroup has three waves per MFMA wave: the MFMA waves load and
// multiply, the other 2 NB waves only rotate (measured per chunk with cycle
// stamps: when the MFMA waves also rotated, the rotation was the longest
// part of their chunk and the other waves waited at the barrier).  Rotating
// thread k rotates the pairs k, k + 128 NB, ... of the chunk's R x 32
// (even, odd) pairs; since 128 NB is a multiple of 32 its pair column k % 32
// is fixed, so its theta follows the chunks by one fp64 multiply
// (theta_{k+32} = theta_k * base^(-64 / dim)).  The angle is reduced in fp64 revolutions
// and rotated with the hardware sine and cosine; the rotated pair is rounded
// to bf16, as the unfused path stores it.  The codes therefore equal those of
// rope_embed + lsh_encode except where a projection lies within rounding
// distance of zero.
constexpr int kRotWaves = 3;  // waves per MFMA wave: 1 multiplies and loads, 2 rotate
template <int NB>  // n_bits / 32 = MFMA waves (2 or 4); twice as many more waves only rotate
__global__ __launch_bounds__(64 * kRotWaves * NB) void rope_lsh_ring_kernel(const uint16_t* __restrict__ x,
                                                                const uint16_t* __restrict__ planes,
                                                                uint32_t* __restrict__ codes32, int64_t n_tok,
                                                                int32_t dim, int32_t rows, int64_t pos0,
                                                                double log2_base) {
    using C = LshCfg<NB>;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[C::kStages * C::kStage];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, l32 = lane & 31;
    const int64_t row0 = (int64_t)blockIdx.x * rows;
    const int64_t last = (row0 + rows < n_tok ? row0 + rows : n_tok) - 1 - row0;  // last live row of the tile
    const uint32_t smem_base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)smem;

    const bool mma_wave = wave < NB;  // waves NB .. 3 NB - 1 load nothing and only rotate
    // direct-load sources as in lsh_encode_ring_kernel; x rows past the
    // tile's last live row repeat it (computed, never stored)
    uint32_t off[C::kLoadsPerWave];
    bool is_x[C::kLoadsPerWave];
#pragma unroll
    for (int j = 0; j < C::kLoadsPerWave; ++j) {
        const int i = (mma_wave ? wave : 0) * C::kLoadsPerWave + j;
        const int r = 8 * i + (lane >> 3);
        const uint32_t chunk = (uint32_t)((lane & 7) ^ ((r >> 1) & 7));
        is_x[j] = r < 32;
        if (r < 32) {
            const int64_t t = r < last ? r : last;
            off[j] = (uint32_t)(t * dim + 8 * chunk) * 2u;
        } else {
            off[j] = (uint32_t)((r - 32) * dim + 8 * chunk) * 2u;
        }
    }
    const uint16_t* xb = x + row0 * (int64_t)dim;
    auto issue = [&](int kt, int st) {
        if (!mma_wave) return;
#pragma unroll
        for (int j = 0; j < C::kLoadsPerWave; ++j) {
            const int i = wave * C::kLoadsPerWave + j;
            g2lds(is_x[j] ? (const void*)(xb + (int64_t)kt * 64) : (const void*)(planes + (int64_t)kt * 64), off[j],
                  smem_base + st * C::kStage + i * 1024);
        }
    };
    const int nk = dim / 64;
    // staggered chunk order, as in lsh_encode_ring_kernel
    const int k0 = (int)((blockIdx.x * 5u) % (unsigned)nk);
    auto chunk_of = [&](int i) { const int c = k0 + (i < nk ? i : nk - 1); return c < nk ? c : c - nk; };
#pragma unroll
    for (int c = 0; c < C::kStages - 1; ++c) issue(chunk_of(c), c);

    // this thread's pair column, its theta (in revolutions: theta / 2 pi) at
    // chunk 0 and at the first chunk it rotates, and the step per chunk
    const int kl = tid & 31;
    const double theta_rev0 = exp2(-(2.0 * (double)kl / (double)dim) * log2_base) * 0.15915494309189535;
    double theta_rev = exp2(-(2.0 * (double)(32 * k0 + kl) / (double)dim) * log2_base) * 0.15915494309189535;
    const double theta_step = exp2(-(64.0 / (double)dim) * log2_base);
    int rot_chunk = k0;
    const int n_pairs = (int)(last + 1) * 32;
    const uint32_t rot_col = (uint32_t)((kl & 3) * 4);
    // rotates the live x rows of the chunk in stage `st_r` in place: the angle
    // m theta in revolutions, reduced in fp64, then v_sin_f32 / v_cos_f32
    // (which take revolutions)
    auto rotate = [&](int st_r) {
        // up to four pairs per thread (R <= 32 rows x 32 pairs over the
        // 128 NB >= 256 rotating threads): all loads first, then independent
        // chains, then the stores, so that their latencies overlap
        const uint32_t sb = smem_base + st_r * C::kStage;
        if (mma_wave) return;
        const int rt = tid - 64 * NB;  // thread index among the rotating waves
        constexpr int kRt = 64 * (kRotWaves - 1) * NB;  // rotating threads
        constexpr int kIt = 32 * 32 / kRt;
        uint32_t w[kIt];
        __attribute__((address_space(3))) uint32_t* q[kIt];
#pragma unroll
        for (int i = 0; i < kIt; ++i) {
            const int r = (rt + kRt * i) >> 5;
            const uint32_t addr = sb + (uint32_t)r * 128u + ((uint32_t)((kl >> 2) ^ ((r >> 1) & 7)) << 4) + rot_col;
            q[i] = (__attribute__((address_space(3))) uint32_t*)(uintptr_t)addr;
            w[i] = rt + kRt * i < n_pairs ? *q[i] : 0u;
        }
#pragma unroll
        for (int i = 0; i < kIt; ++i) {
            const int r = (rt + kRt * i) >> 5;
            const double tr = (double)(pos0 + row0 + r) * theta_rev;
            const float rev = (float)(tr - floor(tr));
            const float sn = __builtin_amdgcn_sinf(rev), cs = __builtin_amdgcn_cosf(rev);
            const float x0 = bf16_lo(w[i]), x1 = bf16_hi(w[i]);
            w[i] = pack_bf16x2(cs * x0 - sn * x1, sn * x0 + cs * x1);
        }
#pragma unroll
        for (int i = 0; i < kIt; ++i)
            if (rt + kRt * i < n_pairs) *q[i] = w[i];
        if (++rot_chunk == nk) {  // the order wraps to chunk 0
            rot_chunk = 0;
            theta_rev = theta_rev0;
        } else {
            theta_rev *= theta_step;
        }
    };

    const uint32_t a_ro = l32 * 128, b_ro = (32 + 32 * wave + l32) * 128;
    uint32_t koff[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) koff[s] = (uint32_t)(((4 * half + s) ^ ((l32 >> 1) & 7)) << 4);

    // pipeline: chunk kt + 1 is rotated while chunk kt is multiplied; one
    // barrier per chunk publishes the rotation and frees the oldest stage
    wait_vmcnt<(C::kStages - 2) * C::kLoadsPerWave>();  // chunk 0 has landed
    ring_barrier();
    rotate(0);
    f32x16_t acc = {};
    int st = 0;
    for (int kt = 0; kt < nk; ++kt) {
        wait_vmcnt<(C::kStages - 3) * C::kLoadsPerWave>();  // chunk kt + 1 has landed
        ring_barrier();  // chunk kt rotated; every wave is done with chunk kt - 1
        issue(chunk_of(kt + C::kStages - 1), st == 0 ? C::kStages - 1 : st - 1);
        if (mma_wave) {
            const uint32_t sb = smem_base + st * C::kStage;
            bf16x8_t a[4], b[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                a[s] = *(lds_bf16x8_t*)(uintptr_t)(sb + a_ro + koff[s]);
                b[s] = *(lds_bf16x8_t*)(uintptr_t)(sb + b_ro + koff[s]);
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], b[s], acc, 0, 0, 0);
        }
        st = st + 1 == C::kStages ? 0 : st + 1;
        if (kt + 1 < nk) rotate(st);
    }
    wait_vmcnt<0>();
    if (!mma_wave) return;

    constexpr int words32 = NB;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const uint64_t bits = __ballot(acc[v] > 0.0f);
        const int r_lo = 8 * (v / 4) + (v % 4);
        if (lane == 0 && r_lo <= last) codes32[(row0 + r_lo) * words32 + wave] = (uint32_t)bits;
        if (lane == 1 && r_lo + 4 <= last) codes32[(row0 + r_lo + 4) * words32 + wave] = (uint32_t)(bits >> 32);
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

hipError_t launch_rope_lsh_encode(const void* x, const void* planes, uint64_t* codes, int64_t n_tok, int32_t dim,
                                  int32_t n_bits, int64_t pos0, double base, hipStream_t s) {
    // rows per workgroup: enough workgroups for every CU (the rotation is
    // per-row VALU work), at most the 32 rows of an MFMA tile
    int64_t rows = (n_tok + kCUs - 1) / kCUs;
    if (rows > 32) rows = 32;
    if (rows < 1) rows = 1;
    const dim3 grid((unsigned)((n_tok + rows - 1) / rows));
    const auto* xp = static_cast<const uint16_t*>(x);
    const auto* pp = static_cast<const uint16_t*>(planes);
    auto* cp = reinterpret_cast<uint32_t*>(codes);
    const double lb = log2(base);
    if (n_bits == 64)
        hipLaunchKernelGGL(rope_lsh_ring_kernel<2>, grid, dim3(64 * kRotWaves * 2), 0, s, xp, pp, cp, n_tok, dim, (int32_t)rows, pos0, lb);
    else
        hipLaunchKernelGGL(rope_lsh_ring_kernel<4>, grid, dim3(64 * kRotWaves * 4), 0, s, xp, pp, cp, n_tok, dim, (int32_t)rows, pos0, lb);
    return hipGetLastError();
}

hipError_t launch_lsh_encode(const void* x, const void* planes, uint64_t* codes, int64_t n_tok,
                             int32_t dim, int32_t n_bits, int dtype, hipStream_t s) {
    if (dtype == SEMSHARE_BF16) {
        const dim3 grid((unsigned)((n_tok + 31) / 32));
        const auto* xp = static_cast<const uint16_t*>(x);
        const auto* pp = static_cast<const uint16_t*>(planes);
        auto* cp = reinterpret_cast<uint32_t*>(codes);
        switch (n_bits) {
        case 64: hipLaunchKernelGGL(lsh_encode_ring_kernel<2>, grid, dim3(128), 0, s, xp, pp, cp, n_tok, dim); break;
        case 128: hipLaunchKernelGGL(lsh_encode_ring_kernel<4>, grid, dim3(256), 0, s, xp, pp, cp, n_tok, dim); break;
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
