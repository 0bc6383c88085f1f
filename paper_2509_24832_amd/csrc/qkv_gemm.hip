// Q/K/V projection of the recomputed tokens (Sections 4.2, 4.3.3) with the
// RoPE / deviation / cache-scatter epilogue, bf16 on v_mfma_f32_32x32x16_bf16.
//
// C[n_sel, Nq + 2 Nkv] = X_sel [n_sel, hidden] . [Wq; Wk; Wv]^T  (all K-major)
//
// Tiling for gfx950: a 256-thread workgroup owns a 128 x BN output tile (BN =
// 256, or 128 when a segment is narrower) and runs alone on its CU; each wave
// owns a 64 x BN/2 sub-tile (2 x BN/64 accumulators of 32x32).  K advances in
// 64-wide tiles through a 3-stage LDS ring filled with direct-to-LDS loads
// (global_load_lds_dwordx4): two tiles are always in flight while the third
// is multiplied, and no VGPRs are spent on staging.  Rows are 128 B in LDS
// with the 16-byte chunk index XOR-swizzled by (row / 2) mod 8, so the 32
// rows a wave reads for one MFMA operand cover all 64 banks twice.  Inside a
// K tile each lane half consumes a contiguous 64-byte run of its row (the K
// order is permuted identically for both operands, which leaves every dot
// product unchanged).
//
// Epilogue through an fp32 LDS tile: RoPE of q/k pairs from the per-row
// (cos, sin) table, bf16 rounding, q to its buffer, k/v scattered to the cache
// rows sel_pos after the squared differences against the old rows are summed
// per tile (the deviation, reduced later in a fixed order).  Workgroups are
// mapped XCD-major: all M tiles of one weight tile run on the same XCD, so the
// weights are fetched from HBM once per XCD.
#include <type_traits>

#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kBM = 128, kBK = 64, kStages = 3;

template <int BN>
struct Cfg {
    static constexpr int kABytes = kBM * kBK * 2;  // 16 KB
    static constexpr int kBBytes = BN * kBK * 2;   // 32 KB (BN = 256)
    static constexpr int kStage = kABytes + kBBytes;
    static constexpr int kLdc = BN + 8;  // floats per epilogue row (acc writes conflict-free)
    static constexpr int kEpi = kBM * kLdc * 4;
    static constexpr int kLds = kStages * kStage > kEpi ? kStages * kStage : kEpi;
    static constexpr int kNB = BN / 64;       // 32-wide column blocks per wave
    static constexpr int kALoads = kBM / 32;  // 1-KB direct loads per wave per K tile
    static constexpr int kBLoads = BN / 32;
    static constexpr int kLoads = kALoads + kBLoads;
};

typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void g2lds(const void* g, unsigned char* lds) {
    __builtin_amdgcn_global_load_lds(g, (lds_void_t*)lds, 16, 0, 0);
}

// s_waitcnt vmcnt(n) (n < 16), other counters left at their maximum.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 16, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ int swz(int row, int chunk) { return ((chunk ^ ((row >> 1) & 7)) << 4); }

// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would wait for every in-flight direct-to-LDS load (vmcnt(0)) and drain the
// ring.  Visibility of a stage is established explicitly instead: each wave
// waits for its own loads of that stage (vmcnt), then all waves meet here.
// The empty asm statements keep the compiler from moving LDS accesses across.
__device__ __forceinline__ void ring_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int BN>
__global__ __launch_bounds__(256, 1) void qkv_gemm_kernel(GemmArgs g) {
    using C = Cfg<BN>;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[C::kLds];

    const int b = blockIdx.x;
    const int xcd = b & 7;
    const int j = b >> 3;
    const int n_idx = xcd + 8 * (j / g.n_mt);
    const int m_idx = j % g.n_mt;
    if (n_idx >= g.n_nt) return;
    int seg = 0, nt = n_idx;
    if (nt >= g.seg_tiles[0]) {
        nt -= g.seg_tiles[0];
        seg = 1;
        if (nt >= g.seg_tiles[1]) { nt -= g.seg_tiles[1]; seg = 2; }
    }
    const uint16_t* wseg = seg == 0 ? g.w[0] : (seg == 1 ? g.w[1] : g.w[2]);
    uint16_t* kvseg = seg == 2 ? g.kv[1] : g.kv[0];
    const int seg_cols = seg == 0 ? g.seg_cols[0] : g.seg_cols[1];
    const int64_t m0 = (int64_t)m_idx * kBM;
    const int32_t ncol0 = nt * BN;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: LDS targets stay scalar
    const int half = lane >> 5, l32 = lane & 31;
    const int wm = wave >> 1, wn = wave & 1;

    // Direct-load sources: instruction i of this wave fills LDS rows
    // [8*grp, 8*grp+8) of its operand; lane -> (row = 8*grp + lane/8, chunk pc = lane%8)
    // and loads the global chunk that the swizzle places there.  Sources are a
    // uniform base (advanced per K tile) plus a fixed per-lane 32-bit offset.
    const int lrow = lane >> 3, lpc = lane & 7;
    int32_t a_off[C::kALoads], b_off[C::kBLoads];
#pragma unroll
    for (int i = 0; i < C::kALoads; ++i) {
        const int row = 8 * (wave * C::kALoads + i) + lrow;
        int64_t grow = m0 + row;
        if (grow > g.n_sel - 1) grow = g.n_sel - 1;  // tail rows: computed, never stored
        a_off[i] = (int32_t)(grow * g.hidden) + 8 * (lpc ^ ((row >> 1) & 7));
    }
#pragma unroll
    for (int i = 0; i < C::kBLoads; ++i) {
        const int row = 8 * (wave * C::kBLoads + i) + lrow;
        b_off[i] = (ncol0 + row) * g.hidden + 8 * (lpc ^ ((row >> 1) & 7));
    }
    // load j (0 .. kLoads-1) of K tile kt into ring stage ST
    auto issue_one = [&](int j, int kt, unsigned char* stage) {
        if (j < C::kALoads)
            g2lds(g.x + (int64_t)kt * kBK + a_off[j], stage + (wave * C::kALoads + j) * 1024);
        else
            g2lds(wseg + (int64_t)kt * kBK + b_off[j - C::kALoads],
                  stage + C::kABytes + (wave * C::kBLoads + (j - C::kALoads)) * 1024);
    };

    f32x16_t acc[2][C::kNB];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int k = 0; k < C::kNB; ++k) acc[i][k] = f32x16_t{};

    // read offsets: rows of both operands are 32-aligned plus l32, so the
    // swizzle term depends on l32 only
    int koff[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) koff[s] = swz(l32, 4 * half + s);
    const int a_row0 = (64 * wm + l32) * 128;
    const int b_row0 = ((BN / 2) * wn + l32) * 128;

    const int nk = g.hidden / kBK;
    for (int j = 0; j < C::kLoads; ++j) issue_one(j, 0, smem);
    if (nk > 1)
        for (int j = 0; j < C::kLoads; ++j) issue_one(j, 1, smem + C::kStage);

    // one K tile on ring stage ST (compile-time, so every LDS address is a constant)
    auto step = [&](auto st_c, int kt) {
        constexpr int ST = decltype(st_c)::value;
        constexpr int NEXT = (ST + 2) % kStages;
        if (kt + 1 < nk) wait_vmcnt<C::kLoads>();
        else wait_vmcnt<0>();
        ring_barrier();  // tile kt visible to all waves; stage NEXT free again
        const bool more = kt + 2 < nk;
        const unsigned char* Ab = smem + ST * C::kStage;
        const unsigned char* Bb = Ab + C::kABytes;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            bf16x8_t av[2], bv[C::kNB];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                av[i] = *reinterpret_cast<const bf16x8_t*>(Ab + a_row0 + i * 32 * 128 + koff[s]);
#pragma unroll
            for (int k = 0; k < C::kNB; ++k)
                bv[k] = *reinterpret_cast<const bf16x8_t*>(Bb + b_row0 + k * 32 * 128 + koff[s]);
            // spread the next-but-one tile's loads over the four k-steps
            if (more) {
#pragma unroll
                for (int j = s * C::kLoads / 4; j < (s + 1) * C::kLoads / 4; ++j)
                    issue_one(j, kt + 2, smem + NEXT * C::kStage);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int k = 0; k < C::kNB; ++k)
                    acc[i][k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[k], acc[i][k], 0, 0, 0);
        }
    };
    for (int kt = 0; kt < nk; kt += kStages) {
        step(std::integral_constant<int, 0>{}, kt);
        if (kt + 1 < nk) step(std::integral_constant<int, 1>{}, kt + 1);
        if (kt + 2 < nk) step(std::integral_constant<int, 2>{}, kt + 2);
    }
    __syncthreads();  // all waves done with the ring before it becomes the epilogue tile

    // ---- epilogue: accumulators -> fp32 LDS tile
    float* Cs = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int k = 0; k < C::kNB; ++k)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r = 64 * wm + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
                const int c = (BN / 2) * wn + 32 * k + l32;
                Cs[r * C::kLdc + c] = acc[i][k][v];
            }
    __syncthreads();

    const int half_d = g.D / 2;
    constexpr int kGroups = BN / 8;  // 8-column groups per row
#pragma unroll 1
    for (int ps = 0; ps < (kBM * kGroups) / 256; ++ps) {
        const int item = ps * 256 + tid;
        const int r = item / kGroups, cg = item % kGroups;
        const int64_t m = m0 + r;
        const int32_t n = ncol0 + 8 * cg;  // column within the segment
        float v8[8];
        {
            const f32x4_t c0 = *reinterpret_cast<const f32x4_t*>(Cs + r * C::kLdc + 8 * cg);
            const f32x4_t c1 = *reinterpret_cast<const f32x4_t*>(Cs + r * C::kLdc + 8 * cg + 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) { v8[e] = c0[e]; v8[4 + e] = c1[e]; }
        }
        float dsum = 0.0f;
        if (m < g.n_sel) {
            const int32_t p = g.pos[m];
            if (seg < 2) {  // RoPE on q and k: pairs (2k, 2k+1) within the head
                const int32_t k0 = (n % g.D) >> 1;
                const float2* cs = g.rope + m * half_d + k0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float2 t = cs[e];
                    const float x0 = v8[2 * e], x1 = v8[2 * e + 1];
                    v8[2 * e] = t.x * x0 - t.y * x1;
                    v8[2 * e + 1] = t.y * x0 + t.x * x1;
                }
            }
            const u32x4_t packed = u32x4_t{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]),
                                           pack_bf16x2(v8[4], v8[5]), pack_bf16x2(v8[6], v8[7])};
            if (seg == 0) {
                *reinterpret_cast<u32x4_t*>(g.q_out + m * seg_cols + n) = packed;
            } else if (p >= 0 && p < g.n_tok) {
                uint16_t* dst = kvseg + (int64_t)p * seg_cols + n;
                if (g.dev_parts) {
                    const u32x4_t old = *reinterpret_cast<const u32x4_t*>(dst);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float d0 = bf16_lo(old[e]) - bf16_lo(packed[e]);
                        const float d1 = bf16_hi(old[e]) - bf16_hi(packed[e]);
                        dsum += d0 * d0 + d1 * d1;
                    }
                }
                *reinterpret_cast<u32x4_t*>(dst) = packed;
            }
        }
        if (g.dev_parts && seg > 0) {
            // the kGroups threads of one tile row are consecutive lanes (kGroups divides 64)
#pragma unroll
            for (int o = kGroups / 2; o >= 1; o >>= 1) dsum += __shfl_xor(dsum, o, kGroups);
            if (cg == 0 && m < g.n_sel) g.dev_parts[(2 * m + (seg - 1)) * (seg_cols / BN) + nt] = dsum;
        }
    }
}

}  // namespace

int32_t qkv_gemm_bn(int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim) {
    const int32_t nq = n_q_heads * head_dim, nkv = n_kv_heads * head_dim;
    return (nq % 256 == 0 && nkv % 256 == 0) ? 256 : 128;
}

hipError_t launch_qkv_gemm(const GemmArgs& g, int32_t bn, hipStream_t s) {
    const int64_t per_xcd = (g.n_nt + 7) / 8;
    const dim3 grid((unsigned)(8 * per_xcd * g.n_mt));
    if (bn == 256)
        hipLaunchKernelGGL(qkv_gemm_kernel<256>, grid, dim3(256), 0, s, g);
    else
        hipLaunchKernelGGL(qkv_gemm_kernel<128>, grid, dim3(256), 0, s, g);
    return hipGetLastError();
}

}  // namespace semshare
