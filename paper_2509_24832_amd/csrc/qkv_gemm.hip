// Q/K/V projection of the recomputed tokens (Sections 4.2, 4.3.3) with the
// RoPE / deviation / cache-scatter epilogue, bf16 on v_mfma_f32_32x32x16_bf16.
//
// C[n_sel, Nq + 2 Nkv] = X_sel [n_sel, hidden] . [Wq; Wk; Wv]^T  (all K-major)
//
// Tiling for gfx950: a 512-thread workgroup owns a 128 x BN output tile (BN =
// 256, or 128 when a segment is narrower) and runs alone on its CU, two waves
// per SIMD, so that one wave's operand reads and loads overlap the other's
// MFMAs (the partial layer's 1280 x 6144 x 4096 product: 65 -> 61.5 us
// against one wave per SIMD).  Waves sit 2 along M and 4 along N; each owns a
// 64 x BN/4 sub-tile (2 x BN/128 accumulators of 32x32).  K advances in
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
// per tile (the deviation, reduced later in a fixed order).  The old rows are
// the cache rows being replaced, or (first layer) the matched rows of the
// reference cache read through the match index.  Workgroups are
// mapped XCD-major: all M tiles of one weight tile run on the same XCD, so the
// weights are fetched from HBM once per XCD.
#include <type_traits>

#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kBM = 128, kBK = 64, kStages = 3;
constexpr int kWaves = 8;  // two per SIMD

template <int BN, int NW>
struct Cfg {
    static constexpr int kThreads = 64 * NW;
    static constexpr int kABytes = kBM * kBK * 2;  // 16 KB
    static constexpr int kBBytes = BN * kBK * 2;   // 32 KB (BN = 256)
    static constexpr int kStage = kABytes + kBBytes;
    static constexpr int kLdc = BN + 8;  // floats per epilogue row (acc writes conflict-free)
    static constexpr int kEpi = kBM * kLdc * 4;
    static constexpr int kLds = kStages * kStage > kEpi ? kStages * kStage : kEpi;
    static constexpr int kWN = NW / 2;             // waves side by side along N (two along M)
    static constexpr int kWCols = BN / kWN;        // columns per wave
    static constexpr int kNB = kWCols / 32;        // 32-wide column blocks per wave
    static constexpr int kALoads = kBM / 8 / NW;   // 1-KB direct loads (8 rows of 128 B) per wave per K tile
    static constexpr int kBLoads = BN / 8 / NW;
    static constexpr int kLoads = kALoads + kBLoads;
    static_assert(kNB >= 1 && kALoads >= 1 && kBLoads >= 1, "tile split");
    // direct loads issued by k-steps 0 .. s-1 of a K tile (spread evenly over its 4 k-steps)
    static constexpr int loads_before(int s) { return (s * kLoads + 3) / 4; }
};

__device__ __forceinline__ int swz(int row, int chunk) { return ((chunk ^ ((row >> 1) & 7)) << 4); }

template <int BN, int NW>
__global__ __launch_bounds__(64 * NW, 1) void qkv_gemm_kernel(GemmArgs g) {
    using C = Cfg<BN, NW>;
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
    const int wm = wave / C::kWN, wn = wave % C::kWN;

    // Direct-load sources: instruction i of this wave fills LDS rows
    // [8*grp, 8*grp+8) of its operand; lane -> (row = 8*grp + lane/8, chunk pc = lane%8)
    // and loads the global chunk that the swizzle places there.  Sources are a
    // uniform base (advanced per K tile) plus a fixed per-lane 32-bit byte
    // offset (operands below 2 GiB, checked by the caller).
    const int lrow = lane >> 3, lpc = lane & 7;
    uint32_t a_off[C::kALoads], b_off[C::kBLoads];
#pragma unroll
    for (int i = 0; i < C::kALoads; ++i) {
        const int row = 8 * (wave * C::kALoads + i) + lrow;
        int64_t grow = m0 + row;
        if (grow > g.n_sel - 1) grow = g.n_sel - 1;  // tail rows: computed, never stored
        if (g.x_rows) {  // the row of x that input row grow reads, kept inside x
            int64_t xr = g.x_rows[grow];
            xr = xr < 0 ? 0 : (xr > g.n_x - 1 ? g.n_x - 1 : xr);
            grow = xr;
        }
        a_off[i] = 2u * (uint32_t)(grow * g.hidden + 8 * (lpc ^ ((row >> 1) & 7)));
    }
#pragma unroll
    for (int i = 0; i < C::kBLoads; ++i) {
        const int row = 8 * (wave * C::kBLoads + i) + lrow;
        b_off[i] = 2u * (uint32_t)((ncol0 + row) * g.hidden + 8 * (lpc ^ ((row >> 1) & 7)));
    }
    const uint32_t smem_base = lds_addr(smem);
    // load j (0 .. kLoads-1) of K tile kt into the ring stage at byte offset st_off
    auto issue_one = [&](int j, int kt, uint32_t st_off) {
        if (j < C::kALoads)
            g2lds(g.x + (int64_t)kt * kBK, a_off[j], smem_base + st_off + (wave * C::kALoads + j) * 1024);
        else
            g2lds(wseg + (int64_t)kt * kBK, b_off[j - C::kALoads],
                  smem_base + st_off + C::kABytes + (wave * C::kBLoads + (j - C::kALoads)) * 1024);
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
    const int b_row0 = (C::kWCols * wn + l32) * 128;

    const int nk = g.hidden / kBK;
    for (int j = 0; j < C::kLoads; ++j) issue_one(j, 0, 0);
    if (nk > 1)
        for (int j = 0; j < C::kLoads; ++j) issue_one(j, 1, C::kStage);

    // MFMA operands of one 16-wide k-step, double-buffered in registers: the
    // LDS reads of step s + 1 are in flight while the MFMAs of step s run
    bf16x8_t av[2][2], bv[2][C::kNB];
    auto read_ops = [&](const unsigned char* Ab, int s, int buf) {
        const unsigned char* Bb = Ab + C::kABytes;
#pragma unroll
        for (int i = 0; i < 2; ++i)
            av[buf][i] = *reinterpret_cast<const bf16x8_t*>(Ab + a_row0 + i * 32 * 128 + koff[s]);
#pragma unroll
        for (int k = 0; k < C::kNB; ++k)
            bv[buf][k] = *reinterpret_cast<const bf16x8_t*>(Bb + b_row0 + k * 32 * 128 + koff[s]);
    };
    if (nk > 1) wait_vmcnt<C::kLoads>();
    else wait_vmcnt<0>();
    ring_barrier();  // tile 0 visible to all waves
    read_ops(smem, 0, 0);

    // one K tile on ring stage ST (compile-time, so every LDS address is a
    // constant).  The loads of tile kt + 2 go to the stage tile kt - 1 left
    // (all waves passed the barrier that ended their reads of it); past the
    // last tile they repeat it into a stage nobody reads any more.  The last
    // k-step waits for tile kt + 1, meets the other waves and starts reading
    // its first operands (after the last tile too, harmlessly, so that no
    // branch splits the step).  Each direct load sits between two MFMAs: a
    // load that waits for the address unit then stalls the issue of this
    // wave while its previous MFMA still runs, not while the pipe is empty.
    auto step = [&](auto st_c, int kt) {
        constexpr int ST = decltype(st_c)::value;
        constexpr int NEXT = (ST + 2) % kStages, FOLLOW = (ST + 1) % kStages;
        constexpr int kM = 2 * C::kNB;  // MFMAs per k-step
        const int kt2 = kt + 2 < nk ? kt + 2 : nk - 1;
        const unsigned char* Ab = smem + ST * C::kStage;
        auto kstep = [&](auto s_c) {
            constexpr int s = decltype(s_c)::value;
            constexpr int cur = s & 1;
            constexpr int j0 = C::loads_before(s), nj = C::loads_before(s + 1) - j0;
            static_assert(nj <= (kM + 1) / 2, "a load after every other MFMA");
            if (s < 3) {
                read_ops(Ab, s + 1, cur ^ 1);
            } else {
                // tile kt + 1 has landed: in flight after it are only the
                // loads of tile kt + 2 issued by the first three k-steps
                wait_vmcnt<C::loads_before(3)>();
                // this wave's reads of tile kt are done: after the barrier the
                // loads of tile kt + 3 refill its stage
                __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
                ring_barrier();
                read_ops(smem + FOLLOW * C::kStage, 0, cur ^ 1);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < kM; ++q) {
                acc[q / C::kNB][q % C::kNB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    av[cur][q / C::kNB], bv[cur][q % C::kNB], acc[q / C::kNB][q % C::kNB], 0, 0, 0);
                if (q % 2 == 0 && q / 2 < nj) issue_one(j0 + q / 2, kt2, NEXT * C::kStage);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        kstep(std::integral_constant<int, 0>{});
        kstep(std::integral_constant<int, 1>{});
        kstep(std::integral_constant<int, 2>{});
        kstep(std::integral_constant<int, 3>{});
    };
    for (int kt = 0; kt < nk; kt += kStages) {
        step(std::integral_constant<int, 0>{}, kt);
        if (kt + 1 < nk) step(std::integral_constant<int, 1>{}, kt + 1);
        if (kt + 2 < nk) step(std::integral_constant<int, 2>{}, kt + 2);
    }
    wait_vmcnt<0>();  // the repeated loads past the last tile have landed
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
                const int c = C::kWCols * wn + 32 * k + l32;
                Cs[r * C::kLdc + c] = acc[i][k][v];
            }
    __syncthreads();

    // Each thread owns one 8-column group (cg) of rows r0, r0 + kRowStep, ...
    // Rows go in batches of kBatch whose global reads (position, RoPE
    // factors, old cache rows) are all issued before any of them is used, so
    // their latencies overlap instead of adding up row by row.  One pass per
    // segment, specialised at compile time (q: RoPE and store; k: RoPE,
    // deviation and scatter; v: deviation and scatter): with the segment a
    // run-time value every optional load became a branch of its own.  Loads
    // read the last row for rows past n_sel (in bounds, never stored).
    const int half_d = g.D / 2;
    constexpr int kGroups = BN / 8;                 // 8-column groups per row
    constexpr int kRowStep = C::kThreads / kGroups; // rows between a thread's items
    constexpr int kItems = kBM / kRowStep;          // items per thread
    constexpr int kBatch = kItems < 8 ? kItems : 8;
    static_assert(kItems % kBatch == 0, "batches divide the items");
    const int cg = tid % kGroups, r0 = tid / kGroups;
    const int32_t n = ncol0 + 8 * cg;           // column within the segment
    const int32_t k0 = (n % g.D) >> 1;          // first RoPE pair of the group (a multiple of 4)
    auto epilogue = [&](auto seg_c) {
        constexpr int SEG = decltype(seg_c)::value;
        constexpr bool kRope = SEG < 2, kKV = SEG > 0;
        const bool dev = kKV && g.dev_parts != nullptr;
#pragma unroll 1
        for (int b0 = 0; b0 < kItems; b0 += kBatch) {
            int64_t mc[kBatch];
            int32_t p[kBatch];
            f32x4_t cs[kBatch][2];  // (cos, sin) of the group's 4 pairs
            u32x4_t old[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int64_t m = m0 + r0 + (b0 + u) * kRowStep;
                mc[u] = m < g.n_sel ? m : g.n_sel - 1;
            }
            if constexpr (kRope) {
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const f32x4_t* rp = reinterpret_cast<const f32x4_t*>(g.rope + mc[u] * half_d + k0);
                    cs[u][0] = rp[0];
                    cs[u][1] = rp[1];
                }
            }
            if constexpr (kKV) {
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int32_t pp = g.pos[mc[u]];
                    p[u] = m0 + r0 + (b0 + u) * kRowStep < g.n_sel && pp >= 0 && pp < g.n_tok ? pp : -1;
                }
                if (dev && g.dev_idx) {  // the deviation against matched reference rows
                    const uint16_t* src = g.dev_src[SEG - 1];
                    int32_t j[kBatch];
#pragma unroll
                    for (int u = 0; u < kBatch; ++u) j[u] = p[u] >= 0 ? g.dev_idx[p[u]] : -1;
#pragma unroll
                    for (int u = 0; u < kBatch; ++u) {
                        old[u] = u32x4_t{0u, 0u, 0u, 0u};
                        if (j[u] >= 0 && j[u] < g.dev_n)
                            old[u] = *reinterpret_cast<const u32x4_t*>(src + (int64_t)j[u] * seg_cols + n);
                    }
                } else if (dev) {  // the deviation against the cache rows being replaced
#pragma unroll
                    for (int u = 0; u < kBatch; ++u) {
                        old[u] = u32x4_t{0u, 0u, 0u, 0u};
                        if (p[u] >= 0) old[u] = *reinterpret_cast<const u32x4_t*>(kvseg + (int64_t)p[u] * seg_cols + n);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int r = r0 + (b0 + u) * kRowStep;
                const int64_t m = m0 + r;
                float v8[8];
                {
                    const f32x4_t c0 = *reinterpret_cast<const f32x4_t*>(Cs + r * C::kLdc + 8 * cg);
                    const f32x4_t c1 = *reinterpret_cast<const f32x4_t*>(Cs + r * C::kLdc + 8 * cg + 4);
#pragma unroll
                    for (int e = 0; e < 4; ++e) { v8[e] = c0[e]; v8[4 + e] = c1[e]; }
                }
                if constexpr (kRope) {  // RoPE on q and k: pairs (2k, 2k+1) within the head
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float2 t = make_float2(cs[u][e >> 1][2 * (e & 1)], cs[u][e >> 1][2 * (e & 1) + 1]);
                        const float x0 = v8[2 * e], x1 = v8[2 * e + 1];
                        // explicit fused forms: the rounding does not depend on how the
                        // compiler contracts the products
                        v8[2 * e] = fmaf(t.x, x0, -(t.y * x1));
                        v8[2 * e + 1] = fmaf(t.y, x0, t.x * x1);
                    }
                }
                const u32x4_t packed = u32x4_t{pack_bf16x2(v8[0], v8[1]), pack_bf16x2(v8[2], v8[3]),
                                               pack_bf16x2(v8[4], v8[5]), pack_bf16x2(v8[6], v8[7])};
                if constexpr (SEG == 0) {
                    if (m < g.n_sel) *reinterpret_cast<u32x4_t*>(g.q_out + m * seg_cols + n) = packed;
                } else {
                    float dsum = 0.0f;
                    if (p[u] >= 0) {
                        if (dev) {
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                const float d0 = bf16_lo(old[u][e]) - bf16_lo(packed[e]);
                                const float d1 = bf16_hi(old[u][e]) - bf16_hi(packed[e]);
                                dsum += d0 * d0 + d1 * d1;
                            }
                        }
                        *reinterpret_cast<u32x4_t*>(kvseg + (int64_t)p[u] * seg_cols + n) = packed;
                    }
                    if (dev) {
                        // the kGroups threads of one tile row are consecutive lanes (kGroups divides 64)
#pragma unroll
                        for (int o = kGroups / 2; o >= 1; o >>= 1) dsum += __shfl_xor(dsum, o, kGroups);
                        if (cg == 0 && m < g.n_sel) g.dev_parts[(2 * m + (SEG - 1)) * (seg_cols / BN) + nt] = dsum;
                    }
                }
            }
        }
    };
    if (seg == 0) epilogue(std::integral_constant<int, 0>{});
    else if (seg == 1) epilogue(std::integral_constant<int, 1>{});
    else epilogue(std::integral_constant<int, 2>{});
}

}  // namespace

int32_t qkv_gemm_bn(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim) {
    const int32_t nq = n_q_heads * head_dim, nkv = n_kv_heads * head_dim;
    if (nq % 256 != 0 || nkv % 256 != 0) return 128;
    // 256-wide tiles, unless so few rows are selected that twice as many
    // 128-wide tiles still fit one pass over the CUs: a tile's K loop takes
    // about the same time whatever its row count, so with few row tiles the
    // narrower ones finish the call in about half the time
    const int64_t n_mt = (n_sel + 127) / 128;
    const int64_t n_nt = (nq + 2 * (int64_t)nkv) / 256;
    return 2 * n_mt * n_nt <= 256 ? 128 : 256;
}

hipError_t launch_qkv_gemm(const GemmArgs& g, int32_t bn, hipStream_t s) {
    const int64_t per_xcd = (g.n_nt + 7) / 8;
    const dim3 grid((unsigned)(8 * per_xcd * g.n_mt));
    if (bn == 256)
        hipLaunchKernelGGL((qkv_gemm_kernel<256, kWaves>), grid, dim3(64 * kWaves), 0, s, g);
    else
        hipLaunchKernelGGL((qkv_gemm_kernel<128, kWaves>), grid, dim3(64 * kWaves), 0, s, g);
    return hipGetLastError();
}

}  // namespace semshare
