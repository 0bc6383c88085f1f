// Causal grouped-query attention of the recomputed tokens over the assembled
// cache (Sections 4.2, 4.3.3), bf16 storage, fp32 accumulation and softmax.
//
// For a selected row at position p and query head h:
//   out = softmax_{j <= p}(q_h . K[j][h/G] * scale) V[j][h/G]
//
// Work decomposition.  A 256-thread workgroup owns one kv head g and 256
// query columns = (256/G selected rows) x (the G query heads of g); it runs
// alone on its CU (one wave per SIMD).  Each wave owns two 32-column blocks,
// so every K or V fragment it reads from LDS feeds two MFMAs (64 flop per LDS
// byte; with one block per wave the matrix cores would wait on LDS).
// S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_32x32x16_bf16: every lane then
// holds one query column.
//
// Data movement.  K and V tiles of 64 keys travel by direct-to-LDS loads
// (global_load_lds_dwordx4) into a 4-stage ring, in their natural [key][d]
// layout with the 16-byte chunk index XOR-swizzled per row (K by row mod D/8,
// V by 2*(row mod D/16)), so the MFMA operand reads below are free of bank
// conflicts.  V^T operands come from ds_read_b64_tr_b16, which transposes
// 4 keys x 4 dims per 16-lane group on the way out of LDS.
//
// Softmax.  Keys run in sub-tiles of 32.  The probabilities of sub-tile u are
// formed while the matrix cores compute S(u+1) and O += V(u-1) P(u-1), which
// keeps the exponentials off the critical path.  No running maximum is taken
// per sub-tile: each column keeps a reference m (a maximum seen earlier) and
// p = 2^((s - m) * scale * log2 e) may exceed 1.  The lane's sum of the
// sub-tile's p bounds their maximum, so while that sum stays below 2^16
// nothing can overflow; otherwise (the first sub-tile, where m is still
// unset, and large upward jumps later) the sub-tile's true maximum becomes
// the new m, O and l are rescaled and the probabilities formed again.  The
// normaliser l sums the fp32 p (the PV product consumes them rounded to bf16;
// a v_dot2c sum of the rounded pairs is a serial chain that cost ~20% here).
//
// Split-KV.  A (row tile, kv head) item whose causal key range is long
// relative to the chip's share of work is cut into equal pieces of whole
// 64-key tiles (the piece count follows from the tile's largest position, so
// short items stay whole); each piece writes its (m, l, O) to the workspace
// in the order its registers hold them (coalesced), and a combine kernel
// merges the pieces by log-sum-exp in piece order.
#include <algorithm>
#include <climits>

#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int KT = 64;       // keys per LDS tile (two sub-tiles)
constexpr int NCOL = 256;    // query columns per workgroup
constexpr int kStages = 4;   // K/V ring depth
constexpr float kSumLimit = 65536.0f;  // 2^16
constexpr int kCUs = 256;        // compute units of the chip
constexpr int kMinPieceKt = 4;   // shortest split-KV piece, in 64-key tiles
constexpr double kSplitShares = 0.75;  // split-KV piece target, in CU shares of work

typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

struct AttnArgs {
    const uint16_t* q;        // [n_sel][Hq][D]
    const int32_t* pos;       // [n_sel]
    const uint16_t* k_cache;  // [n_tok][Hkv][D]
    const uint16_t* v_cache;
    uint16_t* out;            // [n_sel][Hq][D]
    f32x4_t* part_o;          // [items][n_chunks][NCOL * D / 4], register-native order
    float2* part_ml;          // [items][n_chunks][NCOL]  (m, l)
    int32_t* n_used;          // [items]: pieces of the item
    int64_t n_sel, n_tok;
    int32_t Hq, Hkv, G, R;
    int32_t n_tiles;
    int32_t split_units;      // target piece length in 64-key tiles
    int32_t n_chunks;         // most pieces an item can have (grid dimension)
    float cl2;                // sm_scale * log2(e)
};

template <int D>
struct ACfg {
    static constexpr int kNch = D / 8;               // 16-B chunks per key row
    static constexpr int kRowBytes = 2 * D;
    static constexpr int kTileBytes = KT * kRowBytes;  // one tensor
    static constexpr int kStage = 2 * kTileBytes;      // K then V
    static constexpr int kLds = kStages * kStage;
    static constexpr int kRowsPerLoad = 64 / kNch;     // rows one 1-KB direct load covers
    static constexpr int kLoadsPerWave = KT / kRowsPerLoad / 4;  // per tensor
    static constexpr int kLoads = 2 * kLoadsPerWave;   // per wave per tile (K + V)
    static constexpr int kMd = D / 32;                 // 32-row blocks of O^T
    static constexpr int kKs = D / 16;                 // k-steps of S^T
};

// 16 bytes per lane from gbase + off (bytes, per lane) straight into LDS at
// lds_base + 16 * lane (global_load_lds_dwordx4, M0 = the wave-uniform LDS
// base, scalar base address + 32-bit lane offset).  Issued as inline assembly
// on purpose: the compiler then does not treat the transposing LDS reads that
// follow as dependent on these in-flight loads (it would drain the whole ring
// with vmcnt(0) before each of them).  Stage readiness is established
// explicitly instead (wait_vmcnt + ring_barrier), and M0 is written only here
// in this kernel.
__device__ __forceinline__ void g2lds(const void* gbase, uint32_t off, uint32_t lds_base) {
    // the scalar operands are wave-uniform by construction; readfirstlane
    // places them in scalar registers
    // (readfirstlane returns int: both halves go through uint32_t so the low
    // half is zero-extended, never sign-extended into the high half)
    const uint64_t g = reinterpret_cast<uint64_t>(gbase);
    const uint32_t g_hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
    const uint32_t g_lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)g);
    const uint64_t gs = ((uint64_t)g_hi << 32) | (uint64_t)g_lo;
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(reinterpret_cast<const void*>(gs)), "s"((uint32_t)__builtin_amdgcn_readfirstlane(lds_base))
                 : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// s_waitcnt vmcnt(n), other counters left at their maximum; vmcnt is split
// over bits [3:0] and [15:14] of the immediate.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Barrier without the fence of __syncthreads (which would drain the ring of
// in-flight direct loads); stage visibility comes from the explicit vmcnt waits.
__device__ __forceinline__ void ring_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int D>
__global__ __launch_bounds__(256, 1) void attention_kernel(AttnArgs a) {
    using C = ACfg<D>;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[C::kLds];
    __shared__ int32_t s_pos[NCOL];
    __shared__ int32_t s_pmin, s_pmax;

    const int b = blockIdx.x;
    const int g = b % a.Hkv;  // kv head; with 8 kv heads each XCD serves one (its K/V stay in that L2)
    const int jj = b / a.Hkv;
    const int tile = a.n_tiles - 1 - jj / a.n_chunks;  // longest (latest) tiles first
    const int chunk_id = jj % a.n_chunks;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, l32 = lane & 31;

    if (tid < a.R) {
        const int64_t r = (int64_t)tile * a.R + tid;
        int32_t p = r < a.n_sel ? a.pos[r] : -1;
        if (p < 0 || p >= a.n_tok) p = -1;
        s_pos[tid] = p;
    }
    __syncthreads();
    if (wave == 0) {
        int32_t mn = INT_MAX, mx = -1;
        for (int i = lane; i < a.R; i += 64) {
            const int32_t p = s_pos[i];
            if (p >= 0) { mn = min(mn, p); mx = max(mx, p); }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            mn = min(mn, __shfl_xor(mn, o));
            mx = max(mx, __shfl_xor(mx, o));
        }
        if (lane == 0) { s_pmin = mn; s_pmax = mx; }
    }
    __syncthreads();
    const int32_t pmin = __builtin_amdgcn_readfirstlane(s_pmin), pmax = __builtin_amdgcn_readfirstlane(s_pmax);
    // this item's pieces: n_pieces runs of piece_kt whole tiles over [0, pmax]
    const int32_t item_kt = (pmax + KT) / KT;
    int32_t n_pieces = min((item_kt + a.split_units - 1) / a.split_units, a.n_chunks);
    const int32_t piece_kt = (item_kt + n_pieces - 1) / max(n_pieces, 1);
    n_pieces = (item_kt + piece_kt - 1) / max(piece_kt, 1);
    const int64_t item = (int64_t)tile * a.Hkv + g;
    if (chunk_id == 0 && tid == 0 && a.n_chunks > 1) a.n_used[item] = pmax < 0 ? 0 : n_pieces;
    const int32_t kbeg = chunk_id * piece_kt * KT;
    const int32_t kend = min(kbeg + piece_kt * KT, pmax + 1);
    if (pmax < 0 || kbeg >= kend) return;  // no row of the tile reaches this piece

    // this lane's two query columns
    int col[2], head[2];
    int64_t row[2];
    int32_t p_l[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        col[nb] = 64 * wave + 32 * nb + l32;
        const int row_local = col[nb] % a.R;
        row[nb] = (int64_t)tile * a.R + row_local;
        head[nb] = g * a.G + col[nb] / a.R;
        p_l[nb] = s_pos[row_local];
    }
    // Q^T operands: lane half h holds d in [h*D/2, h*D/2 + D/2)
    bf16x8_t qf[2][C::kKs];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const u32x4_t* qp = reinterpret_cast<const u32x4_t*>(
            a.q + ((p_l[nb] >= 0 ? row[nb] : 0) * a.Hq + head[nb]) * (int64_t)D + half * (D / 2));
#pragma unroll
        for (int s = 0; s < C::kKs; ++s) {
            const u32x4_t w = p_l[nb] >= 0 ? qp[s] : u32x4_t{0u, 0u, 0u, 0u};
            qf[nb][s] = __builtin_bit_cast(bf16x8_t, w);
            // kept in accumulation registers (MFMA reads its B operand from
            // there), leaving the vector registers to K/V fragments and softmax
            asm volatile("" : "+a"(qf[nb][s]));
        }
    }

    // ---- direct-load sources.  Load i of this wave (per tensor) fills rows
    // [rpl*(wave*lpw + i), +rpl) of the tile; lane -> (row, physical chunk pc),
    // it fetches the logical chunk that the swizzle stores at pc.
    const int32_t row_stride = a.Hkv * D;
    const uint16_t* kbase = a.k_cache + (int64_t)g * D;
    const uint16_t* vbase = a.v_cache + (int64_t)g * D;
    const int32_t last_key = (int32_t)a.n_tok - 1;
    int ld_row[C::kLoadsPerWave];
    int32_t ld_kc[C::kLoadsPerWave], ld_vc[C::kLoadsPerWave];
#pragma unroll
    for (int i = 0; i < C::kLoadsPerWave; ++i) {
        const int r = C::kRowsPerLoad * (wave * C::kLoadsPerWave + i) + lane / C::kNch;
        const int pc = lane % C::kNch;
        ld_row[i] = r;
        ld_kc[i] = 8 * (pc ^ (r & (C::kNch - 1)));
        ld_vc[i] = 8 * (pc ^ (2 * (r & (C::kNch / 2 - 1))));
    }
    const uint32_t smem_base = lds_addr(smem);
    // Loads of one 64-key tile: scalar bases of its first key row, per-lane
    // byte offsets of this wave's rows (clamped to the last key), LDS base.
    struct TileLoads {
        const uint16_t* kg;
        const uint16_t* vg;
        uint32_t off_k[C::kLoadsPerWave], off_v[C::kLoadsPerWave];
        uint32_t lds;
    };
    auto prep_tile = [&](int t, TileLoads& d) {
        const int32_t key0 = kbeg + t * KT;
        d.kg = kbase + (int64_t)key0 * row_stride;
        d.vg = vbase + (int64_t)key0 * row_stride;
        const int32_t lim = last_key - key0;
#pragma unroll
        for (int i = 0; i < C::kLoadsPerWave; ++i) {
            const uint32_t r = (uint32_t)min(ld_row[i], lim);
            d.off_k[i] = (r * (uint32_t)row_stride + (uint32_t)ld_kc[i]) * 2u;
            d.off_v[i] = (r * (uint32_t)row_stride + (uint32_t)ld_vc[i]) * 2u;
        }
        d.lds = __builtin_amdgcn_readfirstlane(smem_base + (t % kStages) * C::kStage +
                                               wave * C::kLoadsPerWave * 1024);
    };
    // load n of the tile (n in [0, kLoads)): K for even n, V for odd n, rows of load n/2
    auto issue_one = [&](const TileLoads& d, int n) {
        const int i = n >> 1;
        if (n & 1) g2lds(d.vg, d.off_v[i], d.lds + i * 1024 + C::kTileBytes);
        else g2lds(d.kg, d.off_k[i], d.lds + i * 1024);
    };
    auto issue = [&](int t) {
        TileLoads d;
        prep_tile(t, d);
#pragma unroll
        for (int n = 0; n < C::kLoads; ++n) issue_one(d, n);
    };

    // ---- LDS read offsets (bytes within a stage)
    // K (A operand of S^T): key row l32 of the sub-tile, logical chunk half*(D/16) + s
    int k_ro[C::kKs];
#pragma unroll
    for (int s = 0; s < C::kKs; ++s)
        k_ro[s] = l32 * C::kRowBytes + (((half * (C::kNch / 2) + s) ^ (l32 & (C::kNch - 1))) << 4);
    // V^T via transpose reads: 16-lane group gq, lane m in it; rows 16*sp + 8*qh + 4*half + m/4,
    // dims 32*md + 16*(gq%2) + 4*(m%4) .. +3
    const int gq = lane >> 4, m16 = lane & 15;
    const int v_r = 4 * half + (m16 >> 2);  // row within an 8-row group (the swizzle depends on it only)
    int v_ro[C::kMd];
#pragma unroll
    for (int md = 0; md < C::kMd; ++md) {
        const int c = 4 * md + 2 * (gq & 1) + ((m16 & 3) >> 1);
        v_ro[md] = v_r * C::kRowBytes + ((c ^ (2 * (v_r & (C::kNch / 2 - 1)))) << 4) + (m16 & 1) * 8;
    }

    f32x16_t oacc[2][C::kMd];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int i = 0; i < C::kMd; ++i) oacc[nb][i] = f32x16_t{};
    float m_run[2] = {-1.0e30f, -1.0e30f}, l_run[2] = {0.0f, 0.0f};
    const float cl2 = a.cl2;

    // Sub-tile u is half u%2 of the 64-key tile u/2 in ring stage (u/2) % kStages.
    auto stage_of = [&](int u) { return smem + ((u >> 1) % kStages) * C::kStage; };
    // K fragments of sub-tile u (A operand of S^T, k-step s)
    auto read_k = [&](int u, bf16x8_t (&kf)[C::kKs]) {
        const unsigned char* kb = stage_of(u) + (u & 1) * 32 * C::kRowBytes;
#pragma unroll
        for (int s = 0; s < C::kKs; ++s) kf[s] = *reinterpret_cast<const bf16x8_t*>(kb + k_ro[s]);
    };
    // V^T fragments of sub-tile u (A operand of O^T, k-step sp, row block md)
    auto read_v = [&](int u, bf16x8_t (&vf)[2][C::kMd]) {
        const unsigned char* vb = stage_of(u) + C::kTileBytes + (u & 1) * 32 * C::kRowBytes;
#pragma unroll
        for (int sp = 0; sp < 2; ++sp)
#pragma unroll
            for (int md = 0; md < C::kMd; ++md) {
                const unsigned char* p0 = vb + (16 * sp) * C::kRowBytes + v_ro[md];
                const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p0);
                const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p0 + 8 * C::kRowBytes));
                const u32x2_t wl = __builtin_bit_cast(u32x2_t, lo), wh = __builtin_bit_cast(u32x2_t, hi);
                vf[sp][md] = __builtin_bit_cast(bf16x8_t, u32x4_t{wl[0], wl[1], wh[0], wh[1]});
            }
    };
    // S^T for both column blocks (one K fragment feeds both)
    auto s_mfma = [&](const bf16x8_t (&kf)[C::kKs], f32x16_t (&sacc)[2]) {
        sacc[0] = sacc[1] = f32x16_t{};
#pragma unroll
        for (int s = 0; s < C::kKs; ++s)
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
                sacc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[nb][s], sacc[nb], 0, 0, 0);
    };
    // O^T += V^T P^T
    auto pv_mfma = [&](const bf16x8_t (&vf)[2][C::kMd], const bf16x8_t (&pb)[2][2]) {
#pragma unroll
        for (int sp = 0; sp < 2; ++sp)
#pragma unroll
            for (int md = 0; md < C::kMd; ++md)
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    oacc[nb][md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[sp][md], pb[nb][sp], oacc[nb][md], 0, 0, 0);
    };
    // mask keys past a column's position or past the chunk (boundary sub-tiles only)
    auto mask = [&](int u, f32x16_t (&sacc)[2]) {
        const int32_t k0 = kbeg + 32 * u;
        if (k0 + 31 > pmin || k0 + 32 > kend) {
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                // key k0 + 4*half + o is kept iff o <= lim
                const int32_t lim = min(p_l[nb], kend - 1) - k0 - 4 * half;
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (8 * (v >> 2) + (v & 3) > lim) sacc[nb][v] = -INFINITY;
            }
        }
    };
    // probabilities as bf16 MFMA operands (k index 8h+e of step sp is key
    // 16sp + 8(e/4) + 4h + e%4 of the sub-tile, the keys whose S^T values this
    // lane holds) and the lane's sums of them
    auto exp_pack = [&](const f32x16_t (&sacc)[2], bf16x8_t (&pb)[2][2], float (&ts)[2]) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            const float mc = m_run[nb] * cl2;
            ts[nb] = 0.0f;
#pragma unroll
            for (int sp = 0; sp < 2; ++sp) {
                f32x8_t pv;
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = __builtin_amdgcn_exp2f(fmaf(sacc[nb][8 * sp + e], cl2, -mc));
                pb[nb][sp] = __builtin_convertvector(pv, bf16x8_t);
#pragma unroll
                for (int e = 0; e < 8; e += 2) ts[nb] += pv[e] + pv[e + 1];
            }
        }
    };
    // accept the sub-tile's probabilities, or (rare) move the reference to
    // the sub-tile's maximum, rescale O and l, and form them again
    auto settle = [&](const f32x16_t (&sacc)[2], bf16x8_t (&pb)[2][2], float (&ts)[2]) {
        if (__any(!(ts[0] <= kSumLimit) || !(ts[1] <= kSumLimit))) {
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                float mx = sacc[nb][0];
#pragma unroll
                for (int v = 1; v < 16; ++v) mx = fmaxf(mx, sacc[nb][v]);
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const float m_new = fmaxf(m_run[nb], mx);
                const float alpha = __builtin_amdgcn_exp2f((m_run[nb] - m_new) * cl2);
                m_run[nb] = m_new;
                l_run[nb] *= alpha;
#pragma unroll
                for (int i = 0; i < C::kMd; ++i) {
                    // one accumulator at a time: bounded register staging
                    __builtin_amdgcn_sched_barrier(0);
                    oacc[nb][i] *= alpha;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            exp_pack(sacc, pb, ts);
        }
        l_run[0] += ts[0];
        l_run[1] += ts[1];
    };

    const int n_sub = (kend - kbeg + 31) / 32;
    const int n_kt = (n_sub + 1) / 2;
    issue(0);
    if (n_kt > 1) issue(1);
    if (n_kt > 2) issue(2);
    if (n_kt > 2) wait_vmcnt<2 * C::kLoads>();
    else if (n_kt > 1) wait_vmcnt<C::kLoads>();
    else wait_vmcnt<0>();
    ring_barrier();

    f32x16_t sA[2], sB[2];       // scores of even / odd sub-tiles
    bf16x8_t pA[2][2], pB[2][2];  // probabilities of even / odd sub-tiles
    float ts[2];
    {
        bf16x8_t kf[C::kKs];
        read_k(0, kf);
        s_mfma(kf, sA);
        mask(0, sA);
    }
    // Sub-tile u with a successor: S(u+1) and PV(u-1) on the matrix cores
    // while the probabilities of u are formed.  An odd u first opens tile
    // (u+1)/2 (its loads done, the stage of tile (u+1)/2 - 2 free again).
    auto body = [&](int u, f32x16_t (&cur)[2], f32x16_t (&nxt)[2], bf16x8_t (&pc)[2][2],
                    const bf16x8_t (&pp)[2][2], bool has_prev, bool opens) {
        if (opens) {
            const int T = (u + 1) >> 1;
            if (T + 1 < n_kt) wait_vmcnt<C::kLoads>();
            else wait_vmcnt<0>();
            ring_barrier();
            // all loads of tile T+2 at once: spreading them over the MFMA slots
            // costs more (each load holds up the in-order issue of its wave)
            if (T + 2 < n_kt) issue(T + 2);
        }
        if (!has_prev) {
            bf16x8_t kf[C::kKs];
            read_k(u + 1, kf);
            s_mfma(kf, nxt);
            exp_pack(cur, pc, ts);
        } else {
            // Steady state as a software pipeline of 4*kKs slots.  Slot k
            // issues one MFMA, fenced off on its own: k%4 = 0, 1 are S^T
            // k-step k/4 for column blocks 0, 1; k%4 = 2, 3 are PV step k/4.
            // A fenced group of VALU work follows it: the scaled scores of
            // this slot's values, the exponentials of the previous slot's, a
            // bf16 pair conversion and a row-sum update further behind, and
            // one LDS request for step k/4 + 2.  The strict alternation keeps
            // the matrix pipe fed while the softmax arithmetic runs in its
            // shadow, and no operation waits on its immediate predecessor.
            constexpr int kSlots = 4 * C::kKs;
            constexpr int kV = 32 / kSlots;  // probabilities formed per slot (1 or 2)
            auto cvt_slot = [](int q) { return (2 * q + 1) / kV + 2; };
            const unsigned char* kb = stage_of(u + 1) + ((u + 1) & 1) * 32 * C::kRowBytes;
            const unsigned char* vb = stage_of(u - 1) + C::kTileBytes + ((u - 1) & 1) * 32 * C::kRowBytes;
            // one address per K fragment and per V row block; the V half-steps
            // are immediate offsets from it
            const unsigned char* ka[C::kKs];
            const unsigned char* va[C::kMd];
#pragma unroll
            for (int j = 0; j < C::kKs; ++j) ka[j] = kb + k_ro[j];
#pragma unroll
            for (int md = 0; md < C::kMd; ++md) va[md] = vb + v_ro[md];
            auto rk = [&](int j) { return *reinterpret_cast<const bf16x8_t*>(ka[j]); };
            auto rv = [&](int j, int hi) {
                const unsigned char* p0 = va[j % C::kMd] + (16 * (j / C::kMd) + 8 * hi) * C::kRowBytes;
                return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p0));
            };
            const float mc[2] = {m_run[0] * cl2, m_run[1] * cl2};
            float fv[32], ev[32];
            uint32_t pw[16];
            bf16x8_t kf[C::kKs];
            u32x2_t vl[C::kKs], vh[C::kKs];
            ts[0] = ts[1] = 0.0f;
            nxt[0] = nxt[1] = f32x16_t{};
#pragma unroll
            for (int j = 0; j < 2 && j < C::kKs; ++j) {
                kf[j] = rk(j);
                vl[j] = rv(j, 0);
                vh[j] = rv(j, 1);
            }
#pragma unroll
            for (int k = 0; k < kSlots; ++k) {
                const int j = k >> 2, kind = k & 3;
                if (kind < 2) {
                    nxt[kind] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[j], qf[kind][j], nxt[kind], 0, 0, 0);
                } else {
                    const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, u32x4_t{vl[j][0], vl[j][1], vh[j][0], vh[j][1]});
                    f32x16_t& o = oacc[kind - 2][j % C::kMd];
                    o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pp[kind - 2][j / C::kMd], o, 0, 0, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
                if (j + 2 < C::kKs) {
                    if (kind == 0) kf[j + 2] = rk(j + 2);
                    if (kind == 1) vl[j + 2] = rv(j + 2, 0);
                    if (kind == 2) vh[j + 2] = rv(j + 2, 1);
                }
#pragma unroll
                for (int v = 0; v < kV; ++v) {
                    const int f = k * kV + v;  // value f: column block f/16, S^T register f%16
                    fv[f] = fmaf(cur[f >> 4][f & 15], cl2, -mc[f >> 4]);
                    if (k > 0) ev[f - kV] = __builtin_amdgcn_exp2f(fv[f - kV]);
                }
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    if (cvt_slot(q) == k)
                        pw[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{ev[2 * q], ev[2 * q + 1]}, bf16x2_t));
                    if (cvt_slot(q) + 1 == k) ts[q >> 3] += ev[2 * q] + ev[2 * q + 1];
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            // drain: the last slot's exponentials, conversions and sums
#pragma unroll
            for (int f = (kSlots - 1) * kV; f < 32; ++f) ev[f] = __builtin_amdgcn_exp2f(fv[f]);
#pragma unroll
            for (int q = 0; q < 16; ++q)
                if (cvt_slot(q) >= kSlots)
                    pw[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{ev[2 * q], ev[2 * q + 1]}, bf16x2_t));
#pragma unroll
            for (int q = 0; q < 16; ++q)
                if (cvt_slot(q) + 1 >= kSlots) ts[q >> 3] += ev[2 * q] + ev[2 * q + 1];
            // word q = (nb, sp, w) with q = 8 nb + 4 sp + w
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                for (int sp = 0; sp < 2; ++sp)
                    pc[nb][sp] = __builtin_bit_cast(bf16x8_t, u32x4_t{pw[8 * nb + 4 * sp], pw[8 * nb + 4 * sp + 1],
                                                                      pw[8 * nb + 4 * sp + 2], pw[8 * nb + 4 * sp + 3]});
        }
        settle(cur, pc, ts);
        mask(u + 1, nxt);
    };
    // The last sub-tile u: PV(u-1) while its probabilities are formed, then PV(u).
    auto last = [&](int u, f32x16_t (&cur)[2], bf16x8_t (&pc)[2][2], const bf16x8_t (&pp)[2][2],
                    bool has_prev) {
        bf16x8_t vf[2][C::kMd];
        if (has_prev) {
            read_v(u - 1, vf);
            pv_mfma(vf, pp);
        }
        exp_pack(cur, pc, ts);
        settle(cur, pc, ts);
        read_v(u, vf);
        pv_mfma(vf, pc);
    };
    if (n_sub == 1) {
        last(0, sA, pA, pB, false);
    } else {
        body(0, sA, sB, pA, pB, false, false);
        int u = 1;
        for (; u + 2 < n_sub; u += 2) {
            body(u, sB, sA, pB, pA, true, true);
            body(u + 1, sA, sB, pA, pB, true, false);
        }
        if (u + 1 < n_sub) {  // u = n_sub - 2
            body(u, sB, sA, pB, pA, true, true);
            last(u + 1, sA, pA, pB, true);
        } else {  // u = n_sub - 1
            last(u, sB, pB, pA, true);
        }
    }

    // ---- results: oacc[nb][i][4r + e] = O[col][d = 32i + 8r + 4half + e]
    float l_tot[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) l_tot[nb] = l_run[nb] + __shfl_xor(l_run[nb], 32);
    auto store_out = [&](int nb, const f32x16_t (&o)[C::kMd], float inv) {
        uint16_t* op = a.out + (row[nb] * a.Hq + head[nb]) * (int64_t)D;
#pragma unroll
        for (int i = 0; i < C::kMd; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                u32x2_t w;
                w.x = pack_bf16x2(o[i][4 * r] * inv, o[i][4 * r + 1] * inv);
                w.y = pack_bf16x2(o[i][4 * r + 2] * inv, o[i][4 * r + 3] * inv);
                *reinterpret_cast<u32x2_t*>(op + 32 * i + 8 * r + 4 * half) = w;
            }
    };
    if (n_pieces == 1) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
            if (p_l[nb] >= 0) store_out(nb, oacc[nb], 1.0f / l_tot[nb]);
        return;
    }

    // split item: publish this piece's (m, l, O) in register order
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        f32x4_t* po = a.part_o + (((item * a.n_chunks + chunk_id) * 4 + wave) * 2 + nb) * (C::kMd * 4 * 64) + lane;
#pragma unroll
        for (int i = 0; i < C::kMd; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                po[(i * 4 + r) * 64] = f32x4_t{oacc[nb][i][4 * r], oacc[nb][i][4 * r + 1], oacc[nb][i][4 * r + 2],
                                               oacc[nb][i][4 * r + 3]};
        if (half == 0) a.part_ml[(item * a.n_chunks + chunk_id) * NCOL + col[nb]] = make_float2(m_run[nb], l_tot[nb]);
    }
}

// Log-sum-exp merge of an item's pieces, in piece order.  One workgroup per
// (item, wave slice, column block): the 32 columns x D values that attention
// wave `wave` held in block nb, laid out as [i][r][lane] f32x4 per piece, so
// every load is a coalesced 1 KB row.  Thread t handles lane t % 64 and the
// (i, r) pairs t / 64 + 4k.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(AttnArgs a) {
    constexpr int kMd = D / 32;
    constexpr int kPer = kMd;  // (i, r) pairs per thread: 4 * kMd / 4
    const int64_t item = blockIdx.x >> 3;  // tile * Hkv + g
    const int wave = (blockIdx.x >> 1) & 3, nb = blockIdx.x & 1;
    const int32_t nu = a.n_used[item];
    if (nu <= 1) return;
    const int tile = (int)(item / a.Hkv), g = (int)(item % a.Hkv);
    const int tid = threadIdx.x, lane = tid & 63, q4 = tid >> 6;
    const int half = lane >> 5, l32 = lane & 31;
    const int col = 64 * wave + 32 * nb + l32;
    const int64_t row = (int64_t)tile * a.R + col % a.R;
    if (row >= a.n_sel) return;
    const int32_t p = a.pos[row];
    if (p < 0 || p >= a.n_tok) return;
    const int head = g * a.G + col / a.R;
    const float cl2 = a.cl2;
    const float2* ml = a.part_ml + item * a.n_chunks * NCOL + col;
    float M = -1.0e30f;
    for (int c = 0; c < nu; ++c) M = fmaxf(M, ml[c * NCOL].x);
    float L = 0.0f;
    f32x4_t o[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) o[k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < nu; ++c) {
        const float2 mlc = ml[c * NCOL];
        const float w = __builtin_amdgcn_exp2f((mlc.x - M) * cl2);
        L += w * mlc.y;
        const f32x4_t* po = a.part_o + (((item * a.n_chunks + c) * 4 + wave) * 2 + nb) * (kMd * 4 * 64) + lane;
#pragma unroll
        for (int k = 0; k < kPer; ++k) o[k] += w * po[(q4 + 4 * k) * 64];
    }
    const float inv = 1.0f / L;
    uint16_t* op = a.out + (row * a.Hq + head) * (int64_t)D;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int ir = q4 + 4 * k, i = ir >> 2, r = ir & 3;
        const f32x4_t x = o[k] * inv;
        *reinterpret_cast<u32x2_t*>(op + 32 * i + 8 * r + 4 * half) =
            u32x2_t{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
    }
}

template <int D>
hipError_t launch(const AttnArgs& args, hipStream_t s) {
    const int64_t items = (int64_t)args.n_tiles * args.Hkv;
    hipLaunchKernelGGL(attention_kernel<D>, dim3((unsigned)(items * args.n_chunks)), dim3(256), 0, s, args);
    if (args.n_chunks > 1) hipLaunchKernelGGL(combine_kernel<D>, dim3((unsigned)(items * 8)), dim3(256), 0, s, args);
    return hipGetLastError();
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

AttnPlan plan_attention(int64_t n_sel, int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                        int32_t head_dim, int dtype) {
    AttnPlan p{};
    const int32_t G = n_q_heads / n_kv_heads;
    p.rows_per_tile = dtype == SEMSHARE_BF16 ? NCOL / G : 1;
    p.n_tiles = (n_sel + p.rows_per_tile - 1) / p.rows_per_tile;
    const int64_t n_kt = (n_tok + KT - 1) / KT;
    p.split_units = (int32_t)std::max<int64_t>(n_kt, 1);  // one piece per item
    p.n_chunks = 1;
    if (dtype == SEMSHARE_BF16 && n_sel > 0) {
        // Work estimate in 64-key tiles with the selected rows spread over the
        // prompt (a tile's causal range then averages half of it).  Items
        // longer than 3/4 of one CU's share are cut into equal pieces (shorter
        // pieces balance the CUs better but cost partial-result traffic and a
        // prologue each; 3/4 measured best at 5k tokens), never shorter than
        // 4 tiles.
        const double share = (double)p.n_tiles * n_kv_heads * (n_kt + 1) / 2.0 / kCUs;
        const int64_t su = std::max<int64_t>(kMinPieceKt, (int64_t)(share * kSplitShares));
        if (su < n_kt) {
            p.split_units = (int32_t)su;
            p.n_chunks = (int32_t)((n_kt + su - 1) / su);
            // Items with fewer pieces leave their trailing chunk slots empty.
            // At an even stride those empty workgroups line up with the
            // dispatcher's round-robin over the shader engines of an XCD and
            // the real ones all land on half of its CUs (measured 1.6x slower);
            // an odd stride spreads them.
            if (p.n_chunks % 2 == 0) p.n_chunks += 1;
        }
    }
    size_t off = 0;
    p.off_part_o = p.off_part_ml = p.off_used = 0;
    if (p.n_chunks > 1) {
        const size_t pieces = (size_t)p.n_tiles * n_kv_heads * p.n_chunks;
        off = align256(pieces * NCOL * head_dim * sizeof(float));
        p.off_part_ml = off;
        off = align256(off + pieces * NCOL * sizeof(float2));
        p.off_used = off;
        off = align256(off + (size_t)p.n_tiles * n_kv_heads * sizeof(int32_t));
    }
    p.total = off;
    return p;
}

hipError_t launch_attention_bf16(const AttnCall& a, const AttnPlan& p, hipStream_t s) {
    unsigned char* ws = static_cast<unsigned char*>(a.workspace);
    AttnArgs t{};
    t.q = static_cast<const uint16_t*>(a.q);
    t.pos = a.sel_pos;
    t.k_cache = static_cast<const uint16_t*>(a.k_cache);
    t.v_cache = static_cast<const uint16_t*>(a.v_cache);
    t.out = static_cast<uint16_t*>(a.out);
    t.part_o = reinterpret_cast<f32x4_t*>(ws + p.off_part_o);
    t.part_ml = reinterpret_cast<float2*>(ws + p.off_part_ml);
    t.n_used = reinterpret_cast<int32_t*>(ws + p.off_used);
    t.n_sel = a.n_sel;
    t.n_tok = a.n_tok;
    t.Hq = a.n_q_heads;
    t.Hkv = a.n_kv_heads;
    t.G = a.n_q_heads / a.n_kv_heads;
    t.R = p.rows_per_tile;
    t.n_tiles = (int32_t)p.n_tiles;
    t.split_units = p.split_units;
    t.n_chunks = p.n_chunks;
    t.cl2 = a.sm_scale * kLog2e;
    if (a.head_dim == 128) return launch<128>(t, s);
    return launch<64>(t, s);
}

}  // namespace semshare
