// Average attention score per token and the dynamic recompute set (Section 3
// Insight 2 and its Attention Recovery equation; Section 4.3.3: hot / cold
// tokens from AR at a 55% threshold, Recomputed = w_c * c + w_h * h).
//
// Mass of token j at a fully computed layer: the causal softmax attention
// P_h[i][j] of every head h, averaged over the heads and over the query rows
// i (rows before j contribute zero).  Two MFMA passes over the causal score
// matrix, bf16 operands and fp32 accumulation, exponentials in base 2, both
// computing S^T = K Q^T so that each lane owns one query row:
//   mass_lse_kernel  four waves per (8 query blocks of 32, head), two blocks
//                    each, the key tiles streamed: each lane keeps its row's
//                    running reference and sum over its 16 keys per block;
//                    the two lane halves merge at the end -> lse2[h][i].
//   mass_col_kernel  four waves per (8 key blocks of 32, head), two blocks
//                    each, the query tiles streamed with their normalisers:
//                    each lane adds exp2(s - lse2[i]) of its row to a sum per
//                    key row, and the 32 lanes of each half are summed once
//                    at the end -> part[h][j].
//   mass_final_kernel sums the heads in a fixed order and divides by H_q T.
// Each wave keeps the operands of its 2 fixed blocks in VGPRs; the other
// operand streams through a 4-stage LDS ring of 32-row tiles filled by
// direct-to-LDS loads and shared by the workgroup's 4 waves (with one wave
// per workgroup streaming its own tiles from L2, 790 instead of 652 us at
// 5120 tokens, bit-identical).  Where no key of a tile lies past a query
// row, a wave's two blocks are software-pipelined: the MFMAs of one block
// run while the exponentials of the other block's scores (of the same or the
// previous tile) are formed, each MFMA followed by two of them; the (at
// most two) tiles on the diagonal go block by block with their masks.  The
// normaliser pass takes no per-tile maximum: each lane exponentiates against
// a reference it saw earlier and falls back to the tile's maximum only
// while it has none or when the tile's sum exceeds 2^64 (fp32 sums keep
// their relative precision above 1).  At 5120 tokens, 32 / 8 heads: the
// normaliser pass 203 us, the column pass 190 us (365 us with S = Q K^T, a
// key column per lane and 16 bounds-checked normaliser loads per tile; 239
// us transposed; 190 us pipelined, with the normalisers brought in through
// the ring and the fixed operands waited for before the ring starts: the
// compiler had placed memory waits inside the loop that also covered the
// ring's loads).  Pipelining the normaliser pass moved it from 208 us only.
//
// dyn_select_kernel (one workgroup): tokens sorted by mass (descending, lower
// position first on ties); AR is the smallest count whose prefix reaches
// thres of the total, the sums taken in 2^-40 fixed point so that the
// integer decision does not depend on the summation order; the AR first
// tokens are hot.  Then round(w_h AR) hot and round(w_c (T - AR)) cold tokens
// with the largest deviation sigma (lower position first on ties) form the
// recompute set, written in ascending position order.
#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr int kNB = 2;  // fixed 32-blocks per wave (two waves per SIMD fit)
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ bf16x8_t ld8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p));
}

// lane -> row of the 32 x 32 MFMA output held in accumulator v
__device__ __forceinline__ int out_row(int v, int half) { return 8 * (v >> 2) + 4 * half + (v & 3); }

// The streamed operand (K for the normalisers, Q for the column sums) goes
// through a 4-stage LDS ring of 32-row tiles (32 x 128 bf16 = 8 KB) filled by
// direct-to-LDS loads and shared by the 4 waves of a workgroup, which own 8
// consecutive fixed blocks (2 each).  Rows are 256 B; 16-byte chunk c of row
// r sits at chunk c ^ (r & 15), so the 16 rows that one MFMA operand read
// touches at a time cover all banks.
constexpr int kMassWaves = 4;
constexpr int kMassStages = 4;
constexpr int kMassTile = 32 * 128 * 2;                 // bytes
constexpr int kMassLoads = kMassTile / 1024 / kMassWaves;  // 1-KB direct loads per wave per tile (2)

struct MassRing {
    uint32_t off[kMassLoads];  // per-lane byte offsets of this wave's rows within a tile's first row
    uint32_t lds;              // LDS base of the ring
    int wave;
    // lane -> (row 4 i + lane / 16 of the tile, physical chunk lane % 16)
    __device__ void init(int64_t row_stride_bytes, int w, uint32_t lds_base) {
        wave = w;
        lds = lds_base;
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int j = 0; j < kMassLoads; ++j) {
            const int r = 4 * (w * kMassLoads + j) + (lane >> 4);
            const int pc = lane & 15;
            off[j] = (uint32_t)(r * row_stride_bytes) + 16u * (uint32_t)(pc ^ (r & 15));
        }
    }
    // tile whose first row is at `base` (rows past the end clamp to `last`, a
    // row pointer of the operand's last row: computed, never used)
    __device__ void issue(const uint16_t* base, int64_t rows_left, int64_t row_stride_bytes, int stage) {
#pragma unroll
        for (int j = 0; j < kMassLoads; ++j) {
            const int r = 4 * (wave * kMassLoads + j) + ((threadIdx.x & 63) >> 4);
            const uint32_t o = r < rows_left ? off[j]
                                             : off[j] - (uint32_t)((r - (rows_left - 1)) * row_stride_bytes);
            g2lds(base, o, lds + stage * kMassTile + (wave * kMassLoads + j) * 1024);
        }
    }
    // operand fragment of k-step ks for row l32 (dims 8 half + 16 ks ... + 8)
    __device__ bf16x8_t frag(int stage, int l32, int half, int ks) const {
        const uint32_t addr = lds + stage * kMassTile + l32 * 256 + 16u * (uint32_t)((half + 2 * ks) ^ (l32 & 15));
        return *(const __attribute__((address_space(3))) bf16x8_t*)(uintptr_t)addr;
    }
};

// wait until at most N of this wave's tiles are in flight (kPer direct loads
// each), then meet the other waves
template <int N, int kPer = kMassLoads>
__device__ __forceinline__ void ring_wait() {
    wait_vmcnt<N * kPer>();
    ring_barrier();
}

// 4 bytes per lane from gbase + off straight into LDS at lds_base + 4 * lane
// (global_load_lds_dword; the direct-load counterpart of g2lds for one float
// per lane)
__device__ __forceinline__ void g2lds_b32(const void* gbase, uint32_t off, uint32_t lds_base) {
    const uint64_t g = reinterpret_cast<uint64_t>(gbase);
    const uint32_t g_hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
    const uint32_t g_lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)g);
    const uint64_t gs = ((uint64_t)g_hi << 32) | (uint64_t)g_lo;
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
                 :
                 : "v"(off), "s"(reinterpret_cast<const void*>(gs)), "s"((uint32_t)__builtin_amdgcn_readfirstlane(lds_base))
                 : "memory", "m0");
}

__global__ __launch_bounds__(64 * kMassWaves) void mass_lse_kernel(const uint16_t* __restrict__ q,
                                                                   const uint16_t* __restrict__ k, int64_t T,
                                                                   int32_t Hq, int32_t Hkv, float scale_log2e,
                                                                   float* __restrict__ lse2) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[kMassStages * kMassTile];
    const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = blockIdx.y, kvh = h / (Hq / Hkv);
    const int64_t nb = (T + 31) / 32;
    // the workgroups with the longest key ranges first
    const int64_t wg0 = ((int64_t)gridDim.x - 1 - blockIdx.x) * (2 * kMassWaves);
    const int64_t qb0 = wg0 + 2 * wave;
    bf16x8_t bq[kNB][8];
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        int64_t qi = (qb0 + b) * 32 + l32;
        if (qi >= T) qi = T - 1;
        const uint16_t* row = q + (qi * Hq + h) * 128 + 8 * half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) bq[b][ks] = ld8(row + 16 * ks);
    }
    wait_vmcnt<0>();  // the fixed operands are in before the ring's loads start
    float m[kNB], l[kNB];
#pragma unroll
    for (int b = 0; b < kNB; ++b) { m[b] = kNegInf; l[b] = 0.0f; }
    // key tiles of the workgroup: up to its last query block
    const int64_t kb_end = wg0 + 2 * kMassWaves < nb ? wg0 + 2 * kMassWaves : nb;
    const int64_t kstride = (int64_t)Hkv * 128 * 2;  // bytes between key rows
    const uint16_t* kbase = k + (int64_t)kvh * 128;
    MassRing ring;
    ring.init(kstride, wave, lds_addr(smem));
    auto issue = [&](int64_t kb) {
        ring.issue(kbase + kb * 32 * (int64_t)Hkv * 128, T - kb * 32, kstride, (int)(kb & (kMassStages - 1)));
    };
    // tile kb has landed for every wave (and every wave is done with tile
    // kb - 1, whose stage then takes tile kb + 3)
    auto open_tile = [&](int64_t kb) {
        if (kb + 2 < kb_end) ring_wait<2>();
        else if (kb + 1 < kb_end) ring_wait<1>();
        else ring_wait<0>();
        if (kb + kMassStages - 1 < kb_end) issue(kb + kMassStages - 1);
    };
    bf16x8_t ak[8];
    auto read_tile = [&](int64_t kb) {
        const int st = (int)(kb & (kMassStages - 1));
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) ak[ks] = ring.frag(st, l32, half, ks);
    };
    auto s_tile = [&](int b) {
        f32x16_t acc = {};
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak[ks], bq[b][ks], acc, 0, 0, 0);
        return acc;  // acc[v] = S^T[key = 32 kb + out_row(v)][query = 32 (qb0 + b) + l32]
    };
    // Exponentials against the lane's reference m (a maximum seen earlier,
    // scaled): the sum of a tile's 16 is accepted when m is set and the sum
    // shows no value far above it; otherwise (no reference yet, or a large
    // upward jump) the tile's own maximum becomes the reference and l is
    // rescaled.  The max is taken on the raw scores (the scale is positive).
    auto settle = [&](int b, const f32x16_t& acc, float ts) {
        if (m[b] != kNegInf && ts <= 0x1p64f) {
            l[b] += ts;
            return;
        }
        float bm = kNegInf;
#pragma unroll
        for (int v = 0; v < 16; ++v) bm = fmaxf(bm, acc[v]);
        const float mn = fmaxf(m[b], bm * scale_log2e);
        if (mn == kNegInf) return;  // no key of this half seen yet
        float sum = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) sum += __builtin_amdgcn_exp2f(fmaf(acc[v], scale_log2e, -mn));
        l[b] = (m[b] == kNegInf ? 0.0f : l[b] * __builtin_amdgcn_exp2f(m[b] - mn)) + sum;
        m[b] = mn;
    };
    // 8 MFMAs of S^T for block b of the tile in ak into `nxt`, each followed
    // by two exponentials of `cur` against block cb's reference, summed in
    // four partial sums; returns the sum
    auto step = [&](int b, f32x16_t& nxt, const f32x16_t& cur, int cb) {
        nxt = f32x16_t{};
        const float mc = m[cb];
        float e[16], ps[4];
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            nxt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak[ks], bq[b][ks], nxt, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int v = 2 * ks; v < 2 * ks + 2; ++v) e[v] = __builtin_amdgcn_exp2f(fmaf(cur[v], scale_log2e, -mc));
            if (ks > 0) {
#pragma unroll
                for (int v = 2 * ks - 2; v < 2 * ks; ++v) ps[v & 3] = v < 4 ? e[v] : ps[v & 3] + e[v];
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        ps[2] += e[14];
        ps[3] += e[15];
        return (ps[0] + ps[1]) + (ps[2] + ps[3]);
    };
    for (int64_t kb = 0; kb < kMassStages - 1; ++kb)
        if (kb < kb_end) issue(kb);
    // key tiles below both of the wave's query blocks need no mask: there the
    // blocks are pipelined (one block's MFMAs beside the other's
    // exponentials); the diagonal tiles go one block after the other; tiles
    // past the wave's blocks only take part in the ring
    const int64_t p_end = qb0 < kb_end ? qb0 : kb_end;
    int64_t kb = 0;
    if (p_end > 0) {
        open_tile(0);
        read_tile(0);
        f32x16_t accA = s_tile(0), accB;
        for (; kb + 1 < p_end; ++kb) {
            const float t0 = step(1, accB, accA, 0);  // block 1 of tile kb beside block 0's exponentials
            settle(0, accA, t0);
            open_tile(kb + 1);
            read_tile(kb + 1);
            const float t1 = step(0, accA, accB, 1);  // block 0 of tile kb + 1 beside block 1's of tile kb
            settle(1, accB, t1);
        }
        const float t0 = step(1, accB, accA, 0);  // the last unmasked tile
        settle(0, accA, t0);
        float t1 = 0.0f;
        {
            const float mc = m[1];
#pragma unroll
            for (int v = 0; v < 16; ++v) t1 += __builtin_amdgcn_exp2f(fmaf(accB[v], scale_log2e, -mc));
        }
        settle(1, accB, t1);
        ++kb;
    }
    for (; kb < kb_end; ++kb) {
        open_tile(kb);
        if (kb > qb0 + 1) continue;  // wave-uniform: past both blocks
        read_tile(kb);
#pragma unroll
        for (int b = 0; b < kNB; ++b) {
            if (kb > qb0 + b) continue;  // wave-uniform: the block lies above the diagonal
            f32x16_t acc = s_tile(b);
            // only the diagonal block has keys after its queries
            if (kb == qb0 + b) {
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (out_row(v, half) > l32) acc[v] = kNegInf;
            }
            float ts = 0.0f;
            const float mc = m[b];
#pragma unroll
            for (int v = 0; v < 16; ++v) ts += __builtin_amdgcn_exp2f(fmaf(acc[v], scale_log2e, -mc));
            settle(b, acc, ts);
        }
    }
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        const float om = __shfl_xor(m[b], 32), ol = __shfl_xor(l[b], 32);
        const float M = fmaxf(m[b], om);
        const float L = (m[b] == kNegInf ? 0.0f : l[b] * __builtin_amdgcn_exp2f(m[b] - M)) +
                        (om == kNegInf ? 0.0f : ol * __builtin_amdgcn_exp2f(om - M));
        const int64_t qi = (qb0 + b) * 32 + l32;
        if (half == 0 && qi < T) lse2[(int64_t)h * T + qi] = M + log2f(L);
    }
}

// The column pass streams the query tiles together with their rows' normalisers:
// per tile each wave also loads the 32 normalisers (one per lane, the two lane
// halves alike) into its own 256-byte slot of the stage, so they arrive
// through LDS and no wait for a global load sits in the loop.
constexpr int kColLoads = kMassLoads + 1;  // direct loads per wave per tile
constexpr int kLseSlots = kMassStages * kMassTile;  // LDS offset of the normaliser slots

__global__ __launch_bounds__(64 * kMassWaves) void mass_col_kernel(const uint16_t* __restrict__ q,
                                                                   const uint16_t* __restrict__ k, int64_t T,
                                                                   int64_t row_begin, int32_t Hq, int32_t Hkv,
                                                                   float scale_log2e,
                                                                   const float* __restrict__ lse2,
                                                                   float* __restrict__ part) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[kMassStages * kMassTile + kMassStages * kMassWaves * 256];
    const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5, l32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = blockIdx.y, kvh = h / (Hq / Hkv);
    const int64_t nb = (T + 31) / 32;
    const int64_t wg0 = (int64_t)blockIdx.x * (2 * kMassWaves);  // the longest row ranges first
    const int64_t kb0 = wg0 + 2 * wave;
    bf16x8_t bk[kNB][8];
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        int64_t kj = (kb0 + b) * 32 + l32;
        if (kj >= T) kj = T - 1;
        const uint16_t* row = k + (kj * Hkv + kvh) * 128 + 8 * half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) bk[b][ks] = ld8(row + 16 * ks);
    }
    wait_vmcnt<0>();  // the fixed operands are in before the ring's loads start
    // per lane and key row v of each block: the sum over the query rows this
    // lane has held (one per tile); the lanes are summed at the end
    float col[kNB][16];
#pragma unroll
    for (int b = 0; b < kNB; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) col[b][v] = 0.0f;
    const float* lse_h = lse2 + (int64_t)h * T;
    // row tiles of the workgroup: from its first key block (or the window) to the end
    const int64_t qb_first = wg0 > row_begin / 32 ? wg0 : row_begin / 32;
    const int64_t qstride = (int64_t)Hq * 128 * 2;
    const uint16_t* qbase = q + (int64_t)h * 128;
    const uint32_t smem_base = lds_addr(smem);
    MassRing ring;
    ring.init(qstride, wave, smem_base);
    auto stage_of = [&](int64_t qb) { return (int)((qb - qb_first) & (kMassStages - 1)); };
    auto issue = [&](int64_t qb) {
        const int st = stage_of(qb);
        ring.issue(qbase + qb * 32 * (int64_t)Hq * 128, T - qb * 32, qstride, st);
        // the tile's normalisers (rows past T read the last row: replaced below)
        const int64_t r0 = qb * 32;
        const int64_t r = r0 + l32 < T ? r0 + l32 : T - 1;
        g2lds_b32(lse_h + r0, (uint32_t)((r - r0) * 4), smem_base + kLseSlots + (st * kMassWaves + wave) * 256);
    };
    // tile qb has landed for every wave (and every wave is done with tile
    // qb - 1, whose stage then takes tile qb + 3)
    auto open_tile = [&](int64_t qb) {
        if (qb + 2 < nb) ring_wait<2, kColLoads>();
        else if (qb + 1 < nb) ring_wait<1, kColLoads>();
        else ring_wait<0, kColLoads>();
        if (qb + kMassStages - 1 < nb) issue(qb + kMassStages - 1);
    };
    // this lane's query row of tile qb: its operand fragments and its
    // normaliser (+inf outside the window or past T: such rows add 0)
    bf16x8_t aq[8];
    auto read_tile = [&](int64_t qb) {
        const int st = stage_of(qb);
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) aq[ks] = ring.frag(st, l32, half, ks);
        const float x = *(const __attribute__((address_space(3))) float*)(uintptr_t)(
            smem_base + kLseSlots + (st * kMassWaves + wave) * 256 + 4 * lane);
        const int64_t r = qb * 32 + l32;
        return r < T && r >= row_begin ? x : __builtin_inff();
    };
    auto s_tile = [&](int b) {
        f32x16_t acc = {};
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bk[b][ks], aq[ks], acc, 0, 0, 0);
        return acc;  // acc[v] = S^T[key = 32 (kb0 + b) + out_row(v)][query = 32 qb + l32]
    };
    // 8 MFMAs of S^T for block b of the tile in aq into `nxt`, each followed
    // by two scores of `cur` (fma, exponential, sum) under normaliser L
    auto step = [&](int b, f32x16_t& nxt, const f32x16_t& cur, float (&cs)[16], float L) {
        nxt = f32x16_t{};
        float e[16];
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            nxt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bk[b][ks], aq[ks], nxt, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int v = 2 * ks; v < 2 * ks + 2; ++v) e[v] = __builtin_amdgcn_exp2f(fmaf(cur[v], scale_log2e, -L));
            if (ks > 0) {
#pragma unroll
                for (int v = 2 * ks - 2; v < 2 * ks; ++v) cs[v] += e[v];
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        cs[14] += e[14];
        cs[15] += e[15];
    };
    for (int64_t qb = qb_first; qb < qb_first + kMassStages - 1; ++qb)
        if (qb < nb) issue(qb);
    // tiles before the wave's first key block only take part in the ring;
    // the (at most two) tiles where a block's keys reach past a query row go
    // one block after the other with the keys after each row masked; from
    // there on the blocks are pipelined: one block's MFMAs run while the
    // other block's scores are exponentiated and summed
    const int64_t start = kb0 > qb_first ? kb0 : qb_first;
    const int64_t p0 = kb0 + 2 > start ? kb0 + 2 : start;
    int64_t qb = qb_first;
    for (; qb < nb && qb < start; ++qb) open_tile(qb);
    for (; qb < nb && qb < p0; ++qb) {
        open_tile(qb);
        const float L = read_tile(qb);
#pragma unroll
        for (int b = 0; b < kNB; ++b) {
            f32x16_t acc = s_tile(b);
            const int64_t lim = qb * 32 + l32 - (kb0 + b) * 32;  // key row v is kept iff out_row(v) <= lim
#pragma unroll
            for (int v = 0; v < 16; ++v)
                col[b][v] += out_row(v, half) <= lim ? __builtin_amdgcn_exp2f(fmaf(acc[v], scale_log2e, -L)) : 0.0f;
        }
    }
    if (qb < nb) {
        open_tile(qb);
        float L = read_tile(qb);
        f32x16_t accA = s_tile(0), accB;
        for (; qb + 1 < nb; ++qb) {
            step(1, accB, accA, col[0], L);  // block 1 of tile qb beside block 0's scores
            open_tile(qb + 1);
            const float Ln = read_tile(qb + 1);
            step(0, accA, accB, col[1], L);  // block 0 of tile qb + 1 beside block 1's scores of tile qb
            L = Ln;
        }
        step(1, accB, accA, col[0], L);  // the last tile
#pragma unroll
        for (int v = 0; v < 16; ++v) col[1][v] += __builtin_amdgcn_exp2f(fmaf(accB[v], scale_log2e, -L));
    }
    // sum over the 32 query lanes of each half (a fixed butterfly), then lane
    // v of the half writes key row v
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        float c[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) c[v] = col[b][v];
#pragma unroll
        for (int o = 1; o < 32; o <<= 1)
#pragma unroll
            for (int v = 0; v < 16; ++v) c[v] += __shfl_xor(c[v], o);
        float mine = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) mine = l32 == v ? c[v] : mine;
        const int64_t key = (kb0 + b) * 32 + out_row(l32 & 15, half);
        if (l32 < 16 && key < T) part[(int64_t)h * T + key] = mine;
    }
}

__global__ void mass_final_kernel(const float* __restrict__ part, int64_t T, int64_t n_rows, int32_t Hq,
                                  float* __restrict__ mass) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= T) return;
    float s = 0.0f;
    for (int h = 0; h < Hq; ++h) s += part[(int64_t)h * T + j];
    mass[j] = s / ((float)Hq * (float)n_rows);
}

// ------------------------------------------------------------ selection
constexpr int kSelThreads = 1024;

__device__ __forceinline__ void cmp_swap(uint64_t& a, uint64_t& b, bool up) {
    if ((a > b) == up) {
        const uint64_t t = a;
        a = b;
        b = t;
    }
}

// Bitonic sort (ascending) of n2 = 2^k keys in LDS by the whole workgroup.
// Thread t owns elements [8t, 8t + 8) and wave w the 512 elements [512w,
// 512w + 512): passes with stride >= 512 exchange across waves (a workgroup
// barrier each), strides 8 .. 256 stay inside a wave's segment (the wave's
// own LDS traffic is ordered, so no barrier), strides 4, 2, 1 inside a
// thread's registers.
__device__ __forceinline__ void bitonic_sort(uint64_t* key, int n2) {
    const int t = threadIdx.x;
    for (int size = 2; size <= n2; size <<= 1) {
        int stride = size >> 1;
        for (; stride >= 512; stride >>= 1) {  // across waves
            for (int p = t; p < n2 / 2; p += kSelThreads) {
                const int i = 2 * p - (p & (stride - 1));
                cmp_swap(key[i], key[i + stride], (i & size) == 0);
            }
            __syncthreads();
        }
        const int seg = 512 * (t >> 6), lane = t & 63;
        if (seg < n2) {
            for (; stride >= 8; stride >>= 1) {  // inside the wave's segment
                for (int p = lane; p < 256; p += 64) {
                    const int i = seg + 2 * p - (p & (stride - 1));
                    if (i + stride < n2) cmp_swap(key[i], key[i + stride], (i & size) == 0);
                }
                __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
                __builtin_amdgcn_wave_barrier();
            }
            if (8 * t < n2) {  // strides 4, 2, 1 in registers
                uint64_t r[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) r[e] = key[8 * t + e];
#pragma unroll
                for (int st = 4; st >= 1; st >>= 1) {
                    if (st >= size) continue;
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if ((e & st) == 0) cmp_swap(r[e], r[e + st], ((8 * t + e) & size) == 0);
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) key[8 * t + e] = r[e];
            }
        }
        __syncthreads();
    }
}

// exclusive block scan of one int64 per thread; returns the total too
__device__ __forceinline__ int64_t block_scan_i64(int64_t v, int64_t* tot, int64_t* sw) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int64_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(x, d);
        if (lane >= d) x += y;
    }
    if (lane == 63) sw[w] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t run = 0;
        for (int i = 0; i < kSelThreads / 64; ++i) { const int64_t c = sw[i]; sw[i] = run; run += c; }
        sw[kSelThreads / 64] = run;
    }
    __syncthreads();
    const int64_t ex = sw[w] + x - v;
    *tot = sw[kSelThreads / 64];
    __syncthreads();
    return ex;
}

__device__ __forceinline__ float clamp01(float m) { return m > 0.0f ? (m < 1.0f ? m : 1.0f) : 0.0f; }

__global__ __launch_bounds__(kSelThreads) void dyn_select_kernel(const float* __restrict__ mass,
                                                                  const float* __restrict__ sigma, int32_t n,
                                                                  double thres, double w_hot, double w_cold,
                                                                  int32_t* __restrict__ sel_pos,
                                                                  int32_t* __restrict__ counts) {
    __shared__ uint64_t key[kMaxDynTok];
    __shared__ uint8_t hot[kMaxDynTok];
    __shared__ int64_t sw[kSelThreads / 64 + 1];
    __shared__ int s_ar;
    int n2 = 1;
    while (n2 < n) n2 <<= 1;
    // 1. mass descending, lower position first
    for (int i = threadIdx.x; i < n2; i += kSelThreads) {
        if (i < n) {
            const uint32_t mb = __float_as_uint(clamp01(mass[i]));
            key[i] = ((uint64_t)(0xFFFFFFFFu - mb) << 32) | (uint32_t)i;
        } else {
            key[i] = ~0ull;
        }
    }
    if (threadIdx.x == 0) s_ar = n;
    __syncthreads();
    bitonic_sort(key, n2);
    // 2. AR: first count whose fixed-point prefix reaches thres * total
    constexpr int kPer = kMaxDynTok / kSelThreads;
    const int base = threadIdx.x * kPer;
    int64_t fx[kPer];
    int64_t local = 0;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int i = base + e;
        fx[e] = 0;
        if (i < n) {
            const int pos = (int)(key[i] & 0xFFFFFFFFu);
            fx[e] = (int64_t)floor((double)clamp01(mass[pos]) * 1099511627776.0);  // 2^40
        }
        local += fx[e];
    }
    int64_t total;
    int64_t run = block_scan_i64(local, &total, sw);
    const double target = thres * (double)total;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int i = base + e;
        run += fx[e];
        if (i < n && (double)run >= target) {
            atomicMin(&s_ar, i + 1);
            break;
        }
    }
    __syncthreads();
    const int ar = n > 0 ? s_ar : 0;
    for (int i = threadIdx.x; i < n; i += kSelThreads) hot[(int)(key[i] & 0xFFFFFFFFu)] = i < ar ? 1 : 0;
    __syncthreads();
    const int n_hot = (int)floor(w_hot * (double)ar + 0.5);
    const int n_cold = (int)floor(w_cold * (double)(n - ar) + 0.5);
    // 3. hot group first, then cold; sigma descending, lower position first
    for (int i = threadIdx.x; i < n2; i += kSelThreads) {
        if (i < n) {
            const uint32_t sb = __float_as_uint(sigma[i] > 0.0f ? sigma[i] : 0.0f) & 0x7FFFFFFFu;
            key[i] = ((uint64_t)(hot[i] ? 0u : 1u) << 62) | ((uint64_t)(0x7FFFFFFFu - sb) << 20) | (uint32_t)i;
        } else {
            key[i] = ~0ull;
        }
    }
    __syncthreads();
    bitonic_sort(key, n2);
    // hot occupies sorted [0, ar), cold [ar, n): mark the chosen positions
    for (int i = threadIdx.x; i < n; i += kSelThreads) {
        const int pos = (int)(key[i] & 0xFFFFFu);
        const bool take = i < ar ? i < n_hot : i - ar < n_cold;
        hot[pos] = take ? 1 : 0;  // reused: selected flag by position
    }
    __syncthreads();
    // 4. compaction in position order
    int64_t cnt = 0;
#pragma unroll
    for (int e = 0; e < kPer; ++e) cnt += (base + e < n && hot[base + e]) ? 1 : 0;
    int64_t tot2;
    int64_t o = block_scan_i64(cnt, &tot2, sw);
#pragma unroll
    for (int e = 0; e < kPer; ++e)
        if (base + e < n && hot[base + e]) sel_pos[o++] = base + e;
    if (threadIdx.x == 0) {
        counts[0] = ar;
        counts[1] = (int32_t)tot2;
        counts[2] = n_hot;
    }
}

// Retention (Section 4.3.4, Appendix A.6): hot tokens (the AR first by
// mass) and recomputed tokens are never evicted and rank first, in position
// order; the other tokens follow by score (descending, lower position first).
// The first R = max(floor(max(min_keep, AR / T) T + 1/2), forced) are kept.
__global__ __launch_bounds__(kSelThreads) void retention_kernel(const float* __restrict__ mass,
                                                                 const float* __restrict__ score, int32_t n,
                                                                 const int32_t* __restrict__ sel_pos,
                                                                 const int32_t* __restrict__ counts, double min_keep,
                                                                 int32_t* __restrict__ rank,
                                                                 int32_t* __restrict__ kept_pos,
                                                                 int32_t* __restrict__ n_kept) {
    __shared__ uint64_t key[kMaxDynTok];
    __shared__ uint8_t flag[kMaxDynTok];
    __shared__ int64_t sw[kSelThreads / 64 + 1];
    int n2 = 1;
    while (n2 < n) n2 <<= 1;
    const int ar = counts[0] < n ? counts[0] : n;
    const int n_sel = counts[1] < n ? counts[1] : n;
    // hot set: the mass order of the dynamic selection
    for (int i = threadIdx.x; i < n2; i += kSelThreads) {
        if (i < n) {
            const uint32_t mb = __float_as_uint(clamp01(mass[i]));
            key[i] = ((uint64_t)(0xFFFFFFFFu - mb) << 32) | (uint32_t)i;
        } else {
            key[i] = ~0ull;
        }
    }
    __syncthreads();
    bitonic_sort(key, n2);
    for (int i = threadIdx.x; i < n; i += kSelThreads) flag[(int)(key[i] & 0xFFFFFFFFu)] = i < ar ? 1 : 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n_sel; i += kSelThreads) {
        const int p = sel_pos[i];
        if (p >= 0 && p < n) flag[p] = 1;
    }
    __syncthreads();
    // forced first by position, then the rest by score
    for (int i = threadIdx.x; i < n2; i += kSelThreads) {
        if (i < n) {
            if (flag[i]) {
                key[i] = (uint64_t)i;
            } else {
                const uint32_t sb = __float_as_uint(score[i] > 0.0f ? score[i] : 0.0f) & 0x7FFFFFFFu;
                key[i] = (1ull << 62) | ((uint64_t)(0x7FFFFFFFu - sb) << 20) | (uint32_t)i;
            }
        } else {
            key[i] = ~0ull;
        }
    }
    __syncthreads();
    bitonic_sort(key, n2);
    constexpr int kPer = kMaxDynTok / kSelThreads;
    const int base = threadIdx.x * kPer;
    int64_t nf = 0;
#pragma unroll
    for (int e = 0; e < kPer; ++e) nf += (base + e < n && flag[base + e]) ? 1 : 0;
    int64_t n_forced;
    (void)block_scan_i64(nf, &n_forced, sw);
    const double ratio = n > 0 && (double)ar / (double)n > min_keep ? (double)ar / (double)n : min_keep;
    int keep = (int)floor(ratio * (double)n + 0.5);
    if (keep < (int)n_forced) keep = (int)n_forced;
    if (keep > n) keep = n;
    for (int i = threadIdx.x; i < n; i += kSelThreads) {
        const int pos = (int)(key[i] & 0xFFFFFu);
        rank[pos] = i;
        flag[pos] = i < keep ? 1 : 0;  // reused: kept
    }
    __syncthreads();
    int64_t cnt = 0;
#pragma unroll
    for (int e = 0; e < kPer; ++e) cnt += (base + e < n && flag[base + e]) ? 1 : 0;
    int64_t tot;
    int64_t o = block_scan_i64(cnt, &tot, sw);
#pragma unroll
    for (int e = 0; e < kPer; ++e)
        if (base + e < n && flag[base + e]) kept_pos[o++] = base + e;
    if (threadIdx.x == 0) *n_kept = keep;
}

}  // namespace

hipError_t launch_retention(const float* mass, const float* score, int32_t n_tok, const int32_t* sel_pos,
                            const int32_t* counts, double min_keep, int32_t* rank, int32_t* kept_pos, int32_t* n_kept,
                            hipStream_t s) {
    if (n_tok > kMaxDynTok)
        return launch_retention_large(mass, score, n_tok, sel_pos, counts, min_keep, rank, kept_pos, n_kept, s);
    hipLaunchKernelGGL(retention_kernel, dim3(1), dim3(kSelThreads), 0, s, mass, score, n_tok, sel_pos, counts,
                       min_keep, rank, kept_pos, n_kept);
    return hipGetLastError();
}

size_t attention_mass_workspace(int64_t n_tok, int32_t n_q_heads) {
    return (size_t)2 * (size_t)n_q_heads * (size_t)n_tok * sizeof(float);
}

hipError_t launch_attention_mass(const void* q, const void* k, int64_t n_tok, int64_t row_begin, int32_t n_q_heads,
                                 int32_t n_kv_heads, float sm_scale, float* mass, void* workspace, hipStream_t s,
                                 bool reuse_normalisers) {
    float* lse2 = static_cast<float*>(workspace);
    float* part = lse2 + (int64_t)n_q_heads * n_tok;
    const float sl2e = sm_scale * 1.4426950408889634f;
    const int64_t nb = (n_tok + 31) / 32;
    const dim3 grid((unsigned)((nb + 2 * kMassWaves - 1) / (2 * kMassWaves)), (unsigned)n_q_heads);
    const auto* qp = static_cast<const uint16_t*>(q);
    const auto* kp = static_cast<const uint16_t*>(k);
    // the row normalisers do not depend on row_begin: a window pass after a
    // pass over the same q and K finds them in the workspace
    if (!reuse_normalisers)
        hipLaunchKernelGGL(mass_lse_kernel, grid, dim3(64 * kMassWaves), 0, s, qp, kp, n_tok, n_q_heads, n_kv_heads,
                           sl2e, lse2);
    hipLaunchKernelGGL(mass_col_kernel, grid, dim3(64 * kMassWaves), 0, s, qp, kp, n_tok, row_begin, n_q_heads,
                       n_kv_heads, sl2e, lse2, part);
    hipLaunchKernelGGL(mass_final_kernel, dim3((unsigned)((n_tok + 255) / 256)), dim3(256), 0, s, part, n_tok,
                       n_tok - row_begin, n_q_heads, mass);
    return hipGetLastError();
}

hipError_t launch_dynamic_recompute(const float* mass, const float* sigma, int32_t n_tok, double thres, double w_hot,
                                    double w_cold, int32_t* sel_pos, int32_t* counts, hipStream_t s) {
    if (n_tok > kMaxDynTok)
        return launch_dynamic_recompute_large(mass, sigma, n_tok, thres, w_hot, w_cold, sel_pos, counts, s);
    hipLaunchKernelGGL(dyn_select_kernel, dim3(1), dim3(kSelThreads), 0, s, mass, sigma, n_tok, thres, w_hot, w_cold,
                       sel_pos, counts);
    return hipGetLastError();
}

}  // namespace semshare
