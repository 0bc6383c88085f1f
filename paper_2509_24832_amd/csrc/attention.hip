// Causal grouped-query attention of the recomputed tokens over the assembled
// cache (Sections 4.2, 4.3.3), bf16 storage, fp32 accumulation and softmax.
//
// For a selected row at position p and query head h:
//   out = softmax_{j <= p}(q_h . K[j][h/G] * scale) V[j][h/G]
//
// Work decomposition.  A 512-thread workgroup owns one kv head g and 256
// query columns = (256/G selected rows) x (the G query heads of g); it runs
// alone on its CU with two waves per SIMD, each wave owning one 32-column
// block.  The two waves of a SIMD share its matrix core, so the softmax
// arithmetic of one runs while the other's MFMAs execute (with one wave per
// SIMD and two blocks per wave the key loop took ~62 cycles per MFMA, with
// two waves ~51 per MFMA and SIMD; 11% fewer cycles per workgroup at 5120
// tokens, partly given back by a lower clock under the higher MFMA load).
// S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_32x32x16_bf16: every lane then
// holds one query column.  Every MFMA operand and accumulator (Q, the two
// score tiles, O) lives in the architectural vector registers (the file is
// built with the VGPR form of MFMA; 221 registers, two waves per SIMD): with
// scores accumulated in AGPRs, each score had to be copied out
// (v_accvgpr_read) before the softmax could use it, and each masked score
// copied back, 16 to 48 extra vector instructions per 32-key sub-tile.
//
// Data movement.  K and V tiles of 64 keys travel by direct-to-LDS loads
// (global_load_lds_dwordx4) into a 4-stage ring, in their natural [key][d]
// layout with the 16-byte chunk index XOR-swizzled per row (K by row mod D/8;
// V so that the 32 lanes a transposing read serves per pass cover all 64
// banks, ACfg::vswz), so the MFMA operand reads below are free of bank
// conflicts (the SQ_LDS_BANK_CONFLICT counter reads 0; a V swizzle that was
// conflict-free only per 16 lanes cost 1.3 conflict cycles per LDS
// instruction).  V^T operands come from ds_read_b64_tr_b16, which transposes
// 4 keys x 4 dims per 16-lane group on the way out of LDS.  The K tiles of
// all ring stages lie in the lower 64 KB of LDS, the V tiles in the upper;
// the key loop is unrolled over the eight sub-tile positions of the ring, so
// every operand read there is a per-lane base register plus the instruction's
// immediate offset: no address arithmetic is left in the loop (13 of 65 vector
// instructions per 32-key sub-tile before; 5% less time per call).
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
// normaliser l sums the probabilities as the PV product consumes them,
// rounded to bf16, one v_dot2c_f32_bf16 per packed pair against (1, 1): half
// the instructions of two fp32 adds per pair, and the output is then an
// exactly normalised average of V's rows under the rounded weights.
//
// Work division (stream-K over keys).  The unit of work is one 64-key tile
// of one row tile's causal range: a row tile whose largest valid position is
// pmax has pmax/64 + 1 units, the same for every kv head.  A plan kernel lays
// the row tiles end to end, each preceded by kSegCost units standing for the
// fixed cost of starting it (W positions per head), and cuts the line into P
// equal contiguous ranges, one workgroup (one CU) each, so the CUs finish
// together whatever the mix of short and long causal ranges.  A workgroup
// walks its range one segment (the part of a row tile inside it) at a time.  A row
// tile inside a single range writes its output directly; the pieces of a row
// tile that range boundaries cut write (m, l) in fp32 and O / l in bf16, in
// register order (coalesced), to slots the plan assigns, and a combine kernel
// merges them by log-sum-exp in piece order (deterministic).  bf16 pieces
// halve that traffic; each adds one bf16 rounding (relative 2^-9) before the
// output's own.
#include <algorithm>
#include <atomic>
#include <climits>
#include <mutex>
#include <type_traits>

#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int KT = 64;       // keys per LDS tile (two sub-tiles)
constexpr int NCOL = 256;    // query columns per workgroup
constexpr int kNW = 8;       // waves per workgroup (two per SIMD)
constexpr int kNB = NCOL / 32 / kNW;  // 32-column blocks per wave
constexpr int kStages = 4;   // K/V ring depth
constexpr float kSumLimit = 65536.0f;  // 2^16
constexpr int kCUs = 256;        // compute units of the chip
// plan header: W, ranges, split row tiles, slots used, then the sizes it was
// made for (n_sel, n_tok, Hq, Hkv, R), which a launch checks before using it
constexpr int kPlanHdr = 12;
// Fixed cost of a segment (Q and first K/V loads before the key loop, the
// output or partial-result stores after it) in units of one 64-key tile of
// the key loop (measured ~14 us against ~2 us per unit at 256 columns x D 128).
constexpr int32_t kSegCost = 6;

typedef float f32x8_t __attribute__((ext_vector_type(8)));

// acc + the two bf16 values of a packed pair (one v_dot2c_f32_bf16 against (1, 1))
__device__ __forceinline__ float sum_pair(uint32_t pair, float acc) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pair), __builtin_bit_cast(bf16x2_t, 0x3F803F80u),
                                           acc, false);
}
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

struct AttnArgs {
    const uint16_t* q;        // [n_sel][Hq][D]
    const int32_t* pos;       // [n_sel]
    const uint16_t* k_cache;  // [n_tok][Hkv][D]
    const uint16_t* v_cache;
    uint16_t* out;            // [n_sel][Hq][D]
    u32x2_t* part_o;          // [Hkv][max_slots][NCOL * D / 4] bf16 x4 (O / l), register-native order
    float2* part_ml;          // [Hkv][max_slots][NCOL]  (m, l)
    // plan (int32): header [kPlanHdr] = W, ranges P', split row tiles, slots, sizes;
    // ranges [P][4] = first unit, end unit, first row tile, piece index of
    // its first segment; row tiles [n_tiles][8] = first unit, end unit, pmin,
    // pmax, slot base, pieces, -, -; cut row tiles [P][4] = row tile, slot
    // base, pieces, -
    int32_t* plan;
    int64_t n_sel, n_tok;
    int32_t Hq, Hkv, G, R;
    int32_t lgR;              // log2(R): R = 256 / G is a power of two
    int32_t n_tiles;
    int32_t P;                // ranges (workgroups) per kv head
    int32_t max_slots;        // partial-result slots per kv head
    float cl2;                // sm_scale * log2(e)
};

template <int D>
struct ACfg {
    static constexpr int kNch = D / 8;               // 16-B chunks per key row
    static constexpr int kRowBytes = 2 * D;
    static constexpr int kTileBytes = KT * kRowBytes;  // one tensor
    static constexpr int kVBase = kStages * kTileBytes;  // the K tiles of all stages, then the V tiles
    static constexpr int kLds = 2 * kStages * kTileBytes;
    static constexpr int kRowsPerLoad = 64 / kNch;     // rows one 1-KB direct load covers
    static constexpr int kLoadsPerWave = KT / kRowsPerLoad / kNW;  // per tensor
    static constexpr int kLoads = 2 * kLoadsPerWave;   // per wave per tile (K + V)
    static constexpr int kMd = D / 32;                 // 32-row blocks of O^T
    static constexpr int kKs = D / 16;                 // k-steps of S^T
    // V swizzle: chunk c of key row r is stored at chunk c ^ vswz(r).  A
    // transposing read serves 32 lanes per pass: the 4 rows x 4 chunks of one
    // 32-dim block that they read must fill all 64 banks (D = 128: 256-byte
    // rows, so the 4 rows take 4 different 4-chunk blocks; D = 64: 128-byte
    // rows, two per bank sweep, so rows r and r + 2 take different blocks)
    static __host__ __device__ constexpr int vswz(int r) { return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); }
};

// One segment: keys [kbeg, kend) of row tile `tile` for kv head g (kend <=
// pmax + 1; pmin = the tile's smallest valid position).  slot < 0: the
// segment is the whole causal range and writes the output; otherwise it
// writes its (m, l, O) to partial-result slot `slot` of head g.
template <int D>
__device__ __forceinline__ void segment(const AttnArgs& a, unsigned char* smem, const int g, const int tile,
                                        const int32_t kbeg, const int32_t kend, const int32_t pmin, const int slot) {
    using C = ACfg<D>;
    // the lane id through an opaque copy: nothing derived from it is hoisted
    // out of the segment loop (it would stay live through the key loop)
    int tid = (int)threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, l32 = lane & 31;

    // the arguments the prologue needs, requested together: one wait for
    // all of them rather than one per first use
    const int32_t lgR = a.lgR, Hq = a.Hq, G = a.G;
    const int64_t n_sel = a.n_sel;
    const int32_t* const posp = a.pos;
    const uint16_t* const qbase = a.q;
    asm volatile("" ::"s"(lgR), "s"(Hq), "s"(G), "s"(n_sel), "s"(posp), "s"(qbase));
    // this lane's two query columns: column c of the tile is row c % R of
    // it, query head g*G + c / R
    int64_t row[kNB];
    int32_t p_l[kNB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
        const int c = 32 * (kNB * wave + nb) + l32;
        row[nb] = ((int64_t)tile << lgR) + (c & ((1 << lgR) - 1));
        p_l[nb] = row[nb] < n_sel ? posp[row[nb]] : -1;  // checked below, after the Q loads are out
    }
    // Q^T operands: lane half h holds d in [h*D/2, h*D/2 + D/2).  All loads
    // are issued here, together with the positions; they become MFMA
    // operands (zeroed for columns without a position) once the first K/V
    // tile is on its way as well.
    u32x4_t qv[kNB][C::kKs];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
        const int c = 32 * (kNB * wave + nb) + l32;
        const u32x4_t* qp = reinterpret_cast<const u32x4_t*>(
            qbase + ((row[nb] < n_sel ? row[nb] : 0) * Hq + g * G + (c >> lgR)) * (int64_t)D + half * (D / 2));
#pragma unroll
        for (int s = 0; s < C::kKs; ++s) qv[nb][s] = qp[s];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
        if (p_l[nb] < 0 || p_l[nb] >= a.n_tok) p_l[nb] = -1;
    bf16x8_t qf[kNB][C::kKs];

    // ---- direct-load sources.  Load i of this wave (per tensor) fills rows
    // [rpl*(wave*lpw + i), +rpl) of the tile; lane -> (row, physical chunk pc),
    // it fetches the logical chunk that the swizzle stores at pc.
    const int32_t row_stride = a.Hkv * D;
    const uint16_t* kbase = a.k_cache + (int64_t)g * D;
    const uint16_t* vbase = a.v_cache + (int64_t)g * D;
    const int32_t last_key = (int32_t)a.n_tok - 1;
    const uint32_t smem_base = lds_addr(smem);
    // Loads of one 64-key tile: scalar bases of its first key row, per-lane
    // byte offsets of this wave's rows (clamped to the last key), LDS base.
    struct TileLoads {
        const uint16_t* kg;
        const uint16_t* vg;
        uint32_t off_k[C::kLoadsPerWave], off_v[C::kLoadsPerWave];
        uint32_t lds;
    };
    // per-lane byte offsets of this wave's rows for a tile that lies below
    // the last key (the common case), formed once per segment
    uint32_t off_k0[C::kLoadsPerWave], off_v0[C::kLoadsPerWave];
    auto row_offsets = [&](int32_t lim, uint32_t (&ok)[C::kLoadsPerWave], uint32_t (&ov)[C::kLoadsPerWave]) {
        const int pc = lane % C::kNch;
#pragma unroll
        for (int i = 0; i < C::kLoadsPerWave; ++i) {
            const int rw = C::kRowsPerLoad * (wave * C::kLoadsPerWave + i) + lane / C::kNch;
            const uint32_t r = (uint32_t)min(rw, lim);
            ok[i] = (r * (uint32_t)row_stride + 8u * (uint32_t)(pc ^ (rw & (C::kNch - 1)))) * 2u;
            ov[i] = (r * (uint32_t)row_stride + 8u * (uint32_t)(pc ^ C::vswz(rw))) * 2u;
        }
    };
    row_offsets(KT - 1, off_k0, off_v0);
    auto prep_tile = [&](int t, TileLoads& d) {
        const int32_t key0 = kbeg + t * KT;
        d.kg = kbase + (int64_t)key0 * row_stride;
        d.vg = vbase + (int64_t)key0 * row_stride;
        const int32_t lim = last_key - key0;
        if (lim >= KT - 1) {
#pragma unroll
            for (int i = 0; i < C::kLoadsPerWave; ++i) {
                d.off_k[i] = off_k0[i];
                d.off_v[i] = off_v0[i];
            }
        } else {
            row_offsets(lim, d.off_k, d.off_v);  // rows past the last key read the last key
        }
        d.lds = __builtin_amdgcn_readfirstlane(smem_base + (t % kStages) * C::kTileBytes +
                                               wave * C::kLoadsPerWave * 1024);
    };
    // load n of the tile (n in [0, kLoads)): K for even n, V for odd n, rows of load n/2
    auto issue_one = [&](const TileLoads& d, int n) {
        const int i = n >> 1;
        if (n & 1) g2lds(d.vg, d.off_v[i], d.lds + i * 1024 + C::kVBase);
        else g2lds(d.kg, d.off_k[i], d.lds + i * 1024);
    };
    auto issue = [&](int t) {
        TileLoads d;
        prep_tile(t, d);
#pragma unroll
        for (int n = 0; n < C::kLoads; ++n) issue_one(d, n);
    };

    // ---- LDS read offsets (bytes within a stage)
    // K (A operand of S^T): key row l32 of the sub-tile, logical chunk
    // half*(D/16) + s, stored at chunk (half*(D/16) + s) ^ (l32 % (D/8)).
    // With s < D/16 the XOR with s touches bits the half term leaves free, so
    // step s is at k_ro0 ^ (s << 4).
    const uint32_t k_ro0 = l32 * C::kRowBytes + (((half * (C::kNch / 2)) ^ (l32 & (C::kNch - 1))) << 4);
    // V^T via transpose reads: 16-lane group gq, lane m in it; rows 16*sp + 8*qh + 4*half + m/4,
    // dims 32*md + 16*(gq%2) + 4*(m%4) .. +3: chunk c = 4 md + c0 stored at
    // c ^ (2 (row % (D/16))); md sits above c0 and the XOR is bitwise, so row
    // block md is at v_ro0 ^ (md << 6).
    const int gq = lane >> 4, m16 = lane & 15;
    const int v_r = 4 * half + (m16 >> 2);  // row within an 8-row group (the swizzle depends on it only)
    const uint32_t v_ro0 = v_r * C::kRowBytes +
                           (((2 * (gq & 1) + ((m16 & 3) >> 1)) ^ C::vswz(v_r)) << 4) + (m16 & 1) * 8;
    // Stage and sub-tile bases are multiples of 1 KB, above every bit these
    // XORs touch: (base + off0) ^ x == base + (off0 ^ x).
    typedef __attribute__((address_space(3))) const bf16x8_t lds_bf16x8_t;
    auto k_frag = [](uint32_t kb0, int s) { return *(lds_bf16x8_t*)(uintptr_t)(kb0 ^ (uint32_t)(s << 4)); };
    auto v_half = [](uint32_t vb0, int md, int row_off) {
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4_t*)(uintptr_t)((vb0 ^ (uint32_t)(md << 6)) + (uint32_t)row_off * C::kRowBytes));
    };

    f32x16_t oacc[kNB][C::kMd];
    // O is zeroed after the first sub-tile's probabilities (zero_o): before
    // it the registers hold Q and two score tiles only
    auto zero_o = [&]() {
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
            for (int i = 0; i < C::kMd; ++i) {
                oacc[nb][i] = f32x16_t{};
                asm volatile("" : "+v"(oacc[nb][i]));
            }
    };
    float m_run[kNB], l_run[kNB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
        m_run[nb] = -1.0e30f;
        l_run[nb] = 0.0f;
    }
    const float cl2 = a.cl2;
    float mcl[kNB];  // m_run * cl2, formed when m_run changes
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) mcl[nb] = m_run[nb] * cl2;

    // Sub-tile u is half u%2 of the 64-key tile u/2 in ring stage (u/2) % kStages.
    const uint32_t smem_lds = lds_addr(smem);
    // offset of sub-tile u's K rows from the K base (its V rows: the same from the V base)
    auto sub_off = [](uint32_t u) constexpr -> uint32_t {
        return ((u >> 1) & (kStages - 1)) * C::kTileBytes + (u & 1) * 32 * C::kRowBytes;
    };
    auto stage_of = [&](int u) { return smem_lds + sub_off((uint32_t)u); };
    // per-lane read addresses of every K step and V row block at sub-tile
    // offset 0: in the unrolled key loop the sub-tile offset is a constant
    // and becomes the LDS instruction's immediate offset (below 64 KB: the K
    // tiles of all stages, and separately the V tiles, fit in 64 KB)
    uint32_t kro[C::kKs], vro[C::kMd];
#pragma unroll
    for (int s = 0; s < C::kKs; ++s) {
        kro[s] = smem_lds + (k_ro0 ^ (uint32_t)(s << 4));
        asm volatile("" : "+v"(kro[s]));
    }
#pragma unroll
    for (int md = 0; md < C::kMd; ++md) {
        vro[md] = smem_lds + C::kVBase + (v_ro0 ^ (uint32_t)(md << 6));
        asm volatile("" : "+v"(vro[md]));
    }
    // K fragments of sub-tile u (A operand of S^T, k-step s)
    auto read_k = [&](int u, bf16x8_t (&kf)[C::kKs]) {
        const uint32_t kb0 = stage_of(u) + k_ro0;
#pragma unroll
        for (int s = 0; s < C::kKs; ++s) kf[s] = k_frag(kb0, s);
    };
    // V^T fragments of sub-tile u (A operand of O^T, k-step sp, row block md)
    auto read_v = [&](int u, bf16x8_t (&vf)[2][C::kMd]) {
        const uint32_t vb0 = stage_of(u) + C::kVBase + v_ro0;
#pragma unroll
        for (int sp = 0; sp < 2; ++sp)
#pragma unroll
            for (int md = 0; md < C::kMd; ++md) {
                const u32x2_t wl = __builtin_bit_cast(u32x2_t, v_half(vb0, md, 16 * sp));
                const u32x2_t wh = __builtin_bit_cast(u32x2_t, v_half(vb0, md, 16 * sp + 8));
                vf[sp][md] = __builtin_bit_cast(bf16x8_t, u32x4_t{wl[0], wl[1], wh[0], wh[1]});
            }
    };
    // S^T for both column blocks (one K fragment feeds both)
    auto s_mfma = [&](const bf16x8_t (&kf)[C::kKs], f32x16_t (&sacc)[kNB]) {
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) sacc[nb] = f32x16_t{};
#pragma unroll
        for (int s = 0; s < C::kKs; ++s)
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb)
                sacc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s], qf[nb][s], sacc[nb], 0, 0, 0);
    };
    // O^T += V^T P^T
    auto pv_mfma = [&](const bf16x8_t (&vf)[2][C::kMd], const bf16x8_t (&pb)[kNB][2]) {
#pragma unroll
        for (int sp = 0; sp < 2; ++sp)
#pragma unroll
            for (int md = 0; md < C::kMd; ++md)
#pragma unroll
                for (int nb = 0; nb < kNB; ++nb)
                    oacc[nb][md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[sp][md], pb[nb][sp], oacc[nb][md], 0, 0, 0);
    };
    // mask keys past a column's position or past the chunk (boundary sub-tiles only)
    auto mask = [&](int u, f32x16_t (&sacc)[kNB]) {
        const int32_t k0 = kbeg + 32 * u;
        if (k0 + 31 > pmin || k0 + 32 > kend) {
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb) {
                // key k0 + 4*half + o is kept iff o <= lim
                const int32_t lim = min(p_l[nb], kend - 1) - k0 - 4 * half;
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (8 * (v >> 2) + (v & 3) > lim) sacc[nb][v] = -INFINITY;
                // applied here: left to the compiler the selects sink to the
                // next sub-tile's reads and hold 32 lane masks in scalar
                // registers meanwhile
                asm volatile("" : "+v"(sacc[nb]));
            }
        }
    };
    // probabilities as bf16 MFMA operands (k index 8h+e of step sp is key
    // 16sp + 8(e/4) + 4h + e%4 of the sub-tile, the keys whose S^T values this
    // lane holds) and the lane's sums of them
    auto exp_pack = [&](const f32x16_t (&sacc)[kNB], bf16x8_t (&pb)[kNB][2], float (&ts)[kNB]) {
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) {
            const float mc = mcl[nb];
            ts[nb] = 0.0f;
#pragma unroll
            for (int sp = 0; sp < 2; ++sp) {
                f32x8_t pv;
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = __builtin_amdgcn_exp2f(fmaf(sacc[nb][8 * sp + e], cl2, -mc));
                pb[nb][sp] = __builtin_convertvector(pv, bf16x8_t);
                const u32x4_t w = __builtin_bit_cast(u32x4_t, pb[nb][sp]);
#pragma unroll
                for (int e = 0; e < 4; ++e) ts[nb] = sum_pair(w[e], ts[nb]);
            }
        }
    };
    // accept the sub-tile's probabilities, or (rare) move the reference to
    // the sub-tile's maximum, rescale O and l, and form them again
    auto settle = [&](const f32x16_t (&sacc)[kNB], bf16x8_t (&pb)[kNB][2], float (&ts)[kNB], bool o_live) {
        bool over = false;
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) over = over || !(ts[nb] <= kSumLimit);
        if (__any(over)) {
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb) {
                float mx = sacc[nb][0];
#pragma unroll
                for (int v = 1; v < 16; ++v) mx = fmaxf(mx, sacc[nb][v]);
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const float m_new = fmaxf(m_run[nb], mx);
                const float alpha = __builtin_amdgcn_exp2f((m_run[nb] - m_new) * cl2);
                m_run[nb] = m_new;
                mcl[nb] = m_new * cl2;
                if (o_live) {
                    l_run[nb] *= alpha;
#pragma unroll
                    for (int i = 0; i < C::kMd; ++i) {
                        // one accumulator at a time: bounded register staging
                        __builtin_amdgcn_sched_barrier(0);
                        oacc[nb][i] *= alpha;
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            exp_pack(sacc, pb, ts);
        }
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) l_run[nb] += ts[nb];
    };

    const int n_sub = (kend - kbeg + 31) / 32;
    const int n_kt = (n_sub + 1) / 2;
    issue(0);
    // The waits for the Q loads (placed by the compiler, which does not see
    // the direct loads) also cover tile 0, needed next anyway; tiles 1 and 2
    // are issued after them so that those waits do not cover them too.
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int s = 0; s < C::kKs; ++s) {
            const u32x4_t w = p_l[nb] >= 0 ? qv[nb][s] : u32x4_t{0u, 0u, 0u, 0u};
            qf[nb][s] = __builtin_bit_cast(bf16x8_t, w);
        }
    if (n_kt > 1) issue(1);
    if (n_kt > 2) issue(2);
    if (n_kt > 2) wait_vmcnt<2 * C::kLoads>();
    else if (n_kt > 1) wait_vmcnt<C::kLoads>();
    else wait_vmcnt<0>();
    ring_barrier();

    f32x16_t sA[kNB], sB[kNB];       // scores of even / odd sub-tiles
    bf16x8_t pA[kNB][2], pB[kNB][2];  // probabilities of even / odd sub-tiles
    float ts[kNB];
    {
        bf16x8_t kf[C::kKs];
        read_k(0, kf);
        s_mfma(kf, sA);  // Q still in vector registers here
        mask(0, sA);
    }
    // Q stays in the registers it was loaded into for the whole segment
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int s = 0; s < C::kKs; ++s) asm volatile("" : "+v"(qf[nb][s]));
    // Sub-tile u with a successor: S(u+1) and PV(u-1) on the matrix cores
    // while the probabilities of u are formed.  An odd u first opens tile
    // (u+1)/2 (its loads done, the stage of tile (u+1)/2 - 2 free again).
    // U8c: std::integral_constant with u % 8, or -1 where u % 8 is known only at run time
    auto body = [&](auto U8c, int u, f32x16_t (&cur)[kNB], f32x16_t (&nxt)[kNB], bf16x8_t (&pc)[kNB][2],
                    const bf16x8_t (&pp)[kNB][2], bool has_prev, bool opens) {
        constexpr int U8 = decltype(U8c)::value;
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
            // Steady state as a software pipeline of 2*kNB*kKs slots.  Slot k
            // issues one MFMA, fenced off on its own: within the 2*kNB slots
            // of k-step j, the first kNB are S^T step j of the wave's column
            // blocks, the other kNB PV step j.  A fenced group of VALU work
            // follows it: the scaled scores of this slot's values, the
            // exponentials of the previous slot's, a bf16 pair conversion and
            // a row-sum update further behind, and the LDS requests for step
            // j + 2.  The strict alternation keeps the matrix pipe fed while
            // the softmax arithmetic runs in its shadow, and no operation
            // waits on its immediate predecessor.
            constexpr int kPer = 2 * kNB;              // slots per k-step
            constexpr int kSlots = kPer * C::kKs;
            constexpr int kVals = 16 * kNB;            // probabilities per lane per sub-tile
            constexpr int kV = kVals / kSlots;         // formed per slot (1 or 2)
            constexpr int kPairs = kVals / 2;
            constexpr int kRdV0 = kNB == 1 ? 0 : 1;    // slots of the step that request V
            constexpr int kRdV1 = kNB == 1 ? 1 : 2;
            auto cvt_slot = [](int q) { return (2 * q + 1) / kV + 2; };
            // with the ring position a constant, each read is a fixed
            // per-lane address plus an immediate offset; otherwise the
            // sub-tile's base is combined with the lane's offset per read
            constexpr uint32_t ko = sub_off((uint32_t)(U8 + 1) & 7u), vo = sub_off((uint32_t)(U8 + 7) & 7u);
            const uint32_t kb0 = stage_of(u + 1) + k_ro0;
            const uint32_t vb0 = stage_of(u - 1) + C::kVBase + v_ro0;
            auto rk = [&](int j) {
                if constexpr (U8 >= 0) return *(lds_bf16x8_t*)(uintptr_t)(kro[j] + ko);
                else return k_frag(kb0, j);
            };
            auto rv = [&](int j, int hi) {
                if constexpr (U8 >= 0) {
                    const uint32_t at = vro[j % C::kMd] + vo + (uint32_t)(16 * (j / C::kMd) + 8 * hi) * C::kRowBytes;
                    return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(uintptr_t)at));
                } else {
                    return __builtin_bit_cast(u32x2_t, v_half(vb0, j % C::kMd, 16 * (j / C::kMd) + 8 * hi));
                }
            };
            float mc[kNB];
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb) mc[nb] = mcl[nb];
            float fv[kVals], ev[kVals];
            uint32_t pw[kPairs];
            bf16x8_t kf[C::kKs];
            u32x2_t vl[C::kKs], vh[C::kKs];
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb) nxt[nb] = f32x16_t{};
#pragma unroll
            for (int j = 0; j < 2 && j < C::kKs; ++j) {
                kf[j] = rk(j);
                vl[j] = rv(j, 0);
                vh[j] = rv(j, 1);
            }
#pragma unroll
            for (int k = 0; k < kSlots; ++k) {
                const int j = k / kPer, kind = k % kPer;
                if (kind < kNB) {
                    nxt[kind] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[j], qf[kind][j], nxt[kind], 0, 0, 0);
                } else {
                    const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, u32x4_t{vl[j][0], vl[j][1], vh[j][0], vh[j][1]});
                    f32x16_t& o = oacc[kind - kNB][j % C::kMd];
                    o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pp[kind - kNB][j / C::kMd], o, 0, 0, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
                if (j + 2 < C::kKs) {
                    if (kind == 0) kf[j + 2] = rk(j + 2);
                    if (kind == kRdV0) vl[j + 2] = rv(j + 2, 0);
                    if (kind == kRdV1) vh[j + 2] = rv(j + 2, 1);
                }
#pragma unroll
                for (int v = 0; v < kV; ++v) {
                    const int f = k * kV + v;  // value f: column block f/16, S^T register f%16
                    fv[f] = fmaf(cur[f >> 4][f & 15], cl2, -mc[f >> 4]);
                    if (k > 0) ev[f - kV] = __builtin_amdgcn_exp2f(fv[f - kV]);
                }
#pragma unroll
                for (int q = 0; q < kPairs; ++q) {
                    if (cvt_slot(q) == k)
                        pw[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{ev[2 * q], ev[2 * q + 1]}, bf16x2_t));
                    // the first pair of a column block starts its sum
                    if (cvt_slot(q) + 1 == k) ts[q >> 3] = sum_pair(pw[q], (q & 7) ? ts[q >> 3] : 0.0f);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            // drain: the last slot's exponentials, conversions and sums
#pragma unroll
            for (int f = (kSlots - 1) * kV; f < kVals; ++f) ev[f] = __builtin_amdgcn_exp2f(fv[f]);
#pragma unroll
            for (int q = 0; q < kPairs; ++q)
                if (cvt_slot(q) >= kSlots)
                    pw[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{ev[2 * q], ev[2 * q + 1]}, bf16x2_t));
#pragma unroll
            for (int q = 0; q < kPairs; ++q)
                if (cvt_slot(q) + 1 >= kSlots) ts[q >> 3] = sum_pair(pw[q], (q & 7) ? ts[q >> 3] : 0.0f);
            // word q = (nb, sp, w) with q = 8 nb + 4 sp + w
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
                for (int sp = 0; sp < 2; ++sp)
                    pc[nb][sp] = __builtin_bit_cast(bf16x8_t, u32x4_t{pw[8 * nb + 4 * sp], pw[8 * nb + 4 * sp + 1],
                                                                      pw[8 * nb + 4 * sp + 2], pw[8 * nb + 4 * sp + 3]});
        }
        settle(cur, pc, ts, has_prev);
        mask(u + 1, nxt);
    };
    // The last sub-tile u: PV(u-1) while its probabilities are formed, then PV(u).
    auto last = [&](int u, f32x16_t (&cur)[kNB], bf16x8_t (&pc)[kNB][2], const bf16x8_t (&pp)[kNB][2],
                    bool has_prev) {
        bf16x8_t vf[2][C::kMd];
        if (has_prev) {
            read_v(u - 1, vf);
            pv_mfma(vf, pp);
        }
        exp_pack(cur, pc, ts);
        settle(cur, pc, ts, has_prev);
        read_v(u, vf);
        pv_mfma(vf, pc);
    };
    if (n_sub == 1) {
        zero_o();
        last(0, sA, pA, pB, false);
    } else {
        using std::integral_constant;
        body(integral_constant<int, -1>{}, 0, sA, sB, pA, pB, false, false);
        zero_o();
        int u = 1;
        // eight sub-tiles per iteration, u = 1 mod 8 at its start: every
        // sub-tile's ring position is a constant
        for (; u + 8 < n_sub; u += 8) {
            body(integral_constant<int, 1>{}, u, sB, sA, pB, pA, true, true);
            body(integral_constant<int, 2>{}, u + 1, sA, sB, pA, pB, true, false);
            body(integral_constant<int, 3>{}, u + 2, sB, sA, pB, pA, true, true);
            body(integral_constant<int, 4>{}, u + 3, sA, sB, pA, pB, true, false);
            body(integral_constant<int, 5>{}, u + 4, sB, sA, pB, pA, true, true);
            body(integral_constant<int, 6>{}, u + 5, sA, sB, pA, pB, true, false);
            body(integral_constant<int, 7>{}, u + 6, sB, sA, pB, pA, true, true);
            body(integral_constant<int, 0>{}, u + 7, sA, sB, pA, pB, true, false);
        }
        for (; u + 2 < n_sub; u += 2) {
            body(integral_constant<int, -1>{}, u, sB, sA, pB, pA, true, true);
            body(integral_constant<int, -1>{}, u + 1, sA, sB, pA, pB, true, false);
        }
        if (u + 1 < n_sub) {  // u = n_sub - 2
            body(integral_constant<int, -1>{}, u, sB, sA, pB, pA, true, true);
            ++u;
        } else {  // u = n_sub - 1: its scores and the previous probabilities move to where the other path has them
#pragma unroll
            for (int nb = 0; nb < kNB; ++nb) {
                sA[nb] = sB[nb];
#pragma unroll
                for (int sp = 0; sp < 2; ++sp) pB[nb][sp] = pA[nb][sp];
            }
        }
        // one call site for the last sub-tile: the register assignment of
        // the two paths above then agrees where they meet
        last(u, sA, pA, pB, true);
    }

    // ---- results: oacc[nb][i][4r + e] = O[col][d = 32i + 8r + 4half + e]
    float l_tot[kNB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) l_tot[nb] = l_run[nb] + __shfl_xor(l_run[nb], 32);
    // the columns' rows and heads, recomputed rather than held through the loop
    int ln = (int)threadIdx.x & 63;
    asm volatile("" : "+v"(ln));
    auto col_of = [&](int nb) { return 32 * (kNB * wave + nb) + (ln & 31); };
    auto store_out = [&](int nb, const f32x16_t (&o)[C::kMd], float inv) {
        const int c = col_of(nb);
        uint16_t* op =
            a.out + ((((int64_t)tile << a.lgR) + (c & (a.R - 1))) * a.Hq + g * a.G + (c >> a.lgR)) * (int64_t)D;
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
    if (slot < 0) {
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb)
            if (p_l[nb] >= 0) store_out(nb, oacc[nb], 1.0f / l_tot[nb]);
        return;
    }

    // piece of a cut row tile: publish its (m, l) and O / l in register order
    const int64_t sl = (int64_t)g * a.max_slots + slot;
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
        u32x2_t* po = a.part_o + (sl * 8 + kNB * wave + nb) * (C::kMd * 4 * 64) + lane;
        const float inv = l_tot[nb] > 0.0f ? 1.0f / l_tot[nb] : 0.0f;  // l = 0: no key of this piece
#pragma unroll
        for (int i = 0; i < C::kMd; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                po[(i * 4 + r) * 64] = u32x2_t{pack_bf16x2(oacc[nb][i][4 * r] * inv, oacc[nb][i][4 * r + 1] * inv),
                                               pack_bf16x2(oacc[nb][i][4 * r + 2] * inv, oacc[nb][i][4 * r + 3] * inv)};
        if (half == 0) a.part_ml[sl * NCOL + col_of(nb)] = make_float2(m_run[nb], l_tot[nb]);
    }
}

// Plan entries are read as constant memory (the plan kernel wrote them before
// this launch and nothing here writes them), so they come in by scalar loads.
__device__ __forceinline__ int32_t sload(const int32_t* p) {
    return *(const __attribute__((address_space(4))) int32_t*)p;
}

// A plan made for other sizes is not used (it could point past the buffers).
__device__ __forceinline__ bool plan_fits(const AttnArgs& a, const int32_t* hdr) {
    return sload(hdr + 4) == (int32_t)a.n_sel && sload(hdr + 5) == (int32_t)a.n_tok && sload(hdr + 6) == a.Hq &&
           sload(hdr + 7) == a.Hkv && sload(hdr + 8) == a.R;
}

// Workgroup b serves kv head b % Hkv (with 8 kv heads each XCD serves one, so
// its K/V stay in that XCD's L2) and walks range b / Hkv of the plan.
template <int D>
__global__ __launch_bounds__(64 * kNW, 1) void attention_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[ACfg<D>::kLds];
    const int b = blockIdx.x;
    const int g = b % a.Hkv;
    const int jw = b / a.Hkv;
    const int32_t* hdr = a.plan;
    if (!plan_fits(a, hdr) || jw >= sload(hdr + 1)) return;
    const int32_t* rg = hdr + kPlanHdr + 4 * jw;
    int32_t unit = sload(rg);
    const int32_t hi = sload(rg + 1);
    int t = sload(rg + 2);
    int32_t piece = sload(rg + 3);
    const int32_t* til = hdr + kPlanHdr + 4 * a.P;
    for (; t < a.n_tiles; ++t, piece = 0) {
        const int32_t* e = til + 8 * t;
        const int32_t s0 = sload(e), s1 = sload(e + 1);
        if (s1 <= s0) continue;  // no row of the tile has a valid position
        const int32_t seg_lo = max(unit, s0), seg_hi = min(hi, s1);
        if (seg_hi <= seg_lo) break;  // the range ends before the tile's units
        const int32_t pmin = sload(e + 2), pmax = sload(e + 3), pbase = sload(e + 4), npc = sload(e + 5);
        // the arguments and the head through opaque copies: what the segment
        // derives from them is formed inside it, not held in scalar registers
        // through the loop
        auto kp = __builtin_amdgcn_kernarg_segment_ptr();
        int gs = g;
        asm volatile("" : "+s"(kp), "+s"(gs));
        segment<D>(*(const AttnArgs*)kp, smem, gs, t, (seg_lo - s0) * KT, min((seg_hi - s0) * KT, pmax + 1), pmin,
                   npc > 1 ? pbase + piece : -1);
        unit = seg_hi;
        if (unit >= hi) break;
        __syncthreads();  // every wave is done with the ring before the next segment refills it
    }
}

// Log-sum-exp merge of a cut row tile's pieces.  One workgroup per (cut row
// tile, 32-column block, kv head): the 32 columns x D values of block cb
// (attention wave cb held them), laid out as [i][r][lane] f32x4 per piece,
// so every load is a coalesced 1 KB row.  Thread t handles lane
// t % 64 and the (i, r) pairs t / 64 + 4k.  Head g runs on the XCD that
// wrote its pieces (b % 8 == g with 8 kv heads).  Pieces are read kPc at a
// time, all their loads in flight together, and merged into a running
// (max, sum, O) (one group in the common case of at most kPc pieces).
template <int D>
__device__ __forceinline__ void combine_item(const AttnArgs& a, const int32_t* hdr, int item) {
    constexpr int kMd = D / 32;
    constexpr int kPer = kMd;  // (i, r) pairs per thread: 4 * kMd / 4
    constexpr int kPc = 4;
    const int g = item % a.Hkv;
    const int rest = item / a.Hkv;
    const int cb = rest & 7;  // 32-column block of the tile
    const int k = rest >> 3;  // cut row tile
    const int32_t* ent = hdr + kPlanHdr + 4 * a.P + 8 * a.n_tiles + 4 * k;
    const int tile = sload(ent), pbase = sload(ent + 1), nu = sload(ent + 2);
    const int tid = threadIdx.x, lane = tid & 63, q4 = tid >> 6;
    const int half = lane >> 5, l32 = lane & 31;
    const int col = 32 * cb + l32;
    const int64_t row = ((int64_t)tile << a.lgR) + (col & (a.R - 1));
    if (row >= a.n_sel) return;
    const int32_t p = a.pos[row];
    const int head = g * a.G + (col >> a.lgR);
    const float cl2 = a.cl2;
    const int64_t sl0 = (int64_t)g * a.max_slots + pbase;
    const float2* ml = a.part_ml + sl0 * NCOL + col;
    const u32x2_t* po0 = a.part_o + (sl0 * 8 + cb) * (kMd * 4 * 64) + lane;
    constexpr int64_t kPieceStride = 8 * kMd * 4 * 64;  // u32x2 per slot (8 column blocks)
    float M = -1.0e30f, L = 0.0f;
    f32x4_t o[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) o[k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nu; c0 += kPc) {
        float2 mlc[kPc];
        u32x2_t x[kPc][kPer];
#pragma unroll
        for (int c = 0; c < kPc; ++c) {
            mlc[c] = make_float2(-1.0e30f, 0.0f);
            if (c0 + c < nu) {
                mlc[c] = ml[(c0 + c) * NCOL];
#pragma unroll
                for (int k = 0; k < kPer; ++k) x[c][k] = po0[(c0 + c) * kPieceStride + (q4 + 4 * k) * 64];
            }
        }
        float Mn = M;
#pragma unroll
        for (int c = 0; c < kPc; ++c) Mn = fmaxf(Mn, mlc[c].x);
        const float sc = __builtin_amdgcn_exp2f((M - Mn) * cl2);
        M = Mn;
        L *= sc;
#pragma unroll
        for (int k = 0; k < kPer; ++k) o[k] *= sc;
#pragma unroll
        for (int c = 0; c < kPc; ++c) {
            if (c0 + c < nu) {
                const float wl = __builtin_amdgcn_exp2f((mlc[c].x - M) * cl2) * mlc[c].y;  // weight of O_c / l_c
                L += wl;
#pragma unroll
                for (int k = 0; k < kPer; ++k) {
                    // bf16 -> fp32: the 16 bits on top
                    const u32x2_t xx = x[c][k];
                    o[k] += wl * f32x4_t{__builtin_bit_cast(float, xx[0] << 16),
                                         __builtin_bit_cast(float, xx[0] & 0xffff0000u),
                                         __builtin_bit_cast(float, xx[1] << 16),
                                         __builtin_bit_cast(float, xx[1] & 0xffff0000u)};
                }
            }
        }
    }
    if (p < 0 || p >= a.n_tok) return;
    const float inv = 1.0f / L;
    uint16_t* op = a.out + (row * a.Hq + head) * (int64_t)D;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int ir = q4 + 4 * k, i = ir >> 2, r = ir & 3;
        const f32x4_t v = o[k] * inv;
        *reinterpret_cast<u32x2_t*>(op + 32 * i + 8 * r + 4 * half) =
            u32x2_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    }
}

// Items (cut row tile, column block, kv head) in strides of the
// grid, which the launch keeps at a multiple of 8 and far below the item
// bound, so that workgroups are not spent on items a call does not have.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(AttnArgs a) {
    const int32_t* hdr = a.plan;
    if (!plan_fits(a, hdr)) return;
    const int n_items = sload(hdr + 2) * 8 * a.Hkv;
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) combine_item<D>(a, hdr, item);
}

// Inclusive prefix sum over the 1024 threads of a workgroup; *total gets the
// sum of all.  s_w holds 16 wave totals.
__device__ int32_t block_scan(int32_t v, int32_t* s_w, int32_t* total) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int32_t n = __shfl_up(v, o);
        if (lane >= o) v += n;
    }
    if (lane == 63) s_w[w] = v;
    __syncthreads();
    int32_t pre = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int32_t x = s_w[k];
        pre += k < w ? x : 0;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return v + pre;
}

// The plan of a call (one workgroup of 1024 threads; layout at AttnArgs::plan).
// Row tile t with u = pmax/64 + 1 units (0 if no row has a valid position)
// spans [s0 - kSegCost, s1) of the line and its units are [s0, s1); range j
// of P' = min(P, W) is [lo_j, lo_{j+1}) with lo_j = floor(j W / P'), so
// position x lies in range floor(((x + 1) P' - 1) / W), and the ranges
// starting in the span of row tile t are j in
// [ceil((s0 - kSegCost) P' / W), ceil(s1 P' / W)).  A row tile whose units
// ranges cut has one piece per range meeting them, numbered in unit order,
// in slots [slot base, + pieces).  Every step is a parallel pass over the
// row tiles.
__global__ __launch_bounds__(1024) void plan_kernel(AttnArgs a) {
    __shared__ int32_t s_lo[1024], s_hi[1024], s_w[16];
    const int tid = threadIdx.x;
    int32_t* hdr = a.plan;
    int32_t* rng = hdr + kPlanHdr;
    int32_t* til = rng + 4 * a.P;
    int32_t* spl = til + 8 * a.n_tiles;
    // pass 1: each row tile's smallest and largest valid position, its units
    // and their prefix over the row tiles
    int32_t carry = 0;
    for (int32_t base = 0; base < a.n_tiles; base += 1024) {
        s_lo[tid] = INT_MAX;
        s_hi[tid] = -1;
        __syncthreads();
        // each wave's 64 rows are aligned segments of min(R, 64) rows of one
        // row tile: reduced in registers, one LDS update per segment
        const int64_t r0 = (int64_t)base * a.R, r1 = min(a.n_sel, (int64_t)(base + 1024) * a.R);
        const int seg = a.R < 64 ? a.R : 64;
        for (int64_t rb = r0; rb < r1; rb += 1024) {  // the same trip count in every lane
            const int64_t r = rb + tid;
            int32_t lo = INT_MAX, hi = -1;
            if (r < r1) {
                const int32_t p = a.pos[r];
                if (p >= 0 && p < a.n_tok) lo = hi = p;
            }
            for (int o = 1; o < seg; o <<= 1) {
                lo = min(lo, __shfl_xor(lo, o));
                hi = max(hi, __shfl_xor(hi, o));
            }
            if ((tid & (seg - 1)) == 0 && r < r1 && hi >= 0) {
                const int k = (int)(r / a.R - base);
                atomicMin(&s_lo[k], lo);
                atomicMax(&s_hi[k], hi);
            }
        }
        __syncthreads();
        const int32_t t = base + tid;
        const int32_t pmax = s_hi[tid], pmin = s_lo[tid];
        const int32_t units = (t < a.n_tiles && pmax >= 0) ? pmax / KT + 1 : 0;
        const int32_t span = units > 0 ? units + kSegCost : 0;
        int32_t tot;
        const int32_t incl = block_scan(span, s_w, &tot);
        if (t < a.n_tiles) {
            til[8 * t] = carry + incl - units;
            til[8 * t + 1] = carry + incl;
            til[8 * t + 2] = pmax >= 0 ? pmin : -1;
            til[8 * t + 3] = pmax;
        }
        carry += tot;
    }
    const int32_t W = carry;
    const int32_t np = min(a.P, W);
    auto owner = [&](int32_t u) { return (int32_t)(((int64_t)(u + 1) * np - 1) / W); };
    auto first_range = [&](int32_t u) { return (int32_t)(((int64_t)u * np + W - 1) / W); };  // ceil(u P' / W)
    // pass 2: pieces, slot bases, the list of cut row tiles, range starts
    // (each thread reads back only the entries it wrote itself)
    int32_t slots = 0, n_split = 0;
    for (int32_t base = 0; base < a.n_tiles; base += 1024) {
        const int32_t t = base + tid;
        int32_t s0 = 0, s1 = 0, pieces = 0;
        if (t < a.n_tiles) {
            s0 = til[8 * t];
            s1 = til[8 * t + 1];
            if (s1 > s0) pieces = owner(s1 - 1) - owner(s0) + 1;
        }
        const int32_t cut = pieces > 1 ? 1 : 0;
        int32_t tot_slots, tot_cut;
        const int32_t incl_slots = block_scan(cut * pieces, s_w, &tot_slots);
        const int32_t incl_cut = block_scan(cut, s_w, &tot_cut);
        if (t < a.n_tiles) {
            til[8 * t + 4] = slots + incl_slots - cut * pieces;
            til[8 * t + 5] = pieces;
            til[8 * t + 6] = 0;
            til[8 * t + 7] = 0;
            if (cut) {  // the combine reads the three fields at once
                int32_t* e = spl + 4 * (n_split + incl_cut - 1);
                e[0] = t;
                e[1] = slots + incl_slots - cut * pieces;
                e[2] = pieces;
                e[3] = 0;
            }
            if (s1 > s0) {
                const int32_t j1 = first_range(s1);
                for (int32_t j = first_range(s0 - kSegCost); j < j1; ++j) {
                    rng[4 * j] = (int32_t)((int64_t)j * W / np);
                    rng[4 * j + 1] = (int32_t)((int64_t)(j + 1) * W / np);
                    rng[4 * j + 2] = t;
                    rng[4 * j + 3] = max(0, j - owner(s0));
                }
            }
        }
        slots += tot_slots;
        n_split += tot_cut;
    }
    if (tid == 0) {
        hdr[0] = W;
        hdr[1] = np;
        hdr[2] = n_split;
        hdr[3] = slots;
        hdr[4] = (int32_t)a.n_sel;
        hdr[5] = (int32_t)a.n_tok;
        hdr[6] = a.Hq;
        hdr[7] = a.Hkv;
        hdr[8] = a.R;
    }
}

template <int D>
hipError_t launch(const AttnArgs& args, bool make_plan, hipStream_t s) {
    if (make_plan) hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, s, args);
    hipLaunchKernelGGL(attention_kernel<D>, dim3((unsigned)(args.P * args.Hkv)), dim3(64 * kNW), 0, s, args);
    hipLaunchKernelGGL(combine_kernel<D>, dim3((unsigned)std::min(args.P * args.Hkv * 8, 2 * kCUs)), dim3(256), 0, s,
                       args);
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
    p.P = p.max_slots = 0;
    p.off_plan = p.off_part_o = p.off_part_ml = p.total = p.plan_bytes = 0;
    if (dtype == SEMSHARE_BF16 && n_sel > 0) {
        // one range per CU; the cut row tiles hold at most two pieces per
        // range boundary inside them, and at most n_tiles + P pieces in all
        p.P = std::max(1, kCUs / n_kv_heads);
        p.max_slots = (int32_t)std::min<int64_t>(2 * (int64_t)p.P, p.n_tiles + p.P);
        const size_t plan_ints = kPlanHdr + 4 * (size_t)p.P + 8 * (size_t)p.n_tiles + 4 * (size_t)p.P;
        const size_t slots = (size_t)n_kv_heads * p.max_slots;
        p.plan_bytes = plan_ints * sizeof(int32_t);
        p.off_part_o = align256(p.plan_bytes);
        p.off_part_ml = align256(p.off_part_o + slots * NCOL * head_dim * sizeof(uint16_t));
        p.total = align256(p.off_part_ml + slots * NCOL * sizeof(float2));
    }
    return p;
}

namespace {
AttnArgs attn_args(const AttnCall& a, const AttnPlan& p) {
    unsigned char* ws = static_cast<unsigned char*>(a.workspace);
    AttnArgs t{};
    t.q = static_cast<const uint16_t*>(a.q);
    t.pos = a.sel_pos;
    t.k_cache = static_cast<const uint16_t*>(a.k_cache);
    t.v_cache = static_cast<const uint16_t*>(a.v_cache);
    t.out = static_cast<uint16_t*>(a.out);
    t.part_o = reinterpret_cast<u32x2_t*>(ws + p.off_part_o);
    t.part_ml = reinterpret_cast<float2*>(ws + p.off_part_ml);
    t.plan = reinterpret_cast<int32_t*>(ws + p.off_plan);
    t.n_sel = a.n_sel;
    t.n_tok = a.n_tok;
    t.Hq = a.n_q_heads;
    t.Hkv = a.n_kv_heads;
    t.G = a.n_q_heads / a.n_kv_heads;
    t.R = p.rows_per_tile;
    t.lgR = 0;
    while ((1 << (t.lgR + 1)) <= t.R) ++t.lgR;
    t.n_tiles = (int32_t)p.n_tiles;
    t.P = p.P;
    t.max_slots = p.max_slots;
    t.cl2 = a.sm_scale * kLog2e;
    return t;
}
}  // namespace

hipError_t launch_attention_bf16(const AttnCall& a, const AttnPlan& p, hipStream_t s) {
    AttnArgs t = attn_args(a, p);
    const bool make_plan = a.plan == nullptr;
    if (!make_plan) t.plan = static_cast<int32_t*>(const_cast<void*>(a.plan));
    if (a.head_dim == 128) return launch<128>(t, make_plan, s);
    return launch<64>(t, make_plan, s);
}

// ---- the allocation-free attention (semshare_prefill_attention_noalloc)
// Its plan and partial results live in this file-scope device array, one
// copy per GPU, kept until the process ends.  In host code `scratch` names a
// host-side stand-in, never the device memory: every use goes through the
// address hipGetSymbolAddress returns for the current device.
namespace {
__device__ __align__(256) unsigned char scratch[kAttnScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;
}  // namespace

hipError_t attention_scratch(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (!p) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (!p) return hipErrorInvalidSymbol;
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *ptr = p;
    return hipSuccess;
}

hipError_t launch_attention_plan_bf16(const AttnCall& a, const AttnPlan& p, void* plan, hipStream_t s) {
    AttnArgs t = attn_args(a, p);
    t.plan = static_cast<int32_t*>(plan);
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(1024), 0, s, t);
    return hipGetLastError();
}

}  // namespace semshare
