// Internal declarations shared by the HIP kernels and the C ABI layer of
// libsemshare.so.  gfx950 (CDNA4) only: 64-wide wavefronts, MFMA matrix
// cores, 160 KB of LDS per CU, 8 XCDs with one L2 each.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "semshare.h"

namespace semshare {

// ------------------------------------------------------------ bf16 helpers
// bf16 is handled as raw 16-bit patterns; widening is a shift (exact) and
// narrowing rounds to nearest even through the native conversion.

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    __bf16 b = (__bf16)f;
    return __builtin_bit_cast(uint16_t, b);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair (lo in bits 0..15), one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// ------------------------------------------------------------ direct loads into LDS
// Used by the kernels that stream operands through an LDS ring (the QKV GEMM,
// the attention, the LSH encode).

// 16 bytes per lane from gbase + off (bytes, per lane) straight into LDS at
// lds_base + 16 * lane (global_load_lds_dwordx4; M0 = the wave-uniform LDS
// base, scalar base address + 32-bit lane offset).  Inline assembly on
// purpose: the compiler models the builtin form as an LDS access that may
// complete out of order and then waits for every LDS read in flight
// (lgkmcnt(0)) before each MFMA group, or drains the whole ring with
// vmcnt(0) before a transposing LDS read.  Stage readiness is established
// explicitly instead: wait_vmcnt for the wave's own loads, then ring_barrier.
// M0 is written only here.
__device__ __forceinline__ void g2lds(const void* gbase, uint32_t off, uint32_t lds_base) {
    // the scalar operands are wave-uniform by construction; readfirstlane
    // places them in scalar registers (both halves of the address go through
    // uint32_t so the low half is zero-extended, never sign-extended)
    const uint64_t g = reinterpret_cast<uint64_t>(gbase);
    const uint32_t g_hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(g >> 32));
    const uint32_t g_lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)g);
    const uint64_t gs = ((uint64_t)g_hi << 32) | (uint64_t)g_lo;
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(reinterpret_cast<const void*>(gs)), "s"((uint32_t)__builtin_amdgcn_readfirstlane(lds_base))
                 : "memory", "m0");
}

// Byte address of a __shared__ object in the LDS address space.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// s_waitcnt vmcnt(N), the other counters left at their maximum; vmcnt is
// split over bits [3:0] and [15:14] of the immediate.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would wait for every in-flight direct-to-LDS load (vmcnt(0)) and drain the
// ring.  The empty asm statements keep the compiler from moving LDS accesses
// across it.
__device__ __forceinline__ void ring_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// RoPE angle m * theta reduced to [-pi, pi] in fp64 (two-constant
// Cody-Waite reduction).
__device__ __forceinline__ double rope_reduced_angle(double m, double theta) {
    const double a = m * theta;
    const double n = rint(a * 0.15915494309189535);  // 1 / (2 pi)
    double r = fma(-n, 6.283185307179586, a);         // 2 pi, high part
    return fma(-n, 2.4492935982947064e-16, r);        // 2 pi - high part
}

// sin and cos of the RoPE angle m * theta: fp32 sincos of the reduced angle's
// fp32 head, corrected to first order by its fp32 tail (the head alone would
// carry up to 1.2e-7 rad of rounding error).
__device__ __forceinline__ void rope_sincos(double m, double theta, float* s, float* c) {
    const double r = rope_reduced_angle(m, theta);
    const float hi = (float)r;
    const float lo = (float)(r - (double)hi);
    float sh, ch;
    sincosf(hi, &sh, &ch);
    *s = fmaf(ch, lo, sh);
    *c = fmaf(-sh, lo, ch);
}

// ---------------------------------------------------------------- launchers
// Every launcher assumes validated arguments and returns the launch status.

hipError_t launch_rope_embed(const void* x, void* y, int64_t n_tok, int32_t dim, int64_t pos0,
                             double base, int dtype, hipStream_t s);

hipError_t launch_lsh_encode(const void* x, const void* planes, uint64_t* codes, int64_t n_tok,
                             int32_t dim, int32_t n_bits, int dtype, hipStream_t s);

hipError_t launch_rope_lsh_encode(const void* x, const void* planes, uint64_t* codes, int64_t n_tok, int32_t dim,
                                  int32_t n_bits, int64_t pos0, double base, hipStream_t s);

// token count limit of the dynamic recompute selection and first-layer
// retention sorted in one workgroup (keys in LDS); up to kMaxDynTokLarge they
// rank by counting (rank_select.hip)
constexpr int kMaxDynTok = 8192;
constexpr int kMaxDynTokLarge = 65536;
hipError_t launch_dynamic_recompute_large(const float* mass, const float* sigma, int32_t n, double thres,
                                          double w_hot, double w_cold, int32_t* sel_pos, int32_t* counts,
                                          hipStream_t s);
hipError_t launch_retention_large(const float* mass, const float* score, int32_t n, const int32_t* sel_pos,
                                  const int32_t* counts, double min_keep, int32_t* rank, int32_t* kept_pos,
                                  int32_t* n_kept, hipStream_t s);
// token count limit of the per-layer retention (one workgroup, one bit per position in LDS)
constexpr int kMaxRetainTok = 1 << 20;
hipError_t launch_retention_layer(const int32_t* rank, int32_t n_tok, int32_t n_retain, const int32_t* sel_pos,
                                  int32_t n_sel, const int32_t* idx, int32_t* kept_pos, int32_t* src_idx,
                                  int32_t* sel_rows, int32_t* n_kept, hipStream_t s);

size_t attention_mass_workspace(int64_t n_tok, int32_t n_q_heads);
hipError_t launch_attention_mass(const void* q, const void* k, int64_t n_tok, int64_t row_begin, int32_t n_q_heads,
                                 int32_t n_kv_heads, float sm_scale, float* mass, void* workspace, hipStream_t s,
                                 bool reuse_normalisers = false);
hipError_t launch_retention(const float* mass, const float* score, int32_t n_tok, const int32_t* sel_pos,
                            const int32_t* counts, double min_keep, int32_t* rank, int32_t* kept_pos, int32_t* n_kept,
                            hipStream_t s);
hipError_t launch_dynamic_recompute(const float* mass, const float* sigma, int32_t n_tok, double thres, double w_hot,
                                    double w_cold, int32_t* sel_pos, int32_t* counts, hipStream_t s);

hipError_t launch_match(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                        int32_t n_words, int32_t* idx, int32_t* dist, hipStream_t s);

hipError_t launch_match_mfma(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                             int32_t n_words, int32_t* idx, int32_t* dist, hipStream_t s);

hipError_t launch_gather_rows(const void* src_a, const void* src_b, const int32_t* idx,
                              int64_t n_tgt, int64_t n_ref, void* dst_a, void* dst_b,
                              int32_t n_layers, int64_t row_bytes, hipStream_t s,
                              const int32_t* except_pos = nullptr, int64_t n_except = 0);

hipError_t launch_select_recompute(const float* sigma, int64_t n_tok, int64_t n_sel,
                                   int32_t* sel_pos, hipStream_t s, const int32_t* map = nullptr);

size_t bank_similarity_workspace(int64_t n_tgt, int32_t n_prompts);
hipError_t launch_bank_similarity(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                                  const int64_t* offsets, int32_t n_prompts, int32_t n_words, double dmin,
                                  double dmax, int64_t* dist_sum, double* similarity, void* workspace,
                                  hipStream_t s);

// Step 1 of a partial-prefill layer: q/k/v projection, RoPE, deviation and
// the scatter of k/v into the cache.
struct QkvArgs {
    const void* x_sel;
    const int32_t* sel_pos;
    int64_t n_sel;
    const void* wq;
    const void* wk;
    const void* wv;
    void* k_cache;
    void* v_cache;
    int64_t n_tok;
    int32_t hidden, n_q_heads, n_kv_heads, head_dim;
    double rope_base;
    void* q_out;           // [n_sel][Hq][D] or null (K/V only)
    float* deviation_out;  // [n_sel] or null
    void* workspace;       // qkv_workspace_bytes()
    const void* rope_table = nullptr;  // bf16 path: [n_sel][D/2] (cos, sin) made by launch_rope_table, or null
    // bf16 path: the deviation compares with ref_k/ref_v[ref_idx[p]] (rows of
    // a reference cache, [ref_n][Hkv*D]) instead of the cache row p; null:
    // with the cache row
    const void* ref_k = nullptr;
    const void* ref_v = nullptr;
    const int32_t* ref_idx = nullptr;
    int64_t ref_n = 0;
    // bf16 path: input row i is row x_rows[i] of x_sel ([n_x][hidden],
    // entries clamped to [0, n_x)); null: row i of x_sel
    const int32_t* x_rows = nullptr;
    int64_t n_x = 0;
};

// Step 2: causal GQA attention of the selected rows over the cache.
struct AttnCall {
    const void* q;
    const int32_t* sel_pos;
    int64_t n_sel;
    const void* k_cache;
    const void* v_cache;
    int64_t n_tok;
    int32_t n_q_heads, n_kv_heads, head_dim;
    float sm_scale;
    void* out;
    void* workspace;  // plan_attention().total bytes
    const void* plan;  // a plan made by launch_attention_plan_bf16, or null: plan into the workspace
};

// Work decomposition and workspace partition of the attention step.
struct AttnPlan {
    int32_t rows_per_tile;  // selected rows per tile (256 / G for bf16)
    int64_t n_tiles;
    int32_t P;              // workgroups (ranges of the stream-K line) per kv head
    int32_t max_slots;      // partial-result slots per kv head
    size_t off_plan, off_part_o, off_part_ml, total;
    size_t plan_bytes;      // the plan alone (at off_plan)
};

size_t qkv_workspace_bytes(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int dtype);
size_t qkv_workspace_dev_offset(int64_t n_sel, int32_t head_dim, int dtype);
int32_t qkv_dev_parts(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int dtype);

// The bf16 projection GEMM (qkv_gemm.hip).
struct GemmArgs {
    const uint16_t* x;     // [n_sel][hidden], or [n_x][hidden] read through x_rows
    const int32_t* x_rows; // [n_sel] rows of x (clamped to [0, n_x)), or null: row i
    int64_t n_x;
    const int32_t* pos;    // [n_sel]
    const uint16_t* w[3];  // Wq, Wk, Wv (rows = output features)
    int32_t seg_tiles[3];  // BN-wide column tiles per segment (0 for q in K/V-only mode)
    int32_t seg_cols[3];   // output columns per segment
    int32_t n_nt, n_mt;
    int64_t n_sel, n_tok;
    int32_t hidden, D;
    uint16_t* q_out;       // [n_sel][Hq*D]
    uint16_t* kv[2];       // k_cache, v_cache [n_tok][Hkv*D]
    const float2* rope;    // [n_sel][D/2] (cos, sin)
    float* dev_parts;      // [n_sel][2][Hkv*D/BN] squared-difference sums, or null
    const uint16_t* dev_src[2];  // rows the deviation compares with: reference K, V [dev_n][Hkv*D], or null (the cache)
    const int32_t* dev_idx;      // position p -> row dev_idx[p] of dev_src (outside [0, dev_n): a zero row)
    int64_t dev_n;
};
int32_t qkv_gemm_bn(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim);
hipError_t launch_qkv_gemm(const GemmArgs& g, int32_t bn, hipStream_t s);
AttnPlan plan_attention(int64_t n_sel, int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                        int32_t head_dim, int dtype);

hipError_t launch_qkv_bf16(const QkvArgs& a, hipStream_t s);
// The RoPE (cos, sin) table of the bf16 projection, [n_sel][head_dim/2] float2.
hipError_t launch_rope_table(const int32_t* sel_pos, int64_t n_sel, int64_t n_tok, int32_t head_dim,
                             double rope_base, void* table, hipStream_t s);
hipError_t launch_qkv_f32(const QkvArgs& a, hipStream_t s);
hipError_t launch_attention_bf16(const AttnCall& a, const AttnPlan& p, hipStream_t s);
// The plan alone, into `plan` (AttnPlan::plan_bytes bytes).
hipError_t launch_attention_plan_bf16(const AttnCall& a, const AttnPlan& p, void* plan, hipStream_t s);
hipError_t launch_attention_f32(const AttnCall& a, const AttnPlan& p, hipStream_t s);

// Size of the static device array that holds the plan and partial results of
// semshare_prefill_attention_noalloc (plan_attention().total must fit), and
// its address on the current device (looked up once per device).
constexpr size_t kAttnScratchBytes = size_t(40) << 20;
hipError_t attention_scratch(void** ptr);

}  // namespace semshare
