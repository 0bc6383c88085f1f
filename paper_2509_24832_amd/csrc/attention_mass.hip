// Average attention score per token and the dynamic recompute set (Section 3
// Insight 2 and its Attention Recovery equation; Section 4.3.3: hot / cold
// tokens from AR at a 55% threshold, Recomputed = w_c * c + w_h * h).
//
// Mass of token j at a fully computed layer: the causal softmax attention
// P_h[i][j] of every head h, averaged over the heads and over the query rows
// i (rows before j contribute zero).  Two MFMA passes over the causal score
// matrix, bf16 operands and fp32 accumulation, exponentials in base 2:
//   mass_lse_kernel  one wave per (2 query blocks of 32, head): S^T = K Q^T,
//                    so each lane owns a query column and keeps its row's
//                    running max and sum over its 16 keys per block; the
//                    two lane halves merge at the end -> lse2[h][i].
//   mass_col_kernel  one wave per (2 key blocks of 32, head): S = Q K^T, so
//                    each lane owns a key column and sums exp2(s - lse2[i])
//                    over its 16 rows per block -> part[h][j].
//   mass_final_kernel sums the heads in a fixed order and divides by H_q T.
// Each wave keeps the operands of its 2 fixed blocks (queries, resp. keys)
// in VGPRs and streams the other operand from global memory, one 32 x 128
// tile feeding 2 x 8 MFMAs, the next tile's loads in flight meanwhile.
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

__global__ __launch_bounds__(64) void mass_lse_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                       int64_t T, int32_t Hq, int32_t Hkv, float scale_log2e,
                                                       float* __restrict__ lse2) {
    const int lane = threadIdx.x, half = lane >> 5, l32 = lane & 31;
    const int h = blockIdx.y, kvh = h / (Hq / Hkv);
    const int64_t nb = (T + 31) / 32;
    const int64_t qb0 = (int64_t)blockIdx.x * kNB;
    bf16x8_t bq[kNB][8];
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        int64_t qi = (qb0 + b) * 32 + l32;
        if (qi >= T) qi = T - 1;
        const uint16_t* row = q + (qi * Hq + h) * 128 + 8 * half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) bq[b][ks] = ld8(row + 16 * ks);
    }
    float m[kNB], l[kNB];
#pragma unroll
    for (int b = 0; b < kNB; ++b) { m[b] = kNegInf; l[b] = 0.0f; }
    const int64_t kb_end = qb0 + kNB < nb ? qb0 + kNB : nb;
    auto load_k = [&](int64_t kb, bf16x8_t (&ak)[8]) {
        int64_t kj = kb * 32 + l32;
        if (kj >= T) kj = T - 1;
        const uint16_t* krow = k + (kj * Hkv + kvh) * 128 + 8 * half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) ak[ks] = ld8(krow + 16 * ks);
    };
    auto tile = [&](int64_t kb, const bf16x8_t (&ak)[8]) {
#pragma unroll
        for (int b = 0; b < kNB; ++b) {
            if (kb > qb0 + b) continue;  // wave-uniform: the block lies above the diagonal
            f32x16_t acc = {};
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak[ks], bq[b][ks], acc, 0, 0, 0);
            // acc[v] = S^T[key = 32 kb + out_row(v)][query = 32 (qb0 + b) + l32];
            // only the diagonal block has keys after its queries
            // the max is taken on the raw scores (the scale is positive) and
            // the scale folded into one fma per score
            float bm = kNegInf;
            if (kb == qb0 + b) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    if (out_row(v, half) > l32) acc[v] = kNegInf;
                    bm = fmaxf(bm, acc[v]);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) bm = fmaxf(bm, acc[v]);
            }
            const float mn = fmaxf(m[b], bm * scale_log2e);
            if (mn == kNegInf) continue;  // no key of this half seen yet
            float sum = 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) sum += __builtin_amdgcn_exp2f(fmaf(acc[v], scale_log2e, -mn));
            l[b] = l[b] * __builtin_amdgcn_exp2f(m[b] - mn) + sum;
            m[b] = mn;
        }
    };
    // the next tile's loads are in flight while the current one is used
    bf16x8_t ka[8], kc[8];
    load_k(0, ka);
    for (int64_t kb = 0; kb < kb_end; kb += 2) {
        if (kb + 1 < kb_end) load_k(kb + 1, kc);
        tile(kb, ka);
        if (kb + 1 >= kb_end) break;
        if (kb + 2 < kb_end) load_k(kb + 2, ka);
        tile(kb + 1, kc);
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

__global__ __launch_bounds__(64) void mass_col_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                                       int64_t T, int64_t row_begin, int32_t Hq, int32_t Hkv,
                                                       float scale_log2e, const float* __restrict__ lse2,
                                                       float* __restrict__ part) {
    const int lane = threadIdx.x, half = lane >> 5, l32 = lane & 31;
    const int h = blockIdx.y, kvh = h / (Hq / Hkv);
    const int64_t nb = (T + 31) / 32;
    const int64_t kb0 = (int64_t)blockIdx.x * kNB;
    bf16x8_t bk[kNB][8];
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        int64_t kj = (kb0 + b) * 32 + l32;
        if (kj >= T) kj = T - 1;
        const uint16_t* row = k + (kj * Hkv + kvh) * 128 + 8 * half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) bk[b][ks] = ld8(row + 16 * ks);
    }
    float col[kNB];
#pragma unroll
    for (int b = 0; b < kNB; ++b) col[b] = 0.0f;
    const float* lse_h = lse2 + (int64_t)h * T;
    auto load_q = [&](int64_t qb, bf16x8_t (&aq)[8], float (&L)[16]) {
        int64_t qi = qb * 32 + l32;
        if (qi >= T) qi = T - 1;
        const uint16_t* qrow = q + (qi * Hq + h) * 128 + 8 * half;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) aq[ks] = ld8(qrow + 16 * ks);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t r = qb * 32 + out_row(v, half);
            L[v] = r < T && r >= row_begin ? lse_h[r] : __builtin_inff();  // rows outside the window add 0
        }
    };
    auto tile = [&](int64_t qb, const bf16x8_t (&aq)[8], const float (&L)[16]) {
#pragma unroll
        for (int b = 0; b < kNB; ++b) {
            if (qb < kb0 + b) continue;  // wave-uniform: every row of the block precedes the keys
            f32x16_t acc = {};
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq[ks], bk[b][ks], acc, 0, 0, 0);
            // acc[v] = S[query = 32 qb + out_row(v)][key = 32 (kb0 + b) + l32];
            // only the diagonal block has rows before its keys; rows past T
            // carry L = inf and add 0
            if (qb == kb0 + b) {
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    col[b] += l32 <= out_row(v, half) ? __builtin_amdgcn_exp2f(acc[v] * scale_log2e - L[v]) : 0.0f;
            } else {
#pragma unroll
                for (int v = 0; v < 16; ++v) col[b] += __builtin_amdgcn_exp2f(acc[v] * scale_log2e - L[v]);
            }
        }
    };
    bf16x8_t qa[8], qc[8];
    float La[16], Lc[16];
    const int64_t qb_first = kb0 > row_begin / 32 ? kb0 : row_begin / 32;
    if (qb_first < nb) load_q(qb_first, qa, La);
    for (int64_t qb = qb_first; qb < nb; qb += 2) {
        if (qb + 1 < nb) load_q(qb + 1, qc, Lc);
        tile(qb, qa, La);
        if (qb + 1 >= nb) break;
        if (qb + 2 < nb) load_q(qb + 2, qa, La);
        tile(qb + 1, qc, Lc);
    }
#pragma unroll
    for (int b = 0; b < kNB; ++b) {
        const float c = col[b] + __shfl_xor(col[b], 32);
        const int64_t key = (kb0 + b) * 32 + l32;
        if (half == 0 && key < T) part[(int64_t)h * T + key] = c;
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
    const dim3 grid((unsigned)((nb + kNB - 1) / kNB), (unsigned)n_q_heads);
    const auto* qp = static_cast<const uint16_t*>(q);
    const auto* kp = static_cast<const uint16_t*>(k);
    // the row normalisers do not depend on row_begin: a window pass after a
    // pass over the same q and K finds them in the workspace
    if (!reuse_normalisers)
        hipLaunchKernelGGL(mass_lse_kernel, grid, dim3(64), 0, s, qp, kp, n_tok, n_q_heads, n_kv_heads, sl2e, lse2);
    hipLaunchKernelGGL(mass_col_kernel, grid, dim3(64), 0, s, qp, kp, n_tok, row_begin, n_q_heads, n_kv_heads, sl2e,
                       lse2, part);
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
