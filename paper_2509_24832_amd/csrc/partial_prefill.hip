// One attention layer of partial prefill (Sections 4.2, 4.3.3; KV deviation
// of Appendix A.4), bf16 storage with fp32 accumulation.
//
// Kernels, in stream order:
//  1. prep        RoPE (cos, sin) table for the selected positions, one entry
//                 per (row, pair) shared by all heads and by q and k; zeroes
//                 the deviation sums.
//  2. qkv_gemm    projection + RoPE + deviation + cache scatter (qkv_gemm.hip).
//  3. dev_final   sigma = sqrt(sum dK^2) + sqrt(sum dV^2).
//  4. attention   flash-style causal GQA attention of the selected rows over
//                 the assembled cache.  A workgroup owns one kv head and 128
//                 query columns (128/G selected rows x G heads); S^T = K Q^T
//                 and O^T = V^T P^T on MFMA, so every lane holds one query
//                 column and the softmax row statistics need a single
//                 cross-lane exchange.  K and V^T tiles of 64 keys are staged
//                 in LDS (V transposed on the way in).  Long key ranges are
//                 split into chunks (split-KV) when there are too few tiles
//                 to fill the chip.
//  5. combine     log-sum-exp merge of the split-KV partial results.
#include <climits>

#include "semshare_internal.h"

namespace semshare {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// ------------------------------------------------------------------ prep

__global__ void prep_kernel(const int32_t* __restrict__ pos, int64_t n_sel, int64_t n_tok,
                            int32_t half_d, double log2_base, float2* __restrict__ rope) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_sel * half_d) {
        const int64_t m = i / half_d;
        const int32_t k = (int32_t)(i - m * half_d);
        int32_t p = pos[m];
        if (p < 0 || p >= n_tok) p = 0;
        const double theta = exp2(-(2.0 * (double)k / (double)(2 * half_d)) * log2_base);
        float s, c;
        rope_sincos((double)p, theta, &s, &c);
        rope[i] = make_float2(c, s);
    }
}

// sigma = sqrt(sum dK^2) + sqrt(sum dV^2) from per-tile partial sums
// parts[(m * 2 + t) * n_parts + j], summed in a fixed order (deterministic).
__global__ void dev_final_kernel(const float* __restrict__ parts, float* __restrict__ dev, int64_t n_sel,
                                 int32_t n_parts) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_sel) return;
    float sk = 0.0f, sv = 0.0f;
    for (int32_t j = 0; j < n_parts; ++j) {
        sk += parts[(2 * i) * n_parts + j];
        sv += parts[(2 * i + 1) * n_parts + j];
    }
    dev[i] = sqrtf(sk) + sqrtf(sv);
}

// ------------------------------------------------------------------ attention

constexpr int KT = 64;  // keys per LDS tile

struct AttnArgs {
    const uint16_t* q;        // [n_sel][Hq][D]
    const int32_t* pos;       // [n_sel]
    const uint16_t* k_cache;  // [n_tok][Hkv][D]
    const uint16_t* v_cache;
    uint16_t* out;            // [n_sel][Hq][D]
    float* part_o;            // [items][128][D]
    float* part_ml;           // [items][128][2]
    int32_t* n_used;          // [n_tiles * Hkv]
    int64_t n_sel, n_tok;
    int32_t Hq, Hkv, G, R;
    int32_t n_tiles, chunk, n_chunks;
    float cl2;                // sm_scale * log2(e)
};

template <int D>
struct AttnLds {
    static constexpr int KLD = D + 8;   // bf16 per K row  (D=128: 272 B)
    static constexpr int VLD = KT + 4;  // bf16 per V^T row (136 B)
    static constexpr int kBytes = 2 * KT * KLD * 2;
    static constexpr int vBytes = 2 * D * VLD * 2;
    static constexpr int kChunksPerKey = D / 8;              // 16-B chunks per key row
    static constexpr int kKLoads = KT * kChunksPerKey / 256;  // K u32x4_t loads per thread
    static constexpr int kVItems = 16 * (D / 8);              // (key quad, d group) items
};

typedef float f32x8_t __attribute__((ext_vector_type(8)));

// Running-max slack of the online softmax, in log2 units: the output
// accumulators are rescaled only when a column's maximum grows by more than
// this, so probabilities stay <= 2^8 (exact enough in bf16 and fp32) and the
// 64-register rescale is skipped on almost every tile.
constexpr float kRescaleSlack = 8.0f;

template <int D>
__global__ __launch_bounds__(256, 2) void attention_kernel(AttnArgs a) {
    using L = AttnLds<D>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[L::kBytes + L::vBytes];
    __shared__ int32_t s_pos[128];
    __shared__ int32_t s_pmin, s_pmax;
    uint16_t* Ks = reinterpret_cast<uint16_t*>(smem);
    uint16_t* Vt = reinterpret_cast<uint16_t*>(smem + L::kBytes);

    const int b = blockIdx.x;
    const int g = b % a.Hkv;  // kv head: with 8 kv heads, one per XCD (its K/V stay in that L2)
    const int jj = b / a.Hkv;
    const int tile = a.n_tiles - 1 - jj / a.n_chunks;  // longest (latest) tiles first
    const int chunk_id = jj % a.n_chunks;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, l32 = lane & 31;
    const int col = 32 * wave + l32;
    const int row_local = col % a.R, head_local = col / a.R;
    const int64_t row = (int64_t)tile * a.R + row_local;
    const int head = g * a.G + head_local;

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
    const int32_t pmin = s_pmin, pmax = s_pmax;
    const int32_t p_l = s_pos[row_local];
    if (chunk_id == 0 && tid == 0 && a.n_chunks > 1)
        a.n_used[tile * a.Hkv + g] = pmax < 0 ? 0 : pmax / a.chunk + 1;
    const int32_t kbeg = chunk_id * a.chunk;
    const int32_t kend = min(kbeg + a.chunk, pmax + 1);
    if (kbeg >= kend) return;

    // Q^T operand: lane half h holds d in [h*D/2, h*D/2 + D/2)
    bf16x8_t qf[D / 16];
    {
        const u32x4_t* qp = reinterpret_cast<const u32x4_t*>(a.q + ((p_l >= 0 ? row : 0) * a.Hq + head) * (int64_t)D +
                                                             half * (D / 2));
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
            const u32x4_t w = p_l >= 0 ? qp[s] : u32x4_t{0u, 0u, 0u, 0u};
            qf[s] = __builtin_bit_cast(bf16x8_t, w);
        }
    }

    // Per-thread global offsets (elements) of its K/V tile loads, relative to
    // the tile's first key; consecutive keys are row_stride elements apart.
    const int32_t row_stride = a.Hkv * D;
    const uint16_t* kbase = a.k_cache + (int64_t)g * D;
    const uint16_t* vbase = a.v_cache + (int64_t)g * D;
    const int32_t last_key = (int32_t)a.n_tok - 1;
    int32_t k_key[L::kKLoads], k_off[L::kKLoads];
#pragma unroll
    for (int i = 0; i < L::kKLoads; ++i) {
        const int item = i * 256 + tid;
        k_key[i] = item / L::kChunksPerKey;
        k_off[i] = k_key[i] * row_stride + (item % L::kChunksPerKey) * 8;
    }
    // V: thread -> (key quad kq = tid % 16, d group dg = tid / 16): the
    // transposed LDS writes of a wave then cover every bank exactly twice.
    const bool v_owner = tid < L::kVItems;
    const int v_kq = tid & 15, v_dg = tid >> 4;
    const int32_t v_off = 4 * v_kq * row_stride + v_dg * 8;

    u32x4_t rk[L::kKLoads];
    u32x4_t rv[4];
    auto load_regs = [&](int32_t k0) {
        const int64_t base = (int64_t)k0 * row_stride;
        if (k0 + KT <= (int32_t)a.n_tok) {
#pragma unroll
            for (int i = 0; i < L::kKLoads; ++i) rk[i] = *reinterpret_cast<const u32x4_t*>(kbase + base + k_off[i]);
            if (v_owner) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    rv[i] = *reinterpret_cast<const u32x4_t*>(vbase + base + v_off + i * row_stride);
            }
        } else {  // tail tile: clamp rows past the end (their scores are masked)
#pragma unroll
            for (int i = 0; i < L::kKLoads; ++i) {
                const int32_t kk = min(k0 + k_key[i], last_key);
                rk[i] = *reinterpret_cast<const u32x4_t*>(kbase + (int64_t)kk * row_stride + (k_off[i] - k_key[i] * row_stride));
            }
            if (v_owner) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int32_t kk = min(k0 + 4 * v_kq + i, last_key);
                    rv[i] = *reinterpret_cast<const u32x4_t*>(vbase + (int64_t)kk * row_stride + v_dg * 8);
                }
            }
        }
    };
    auto store_lds = [&](int buf) {
        uint16_t* kb = Ks + buf * KT * L::KLD;
#pragma unroll
        for (int i = 0; i < L::kKLoads; ++i) {
            const int item = i * 256 + tid;
            *reinterpret_cast<u32x4_t*>(kb + k_key[i] * L::KLD + (item % L::kChunksPerKey) * 8) = rk[i];
        }
        if (v_owner) {
            uint16_t* vb = Vt + buf * D * L::VLD + (8 * v_dg) * L::VLD + 4 * v_kq;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // d = 8*dg + 2e (low halves) and 2e+1 (high halves), keys 4kq .. 4kq+3
                u32x2_t lo, hi;
                lo.x = __builtin_amdgcn_perm(rv[1][e], rv[0][e], 0x05040100u);
                lo.y = __builtin_amdgcn_perm(rv[3][e], rv[2][e], 0x05040100u);
                hi.x = __builtin_amdgcn_perm(rv[1][e], rv[0][e], 0x07060302u);
                hi.y = __builtin_amdgcn_perm(rv[3][e], rv[2][e], 0x07060302u);
                *reinterpret_cast<u32x2_t*>(vb + (2 * e) * L::VLD) = lo;
                *reinterpret_cast<u32x2_t*>(vb + (2 * e + 1) * L::VLD) = hi;
            }
        }
    };

    f32x16_t oacc[D / 32];
#pragma unroll
    for (int i = 0; i < D / 32; ++i) oacc[i] = f32x16_t{};
    float m_run = -1.0e30f, l_run = 0.0f;
    const float cl2 = a.cl2;

    load_regs(kbeg);
    store_lds(0);
    __syncthreads();
    const int n_kt = (kend - kbeg + KT - 1) / KT;
    for (int it = 0; it < n_kt; ++it) {
        const int32_t kt = kbeg + it * KT;
        const int buf = it & 1;
        const bool more = it + 1 < n_kt;
        if (more) load_regs(kt + KT);

        const uint16_t* kb = Ks + buf * KT * L::KLD;
        f32x16_t sacc[2] = {f32x16_t{}, f32x16_t{}};
#pragma unroll
        for (int s = 0; s < D / 16; ++s) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                const bf16x8_t kv = *reinterpret_cast<const bf16x8_t*>(kb + (32 * mb + l32) * L::KLD + half * (D / 2) + 8 * s);
                sacc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kv, qf[s], sacc[mb], 0, 0, 0);
            }
        }
        // sacc[mb][v] = score of key kt + 32mb + 8(v/4) + 4half + (v%4) for this lane's column
        if (kt + KT - 1 > pmin || kt + KT > kend) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int32_t key = kt + 32 * mb + 8 * (v >> 2) + 4 * half + (v & 3);
                    if (key > p_l || key >= kend) sacc[mb][v] = -INFINITY;
                }
        }
        float mx = fmaxf(sacc[0][0], sacc[0][1]);
#pragma unroll
        for (int v = 2; v < 16; v += 2) mx = fmaxf(mx, fmaxf(sacc[0][v], sacc[0][v + 1]));
#pragma unroll
        for (int v = 0; v < 16; v += 2) mx = fmaxf(mx, fmaxf(sacc[1][v], sacc[1][v + 1]));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        if (__any((m_new - m_run) * cl2 > kRescaleSlack)) {  // rare: the first tile, then big jumps only
            const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * cl2);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int i = 0; i < D / 32; ++i) oacc[i] *= alpha;
        }
        const float mc = m_run * cl2;
        float lsum = 0.0f;
        bf16x8_t pb[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {  // keys 16s .. 16s+15 of the tile (permuted, see below)
            f32x8_t pv;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float x = __builtin_amdgcn_exp2f(fmaf(sacc[s >> 1][8 * (s & 1) + e], cl2, -mc));
                pv[e] = x;
                lsum += x;
            }
            pb[s] = __builtin_convertvector(pv, bf16x8_t);
        }
        l_run += lsum;

        // O^T += V^T P^T.  MFMA k index 8h+e of step s is key 16s + 8(e/4) + 4h + e%4:
        // exactly the keys this lane's P values (above) belong to.
        const uint16_t* vb = Vt + buf * D * L::VLD;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
#pragma unroll
            for (int i = 0; i < D / 32; ++i) {
                const uint16_t* vr = vb + (32 * i + l32) * L::VLD + 16 * s + 4 * half;
                const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(vr);
                const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(vr + 8);
                const u32x4_t w = u32x4_t{lo.x, lo.y, hi.x, hi.y};
                oacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, w), pb[s], oacc[i], 0, 0, 0);
            }
        }
        if (more) store_lds(buf ^ 1);
        __syncthreads();
    }

    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (p_l < 0) return;
    // oacc[i][v] = O[col][d = 32i + 8(v/4) + 4half + (v%4)]
    if (pmax + 1 <= a.chunk) {
        const float inv = 1.0f / l_tot;
        uint16_t* op = a.out + (row * a.Hq + head) * (int64_t)D;
#pragma unroll
        for (int i = 0; i < D / 32; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int d0 = 32 * i + 8 * r + 4 * half;
                u32x2_t w;
                w.x = pack_bf16x2(oacc[i][4 * r] * inv, oacc[i][4 * r + 1] * inv);
                w.y = pack_bf16x2(oacc[i][4 * r + 2] * inv, oacc[i][4 * r + 3] * inv);
                *reinterpret_cast<u32x2_t*>(op + d0) = w;
            }
    } else {
        const int64_t item = ((int64_t)tile * a.Hkv + g) * a.n_chunks + chunk_id;
        float* po = a.part_o + (item * 128 + col) * D;
#pragma unroll
        for (int i = 0; i < D / 32; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int d0 = 32 * i + 8 * r + 4 * half;
                *reinterpret_cast<f32x4_t*>(po + d0) =
                    f32x4_t{oacc[i][4 * r], oacc[i][4 * r + 1], oacc[i][4 * r + 2], oacc[i][4 * r + 3]};
            }
        if (half == 0) *reinterpret_cast<float2*>(a.part_ml + (item * 128 + col) * 2) = make_float2(m_run, l_tot);
    }
}

// Log-sum-exp merge of split-KV partial results: one workgroup per
// (tile, kv head); thread t owns column t/2 and half of its head dim.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(AttnArgs a) {
    const int64_t tg = blockIdx.x;  // tile * Hkv + g
    const int32_t nu = a.n_used[tg];
    if (nu <= 1) return;
    const int tid = threadIdx.x;
    const int col = tid >> 1, dh = tid & 1;
    const int tile = (int)(tg / a.Hkv), g = (int)(tg % a.Hkv);
    const int row_local = col % a.R, head_local = col / a.R;
    const int64_t row = (int64_t)tile * a.R + row_local;
    if (row >= a.n_sel) return;
    const int32_t p = a.pos[row];
    if (p < 0 || p >= a.n_tok) return;
    const int head = g * a.G + head_local;
    const int64_t item0 = tg * a.n_chunks;
    constexpr int PER = D / 2;
    float M = -1.0e30f;
    for (int c = 0; c < nu; ++c) M = fmaxf(M, a.part_ml[((item0 + c) * 128 + col) * 2]);
    f32x4_t acc[PER / 4];
#pragma unroll
    for (int e = 0; e < PER / 4; ++e) acc[e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float Lsum = 0.0f;
    for (int c = 0; c < nu; ++c) {
        const float2 ml = *reinterpret_cast<const float2*>(a.part_ml + ((item0 + c) * 128 + col) * 2);
        const float w = __builtin_amdgcn_exp2f((ml.x - M) * a.cl2);
        Lsum += w * ml.y;
        const f32x4_t* po = reinterpret_cast<const f32x4_t*>(a.part_o + ((item0 + c) * 128 + col) * D + dh * PER);
#pragma unroll
        for (int e = 0; e < PER / 4; ++e) acc[e] += w * po[e];
    }
    const float inv = 1.0f / Lsum;
    u32x4_t* op = reinterpret_cast<u32x4_t*>(a.out + (row * a.Hq + head) * (int64_t)D + dh * PER);
#pragma unroll
    for (int e = 0; e < PER / 8; ++e) {
        const f32x4_t x0 = acc[2 * e] * inv, x1 = acc[2 * e + 1] * inv;
        op[e] = u32x4_t{pack_bf16x2(x0[0], x0[1]), pack_bf16x2(x0[2], x0[3]), pack_bf16x2(x1[0], x1[1]),
                        pack_bf16x2(x1[2], x1[3])};
    }
}

template <int D>
hipError_t launch_attention(const AttnArgs& args, hipStream_t s) {
    const unsigned grid = (unsigned)((int64_t)args.n_tiles * args.Hkv * args.n_chunks);
    hipLaunchKernelGGL(attention_kernel<D>, dim3(grid), dim3(256), 0, s, args);
    if (args.n_chunks > 1)
        hipLaunchKernelGGL(combine_kernel<D>, dim3((unsigned)((int64_t)args.n_tiles * args.Hkv)), dim3(256), 0, s, args);
    return hipGetLastError();
}

}  // namespace

size_t qkv_workspace_dev_offset(int64_t n_sel, int32_t head_dim, int dtype) {
    return dtype == SEMSHARE_BF16 ? align256((size_t)n_sel * (head_dim / 2) * sizeof(float2)) : 0;
}

int32_t qkv_dev_parts(int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int dtype) {
    const int32_t cols = n_kv_heads * head_dim;
    return dtype == SEMSHARE_BF16 ? cols / qkv_gemm_bn(n_q_heads, n_kv_heads, head_dim) : cols / 2;
}

size_t qkv_workspace_bytes(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int dtype) {
    return qkv_workspace_dev_offset(n_sel, head_dim, dtype) +
           align256((size_t)n_sel * 2 * qkv_dev_parts(n_q_heads, n_kv_heads, head_dim, dtype) * sizeof(float));
}

AttnPlan plan_attention(int64_t n_sel, int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                        int32_t head_dim, int dtype) {
    AttnPlan p{};
    const int32_t G = n_q_heads / n_kv_heads;
    p.rows_per_tile = dtype == SEMSHARE_BF16 ? 128 / G : 1;
    p.n_tiles = (n_sel + p.rows_per_tile - 1) / p.rows_per_tile;
    p.chunk = (int32_t)((n_tok + 63) / 64 * 64);
    p.n_chunks = 1;
    if (dtype == SEMSHARE_BF16 && n_sel > 0) {
        // split the key range when there are too few (tile, kv head) items to
        // fill the chip; each chunk keeps >= 256 keys
        const int64_t items = p.n_tiles * n_kv_heads;
        int64_t want = (1024 + items - 1) / items;
        const int64_t cap = (n_tok + 255) / 256;
        if (want > cap) want = cap;
        if (want < 1) want = 1;
        const int64_t per = (n_tok + want - 1) / want;
        p.chunk = (int32_t)((per + 63) / 64 * 64);
        p.n_chunks = (int32_t)((n_tok + p.chunk - 1) / p.chunk);
        if (p.n_chunks < 1) p.n_chunks = 1;
    }
    size_t off = 0;
    p.off_part_o = p.off_part_ml = p.off_used = 0;
    if (p.n_chunks > 1) {
        const size_t items = (size_t)p.n_tiles * n_kv_heads * p.n_chunks;
        off = align256(items * 128 * head_dim * sizeof(float));
        p.off_part_ml = off;
        off = align256(off + items * 128 * 2 * sizeof(float));
        p.off_used = off;
        off = align256(off + (size_t)p.n_tiles * n_kv_heads * sizeof(int32_t));
    }
    p.total = off;
    return p;
}

hipError_t launch_qkv_bf16(const QkvArgs& a, hipStream_t s) {
    unsigned char* ws = static_cast<unsigned char*>(a.workspace);
    float2* rope = reinterpret_cast<float2*>(ws);
    float* dev_parts = a.deviation_out
                           ? reinterpret_cast<float*>(ws + qkv_workspace_dev_offset(a.n_sel, a.head_dim, SEMSHARE_BF16))
                           : nullptr;
    const int32_t half_d = a.head_dim / 2;
    {
        const int64_t n = a.n_sel * half_d;
        hipLaunchKernelGGL(prep_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a.sel_pos, a.n_sel,
                           a.n_tok, half_d, log2(a.rope_base), rope);
    }
    const int32_t bn = qkv_gemm_bn(a.n_q_heads, a.n_kv_heads, a.head_dim);
    GemmArgs g{};
    g.x = static_cast<const uint16_t*>(a.x_sel);
    g.pos = a.sel_pos;
    g.w[0] = static_cast<const uint16_t*>(a.wq);
    g.w[1] = static_cast<const uint16_t*>(a.wk);
    g.w[2] = static_cast<const uint16_t*>(a.wv);
    g.seg_cols[0] = a.n_q_heads * a.head_dim;
    g.seg_cols[1] = g.seg_cols[2] = a.n_kv_heads * a.head_dim;
    g.seg_tiles[0] = a.q_out ? g.seg_cols[0] / bn : 0;
    g.seg_tiles[1] = g.seg_tiles[2] = g.seg_cols[1] / bn;
    g.n_nt = g.seg_tiles[0] + g.seg_tiles[1] + g.seg_tiles[2];
    g.n_mt = (int32_t)((a.n_sel + 127) / 128);
    g.n_sel = a.n_sel;
    g.n_tok = a.n_tok;
    g.hidden = a.hidden;
    g.D = a.head_dim;
    g.q_out = static_cast<uint16_t*>(a.q_out);
    g.kv[0] = static_cast<uint16_t*>(a.k_cache);
    g.kv[1] = static_cast<uint16_t*>(a.v_cache);
    g.rope = rope;
    g.dev_parts = dev_parts;
    launch_qkv_gemm(g, bn, s);
    if (a.deviation_out)
        hipLaunchKernelGGL(dev_final_kernel, dim3((unsigned)((a.n_sel + 255) / 256)), dim3(256), 0, s, dev_parts,
                           a.deviation_out, a.n_sel,
                           qkv_dev_parts(a.n_q_heads, a.n_kv_heads, a.head_dim, SEMSHARE_BF16));
    return hipGetLastError();
}

hipError_t launch_attention_bf16(const AttnCall& a, const AttnPlan& p, hipStream_t s) {
    unsigned char* ws = static_cast<unsigned char*>(a.workspace);
    AttnArgs t{};
    t.q = static_cast<const uint16_t*>(a.q);
    t.pos = a.sel_pos;
    t.k_cache = static_cast<const uint16_t*>(a.k_cache);
    t.v_cache = static_cast<const uint16_t*>(a.v_cache);
    t.out = static_cast<uint16_t*>(a.out);
    t.part_o = reinterpret_cast<float*>(ws + p.off_part_o);
    t.part_ml = reinterpret_cast<float*>(ws + p.off_part_ml);
    t.n_used = reinterpret_cast<int32_t*>(ws + p.off_used);
    t.n_sel = a.n_sel;
    t.n_tok = a.n_tok;
    t.Hq = a.n_q_heads;
    t.Hkv = a.n_kv_heads;
    t.G = a.n_q_heads / a.n_kv_heads;
    t.R = p.rows_per_tile;
    t.n_tiles = (int32_t)p.n_tiles;
    t.chunk = p.chunk;
    t.n_chunks = p.n_chunks;
    t.cl2 = a.sm_scale * kLog2e;
    if (a.head_dim == 128) return launch_attention<128>(t, s);
    return launch_attention<64>(t, s);
}

}  // namespace semshare
