// One attention layer of partial prefill, fp32 storage and arithmetic
// (Sections 4.2, 4.3.3; KV deviation of Appendix A.4).  Meant for small
// fp32 problems: fp32 has no MFMA advantage over the VALU on this chip (both
// 157.3 TFLOP/s), so the projections and the attention run on the vector
// units, tiled through LDS so that each operand read from L2 feeds many
// fused multiply-adds.
//  1. qkv_f32   a 64 x 64 output tile per workgroup (each thread 4 rows x 4
//               columns, K in chunks of 16 staged in LDS), then per column
//               pair: RoPE of q/k pairs (fp64 angle, fp32 rotation), q to
//               its buffer, k/v to the cache rows sel_pos after the old row's
//               squared differences are added to the deviation sums.
//  2. dev_final sigma = sqrt(sum dK^2) + sqrt(sum dV^2).
//  3. attn_f32  with enough rows to fill the chip: one workgroup per (16
//               selected rows, query head), the rows sharing every 32-key
//               tile of K and V in LDS, online softmax; otherwise one
//               workgroup per (selected row, query head): scores of all
//               causal keys in LDS, exact softmax, then P V.
#include <climits>

#include "semshare_internal.h"

namespace semshare {
namespace {

struct QkvF32Args {
    const float* x;
    const int32_t* pos;
    const float* w[3];
    int32_t seg_cols[3];
    int32_t first_seg;
    int64_t n_sel, n_tok;
    int32_t hidden, D;
    double log2_base;
    float* q_out;
    float* kv[2];
    float* dev_parts;  // [n_sel][2][Hkv*D/2] squared differences per pair, or null
};

constexpr int kTM = 64, kTN = 64, kTK = 16;

// Column c (over the segments in use) -> its segment, its column within the
// segment; segments are [q (when written)][k][v].
__device__ __forceinline__ int seg_of(const QkvF32Args& a, int32_t c, int32_t* cin) {
    const int32_t nq = a.first_seg == 0 ? a.seg_cols[0] : 0, nkv = a.seg_cols[1];
    if (c < nq) { *cin = c; return 0; }
    if (c < nq + nkv) { *cin = c - nq; return 1; }
    *cin = c - nq - nkv;
    return 2;
}

__global__ __launch_bounds__(256) void qkv_f32_kernel(QkvF32Args a, int32_t cols) {
    __shared__ __attribute__((aligned(16))) float As[kTK][kTM + 4];  // x rows, k-major
    __shared__ __attribute__((aligned(16))) float Bs[kTK][kTN + 4];  // weight rows (output columns), k-major
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int64_t m0 = (int64_t)blockIdx.y * kTM;
    const int32_t n0 = (int32_t)blockIdx.x * kTN;
    // loader rows: element tid + 256 i of a 64 x 16 tile is (row (tid >> 4) + 16 i, k tid & 15)
    const int kk = tid & 15;
    const float* xrow[4];
    const float* wrow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = (tid >> 4) + 16 * i;
        xrow[i] = m0 + r < a.n_sel ? a.x + (m0 + r) * a.hidden : nullptr;
        const int32_t c = n0 + r;
        wrow[i] = nullptr;
        if (c < cols) {
            int32_t cin;
            const int sg = seg_of(a, c, &cin);
            wrow[i] = a.w[sg] + (int64_t)cin * a.hidden;
        }
    }
    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0f;
    // the next chunk's elements are fetched into registers while the current
    // one is multiplied, so the global latency overlaps the arithmetic
    float ra[4], rb[4];
    auto fetch = [&](int32_t k0) {
        const bool kin = k0 + kk < a.hidden;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            ra[i] = xrow[i] && kin ? xrow[i][k0 + kk] : 0.0f;
            rb[i] = wrow[i] && kin ? wrow[i][k0 + kk] : 0.0f;
        }
    };
    fetch(0);
    for (int32_t k0 = 0; k0 < a.hidden; k0 += kTK) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = (tid >> 4) + 16 * i;
            As[kk][r] = ra[i];
            Bs[kk][r] = rb[i];
        }
        __syncthreads();
        if (k0 + kTK < a.hidden) fetch(k0 + kTK);
#pragma unroll
        for (int k = 0; k < kTK; ++k) {
            const float4 av = *reinterpret_cast<const float4*>(&As[k][4 * ty]);
            const float4 bv = *reinterpret_cast<const float4*>(&Bs[k][4 * tx]);
            const float ar[4] = {av.x, av.y, av.z, av.w}, br[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], br[j], acc[i][j]);
        }
        __syncthreads();
    }
    // epilogue: this thread's 4 rows x 2 column pairs (segment sizes are even,
    // so a pair never straddles two segments)
    const int32_t nkv = a.seg_cols[1];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t m = m0 + 4 * ty + i;
        if (m >= a.n_sel) continue;
        const int32_t p = a.pos[m];
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
            const int32_t cg = n0 + 4 * tx + 2 * pp;
            if (cg >= cols) continue;
            int32_t c;
            const int seg = seg_of(a, cg, &c);
            const int32_t seg_cols = seg == 0 ? a.seg_cols[0] : nkv;
            const float s0 = acc[i][2 * pp], s1 = acc[i][2 * pp + 1];
            float y0 = s0, y1 = s1;
            if (seg < 2) {
                const int32_t k = (c % a.D) / 2;
                const double theta = exp2(-(2.0 * (double)k / (double)a.D) * a.log2_base);
                float sn, cs;
                rope_sincos((double)(p >= 0 && p < a.n_tok ? p : 0), theta, &sn, &cs);
                y0 = cs * s0 - sn * s1;
                y1 = sn * s0 + cs * s1;
            }
            if (seg == 0) {
                float* q = a.q_out + m * seg_cols + c;
                q[0] = y0;
                q[1] = y1;
                continue;
            }
            float* part = a.dev_parts ? a.dev_parts + (2 * m + (seg - 1)) * (int64_t)(nkv / 2) + c / 2 : nullptr;
            if (p < 0 || p >= a.n_tok) {
                if (part) *part = 0.0f;
                continue;
            }
            float* dst = (seg == 1 ? a.kv[0] : a.kv[1]) + (int64_t)p * seg_cols + c;
            if (part) {
                const float d0 = dst[0] - y0, d1 = dst[1] - y1;
                *part = d0 * d0 + d1 * d1;
            }
            dst[0] = y0;
            dst[1] = y1;
        }
    }
}

__global__ void dev_final_f32_kernel(const float* __restrict__ parts, float* __restrict__ dev, int64_t n_sel,
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

constexpr int kAttnThreads = 128;

__device__ __forceinline__ float block_reduce(float v, float* red, bool is_max) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float u = __shfl_xor(v, o);
        v = is_max ? fmaxf(v, u) : v + u;
    }
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float r = red[0];
    for (int w = 1; w < kAttnThreads / 64; ++w) r = is_max ? fmaxf(r, red[w]) : r + red[w];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kAttnThreads) void attn_f32_row_kernel(const float* __restrict__ q,
                                                                const int32_t* __restrict__ pos,
                                                                const float* __restrict__ k_cache,
                                                                const float* __restrict__ v_cache,
                                                                float* __restrict__ out, int64_t n_tok,
                                                                int32_t Hq, int32_t Hkv, int32_t D,
                                                                float scale) {
    extern __shared__ float sc[];  // [n_tok] scores / probabilities
    __shared__ float red[kAttnThreads / 64];
    __shared__ float qs[128];
    const int64_t m = blockIdx.x / Hq;
    const int h = blockIdx.x % Hq;
    const int g = h / (Hq / Hkv);
    const int32_t p = pos[m];
    if (p < 0 || p >= n_tok) return;
    for (int d = threadIdx.x; d < D; d += kAttnThreads) qs[d] = q[(m * Hq + h) * D + d];
    __syncthreads();
    const int64_t stride = (int64_t)Hkv * D;
    float mx = -INFINITY;
    for (int32_t j = threadIdx.x; j <= p; j += kAttnThreads) {
        const float* kr = k_cache + j * stride + (int64_t)g * D;
        float s = 0.f;
        for (int d = 0; d < D; ++d) s = fmaf(qs[d], kr[d], s);
        s *= scale;
        sc[j] = s;
        mx = fmaxf(mx, s);
    }
    mx = block_reduce(mx, red, true);
    float sum = 0.f;
    for (int32_t j = threadIdx.x; j <= p; j += kAttnThreads) {
        const float e = expf(sc[j] - mx);
        sc[j] = e;
        sum += e;
    }
    sum = block_reduce(sum, red, false);
    const float inv = 1.0f / sum;
    for (int d = threadIdx.x; d < D; d += kAttnThreads) {
        const float* vc = v_cache + (int64_t)g * D + d;
        float acc = 0.f;
        for (int32_t j = 0; j <= p; ++j) acc = fmaf(sc[j], vc[j * stride], acc);
        out[(m * Hq + h) * D + d] = acc * inv;
    }
}

constexpr int kRowsF32 = 16;  // selected rows per workgroup (same query head)
constexpr int kKeysF32 = 32;  // keys per LDS tile

// The tiled form, for calls with enough (16-row block, head) pairs to fill
// the chip: one workgroup per 16 selected rows of one query head, which share
// every 32-key tile of K and V in LDS.  Thread t serves row qi = t / 16; as
// lane kk = t % 16 of its row it holds the row's q in registers, computes the
// scores of keys kk and kk + 16 of each tile and owns the output dims
// [kk D/16, (kk + 1) D/16).  Online softmax (running max and sum per row).
// Rows are in ascending position order, so the tiles run up to the last
// valid row's position.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_tiled_kernel(const float* __restrict__ q,
                                                             const int32_t* __restrict__ pos,
                                                             const float* __restrict__ k_cache,
                                                             const float* __restrict__ v_cache,
                                                             float* __restrict__ out, int64_t n_sel, int64_t n_tok,
                                                             int32_t Hq, int32_t Hkv, float scale) {
    constexpr int kDpt = D / 16;  // output dims per thread
    constexpr int kLdk = D + 4;   // K row stride in LDS (16-byte rows, banks spread)
    __shared__ __attribute__((aligned(16))) float Ks[kKeysF32][kLdk];
    __shared__ __attribute__((aligned(16))) float Vs[kKeysF32][D];
    __shared__ __attribute__((aligned(16))) float Ps[kRowsF32][kKeysF32];
    __shared__ int32_t s_pmax;
    const int tid = threadIdx.x, qi = tid >> 4, kk = tid & 15;
    const int64_t r0 = (int64_t)(blockIdx.x / Hq) * kRowsF32;
    const int h = blockIdx.x % Hq;
    const int g = h / (Hq / Hkv);
    const int64_t row = r0 + qi;
    int32_t p = row < n_sel ? pos[row] : -1;
    if (p >= n_tok) p = -1;
    float qr[D];
    {
        const float* qp = q + ((row < n_sel ? row : 0) * Hq + h) * (int64_t)D;
#pragma unroll
        for (int d = 0; d < D; d += 4) {
            const float4 v = *reinterpret_cast<const float4*>(qp + d);
            qr[d] = v.x; qr[d + 1] = v.y; qr[d + 2] = v.z; qr[d + 3] = v.w;
        }
    }
    if (tid == 0) s_pmax = -1;
    __syncthreads();
    if (kk == 0 && p >= 0) atomicMax(&s_pmax, p);
    __syncthreads();
    const int32_t pmax = s_pmax;
    if (pmax < 0) return;  // no row of the block has a valid position (uniform)
    const int64_t stride = (int64_t)Hkv * D;
    float m = -1.0e30f, l = 0.0f;
    float o[kDpt];
#pragma unroll
    for (int i = 0; i < kDpt; ++i) o[i] = 0.0f;
    for (int32_t j0 = 0; j0 <= pmax; j0 += kKeysF32) {
        // the tile: 32 rows of D floats each for K and V, 16-byte loads
        for (int e = tid; e < kKeysF32 * D / 4; e += 256) {
            const int r = e / (D / 4), d = 4 * (e % (D / 4));
            const int64_t j = j0 + r;
            float4 kv4 = make_float4(0.f, 0.f, 0.f, 0.f), vv4 = kv4;
            if (j < n_tok) {
                kv4 = *reinterpret_cast<const float4*>(k_cache + j * stride + (int64_t)g * D + d);
                vv4 = *reinterpret_cast<const float4*>(v_cache + j * stride + (int64_t)g * D + d);
            }
            *reinterpret_cast<float4*>(&Ks[r][d]) = kv4;
            *reinterpret_cast<float4*>(&Vs[r][d]) = vv4;
        }
        __syncthreads();
        float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
        for (int d = 0; d < D; d += 4) {
            const float4 a = *reinterpret_cast<const float4*>(&Ks[kk][d]);
            const float4 b = *reinterpret_cast<const float4*>(&Ks[kk + 16][d]);
            s0 = fmaf(qr[d], a.x, s0); s0 = fmaf(qr[d + 1], a.y, s0); s0 = fmaf(qr[d + 2], a.z, s0); s0 = fmaf(qr[d + 3], a.w, s0);
            s1 = fmaf(qr[d], b.x, s1); s1 = fmaf(qr[d + 1], b.y, s1); s1 = fmaf(qr[d + 2], b.z, s1); s1 = fmaf(qr[d + 3], b.w, s1);
        }
        s0 = j0 + kk <= p ? s0 * scale : -INFINITY;
        s1 = j0 + kk + 16 <= p ? s1 * scale : -INFINITY;
        // the row's tile maximum and sum over its 16 lanes (consecutive lanes of one wave)
        float tmax = fmaxf(s0, s1);
#pragma unroll
        for (int o2 = 8; o2 >= 1; o2 >>= 1) tmax = fmaxf(tmax, __shfl_xor(tmax, o2, 16));
        const float m_new = fmaxf(m, tmax);
        const float alpha = expf(m - m_new);
        const float e0 = expf(s0 - m_new), e1 = expf(s1 - m_new);
        float ts = e0 + e1;
#pragma unroll
        for (int o2 = 8; o2 >= 1; o2 >>= 1) ts += __shfl_xor(ts, o2, 16);
        l = l * alpha + ts;
        m = m_new;
        Ps[qi][kk] = e0;
        Ps[qi][kk + 16] = e1;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kDpt; ++i) o[i] *= alpha;
        for (int key = 0; key < kKeysF32; key += 4) {
            const float4 p4 = *reinterpret_cast<const float4*>(&Ps[qi][key]);
            const float pk[4] = {p4.x, p4.y, p4.z, p4.w};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float* vr = &Vs[key + u][kDpt * kk];
#pragma unroll
                for (int i = 0; i < kDpt; ++i) o[i] = fmaf(pk[u], vr[i], o[i]);
            }
        }
        __syncthreads();
    }
    if (p < 0) return;
    const float inv = 1.0f / l;
    float* op = out + (row * Hq + h) * (int64_t)D + kDpt * kk;
#pragma unroll
    for (int i = 0; i < kDpt; ++i) op[i] = o[i] * inv;
}

}  // namespace

hipError_t launch_qkv_f32(const QkvArgs& a, hipStream_t s) {
    unsigned char* ws = static_cast<unsigned char*>(a.workspace);
    float* dev_parts = a.deviation_out
                           ? reinterpret_cast<float*>(ws + qkv_workspace_dev_offset(a.n_sel, a.head_dim, SEMSHARE_FP32))
                           : nullptr;
    QkvF32Args q{};
    q.x = static_cast<const float*>(a.x_sel);
    q.pos = a.sel_pos;
    q.w[0] = static_cast<const float*>(a.wq);
    q.w[1] = static_cast<const float*>(a.wk);
    q.w[2] = static_cast<const float*>(a.wv);
    q.seg_cols[0] = a.n_q_heads * a.head_dim;
    q.seg_cols[1] = q.seg_cols[2] = a.n_kv_heads * a.head_dim;
    q.first_seg = a.q_out ? 0 : 1;
    q.n_sel = a.n_sel;
    q.n_tok = a.n_tok;
    q.hidden = a.hidden;
    q.D = a.head_dim;
    q.log2_base = log2(a.rope_base);
    q.q_out = static_cast<float*>(a.q_out);
    q.kv[0] = static_cast<float*>(a.k_cache);
    q.kv[1] = static_cast<float*>(a.v_cache);
    q.dev_parts = dev_parts;
    const int32_t cols = (a.q_out ? q.seg_cols[0] : 0) + 2 * q.seg_cols[1];
    const dim3 grid((unsigned)((cols + kTN - 1) / kTN), (unsigned)((a.n_sel + kTM - 1) / kTM));
    hipLaunchKernelGGL(qkv_f32_kernel, grid, dim3(256), 0, s, q, cols);
    if (dev_parts)
        hipLaunchKernelGGL(dev_final_f32_kernel, dim3((unsigned)((a.n_sel + 255) / 256)), dim3(256), 0, s, dev_parts,
                           a.deviation_out, a.n_sel, qkv_dev_parts(a.n_sel, a.n_q_heads, a.n_kv_heads, a.head_dim, SEMSHARE_FP32));
    return hipGetLastError();
}

hipError_t launch_attention_f32(const AttnCall& a, const AttnPlan& p, hipStream_t s) {
    (void)p;
    const int64_t blocks = (a.n_sel + kRowsF32 - 1) / kRowsF32;
    // the tiled form once it has at least one workgroup per CU
    const bool tiled = blocks * a.n_q_heads >= 256 && (a.head_dim == 32 || a.head_dim == 64 || a.head_dim == 128);
    const auto* qp = static_cast<const float*>(a.q);
    const auto* kp = static_cast<const float*>(a.k_cache);
    const auto* vp = static_cast<const float*>(a.v_cache);
    auto* op = static_cast<float*>(a.out);
    if (tiled) {
        const dim3 grid((unsigned)(blocks * a.n_q_heads));
        if (a.head_dim == 32)
            hipLaunchKernelGGL(attn_f32_tiled_kernel<32>, grid, dim3(256), 0, s, qp, a.sel_pos, kp, vp, op, a.n_sel,
                               a.n_tok, a.n_q_heads, a.n_kv_heads, a.sm_scale);
        else if (a.head_dim == 64)
            hipLaunchKernelGGL(attn_f32_tiled_kernel<64>, grid, dim3(256), 0, s, qp, a.sel_pos, kp, vp, op, a.n_sel,
                               a.n_tok, a.n_q_heads, a.n_kv_heads, a.sm_scale);
        else
            hipLaunchKernelGGL(attn_f32_tiled_kernel<128>, grid, dim3(256), 0, s, qp, a.sel_pos, kp, vp, op, a.n_sel,
                               a.n_tok, a.n_q_heads, a.n_kv_heads, a.sm_scale);
    } else {
        // few rows: one workgroup per (selected row, head) keeps more CUs busy
        const size_t lds = (size_t)a.n_tok * sizeof(float);
        hipLaunchKernelGGL(attn_f32_row_kernel, dim3((unsigned)(a.n_sel * a.n_q_heads)), dim3(kAttnThreads), lds, s,
                           qp, a.sel_pos, kp, vp, op, a.n_tok, a.n_q_heads, a.n_kv_heads, a.head_dim, a.sm_scale);
    }
    return hipGetLastError();
}

}  // namespace semshare
