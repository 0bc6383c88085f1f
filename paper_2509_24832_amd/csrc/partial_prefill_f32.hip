// One attention layer of partial prefill, fp32 storage and arithmetic
// (Sections 4.2, 4.3.3; KV deviation of Appendix A.4).  Meant for small
// fp32 problems: fp32 has no MFMA advantage over the VALU on this chip, so the
// projections and the attention run on the vector units.
//  1. qkv_f32   one thread per (selected row, output pair): two dot products,
//               RoPE of q/k pairs (fp64 angle, fp32 rotation), q to the
//               workspace, k/v to the cache rows sel_pos after the old row's
//               squared differences are added to the deviation sums.
//  2. dev_final sigma = sqrt(sum dK^2) + sqrt(sum dV^2).
//  3. attn_f32  one workgroup per (selected row, query head): scores of all
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

__global__ __launch_bounds__(256) void qkv_f32_kernel(QkvF32Args a, int32_t pairs_per_row) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.n_sel * pairs_per_row) return;
    const int64_t m = i / pairs_per_row;
    int32_t c = 2 * (int32_t)(i - m * pairs_per_row);  // column over the used segments
    const int32_t nq = a.first_seg == 0 ? a.seg_cols[0] : 0, nkv = a.seg_cols[1];
    int seg;
    if (c < nq) {
        seg = 0;
    } else if (c < nq + nkv) {
        seg = 1;
        c -= nq;
    } else {
        seg = 2;
        c -= nq + nkv;
    }
    const float* wseg = seg == 0 ? a.w[0] : (seg == 1 ? a.w[1] : a.w[2]);
    const int32_t seg_cols = seg == 0 ? a.seg_cols[0] : nkv;
    const float4* xr = reinterpret_cast<const float4*>(a.x + m * a.hidden);
    const float4* w0 = reinterpret_cast<const float4*>(wseg + (int64_t)c * a.hidden);
    const float4* w1 = reinterpret_cast<const float4*>(wseg + (int64_t)(c + 1) * a.hidden);
    float s0 = 0.f, s1 = 0.f;
    for (int32_t k = 0; k < a.hidden / 4; ++k) {
        const float4 xv = xr[k], u = w0[k], v = w1[k];
        s0 = fmaf(xv.x, u.x, fmaf(xv.y, u.y, fmaf(xv.z, u.z, fmaf(xv.w, u.w, s0))));
        s1 = fmaf(xv.x, v.x, fmaf(xv.y, v.y, fmaf(xv.z, v.z, fmaf(xv.w, v.w, s1))));
    }
    const int32_t p = a.pos[m];
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
        return;
    }
    float* part = a.dev_parts ? a.dev_parts + (2 * m + (seg - 1)) * (int64_t)(nkv / 2) + c / 2 : nullptr;
    if (p < 0 || p >= a.n_tok) {
        if (part) *part = 0.0f;
        return;
    }
    float* dst = (seg == 1 ? a.kv[0] : a.kv[1]) + (int64_t)p * seg_cols + c;
    if (part) {
        const float d0 = dst[0] - y0, d1 = dst[1] - y1;
        *part = d0 * d0 + d1 * d1;
    }
    dst[0] = y0;
    dst[1] = y1;
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

__global__ __launch_bounds__(kAttnThreads) void attn_f32_kernel(const float* __restrict__ q,
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
    const int32_t pairs = cols / 2;
    const int64_t n = a.n_sel * pairs;
    hipLaunchKernelGGL(qkv_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, q, pairs);
    if (dev_parts)
        hipLaunchKernelGGL(dev_final_f32_kernel, dim3((unsigned)((a.n_sel + 255) / 256)), dim3(256), 0, s, dev_parts,
                           a.deviation_out, a.n_sel, qkv_dev_parts(a.n_q_heads, a.n_kv_heads, a.head_dim, SEMSHARE_FP32));
    return hipGetLastError();
}

hipError_t launch_attention_f32(const AttnCall& a, const AttnPlan& p, hipStream_t s) {
    (void)p;
    const size_t lds = (size_t)a.n_tok * sizeof(float);
    hipLaunchKernelGGL(attn_f32_kernel, dim3((unsigned)(a.n_sel * a.n_q_heads)), dim3(kAttnThreads), lds, s,
                       static_cast<const float*>(a.q), a.sel_pos, static_cast<const float*>(a.k_cache),
                       static_cast<const float*>(a.v_cache), static_cast<float*>(a.out), a.n_tok, a.n_q_heads,
                       a.n_kv_heads, a.head_dim, a.sm_scale);
    return hipGetLastError();
}

}  // namespace semshare
