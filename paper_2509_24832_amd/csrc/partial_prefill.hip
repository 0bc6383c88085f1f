// Projection half of one partial-prefill layer (Sections 4.2, 4.3.3; KV
// deviation of Appendix A.4), bf16 storage with fp32 accumulation.
//
// Kernels, in stream order:
//  1. prep        RoPE (cos, sin) table for the selected positions (skipped
//                 when the caller passes one made beforehand), one entry
//                 per (row, pair) shared by all heads and by q and k.
//  2. qkv_gemm    projection + RoPE + deviation partials + cache scatter
//                 (qkv_gemm.hip).
//  3. dev_final   sigma = sqrt(sum dK^2) + sqrt(sum dV^2), partials summed in
//                 a fixed order.
// The attention half lives in attention.hip.
#include "semshare_internal.h"

namespace semshare {
namespace {

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

}  // namespace

size_t qkv_workspace_dev_offset(int64_t n_sel, int32_t head_dim, int dtype) {
    return dtype == SEMSHARE_BF16 ? align256((size_t)n_sel * (head_dim / 2) * sizeof(float2)) : 0;
}

int32_t qkv_dev_parts(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int dtype) {
    const int32_t cols = n_kv_heads * head_dim;
    return dtype == SEMSHARE_BF16 ? cols / qkv_gemm_bn(n_sel, n_q_heads, n_kv_heads, head_dim) : cols / 2;
}

// The deviation parts are sized for the narrowest tiles (128 columns) whatever
// the call's tile width, so that the size grows with n_sel: a workspace sized
// for n rows serves every call with fewer.
size_t qkv_workspace_bytes(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int dtype) {
    const int32_t cols = n_kv_heads * head_dim;
    const int32_t max_parts = dtype == SEMSHARE_BF16 ? (cols + 127) / 128 : cols / 2;
    return qkv_workspace_dev_offset(n_sel, head_dim, dtype) + align256((size_t)n_sel * 2 * max_parts * sizeof(float));
}

hipError_t launch_rope_table(const int32_t* sel_pos, int64_t n_sel, int64_t n_tok, int32_t head_dim,
                             double rope_base, void* table, hipStream_t s) {
    const int32_t half_d = head_dim / 2;
    const int64_t n = n_sel * half_d;
    if (n > 0)
        hipLaunchKernelGGL(prep_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, sel_pos, n_sel, n_tok,
                           half_d, log2(rope_base), static_cast<float2*>(table));
    return hipGetLastError();
}

hipError_t launch_qkv_bf16(const QkvArgs& a, hipStream_t s) {
    unsigned char* ws = static_cast<unsigned char*>(a.workspace);
    // a table made beforehand (shared by the layers of one selection), else
    // one made here in the workspace
    const float2* rope = a.rope_table ? static_cast<const float2*>(a.rope_table) : reinterpret_cast<float2*>(ws);
    float* dev_parts = a.deviation_out
                           ? reinterpret_cast<float*>(ws + qkv_workspace_dev_offset(a.n_sel, a.head_dim, SEMSHARE_BF16))
                           : nullptr;
    if (!a.rope_table) launch_rope_table(a.sel_pos, a.n_sel, a.n_tok, a.head_dim, a.rope_base, ws, s);
    const int32_t bn = qkv_gemm_bn(a.n_sel, a.n_q_heads, a.n_kv_heads, a.head_dim);
    GemmArgs g{};
    g.x = static_cast<const uint16_t*>(a.x_sel);
    g.x_rows = a.x_rows;
    g.n_x = a.n_x;
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
    g.dev_src[0] = static_cast<const uint16_t*>(a.ref_k);
    g.dev_src[1] = static_cast<const uint16_t*>(a.ref_v);
    g.dev_idx = a.ref_idx;
    g.dev_n = a.ref_n;
    launch_qkv_gemm(g, bn, s);
    if (a.deviation_out)
        hipLaunchKernelGGL(dev_final_kernel, dim3((unsigned)((a.n_sel + 255) / 256)), dim3(256), 0, s, dev_parts,
                           a.deviation_out, a.n_sel,
                           qkv_dev_parts(a.n_sel, a.n_q_heads, a.n_kv_heads, a.head_dim, SEMSHARE_BF16));
    return hipGetLastError();
}

}  // namespace semshare
