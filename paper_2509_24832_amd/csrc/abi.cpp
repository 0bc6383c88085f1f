// C ABI of libsemshare.so: host-side argument validation, workspace
// planning and dispatch to the HIP launchers.  Nothing here allocates
// device memory or synchronizes the device.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "semshare_internal.h"

namespace {

thread_local char g_err[512] = "";

semshare_status_t fail(semshare_status_t code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

semshare_status_t ok() {
    g_err[0] = '\0';
    return SEMSHARE_OK;
}

semshare_status_t from_hip(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(SEMSHARE_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool dtype_ok(semshare_dtype_t dt) { return dt == SEMSHARE_FP32 || dt == SEMSHARE_BF16; }
bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }
size_t dtype_size(semshare_dtype_t dt) { return dt == SEMSHARE_BF16 ? 2 : 4; }

}  // namespace

extern "C" {

const char* semshare_last_error(void) { return g_err; }

int32_t semshare_version(void) { return 10000; }

semshare_status_t semshare_rope_embed(const void* x, void* y, int64_t n_tok, int32_t dim,
                                      int64_t pos0, double base, semshare_dtype_t dtype,
                                      void* stream) {
    if (!dtype_ok(dtype)) return fail(SEMSHARE_E_INVAL, "rope_embed: unknown dtype %d", dtype);
    if (n_tok < 0) return fail(SEMSHARE_E_INVAL, "rope_embed: n_tok < 0");
    if (dim <= 0 || (dim & 1)) return fail(SEMSHARE_E_INVAL, "rope_embed: dim must be even and > 0 (got %d)", dim);
    if (!(base > 0.0) || !std::isfinite(base)) return fail(SEMSHARE_E_INVAL, "rope_embed: base must be finite and > 0");
    if (pos0 < 0) return fail(SEMSHARE_E_INVAL, "rope_embed: pos0 < 0");
    if (pos0 + n_tok > (int64_t(1) << 40)) return fail(SEMSHARE_E_INVAL, "rope_embed: positions exceed 2^40");
    if (n_tok == 0) return ok();
    if (!x || !y) return fail(SEMSHARE_E_INVAL, "rope_embed: null buffer");
    return from_hip(semshare::launch_rope_embed(x, y, n_tok, dim, pos0, base, dtype, (hipStream_t)stream),
                    "rope_embed launch");
}

semshare_status_t semshare_lsh_encode(const void* x, const void* planes, uint64_t* codes,
                                      int64_t n_tok, int32_t dim, int32_t n_bits,
                                      semshare_dtype_t dtype, void* stream) {
    if (!dtype_ok(dtype)) return fail(SEMSHARE_E_INVAL, "lsh_encode: unknown dtype %d", dtype);
    if (n_tok < 0) return fail(SEMSHARE_E_INVAL, "lsh_encode: n_tok < 0");
    if (n_bits != 64 && n_bits != 128 && n_bits != 256)
        return fail(SEMSHARE_E_INVAL, "lsh_encode: n_bits must be 64, 128 or 256 (got %d)", n_bits);
    if (dim <= 0) return fail(SEMSHARE_E_INVAL, "lsh_encode: dim must be > 0");
    if (dtype == SEMSHARE_BF16 && dim % 64)
        return fail(SEMSHARE_E_UNSUPPORTED, "lsh_encode: bf16 needs dim %% 64 == 0 (got %d)", dim);
    // the bf16 kernel addresses 32 rows of x and the n_bits planes by 32-bit byte offsets
    if (dtype == SEMSHARE_BF16 && dim > (1 << 20))
        return fail(SEMSHARE_E_UNSUPPORTED, "lsh_encode: bf16 needs dim <= 2^20 (got %d)", dim);
    if (dtype == SEMSHARE_FP32 && dim % 4)
        return fail(SEMSHARE_E_UNSUPPORTED, "lsh_encode: fp32 needs dim %% 4 == 0 (got %d)", dim);
    if (n_tok > (int64_t(1) << 31) - 64) return fail(SEMSHARE_E_UNSUPPORTED, "lsh_encode: n_tok too large");
    if (n_tok == 0) return ok();
    if (!x || !planes || !codes) return fail(SEMSHARE_E_INVAL, "lsh_encode: null buffer");
    if (!aligned16(x) || !aligned16(planes) || !aligned16(codes))
        return fail(SEMSHARE_E_INVAL, "lsh_encode: buffers must be 16-byte aligned");
    return from_hip(semshare::launch_lsh_encode(x, planes, codes, n_tok, dim, n_bits, dtype, (hipStream_t)stream),
                    "lsh_encode launch");
}

semshare_status_t semshare_rope_lsh_encode(const void* x, const void* planes, uint64_t* codes, int64_t n_tok,
                                          int32_t dim, int32_t n_bits, int64_t pos0, double base,
                                          semshare_dtype_t dtype, void* stream) {
    if (!dtype_ok(dtype)) return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: unknown dtype %d", dtype);
    if (n_tok < 0) return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: n_tok < 0");
    if (n_bits != 64 && n_bits != 128 && n_bits != 256)
        return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: n_bits must be 64, 128 or 256 (got %d)", n_bits);
    if (dim <= 0 || (dim & 1)) return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: dim must be even and > 0 (got %d)", dim);
    if (!(base > 0.0) || !std::isfinite(base)) return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: base must be finite and > 0");
    if (pos0 < 0) return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: pos0 < 0");
    if (pos0 + n_tok > (int64_t(1) << 40)) return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: positions exceed 2^40");
    if (dtype != SEMSHARE_BF16 || n_bits == 256)
        return fail(SEMSHARE_E_UNSUPPORTED, "rope_lsh_encode: built for bf16 with 64 or 128 bits "
                                            "(use rope_embed + lsh_encode otherwise)");
    if (dim % 64) return fail(SEMSHARE_E_UNSUPPORTED, "rope_lsh_encode: needs dim %% 64 == 0 (got %d)", dim);
    if (dim > (1 << 20)) return fail(SEMSHARE_E_UNSUPPORTED, "rope_lsh_encode: needs dim <= 2^20 (got %d)", dim);
    if (n_tok > (int64_t(1) << 31) - 64) return fail(SEMSHARE_E_UNSUPPORTED, "rope_lsh_encode: n_tok too large");
    if (n_tok == 0) return ok();
    if (!x || !planes || !codes) return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: null buffer");
    if (!aligned16(x) || !aligned16(planes) || !aligned16(codes))
        return fail(SEMSHARE_E_INVAL, "rope_lsh_encode: buffers must be 16-byte aligned");
    return from_hip(semshare::launch_rope_lsh_encode(x, planes, codes, n_tok, dim, n_bits, pos0, base,
                                                     (hipStream_t)stream),
                    "rope_lsh_encode launch");
}

size_t semshare_attention_mass_workspace(int64_t n_tok, int32_t n_q_heads) {
    if (n_tok < 0 || n_q_heads <= 0) return 0;
    return semshare::attention_mass_workspace(n_tok, n_q_heads);
}

// semshare_attention_mass (reuse = false) and semshare_attention_mass_window
// (reuse = true: the row normalisers are taken from the workspace)
static semshare_status_t attention_mass_impl(const char* name, bool reuse, const void* q, const void* k_cache,
                                             int64_t n_tok, int64_t row_begin, int32_t n_q_heads, int32_t n_kv_heads,
                                             int32_t head_dim, float sm_scale, float* mass, void* workspace,
                                             size_t workspace_bytes, semshare_dtype_t dtype, void* stream) {
    if (!dtype_ok(dtype)) return fail(SEMSHARE_E_INVAL, "%s: unknown dtype %d", name, dtype);
    if (n_tok < 0) return fail(SEMSHARE_E_INVAL, "%s: n_tok < 0", name);
    if (row_begin < 0 || (n_tok > 0 && row_begin >= n_tok))
        return fail(SEMSHARE_E_INVAL, "%s: row_begin must lie in [0, n_tok)", name);
    if (n_q_heads <= 0 || n_kv_heads <= 0 || n_q_heads % n_kv_heads)
        return fail(SEMSHARE_E_INVAL, "%s: n_q_heads must be a positive multiple of n_kv_heads", name);
    if (!(sm_scale >= 0.0f) || !std::isfinite(sm_scale))
        return fail(SEMSHARE_E_INVAL, "%s: sm_scale must be finite and >= 0", name);
    if (dtype != SEMSHARE_BF16 || head_dim != 128)
        return fail(SEMSHARE_E_UNSUPPORTED, "%s: built for bf16 with head_dim 128", name);
    if (n_tok > (int64_t(1) << 24) || (int64_t)n_q_heads * n_tok > (int64_t(1) << 31))
        return fail(SEMSHARE_E_UNSUPPORTED, "%s: too many tokens", name);
    if (n_tok == 0) return ok();
    if (!q || !k_cache || !mass || !workspace) return fail(SEMSHARE_E_INVAL, "%s: null buffer", name);
    if (!aligned16(q) || !aligned16(k_cache) || reinterpret_cast<uintptr_t>(workspace) % 4 ||
        reinterpret_cast<uintptr_t>(mass) % 4)
        return fail(SEMSHARE_E_INVAL, "%s: q and k_cache must be 16-byte aligned, mass and workspace 4-byte", name);
    if (workspace_bytes < semshare::attention_mass_workspace(n_tok, n_q_heads))
        return fail(SEMSHARE_E_INVAL, "%s: workspace too small (%zu < %zu)", name, workspace_bytes,
                    semshare::attention_mass_workspace(n_tok, n_q_heads));
    const float scale = sm_scale == 0.0f ? 1.0f / sqrtf((float)head_dim) : sm_scale;
    return from_hip(semshare::launch_attention_mass(q, k_cache, n_tok, row_begin, n_q_heads, n_kv_heads, scale, mass,
                                                    workspace, (hipStream_t)stream, reuse),
                    name);
}

semshare_status_t semshare_attention_mass(const void* q, const void* k_cache, int64_t n_tok, int64_t row_begin,
                                          int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, float sm_scale,
                                          float* mass, void* workspace, size_t workspace_bytes,
                                          semshare_dtype_t dtype, void* stream) {
    return attention_mass_impl("attention_mass", false, q, k_cache, n_tok, row_begin, n_q_heads, n_kv_heads, head_dim,
                               sm_scale, mass, workspace, workspace_bytes, dtype, stream);
}

semshare_status_t semshare_attention_mass_window(const void* q, const void* k_cache, int64_t n_tok, int64_t row_begin,
                                                 int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                 float sm_scale, float* mass, void* workspace, size_t workspace_bytes,
                                                 semshare_dtype_t dtype, void* stream) {
    return attention_mass_impl("attention_mass_window", true, q, k_cache, n_tok, row_begin, n_q_heads, n_kv_heads,
                               head_dim, sm_scale, mass, workspace, workspace_bytes, dtype, stream);
}

semshare_status_t semshare_retention(const float* mass, const float* score, int32_t n_tok, const int32_t* sel_pos,
                                     const int32_t* counts, double min_keep, int32_t* rank, int32_t* kept_pos,
                                     int32_t* n_kept, void* stream) {
    if (n_tok < 0 || n_tok > semshare::kMaxDynTokLarge)
        return fail(n_tok < 0 ? SEMSHARE_E_INVAL : SEMSHARE_E_UNSUPPORTED, "retention: n_tok must be in [0, %d]",
                    semshare::kMaxDynTokLarge);
    if (!(min_keep >= 0.0 && min_keep <= 1.0)) return fail(SEMSHARE_E_INVAL, "retention: min_keep must lie in [0, 1]");
    if (!counts || !n_kept || (n_tok > 0 && (!mass || !score || !sel_pos || !rank || !kept_pos)))
        return fail(SEMSHARE_E_INVAL, "retention: null buffer");
    return from_hip(semshare::launch_retention(mass, score, n_tok, sel_pos, counts, min_keep, rank, kept_pos, n_kept,
                                               (hipStream_t)stream),
                    "retention launch");
}

semshare_status_t semshare_retention_layer(const int32_t* rank, int32_t n_tok, int32_t n_retain,
                                           const int32_t* sel_pos, int32_t n_sel, const int32_t* idx,
                                           int32_t* kept_pos, int32_t* src_idx, int32_t* sel_rows, int32_t* n_kept,
                                           void* stream) {
    const char* fn = "retention_layer";
    if (n_tok < 0 || n_sel < 0 || n_retain < 0) return fail(SEMSHARE_E_INVAL, "%s: negative size", fn);
    if (n_tok > semshare::kMaxRetainTok)
        return fail(SEMSHARE_E_UNSUPPORTED, "%s: n_tok must be <= %d", fn, semshare::kMaxRetainTok);
    if (n_sel > n_tok) return fail(SEMSHARE_E_INVAL, "%s: n_sel > n_tok", fn);
    if (!n_kept || (n_tok > 0 && (!rank || !kept_pos)) || (n_sel > 0 && (!sel_pos || !sel_rows)) ||
        ((idx == nullptr) != (src_idx == nullptr)))
        return fail(SEMSHARE_E_INVAL, "%s: null buffer (idx and src_idx go together)", fn);
    return from_hip(semshare::launch_retention_layer(rank, n_tok, n_retain, sel_pos, n_sel, idx, kept_pos, src_idx,
                                                     sel_rows, n_kept, (hipStream_t)stream),
                    "retention_layer launch");
}

semshare_status_t semshare_dynamic_recompute(const float* mass, const float* sigma, int32_t n_tok, double thres,
                                             double w_hot, double w_cold, int32_t* sel_pos, int32_t* counts,
                                             void* stream) {
    if (n_tok < 0 || n_tok > semshare::kMaxDynTokLarge)
        return fail(n_tok < 0 ? SEMSHARE_E_INVAL : SEMSHARE_E_UNSUPPORTED, "dynamic_recompute: n_tok must be in [0, %d]",
                    semshare::kMaxDynTokLarge);
    if (!(thres >= 0.0 && thres <= 1.0) || !(w_hot >= 0.0 && w_hot <= 1.0) || !(w_cold >= 0.0 && w_cold <= 1.0))
        return fail(SEMSHARE_E_INVAL, "dynamic_recompute: thres, w_hot and w_cold must lie in [0, 1]");
    if (!counts || (n_tok > 0 && (!mass || !sigma || !sel_pos)))
        return fail(SEMSHARE_E_INVAL, "dynamic_recompute: null buffer");
    return from_hip(semshare::launch_dynamic_recompute(mass, sigma, n_tok, thres, w_hot, w_cold, sel_pos, counts,
                                                       (hipStream_t)stream),
                    "dynamic_recompute launch");
}

}  // extern "C"

namespace {
// The arguments both matchers take, checked alike; `ok_to_launch` is false
// when there is nothing to do (or an error was recorded).
semshare_status_t check_match(const char* who, const uint64_t* tgt_codes, int64_t n_tgt, const uint64_t* ref_codes,
                              int64_t n_ref, int32_t n_words, const int32_t* idx, bool* ok_to_launch) {
    *ok_to_launch = false;
    if (n_tgt < 0) return fail(SEMSHARE_E_INVAL, "%s: n_tgt < 0", who);
    if (n_words < 1 || n_words > 4) return fail(SEMSHARE_E_INVAL, "%s: n_words must be 1..4 (got %d)", who, n_words);
    if (n_ref < 1) return fail(SEMSHARE_E_INVAL, "%s: n_ref must be >= 1", who);
    if (n_ref >= (int64_t(1) << 23)) return fail(SEMSHARE_E_UNSUPPORTED, "%s: n_ref must be < 2^23", who);
    if (n_tgt > (int64_t(1) << 31) - 1024) return fail(SEMSHARE_E_UNSUPPORTED, "%s: n_tgt too large", who);
    if (n_tgt == 0) return ok();
    if (!tgt_codes || !ref_codes || !idx) return fail(SEMSHARE_E_INVAL, "%s: null buffer", who);
    *ok_to_launch = true;
    return ok();
}
}  // namespace

extern "C" {

semshare_status_t semshare_match(const uint64_t* tgt_codes, int64_t n_tgt,
                                 const uint64_t* ref_codes, int64_t n_ref, int32_t n_words,
                                 int32_t* idx, int32_t* dist, void* stream) {
    bool go;
    const semshare_status_t st = check_match("match", tgt_codes, n_tgt, ref_codes, n_ref, n_words, idx, &go);
    if (!go) return st;
    return from_hip(semshare::launch_match(tgt_codes, n_tgt, ref_codes, n_ref, n_words, idx, dist, (hipStream_t)stream),
                    "match launch");
}

semshare_status_t semshare_match_mfma(const uint64_t* tgt_codes, int64_t n_tgt,
                                      const uint64_t* ref_codes, int64_t n_ref, int32_t n_words,
                                      int32_t* idx, int32_t* dist, void* stream) {
    bool go;
    const semshare_status_t st = check_match("match_mfma", tgt_codes, n_tgt, ref_codes, n_ref, n_words, idx, &go);
    if (!go) return st;
    return from_hip(
        semshare::launch_match_mfma(tgt_codes, n_tgt, ref_codes, n_ref, n_words, idx, dist, (hipStream_t)stream),
        "match_mfma launch");
}

semshare_status_t semshare_gather_kv(const void* ref_k, const void* ref_v, const int32_t* idx,
                                     int64_t n_tgt, int64_t n_ref, void* out_k, void* out_v,
                                     int32_t n_layers, int32_t n_kv_heads, int32_t head_dim,
                                     semshare_dtype_t dtype, void* stream) {
    if (!dtype_ok(dtype)) return fail(SEMSHARE_E_INVAL, "gather_kv: unknown dtype %d", dtype);
    if (n_tgt < 0 || n_ref < 0 || n_layers < 0) return fail(SEMSHARE_E_INVAL, "gather_kv: negative size");
    if (n_kv_heads <= 0 || head_dim <= 0) return fail(SEMSHARE_E_INVAL, "gather_kv: n_kv_heads and head_dim must be > 0");
    if ((ref_v == nullptr) != (out_v == nullptr))
        return fail(SEMSHARE_E_INVAL, "gather_kv: ref_v and out_v must both be set or both be NULL");
    const int64_t row_bytes = (int64_t)n_kv_heads * head_dim * (int64_t)dtype_size(dtype);
    if (row_bytes % 16) return fail(SEMSHARE_E_UNSUPPORTED, "gather_kv: row size %lld bytes is not a multiple of 16", (long long)row_bytes);
    if ((int64_t)n_layers * n_tgt > (int64_t(1) << 30) || n_ref > (int64_t(1) << 31) - 1)
        return fail(SEMSHARE_E_UNSUPPORTED, "gather_kv: too many rows");
    if (n_tgt == 0 || n_layers == 0) return ok();
    if (!ref_k || !out_k || !idx) return fail(SEMSHARE_E_INVAL, "gather_kv: null buffer");
    if (!aligned16(ref_k) || !aligned16(out_k) || (ref_v && (!aligned16(ref_v) || !aligned16(out_v))))
        return fail(SEMSHARE_E_INVAL, "gather_kv: buffers must be 16-byte aligned");
    return from_hip(semshare::launch_gather_rows(ref_k, ref_v, idx, n_tgt, n_ref, out_k, out_v, n_layers, row_bytes,
                                                 (hipStream_t)stream),
                    "gather_kv launch");
}

semshare_status_t semshare_gather_kv_except(const void* ref_k, const void* ref_v, const int32_t* idx,
                                     int64_t n_tgt, int64_t n_ref, void* out_k, void* out_v,
                                     int32_t n_layers, int32_t n_kv_heads, int32_t head_dim,
                                     semshare_dtype_t dtype, const int32_t* except_pos,
                                            int64_t n_except, void* stream) {
    if (n_except < 0 || n_except > n_tgt || (n_except > 0 && !except_pos))
        return fail(SEMSHARE_E_INVAL, "gather_kv_except: n_except must lie in [0, n_tgt] with a list");
    if (!dtype_ok(dtype)) return fail(SEMSHARE_E_INVAL, "gather_kv_except: unknown dtype %d", dtype);
    if (n_tgt < 0 || n_ref < 0 || n_layers < 0) return fail(SEMSHARE_E_INVAL, "gather_kv_except: negative size");
    if (n_kv_heads <= 0 || head_dim <= 0) return fail(SEMSHARE_E_INVAL, "gather_kv_except: n_kv_heads and head_dim must be > 0");
    if ((ref_v == nullptr) != (out_v == nullptr))
        return fail(SEMSHARE_E_INVAL, "gather_kv_except: ref_v and out_v must both be set or both be NULL");
    const int64_t row_bytes = (int64_t)n_kv_heads * head_dim * (int64_t)dtype_size(dtype);
    if (row_bytes % 16) return fail(SEMSHARE_E_UNSUPPORTED, "gather_kv_except: row size %lld bytes is not a multiple of 16", (long long)row_bytes);
    if ((int64_t)n_layers * n_tgt > (int64_t(1) << 30) || n_ref > (int64_t(1) << 31) - 1)
        return fail(SEMSHARE_E_UNSUPPORTED, "gather_kv_except: too many rows");
    if (n_tgt == 0 || n_layers == 0) return ok();
    if (!ref_k || !out_k || !idx) return fail(SEMSHARE_E_INVAL, "gather_kv_except: null buffer");
    if (!aligned16(ref_k) || !aligned16(out_k) || (ref_v && (!aligned16(ref_v) || !aligned16(out_v))))
        return fail(SEMSHARE_E_INVAL, "gather_kv_except: buffers must be 16-byte aligned");
    return from_hip(semshare::launch_gather_rows(ref_k, ref_v, idx, n_tgt, n_ref, out_k, out_v, n_layers, row_bytes,
                                                 (hipStream_t)stream, except_pos, n_except),
                    "gather_kv_except launch");
}

}  // extern "C"

namespace {

// Shape checks shared by the partial-prefill calls.  Returns SEMSHARE_OK or
// the failing status (message already set).
semshare_status_t check_prefill_shapes(const char* fn, int64_t n_sel, int64_t n_tok, int32_t hidden,
                                       int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                       semshare_dtype_t dtype, bool need_hidden) {
    if (!dtype_ok(dtype)) return fail(SEMSHARE_E_INVAL, "%s: unknown dtype %d", fn, dtype);
    if (n_sel < 0 || n_tok < 0) return fail(SEMSHARE_E_INVAL, "%s: negative size", fn);
    if (n_sel > n_tok) return fail(SEMSHARE_E_INVAL, "%s: n_sel (%lld) > n_tok (%lld)", fn, (long long)n_sel, (long long)n_tok);
    if ((need_hidden && hidden <= 0) || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0)
        return fail(SEMSHARE_E_INVAL, "%s: sizes must be > 0", fn);
    if (n_q_heads % n_kv_heads) return fail(SEMSHARE_E_INVAL, "%s: n_q_heads %% n_kv_heads != 0", fn);
    if (head_dim & 1) return fail(SEMSHARE_E_INVAL, "%s: head_dim must be even", fn);
    if (n_tok > (int64_t(1) << 30) || (int64_t)n_kv_heads * head_dim * n_tok > (int64_t(1) << 40))
        return fail(SEMSHARE_E_UNSUPPORTED, "%s: cache too large", fn);
    const int32_t G = n_q_heads / n_kv_heads;
    if (need_hidden && hidden % 64) return fail(SEMSHARE_E_UNSUPPORTED, "%s: hidden %% 64 != 0", fn);
    if (dtype == SEMSHARE_BF16) {
        if (head_dim != 128 && head_dim != 64)
            return fail(SEMSHARE_E_UNSUPPORTED, "%s: bf16 supports head_dim 64 or 128 (got %d)", fn, head_dim);
        if (128 % G) return fail(SEMSHARE_E_UNSUPPORTED, "%s: bf16 needs 128 %% (n_q_heads/n_kv_heads) == 0", fn);
        if (((int64_t)n_kv_heads * head_dim) % 128)
            return fail(SEMSHARE_E_UNSUPPORTED, "%s: bf16 needs n_kv_heads*head_dim %% 128 == 0", fn);
        // the projection addresses its operands by 32-bit byte offsets
        if (need_hidden && (2 * n_sel * hidden >= (int64_t(1) << 31) ||
                            2 * (int64_t)n_q_heads * head_dim * hidden >= (int64_t(1) << 31)))
            return fail(SEMSHARE_E_UNSUPPORTED, "%s: bf16 x_sel or a weight matrix of 2 GiB or more", fn);
    } else {
        if (head_dim > 128) return fail(SEMSHARE_E_UNSUPPORTED, "%s: fp32 supports head_dim <= 128", fn);
        if (n_tok > 8192) return fail(SEMSHARE_E_UNSUPPORTED, "%s: fp32 path supports n_tok <= 8192", fn);
    }
    return SEMSHARE_OK;
}

struct PrefillLayout {
    size_t off_q, off_qkv, off_attn, total;
};

PrefillLayout prefill_layout(int64_t n_sel, int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                             int32_t head_dim, semshare_dtype_t dtype) {
    auto a256 = [](size_t x) { return (x + 255) & ~size_t(255); };
    PrefillLayout l{};
    l.off_q = 0;
    l.off_qkv = a256((size_t)n_sel * n_q_heads * head_dim * dtype_size(dtype));
    l.off_attn = l.off_qkv + semshare::qkv_workspace_bytes(n_sel, n_q_heads, n_kv_heads, head_dim, dtype);
    l.total = l.off_attn + semshare::plan_attention(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype).total;
    return l;
}

semshare_status_t check_workspace(const char* fn, const void* ws, size_t have, size_t need) {
    if (need == 0) return SEMSHARE_OK;
    if (!ws || have < need)
        return fail(SEMSHARE_E_INVAL, "%s: workspace of %zu bytes is smaller than the %zu required", fn, have, need);
    if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(SEMSHARE_E_INVAL, "%s: workspace not 256-byte aligned", fn);
    return SEMSHARE_OK;
}

// plan argument of prefill_attention_impl: make the plan in the workspace
const void* const PLAN_IN_WORKSPACE = reinterpret_cast<const void*>(uintptr_t(1));

float default_scale(float sm_scale, int32_t head_dim) {
    return sm_scale > 0.0f ? sm_scale : (float)(1.0 / std::sqrt((double)head_dim));
}

}  // namespace

extern "C" {

size_t semshare_qkv_rope_workspace(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                   semshare_dtype_t dtype) {
    if (!dtype_ok(dtype) || n_sel < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0) return 0;
    return semshare::qkv_workspace_bytes(n_sel, n_q_heads, n_kv_heads, head_dim, dtype);
}

size_t semshare_prefill_attention_workspace(int64_t n_sel, int64_t n_tok, int32_t n_q_heads,
                                            int32_t n_kv_heads, int32_t head_dim, semshare_dtype_t dtype) {
    if (!dtype_ok(dtype) || n_sel < 0 || n_tok < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0 ||
        n_q_heads % n_kv_heads)
        return 0;
    return semshare::plan_attention(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype).total;
}

size_t semshare_partial_prefill_workspace(int64_t n_sel, int64_t n_tok, int32_t hidden,
                                          int32_t n_q_heads, int32_t n_kv_heads,
                                          int32_t head_dim, semshare_dtype_t dtype) {
    if (!dtype_ok(dtype) || n_sel < 0 || n_tok < 0 || hidden <= 0 || n_q_heads <= 0 || n_kv_heads <= 0 ||
        head_dim <= 0 || n_q_heads % n_kv_heads)
        return 0;
    return prefill_layout(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype).total;
}

namespace {
// rope_table == nullptr: semshare_qkv_rope (the table is made in the workspace)
struct DevRef {  // the first-layer deviation source of semshare_qkv_rope_dev_ref
    const void* k;
    const void* v;
    const int32_t* idx;
    int64_t n_ref;
};

semshare_status_t qkv_rope_impl(const char* fn, const void* rope_table, size_t rope_table_bytes, const void* x_sel,
                                const int32_t* sel_pos, int64_t n_sel, const void* wq, const void* wk,
                                const void* wv, void* k_cache, void* v_cache, int64_t n_tok, int32_t hidden,
                                int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, double rope_base,
                                void* q_out, float* deviation_out, void* workspace, size_t workspace_bytes,
                                semshare_dtype_t dtype, void* stream, const DevRef* ref = nullptr,
                                const int32_t* x_rows = nullptr, int64_t n_x = 0) {
    semshare_status_t st = check_prefill_shapes(fn, n_sel, n_tok, hidden, n_q_heads, n_kv_heads, head_dim, dtype, true);
    if (st != SEMSHARE_OK) return st;
    if (!(rope_base > 0.0) || !std::isfinite(rope_base)) return fail(SEMSHARE_E_INVAL, "%s: rope_base must be finite and > 0", fn);
    if (n_sel == 0) return ok();
    if (!x_sel || !sel_pos || !wk || !wv || !k_cache || !v_cache) return fail(SEMSHARE_E_INVAL, "%s: null buffer", fn);
    if (q_out && !wq) return fail(SEMSHARE_E_INVAL, "%s: wq is NULL but q_out is requested", fn);
    if (!aligned16(x_sel) || !aligned16(wk) || !aligned16(wv) || !aligned16(k_cache) || !aligned16(v_cache) ||
        (q_out && (!aligned16(wq) || !aligned16(q_out))))
        return fail(SEMSHARE_E_INVAL, "%s: buffers must be 16-byte aligned", fn);
    st = check_workspace(fn, workspace, workspace_bytes, semshare::qkv_workspace_bytes(n_sel, n_q_heads, n_kv_heads, head_dim, dtype));
    if (st != SEMSHARE_OK) return st;
    semshare::QkvArgs a{x_sel, sel_pos, n_sel, wq, wk, wv, k_cache, v_cache, n_tok, hidden, n_q_heads,
                        n_kv_heads, head_dim, rope_base, q_out, deviation_out, workspace};
    if (x_rows) {
        if (dtype != SEMSHARE_BF16) return fail(SEMSHARE_E_UNSUPPORTED, "%s: bf16 only", fn);
        if (n_x <= 0) return fail(SEMSHARE_E_INVAL, "%s: n_x must be > 0", fn);
        if (2 * n_x * hidden >= (int64_t(1) << 31))
            return fail(SEMSHARE_E_UNSUPPORTED, "%s: bf16 x of 2 GiB or more", fn);
        a.x_rows = x_rows;
        a.n_x = n_x;
    }
    if (rope_table) {
        if (dtype != SEMSHARE_BF16) return fail(SEMSHARE_E_UNSUPPORTED, "%s: the RoPE table is for bf16 only", fn);
        if (!aligned16(rope_table)) return fail(SEMSHARE_E_INVAL, "%s: rope_table must be 16-byte aligned", fn);
        if (rope_table_bytes < semshare_rope_table_bytes(n_sel, head_dim))
            return fail(SEMSHARE_E_INVAL, "%s: rope_table of %zu bytes, %zu needed", fn, rope_table_bytes,
                        semshare_rope_table_bytes(n_sel, head_dim));
        a.rope_table = rope_table;
    }
    if (ref) {
        if (dtype != SEMSHARE_BF16) return fail(SEMSHARE_E_UNSUPPORTED, "%s: bf16 only", fn);
        if (!deviation_out || !ref->k || !ref->v || !ref->idx)
            return fail(SEMSHARE_E_INVAL, "%s: deviation_out, ref_k, ref_v and idx are required", fn);
        if (ref->n_ref < 0 || ref->n_ref > (int64_t(1) << 31) - 1) return fail(SEMSHARE_E_INVAL, "%s: n_ref out of range", fn);
        if (!aligned16(ref->k) || !aligned16(ref->v)) return fail(SEMSHARE_E_INVAL, "%s: ref_k and ref_v must be 16-byte aligned", fn);
        a.ref_k = ref->k;
        a.ref_v = ref->v;
        a.ref_idx = ref->idx;
        a.ref_n = ref->n_ref;
    }
    hipError_t e = dtype == SEMSHARE_BF16 ? semshare::launch_qkv_bf16(a, (hipStream_t)stream)
                                          : semshare::launch_qkv_f32(a, (hipStream_t)stream);
    return from_hip(e, "qkv_rope launch");
}
}  // namespace

semshare_status_t semshare_qkv_rope(const void* x_sel, const int32_t* sel_pos, int64_t n_sel,
                                    const void* wq, const void* wk, const void* wv, void* k_cache,
                                    void* v_cache, int64_t n_tok, int32_t hidden, int32_t n_q_heads,
                                    int32_t n_kv_heads, int32_t head_dim, double rope_base, void* q_out,
                                    float* deviation_out, void* workspace, size_t workspace_bytes,
                                    semshare_dtype_t dtype, void* stream) {
    return qkv_rope_impl("qkv_rope", nullptr, 0, x_sel, sel_pos, n_sel, wq, wk, wv, k_cache, v_cache, n_tok, hidden,
                         n_q_heads, n_kv_heads, head_dim, rope_base, q_out, deviation_out, workspace,
                         workspace_bytes, dtype, stream);
}

semshare_status_t semshare_qkv_rope_dev_ref(const void* x_sel, const int32_t* sel_pos, int64_t n_sel, const void* wq,
                                            const void* wk, const void* wv, void* k_cache, void* v_cache, int64_t n_tok,
                                            int32_t hidden, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                            double rope_base, void* q_out, float* deviation_out, const void* ref_k,
                                            const void* ref_v, const int32_t* idx, int64_t n_ref, void* workspace,
                                            size_t workspace_bytes, semshare_dtype_t dtype, void* stream) {
    const DevRef ref{ref_k, ref_v, idx, n_ref};
    return qkv_rope_impl("qkv_rope_dev_ref", nullptr, 0, x_sel, sel_pos, n_sel, wq, wk, wv, k_cache, v_cache, n_tok,
                         hidden, n_q_heads, n_kv_heads, head_dim, rope_base, q_out, deviation_out, workspace,
                         workspace_bytes, dtype, stream, &ref);
}

size_t semshare_rope_table_bytes(int64_t n_sel, int32_t head_dim) {
    if (n_sel <= 0 || head_dim <= 0 || (head_dim & 1)) return 0;
    return (size_t)n_sel * (size_t)(head_dim / 2) * 2 * sizeof(float);
}

semshare_status_t semshare_rope_table(const int32_t* sel_pos, int64_t n_sel, int64_t n_tok, int32_t head_dim,
                                      double rope_base, void* table, size_t table_bytes, void* stream) {
    const char* fn = "rope_table";
    if (n_sel < 0 || n_tok < 0) return fail(SEMSHARE_E_INVAL, "%s: negative size", fn);
    if (head_dim <= 0 || (head_dim & 1)) return fail(SEMSHARE_E_INVAL, "%s: head_dim must be even and > 0", fn);
    if (!(rope_base > 0.0) || !std::isfinite(rope_base)) return fail(SEMSHARE_E_INVAL, "%s: rope_base must be finite and > 0", fn);
    if (n_sel == 0) return ok();
    if (!sel_pos || !table) return fail(SEMSHARE_E_INVAL, "%s: null buffer", fn);
    if (!aligned16(table)) return fail(SEMSHARE_E_INVAL, "%s: table must be 16-byte aligned", fn);
    if (table_bytes < semshare_rope_table_bytes(n_sel, head_dim))
        return fail(SEMSHARE_E_INVAL, "%s: table of %zu bytes, %zu needed", fn, table_bytes,
                    semshare_rope_table_bytes(n_sel, head_dim));
    return from_hip(semshare::launch_rope_table(sel_pos, n_sel, n_tok, head_dim, rope_base, table, (hipStream_t)stream),
                    "rope_table launch");
}

semshare_status_t semshare_qkv_rope_tabled(const void* rope_table, size_t rope_table_bytes, const void* x_sel,
                                           const int32_t* sel_pos, int64_t n_sel, const void* wq, const void* wk,
                                           const void* wv, void* k_cache, void* v_cache, int64_t n_tok,
                                           int32_t hidden, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                           void* q_out, float* deviation_out, void* workspace,
                                           size_t workspace_bytes, semshare_dtype_t dtype, void* stream) {
    const char* fn = "qkv_rope_tabled";
    if (!rope_table && n_sel > 0) return fail(SEMSHARE_E_INVAL, "%s: null rope_table", fn);
    // rope_base only passes the shared checks: the table holds the factors
    return qkv_rope_impl(fn, rope_table, rope_table_bytes, x_sel, sel_pos, n_sel, wq, wk, wv, k_cache, v_cache,
                         n_tok, hidden, n_q_heads, n_kv_heads, head_dim, 10000.0, q_out, deviation_out, workspace,
                         workspace_bytes, dtype, stream);
}

semshare_status_t semshare_qkv_rope_tabled_rows(const void* rope_table, size_t rope_table_bytes, const void* x,
                                                int64_t n_x, const int32_t* x_rows, const int32_t* sel_pos,
                                                int64_t n_sel, const void* wq, const void* wk, const void* wv,
                                                void* k_cache, void* v_cache, int64_t n_tok, int32_t hidden,
                                                int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, void* q_out,
                                                float* deviation_out, void* workspace, size_t workspace_bytes,
                                                semshare_dtype_t dtype, void* stream) {
    const char* fn = "qkv_rope_tabled_rows";
    if (n_x < 0) return fail(SEMSHARE_E_INVAL, "%s: negative n_x", fn);
    if (n_sel > 0 && (!rope_table || !x_rows)) return fail(SEMSHARE_E_INVAL, "%s: null rope_table or x_rows", fn);
    return qkv_rope_impl(fn, rope_table, rope_table_bytes, x, sel_pos, n_sel, wq, wk, wv, k_cache, v_cache, n_tok,
                         hidden, n_q_heads, n_kv_heads, head_dim, 10000.0, q_out, deviation_out, workspace,
                         workspace_bytes, dtype, stream, nullptr, x_rows, n_x);
}

namespace {
semshare_status_t prefill_attention_impl(const char* fn, const void* plan_buf, size_t plan_bytes, const void* q,
                                          const int32_t* sel_pos, int64_t n_sel, const void* k_cache,
                                          const void* v_cache, int64_t n_tok, int32_t n_q_heads,
                                          int32_t n_kv_heads, int32_t head_dim, float sm_scale, void* out,
                                          void* workspace, size_t workspace_bytes, semshare_dtype_t dtype,
                                          void* stream) {
    semshare_status_t st = check_prefill_shapes(fn, n_sel, n_tok, 0, n_q_heads, n_kv_heads, head_dim, dtype, false);
    if (st != SEMSHARE_OK) return st;
    if (!(sm_scale >= 0.0f) || !std::isfinite(sm_scale)) return fail(SEMSHARE_E_INVAL, "%s: sm_scale must be finite and >= 0", fn);
    if (n_sel == 0) return ok();
    if (!q || !sel_pos || !k_cache || !v_cache || !out) return fail(SEMSHARE_E_INVAL, "%s: null buffer", fn);
    if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
        return fail(SEMSHARE_E_INVAL, "%s: buffers must be 16-byte aligned", fn);
    const semshare::AttnPlan plan = semshare::plan_attention(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype);
    st = check_workspace(fn, workspace, workspace_bytes, plan.total);
    if (st != SEMSHARE_OK) return st;
    if (plan_buf == PLAN_IN_WORKSPACE) {
        plan_buf = nullptr;
    } else if (plan.plan_bytes > 0) {
        if (!plan_buf || plan_bytes < plan.plan_bytes)
            return fail(SEMSHARE_E_INVAL, "%s: plan of %zu bytes is smaller than the %zu required", fn, plan_bytes,
                        plan.plan_bytes);
        if (reinterpret_cast<uintptr_t>(plan_buf) % 256) return fail(SEMSHARE_E_INVAL, "%s: plan not 256-byte aligned", fn);
    }
    const semshare::AttnCall a{q, sel_pos, n_sel, k_cache, v_cache, n_tok, n_q_heads, n_kv_heads, head_dim,
                               default_scale(sm_scale, head_dim), out, workspace, plan_buf};
    hipError_t e = dtype == SEMSHARE_BF16 ? semshare::launch_attention_bf16(a, plan, (hipStream_t)stream)
                                          : semshare::launch_attention_f32(a, plan, (hipStream_t)stream);
    return from_hip(e, "prefill_attention launch");
}
}  // namespace

semshare_status_t semshare_prefill_attention(const void* q, const int32_t* sel_pos, int64_t n_sel,
                                             const void* k_cache, const void* v_cache, int64_t n_tok,
                                             int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                             float sm_scale, void* out, void* workspace,
                                             size_t workspace_bytes, semshare_dtype_t dtype, void* stream) {
    return prefill_attention_impl("prefill_attention", PLAN_IN_WORKSPACE, 0, q, sel_pos, n_sel, k_cache, v_cache,
                                  n_tok, n_q_heads, n_kv_heads, head_dim, sm_scale, out, workspace, workspace_bytes,
                                  dtype, stream);
}

semshare_status_t semshare_prefill_attention_noalloc(const void* q, const int32_t* sel_pos, int64_t n_sel,
                                                     const void* k_cache, const void* v_cache, int64_t n_tok,
                                                     int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                     float sm_scale, void* out, semshare_dtype_t dtype, void* stream) {
    const char* fn = "prefill_attention_noalloc";
    semshare_status_t st = check_prefill_shapes(fn, n_sel, n_tok, 0, n_q_heads, n_kv_heads, head_dim, dtype, false);
    if (st != SEMSHARE_OK) return st;
    // the argument checks of semshare_prefill_attention come first, so that a
    // bad call is rejected before the device is touched
    if (!(sm_scale >= 0.0f) || !std::isfinite(sm_scale)) return fail(SEMSHARE_E_INVAL, "%s: sm_scale must be finite and >= 0", fn);
    if (n_sel == 0) return ok();
    if (!q || !sel_pos || !k_cache || !v_cache || !out) return fail(SEMSHARE_E_INVAL, "%s: null buffer", fn);
    if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
        return fail(SEMSHARE_E_INVAL, "%s: buffers must be 16-byte aligned", fn);
    const size_t need = semshare::plan_attention(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype).total;
    if (need > semshare::kAttnScratchBytes)
        return fail(SEMSHARE_E_UNSUPPORTED,
                    "%s: these sizes need %zu bytes of scratch, more than the %zu bytes of the library's static "
                    "scratch; use semshare_prefill_attention with a workspace",
                    fn, need, semshare::kAttnScratchBytes);
    if (need == 0)  // the fp32 path uses no scratch
        return prefill_attention_impl(fn, PLAN_IN_WORKSPACE, 0, q, sel_pos, n_sel, k_cache, v_cache, n_tok, n_q_heads,
                                      n_kv_heads, head_dim, sm_scale, out, nullptr, 0, dtype, stream);
    void* ws = nullptr;
    const hipError_t e = semshare::attention_scratch(&ws);
    if (e != hipSuccess) return from_hip(e, "prefill_attention_noalloc: scratch address");
    return prefill_attention_impl(fn, PLAN_IN_WORKSPACE, 0, q, sel_pos, n_sel, k_cache, v_cache, n_tok, n_q_heads,
                                  n_kv_heads, head_dim, sm_scale, out, ws, semshare::kAttnScratchBytes, dtype, stream);
}

size_t semshare_attention_plan_bytes(int64_t n_sel, int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                                     int32_t head_dim, semshare_dtype_t dtype) {
    if (!dtype_ok(dtype) || n_sel < 0 || n_tok < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || head_dim <= 0 ||
        n_q_heads % n_kv_heads)
        return 0;
    return semshare::plan_attention(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype).plan_bytes;
}

semshare_status_t semshare_attention_plan(const int32_t* sel_pos, int64_t n_sel, int64_t n_tok, int32_t n_q_heads,
                                          int32_t n_kv_heads, int32_t head_dim, semshare_dtype_t dtype, void* plan,
                                          size_t plan_bytes, void* stream) {
    const char* fn = "attention_plan";
    semshare_status_t st = check_prefill_shapes(fn, n_sel, n_tok, 0, n_q_heads, n_kv_heads, head_dim, dtype, false);
    if (st != SEMSHARE_OK) return st;
    const semshare::AttnPlan p = semshare::plan_attention(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype);
    if (p.plan_bytes == 0) return ok();  // nothing to plan (no rows, or the fp32 path)
    if (!sel_pos) return fail(SEMSHARE_E_INVAL, "%s: null buffer", fn);
    if (!plan || plan_bytes < p.plan_bytes)
        return fail(SEMSHARE_E_INVAL, "%s: plan of %zu bytes is smaller than the %zu required", fn, plan_bytes,
                    p.plan_bytes);
    if (reinterpret_cast<uintptr_t>(plan) % 256) return fail(SEMSHARE_E_INVAL, "%s: plan not 256-byte aligned", fn);
    const semshare::AttnCall a{nullptr, sel_pos, n_sel, nullptr, nullptr, n_tok, n_q_heads, n_kv_heads, head_dim,
                               0.0f, nullptr, nullptr, nullptr};
    return from_hip(semshare::launch_attention_plan_bf16(a, p, plan, (hipStream_t)stream), "attention_plan launch");
}

semshare_status_t semshare_prefill_attention_planned(const void* plan, size_t plan_bytes, const void* q,
                                                     const int32_t* sel_pos, int64_t n_sel, const void* k_cache,
                                                     const void* v_cache, int64_t n_tok, int32_t n_q_heads,
                                                     int32_t n_kv_heads, int32_t head_dim, float sm_scale, void* out,
                                                     void* workspace, size_t workspace_bytes,
                                                     semshare_dtype_t dtype, void* stream) {
    return prefill_attention_impl("prefill_attention_planned", plan, plan_bytes, q, sel_pos, n_sel, k_cache,
                                  v_cache, n_tok, n_q_heads, n_kv_heads, head_dim, sm_scale, out, workspace,
                                  workspace_bytes, dtype, stream);
}

semshare_status_t semshare_partial_prefill(
    const void* x_sel, const int32_t* sel_pos, int64_t n_sel, const void* wq, const void* wk,
    const void* wv, void* k_cache, void* v_cache, int64_t n_tok, int32_t hidden,
    int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, double rope_base, float sm_scale,
    void* out, float* deviation_out, void* workspace, size_t workspace_bytes,
    semshare_dtype_t dtype, void* stream) {
    const char* fn = "partial_prefill";
    semshare_status_t st = check_prefill_shapes(fn, n_sel, n_tok, hidden, n_q_heads, n_kv_heads, head_dim, dtype, true);
    if (st != SEMSHARE_OK) return st;
    if (!(rope_base > 0.0) || !std::isfinite(rope_base)) return fail(SEMSHARE_E_INVAL, "%s: rope_base must be finite and > 0", fn);
    if (!(sm_scale >= 0.0f) || !std::isfinite(sm_scale)) return fail(SEMSHARE_E_INVAL, "%s: sm_scale must be finite and >= 0", fn);
    if (n_sel == 0) return ok();
    if (!x_sel || !sel_pos || !wk || !wv || !k_cache || !v_cache) return fail(SEMSHARE_E_INVAL, "%s: null buffer", fn);
    if (out && !wq) return fail(SEMSHARE_E_INVAL, "%s: wq is NULL but out is requested", fn);
    if (!aligned16(x_sel) || !aligned16(wk) || !aligned16(wv) || !aligned16(k_cache) || !aligned16(v_cache) ||
        (out && (!aligned16(wq) || !aligned16(out))))
        return fail(SEMSHARE_E_INVAL, "%s: buffers must be 16-byte aligned", fn);
    const PrefillLayout lay = prefill_layout(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype);
    st = check_workspace(fn, workspace, workspace_bytes, lay.total);
    if (st != SEMSHARE_OK) return st;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    void* q_ws = out ? ws + lay.off_q : nullptr;
    const semshare::QkvArgs qa{x_sel, sel_pos, n_sel, wq, wk, wv, k_cache, v_cache, n_tok, hidden, n_q_heads,
                               n_kv_heads, head_dim, rope_base, q_ws, deviation_out, ws + lay.off_qkv};
    hipError_t e = dtype == SEMSHARE_BF16 ? semshare::launch_qkv_bf16(qa, (hipStream_t)stream)
                                          : semshare::launch_qkv_f32(qa, (hipStream_t)stream);
    if (e != hipSuccess || !out) return from_hip(e, "partial_prefill launch");
    const semshare::AttnPlan plan = semshare::plan_attention(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype);
    const semshare::AttnCall aa{q_ws, sel_pos, n_sel, k_cache, v_cache, n_tok, n_q_heads, n_kv_heads, head_dim,
                                default_scale(sm_scale, head_dim), out, ws + lay.off_attn, nullptr};
    e = dtype == SEMSHARE_BF16 ? semshare::launch_attention_bf16(aa, plan, (hipStream_t)stream)
                               : semshare::launch_attention_f32(aa, plan, (hipStream_t)stream);
    return from_hip(e, "partial_prefill launch");
}

semshare_status_t semshare_select_recompute(const float* sigma, int64_t n_tok, int64_t n_sel,
                                            int32_t* sel_pos, void* stream) {
    if (n_tok < 0 || n_sel < 0 || n_sel > n_tok)
        return fail(SEMSHARE_E_INVAL, "select_recompute: need 0 <= n_sel <= n_tok");
    if (n_tok > (int64_t(1) << 20)) return fail(SEMSHARE_E_UNSUPPORTED, "select_recompute: n_tok must be <= 2^20");
    if (n_sel == 0) return ok();
    if (!sigma || !sel_pos) return fail(SEMSHARE_E_INVAL, "select_recompute: null buffer");
    return from_hip(semshare::launch_select_recompute(sigma, n_tok, n_sel, sel_pos, (hipStream_t)stream),
                    "select_recompute launch");
}

semshare_status_t semshare_select_recompute_nested(const float* sigma, const int32_t* cand_pos, int64_t n_cand,
                                                   int64_t n_sel, int32_t* sel_pos, void* stream) {
    if (n_cand < 0 || n_sel < 0 || n_sel > n_cand)
        return fail(SEMSHARE_E_INVAL, "select_recompute_nested: need 0 <= n_sel <= n_cand");
    if (n_cand > (int64_t(1) << 20)) return fail(SEMSHARE_E_UNSUPPORTED, "select_recompute_nested: n_cand must be <= 2^20");
    if (n_sel == 0) return ok();
    if (!sigma || !cand_pos || !sel_pos) return fail(SEMSHARE_E_INVAL, "select_recompute_nested: null buffer");
    return from_hip(semshare::launch_select_recompute(sigma, n_cand, n_sel, sel_pos, (hipStream_t)stream, cand_pos),
                    "select_recompute_nested launch");
}

size_t semshare_bank_similarity_workspace(int64_t n_tgt, int32_t n_prompts) {
    if (n_tgt <= 0 || n_prompts <= 0) return 0;
    return semshare::bank_similarity_workspace(n_tgt, n_prompts);
}

semshare_status_t semshare_bank_similarity(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                                           const int64_t* ref_offsets, int32_t n_prompts, int32_t n_words,
                                           double dmin, double dmax, int64_t* dist_sum, double* similarity,
                                           void* workspace, size_t workspace_bytes, void* stream) {
    const char* fn = "bank_similarity";
    if (n_tgt < 0 || n_ref < 0 || n_prompts < 0) return fail(SEMSHARE_E_INVAL, "%s: negative size", fn);
    if (n_words < 1 || n_words > 4) return fail(SEMSHARE_E_INVAL, "%s: n_words must be 1..4 (got %d)", fn, n_words);
    if (n_prompts > 65535) return fail(SEMSHARE_E_UNSUPPORTED, "%s: n_prompts must be <= 65535", fn);
    if (n_tgt > (int64_t(1) << 31) - 256) return fail(SEMSHARE_E_UNSUPPORTED, "%s: n_tgt too large", fn);
    if (!std::isfinite(dmin) || !std::isfinite(dmax) || !(dmax > dmin))
        return fail(SEMSHARE_E_INVAL, "%s: need finite dmin < dmax", fn);
    if (n_prompts == 0) return ok();
    if (!ref_offsets || !dist_sum || !similarity || (n_tgt > 0 && !tgt) || (n_ref > 0 && !ref))
        return fail(SEMSHARE_E_INVAL, "%s: null buffer", fn);
    const size_t need = semshare_bank_similarity_workspace(n_tgt, n_prompts);
    if (workspace_bytes < need || (need > 0 && (!workspace || reinterpret_cast<uintptr_t>(workspace) % 8)))
        return fail(SEMSHARE_E_INVAL, "%s: workspace of %zu bytes (8-byte aligned) needed, %zu given", fn, need,
                    workspace_bytes);
    return from_hip(semshare::launch_bank_similarity(tgt, n_tgt, ref, n_ref, ref_offsets, n_prompts, n_words, dmin,
                                                     dmax, dist_sum, similarity, workspace, (hipStream_t)stream),
                    "bank_similarity launch");
}

}  // extern "C"
