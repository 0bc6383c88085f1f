/*
 * semshare.h -- C ABI of libsemshare.so, the MI355X (gfx950) hot path of
 * SemShareKV: fuzzy token matching and KV reuse for one target prompt
 * against a cached reference prompt (Zhao & Mastorakis, "SemShareKV:
 * Efficient KVCache Sharing for Semantically Similar Prompts via Token-Level
 * LSH Matching", arXiv 2509.24832).
 *
 * Common contract of every call
 *  - Buffer pointers are DEVICE pointers owned by the caller.  The library
 *    never allocates, frees or keeps them after the call returns.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued
 *    asynchronously on it; no call synchronizes the device.
 *  - Arguments are validated on the host before anything is enqueued.  On a
 *    bad argument the call returns SEMSHARE_E_INVAL (or
 *    SEMSHARE_E_UNSUPPORTED for a valid shape this build has no kernel for)
 *    and enqueues nothing.  SEMSHARE_E_DEVICE reports a HIP launch error.
 *    semshare_last_error() then returns a message (thread-local).
 *  - Layouts are row-major and dense.  "dtype" is the storage type of the
 *    floating-point buffers of the call; arithmetic accumulates in fp32.
 *  - Buffers are aligned to their element size; the LSH, gather and
 *    partial-prefill calls also need 16-byte aligned buffers (as any
 *    allocator returns) and reject others with SEMSHARE_E_INVAL.
 *  - A call with an empty problem (zero tokens) succeeds and enqueues
 *    nothing.
 */
#ifndef SEMSHARE_H
#define SEMSHARE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t semshare_status_t;
enum {
    SEMSHARE_OK = 0,
    SEMSHARE_E_INVAL = -1,
    SEMSHARE_E_UNSUPPORTED = -2,
    SEMSHARE_E_DEVICE = -3
};

typedef int32_t semshare_dtype_t;
enum { SEMSHARE_FP32 = 0, SEMSHARE_BF16 = 1 };

/* Message describing the last failed call on this thread ("" if none). */
const char* semshare_last_error(void);

/* ABI version: major * 10000 + minor * 100 + patch. */
int32_t semshare_version(void);

/*
 * RoPE injected into token embeddings (Section 4.3.1; Appendix A.1 Eq. 1,
 * read as the standard rotary embedding): the row at position m has every
 * pair (x[2k], x[2k+1]) rotated by the angle m * theta_k with
 * theta_k = base^(-2k/dim), k = 0 .. dim/2-1.  Row r of x sits at position
 * pos0 + r.  Angles are formed in fp64, reduced modulo 2*pi, then rotated in
 * fp32 and rounded to `dtype`.
 *   x, y   [n_tok][dim] dtype.  y may equal x (in place); no other overlap.
 *   dim    even, > 0.   base > 0.   pos0 >= 0.
 */
semshare_status_t semshare_rope_embed(const void* x, void* y, int64_t n_tok, int32_t dim,
                                      int64_t pos0, double base, semshare_dtype_t dtype,
                                      void* stream);

/*
 * Random-hyperplane LSH of embeddings (Section 4.3 and Appendix A.2; the
 * sign-bit family of the FAISS LSH index the implementation uses, Appendix D):
 * bit j of row t is 1 iff <x_t, planes_j> > 0, computed with fp32
 * accumulation of exact bf16/fp32 products.  Bit j is stored at bit (j % 64)
 * of word j / 64.
 *   x       [n_tok][dim] dtype
 *   planes  [n_bits][dim] dtype (row j = hyperplane j)
 *   codes   [n_tok][n_bits / 64] uint64 (output)
 *   n_bits  64, 128 or 256.   dim: multiple of 64 (bf16) or of 4 (fp32).
 */
semshare_status_t semshare_lsh_encode(const void* x, const void* planes, uint64_t* codes,
                                      int64_t n_tok, int32_t dim, int32_t n_bits,
                                      semshare_dtype_t dtype, void* stream);

/*
 * RoPE and LSH in one pass (Section 4.3: the codes of the RoPE-embedded
 * embeddings; Appendix A.1 Eq. (1) and A.2): the codes that
 * semshare_rope_embed (row t at position pos0 + t, RoPE base `base`)
 * followed by semshare_lsh_encode give, without writing the rotated rows
 * to memory.  Each rotated pair is rounded to bf16 before the projection,
 * as the stored rows would be.
 *   x       [n_tok][dim] bf16, raw (not yet rotated) embeddings
 *   planes  [n_bits][dim] bf16;   codes [n_tok][n_bits / 64] uint64 (output)
 *   n_bits  64 or 128; 256 and fp32 return SEMSHARE_E_UNSUPPORTED.
 *   dim: multiple of 64, <= 2^20.   pos0 >= 0, pos0 + n_tok <= 2^40.
 *   Buffers 16-byte aligned.
 */
semshare_status_t semshare_rope_lsh_encode(const void* x, const void* planes, uint64_t* codes,
                                          int64_t n_tok, int32_t dim, int32_t n_bits, int64_t pos0,
                                          double base, semshare_dtype_t dtype, void* stream);

/*
 * Fuzzy token matching (Sections 4.2 and 4.3): for every target token, the
 * reference token whose LSH code is nearest in Hamming distance; on equal
 * distance the lowest reference index wins, so the answer is unique.  A
 * bank of several reference prompts is their concatenation along the token
 * axis (index b * n_per_ref + j).
 *   tgt_codes  [n_tgt][n_words] uint64;   ref_codes [n_ref][n_words] uint64
 *   n_words    1 .. 4.   n_ref in [1, 2^23).
 *   idx        [n_tgt] int32 (output): matched reference index.
 *   dist       [n_tgt] int32 (output, may be NULL): its Hamming distance.
 */
semshare_status_t semshare_match(const uint64_t* tgt_codes, int64_t n_tgt,
                                 const uint64_t* ref_codes, int64_t n_ref, int32_t n_words,
                                 int32_t* idx, int32_t* dist, void* stream);

/*
 * The same match on the matrix cores (Sections 4.2 and 4.3; same contract,
 * outputs bit-identical to semshare_match).  With the bits of a code read as
 * +-1, the dot product of two codes of n_b bits is n_b - 2 * (Hamming
 * distance), so the nearest code is the one with the largest dot product; the
 * kernel computes those with int8 MFMAs over bits expanded to bytes and keeps
 * the largest (lowest index on ties).  Arguments, limits and errors as
 * semshare_match; the library allocates nothing.
 */
semshare_status_t semshare_match_mfma(const uint64_t* tgt_codes, int64_t n_tgt,
                                      const uint64_t* ref_codes, int64_t n_ref, int32_t n_words,
                                      int32_t* idx, int32_t* dist, void* stream);

/*
 * KV rearrangement (Section 4.3; Section 4.3.2 for keeping K post-RoPE):
 * out[l][t] = ref[l][idx[t]] for every layer l, where a row is all kv heads
 * of one token (n_kv_heads * head_dim elements), copied bit for bit.  Keys
 * are not re-rotated to the target positions.
 *   ref_k, ref_v  [n_layers][n_ref][n_kv_heads][head_dim] dtype
 *   out_k, out_v  [n_layers][n_tgt][n_kv_heads][head_dim] dtype
 *   idx           [n_tgt] int32.  A row whose index lies outside [0, n_ref)
 *                 is written as zeros instead of being read.
 *   ref_v and out_v may both be NULL (gathers K only), which also serves as
 *   a plain row gather.  Row size n_kv_heads * head_dim * sizeof(dtype)
 *   must be a multiple of 16 bytes.
 */
semshare_status_t semshare_gather_kv(const void* ref_k, const void* ref_v, const int32_t* idx,
                                     int64_t n_tgt, int64_t n_ref, void* out_k, void* out_v,
                                     int32_t n_layers, int32_t n_kv_heads, int32_t head_dim,
                                     semshare_dtype_t dtype, void* stream);

/*
 * semshare_gather_kv for every target row except those listed: the rows
 * except_pos[0 .. n_except) (ascending target positions) of every layer are
 * left as they are.  Once the recompute set is known (Section 4.3.3), the
 * layers after the first need not copy the rows their partial prefill
 * overwrites.  Arguments and errors as semshare_gather_kv; 0 <= n_except <=
 * n_tgt, except_pos sorted ascending (device), may be NULL when n_except = 0.
 */
semshare_status_t semshare_gather_kv_except(const void* ref_k, const void* ref_v, const int32_t* idx,
                                            int64_t n_tgt, int64_t n_ref, void* out_k, void* out_v,
                                            int32_t n_layers, int32_t n_kv_heads, int32_t head_dim,
                                            semshare_dtype_t dtype, const int32_t* except_pos,
                                            int64_t n_except, void* stream);

/*
 * One attention layer of partial prefill (Sections 4.2 and 4.3.3): only the
 * selected tokens are recomputed, against the assembled (rearranged) cache.
 *  1. q = RoPE_p(x Wq^T), k = RoPE_p(x Wk^T) per head and v = x Wv^T for
 *     every selected row (position p = sel_pos[i]); RoPE is the standard
 *     rotation of interleaved pairs within each head (theta_k =
 *     rope_base^(-2k/head_dim)).
 *  2. If deviation_out != NULL: deviation_out[i] = ||K_cache[p] - k||_2 +
 *     ||V_cache[p] - v||_2 over the row's n_kv_heads*head_dim entries, against
 *     the row held before step 3 (KV deviation, Appendix A.4), with k and v
 *     as rounded to dtype.  The sums are formed in a fixed order, so the
 *     result is reproducible bit for bit (the order depends on n_sel and
 *     the head shape, which set the projection's tile width).
 *  3. Cache rows sel_pos[i] are overwritten with k (post-RoPE) and v.
 *  4. If out != NULL: for every selected row and query head h,
 *     out = softmax_{j <= p}(q_h . K[j][h/G] * sm_scale) V[j][h/G] over the
 *     updated cache, G = n_q_heads / n_kv_heads (grouped-query attention).
 *     out == NULL builds cache rows only (e.g. a prompt's own cache).
 *   x_sel      [n_sel][hidden] dtype: layer input of the selected tokens.
 *   sel_pos    [n_sel] int32, strictly ascending, in [0, n_tok).  Rows whose
 *              position lies outside [0, n_tok) are skipped (not written,
 *              not attended); ordering is the caller's contract.
 *   wq         [n_q_heads*head_dim][hidden] dtype (nn.Linear layout)
 *   wk, wv     [n_kv_heads*head_dim][hidden] dtype
 *   k_cache, v_cache  [n_tok][n_kv_heads][head_dim] dtype of THIS layer.
 *   sm_scale   0 means 1/sqrt(head_dim).
 *   out        [n_sel][n_q_heads][head_dim] dtype, or NULL.
 *   deviation_out  [n_sel] float32, or NULL.
 *   workspace  device scratch of at least semshare_partial_prefill_workspace()
 *              bytes, 256-byte aligned; contents on entry are ignored.
 *   Supported: hidden % 64 == 0; bf16 with head_dim 128 or 64, 128 % G == 0
 *   and n_kv_heads*head_dim % 128 == 0; fp32 with even head_dim <= 128 and
 *   n_tok <= 8192.
 */
semshare_status_t semshare_partial_prefill(
    const void* x_sel, const int32_t* sel_pos, int64_t n_sel, const void* wq, const void* wk,
    const void* wv, void* k_cache, void* v_cache, int64_t n_tok, int32_t hidden,
    int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, double rope_base, float sm_scale,
    void* out, float* deviation_out, void* workspace, size_t workspace_bytes,
    semshare_dtype_t dtype, void* stream);

/* Workspace bytes semshare_partial_prefill needs for these sizes (with an
 * attention output requested and deviation requested -- an upper bound for
 * the calls that request less).  Returns 0 for invalid sizes. */
size_t semshare_partial_prefill_workspace(int64_t n_sel, int64_t n_tok, int32_t hidden,
                                          int32_t n_q_heads, int32_t n_kv_heads,
                                          int32_t head_dim, semshare_dtype_t dtype);

/*
 * Step 1 of semshare_partial_prefill on its own (same kernels): steps 1-3
 * above -- projection, RoPE, deviation and the scatter of k/v into the
 * cache rows sel_pos -- writing the RoPE'd q to q_out instead of attending.
 *   q_out      [n_sel][n_q_heads][head_dim] dtype, or NULL (K/V only; wq may
 *              then be NULL too).
 *   workspace  at least semshare_qkv_rope_workspace() bytes, 256-byte
 *              aligned (may be NULL when that size is 0).
 *   Other arguments and limits as for semshare_partial_prefill.
 */
semshare_status_t semshare_qkv_rope(const void* x_sel, const int32_t* sel_pos, int64_t n_sel,
                                    const void* wq, const void* wk, const void* wv, void* k_cache,
                                    void* v_cache, int64_t n_tok, int32_t hidden, int32_t n_q_heads,
                                    int32_t n_kv_heads, int32_t head_dim, double rope_base,
                                    void* q_out, float* deviation_out, void* workspace,
                                    size_t workspace_bytes, semshare_dtype_t dtype, void* stream);
size_t semshare_qkv_rope_workspace(int64_t n_sel, int32_t n_q_heads, int32_t n_kv_heads,
                                   int32_t head_dim, semshare_dtype_t dtype);

/*
 * semshare_qkv_rope for the first layer, whose deviation compares each
 * recomputed row with the matched reference row directly (Section 4.2: the
 * first layer is recomputed in full and its KV deviation against the
 * rearranged reference cache picks the tokens to recompute; Appendix A.4):
 * deviation_out[i] = ||ref_k[idx[p]] - k||_2 + ||ref_v[idx[p]] - v||_2 with
 * p = sel_pos[i], i.e. against the row semshare_gather_kv would have placed
 * at p (an index outside [0, n_ref) counts as the zero row that the gather
 * writes).  When every row of the layer is recomputed, its gathered rows are
 * read by nothing but the deviation, so this call spares that layer's gather.
 * Cache rows sel_pos[i] are written as by semshare_qkv_rope; the others are
 * left as they are.  Results are bit for bit those of semshare_gather_kv of
 * this layer followed by semshare_qkv_rope with deviation.
 *   ref_k, ref_v  [n_ref][n_kv_heads][head_dim] dtype: the reference cache of
 *                 this layer (16-byte aligned; must not overlap k_cache or
 *                 v_cache).   idx [n_tok] int32: the match index.
 *   deviation_out [n_sel] float32, required.   bf16 only (fp32:
 *   SEMSHARE_E_UNSUPPORTED).  Other arguments, workspace and limits as for
 *   semshare_qkv_rope.
 */
semshare_status_t semshare_qkv_rope_dev_ref(const void* x_sel, const int32_t* sel_pos, int64_t n_sel, const void* wq,
                                            const void* wk, const void* wv, void* k_cache, void* v_cache, int64_t n_tok,
                                            int32_t hidden, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                            double rope_base, void* q_out, float* deviation_out, const void* ref_k,
                                            const void* ref_v, const int32_t* idx, int64_t n_ref, void* workspace,
                                            size_t workspace_bytes, semshare_dtype_t dtype, void* stream);

/*
 * The RoPE factor table of semshare_qkv_rope for one set of selected
 * positions, made once and reused.  RoPE (Section 4.3.3: the recomputed q
 * and k are rotated by their own positions) depends on the position and the
 * pair index only, and the same tokens are recomputed in every layer
 * (Section 4.2), so the layers of one selection can share one table.
 *   table  device buffer of at least semshare_rope_table_bytes() bytes,
 *          16-byte aligned; [n_sel][head_dim/2] float32 pairs (cos, sin) of
 *          the angle sel_pos[i] * rope_base^(-2k/head_dim), computed in
 *          float64 and rounded (positions outside [0, n_tok) use 0).
 *          Written on `stream`.  bf16 projection only.
 */
size_t semshare_rope_table_bytes(int64_t n_sel, int32_t head_dim);
semshare_status_t semshare_rope_table(const int32_t* sel_pos, int64_t n_sel, int64_t n_tok, int32_t head_dim,
                                      double rope_base, void* table, size_t table_bytes, void* stream);

/*
 * semshare_qkv_rope (bf16) with the RoPE factors from semshare_rope_table
 * (n_sel and head_dim as the table's; rope_base is the table's).  The table
 * stays owned by the caller and is only read.  With a table of the same
 * sel_pos values: the results of semshare_qkv_rope with that rope_base, bit
 * for bit.  The rows the call writes are sel_pos; the rotation is the
 * table's, so a table of the tokens' positions with sel_pos holding their
 * rows in a compacted cache (semshare_retention_layer) recomputes the tokens
 * of a layer whose cache holds the kept tokens only.  The workspace is the
 * one semshare_qkv_rope_workspace() sizes.  dtype FP32: SEMSHARE_E_UNSUPPORTED.
 */
semshare_status_t semshare_qkv_rope_tabled(const void* rope_table, size_t rope_table_bytes, const void* x_sel,
                                           const int32_t* sel_pos, int64_t n_sel, const void* wq, const void* wk,
                                           const void* wv, void* k_cache, void* v_cache, int64_t n_tok,
                                           int32_t hidden, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                           void* q_out, float* deviation_out, void* workspace,
                                           size_t workspace_bytes, semshare_dtype_t dtype, void* stream);

/*
 * semshare_qkv_rope_tabled with the selected rows read in place: input row i
 * is row x_rows[i] of x ([n_x][hidden] bf16, 16-byte aligned, under 2 GiB),
 * so the recomputed tokens' embeddings need not be gathered into a separate
 * x_sel first (Section 4.2: the recomputed tokens are a subset of the
 * target's).  Results equal gathering x_sel[i] = x[x_rows[i]] and calling
 * semshare_qkv_rope_tabled, bit for bit.  x_rows [n_sel] int32 (device);
 * entries outside [0, n_x) read row 0 or row n_x - 1 (never out of bounds).
 * dtype FP32: SEMSHARE_E_UNSUPPORTED.
 */
semshare_status_t semshare_qkv_rope_tabled_rows(const void* rope_table, size_t rope_table_bytes, const void* x,
                                                int64_t n_x, const int32_t* x_rows, const int32_t* sel_pos,
                                                int64_t n_sel, const void* wq, const void* wk, const void* wv,
                                                void* k_cache, void* v_cache, int64_t n_tok, int32_t hidden,
                                                int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, void* q_out,
                                                float* deviation_out, void* workspace, size_t workspace_bytes,
                                                semshare_dtype_t dtype, void* stream);

/*
 * Step 2 of semshare_partial_prefill on its own (same kernels): causal
 * grouped-query attention of the selected rows over the cache (step 4
 * above), for q as semshare_qkv_rope writes it.  Keys j <= sel_pos[i] of kv
 * head h / G are attended; rows with a position outside [0, n_tok) are not
 * written.
 *   q          [n_sel][n_q_heads][head_dim] dtype (RoPE'd)
 *   out        [n_sel][n_q_heads][head_dim] dtype
 *   workspace  at least semshare_prefill_attention_workspace() bytes,
 *              256-byte aligned (split-KV partial results; may be NULL when
 *              that size is 0).
 */
semshare_status_t semshare_prefill_attention(const void* q, const int32_t* sel_pos, int64_t n_sel,
                                             const void* k_cache, const void* v_cache,
                                             int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                                             int32_t head_dim, float sm_scale, void* out,
                                             void* workspace, size_t workspace_bytes,
                                             semshare_dtype_t dtype, void* stream);
size_t semshare_prefill_attention_workspace(int64_t n_sel, int64_t n_tok, int32_t n_q_heads,
                                            int32_t n_kv_heads, int32_t head_dim,
                                            semshare_dtype_t dtype);

/*
 * semshare_prefill_attention for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same kernels and results, bit for bit, with no workspace
 * argument.  The work plan and the partial results of cut row tiles live in a
 * static device array of the library, 40 MiB per GPU, held from the
 * library's first use on that GPU until the process ends; this call
 * allocates nothing.  Sizes whose workspace
 * (semshare_prefill_attention_workspace) exceeds 40 MiB return
 * SEMSHARE_E_UNSUPPORTED (with 8 kv heads and head_dim 128 the need is about
 * 34 MiB whatever n_tok, so every size the other call takes fits).  The
 * array is shared by every call on the same GPU and keeps the last call's
 * contents (nothing in it needs to start at zero): calls that overlap on one
 * GPU, from several streams or threads, race and must be serialised by the
 * caller.  Arguments, limits and errors otherwise as
 * semshare_prefill_attention.
 */
semshare_status_t semshare_prefill_attention_noalloc(const void* q, const int32_t* sel_pos, int64_t n_sel,
                                                     const void* k_cache, const void* v_cache, int64_t n_tok,
                                                     int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                     float sm_scale, void* out, semshare_dtype_t dtype, void* stream);

/*
 * The work plan of semshare_prefill_attention for one set of selected
 * positions, made once and reused.  The selection is made once per prompt
 * (Section 4.2: the same high-deviation tokens are recomputed in every layer
 * after the first), so every later layer's attention can share one plan
 * instead of making its own.  The plan depends on sel_pos (its values),
 * n_sel, n_tok, n_q_heads, n_kv_heads, head_dim and dtype only.
 *   plan   device buffer of at least semshare_attention_plan_bytes() bytes,
 *          256-byte aligned; written on `stream`.  0 bytes (nothing to do)
 *          for dtype FP32 or n_sel == 0.
 */
size_t semshare_attention_plan_bytes(int64_t n_sel, int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                                     int32_t head_dim, semshare_dtype_t dtype);
semshare_status_t semshare_attention_plan(const int32_t* sel_pos, int64_t n_sel, int64_t n_tok,
                                          int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                          semshare_dtype_t dtype, void* plan, size_t plan_bytes,
                                          void* stream);

/*
 * semshare_prefill_attention with a plan from semshare_attention_plan (same
 * sel_pos values and sizes; the buffer stays owned by the caller and is only
 * read).  Same results as semshare_prefill_attention, bit for bit.  A plan
 * made for other sizes is detected on the device and nothing is written; a
 * plan made for other positions of the same sizes gives wrong results.  The
 * workspace is the one semshare_prefill_attention_workspace() sizes.
 */
semshare_status_t semshare_prefill_attention_planned(const void* plan, size_t plan_bytes, const void* q,
                                                     const int32_t* sel_pos, int64_t n_sel,
                                                     const void* k_cache, const void* v_cache,
                                                     int64_t n_tok, int32_t n_q_heads, int32_t n_kv_heads,
                                                     int32_t head_dim, float sm_scale, void* out,
                                                     void* workspace, size_t workspace_bytes,
                                                     semshare_dtype_t dtype, void* stream);

/*
 * High-deviation token selection (Section 3 Insight 1; Section 4.2): the
 * n_sel positions with the largest deviation sigma (ties: the lower
 * position first), written in ascending position order.  One workgroup
 * selects by radix over the float bits; sigma must hold non-negative finite
 * values (as deviation_out produces).
 *   sigma    [n_tok] float32.   n_tok <= 2^20.   0 <= n_sel <= n_tok.
 *   sel_pos  [n_sel] int32 (output).
 */
semshare_status_t semshare_select_recompute(const float* sigma, int64_t n_tok, int64_t n_sel,
                                            int32_t* sel_pos, void* stream);

/*
 * The recompute set of a later layer, drawn from the previous layer's
 * (Section 4.3.3: starting from the second layer, the tokens of a layer are
 * chosen among those of the previous layer, Recomp[i] = T prod alpha_recomp[j]
 * of Appendix A.5; by Insight 1 of Section 3 the ones with the largest KV
 * deviation): of the n_cand candidates cand_pos (the previous layer's
 * recomputed positions, strictly ascending) with deviations sigma (that
 * layer's deviation_out, aligned with cand_pos), the n_sel with the largest
 * deviation (ties: the lower position first), their positions written in
 * ascending order.  The same one-workgroup radix selection as
 * semshare_select_recompute.
 *   sigma  [n_cand] float32 (non-negative, finite).   cand_pos [n_cand] int32.
 *   sel_pos [n_sel] int32 (output; may not alias cand_pos).
 *   n_cand <= 2^20;  0 <= n_sel <= n_cand.
 */
semshare_status_t semshare_select_recompute_nested(const float* sigma, const int32_t* cand_pos, int64_t n_cand,
                                                   int64_t n_sel, int32_t* sel_pos, void* stream);

/*
 * Average attention score of every token at a fully computed layer (Section
 * 3, Insight 2: the attention of each head averaged over the heads, then
 * over the query rows): mass[j] = sum_h sum_{i >= max(j, row_begin)}
 * P_h[i][j] / (n_q_heads (n_tok - row_begin)), P_h the causal softmax of
 * q_i . k_j * sm_scale (GQA: head h reads kv head h / (n_q_heads /
 * n_kv_heads)).  row_begin = 0 averages every row (the masses sum to 1);
 * row_begin > 0 averages the last n_tok - row_begin rows only, the window
 * the retention step ranks by (Section 4.3.4).  0 <= row_begin < n_tok.
 *   q        [n_tok][n_q_heads][head_dim] bf16 (RoPE'd queries of every row)
 *   k_cache  [n_tok][n_kv_heads][head_dim] bf16
 *   mass     [n_tok] float32 (output)
 *   sm_scale 0 => 1/sqrt(head_dim).   bf16 and head_dim 128 only, else
 *   SEMSHARE_E_UNSUPPORTED.   workspace: semshare_attention_mass_workspace()
 *   bytes, 4-byte aligned; q and k_cache 16-byte aligned.
 */
size_t semshare_attention_mass_workspace(int64_t n_tok, int32_t n_q_heads);
semshare_status_t semshare_attention_mass(const void* q, const void* k_cache, int64_t n_tok, int64_t row_begin,
                                          int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, float sm_scale,
                                          float* mass, void* workspace, size_t workspace_bytes,
                                          semshare_dtype_t dtype, void* stream);

/*
 * The same average over the rows >= row_begin (the retention window of
 * Section 4.3.4), reusing the per-row softmax normalisers that a previous
 * semshare_attention_mass call left in `workspace`: a row's normaliser sums
 * over all its keys whatever row_begin is, so the window pass only sums the
 * columns (about 40% less work at 5120 tokens).  Precondition (not checked on
 * the device): workspace is the buffer of a semshare_attention_mass call with
 * the same q, k_cache, n_tok, heads, head_dim and sm_scale, on the same
 * stream, not written since.  Arguments and errors as semshare_attention_mass.
 */
semshare_status_t semshare_attention_mass_window(const void* q, const void* k_cache, int64_t n_tok, int64_t row_begin,
                                                 int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                 float sm_scale, float* mass, void* workspace, size_t workspace_bytes,
                                                 semshare_dtype_t dtype, void* stream);

/*
 * Token retention on the first layer (Section 4.3.4; Appendix A.6 gives the
 * per-layer counts Retain[i] = T prod alpha[j]): hot tokens (the counts[0]
 * first by mass, as semshare_dynamic_recompute orders them) and the
 * recomputed tokens sel_pos[0 .. counts[1]) are never evicted; they rank
 * first, in position order, followed by every other token by score
 * (descending, lower position first on ties), score being the average
 * attention over the last (1 - AR / T) of the rows (semshare_attention_mass
 * with row_begin).  Kept are the first R = max(floor(max(min_keep, AR / T)
 * n_tok + 1/2), number of never-evicted tokens) of that ranking (the paper:
 * min_keep = 0.8), written to kept_pos in ascending order; *n_kept = R.
 * rank[p] is the place of position p in the ranking, so a later layer that
 * keeps Retain[i] tokens keeps those with rank < Retain[i] (nested sets).
 * Compacting the cache is semshare_gather_kv with idx = kept_pos.
 *   mass, score  [n_tok] float32;  sel_pos, counts: the outputs of
 *   semshare_dynamic_recompute (device).   rank, kept_pos [n_tok] int32,
 *   n_kept [1] int32 (outputs, device).   n_tok <= 65536 (beyond 8192 the
 *   ranking is counted by many workgroups, same results).
 */
semshare_status_t semshare_retention(const float* mass, const float* score, int32_t n_tok, const int32_t* sel_pos,
                                     const int32_t* counts, double min_keep, int32_t* rank, int32_t* kept_pos,
                                     int32_t* n_kept, void* stream);

/*
 * Retention on a later layer (Section 4.3.4: later layers keep fewer tokens;
 * Appendix A.6: Retain[i] = T prod alpha_retain[j]) and the compaction plan of
 * its cache.  Kept are the tokens whose first-layer rank (semshare_retention)
 * is below n_retain, plus this layer's recomputed tokens sel_pos (never
 * evicted: recomputing a token that is then dropped would waste the work), so
 * the kept sets of layers with falling n_retain are nested apart from the
 * recomputed tokens.  Written in ascending position order:
 *   kept_pos[0 .. *n_kept)  the kept positions;
 *   src_idx[j] = idx[kept_pos[j]]  the reference row each compacted cache row
 *                copies (semshare_gather_kv with idx = src_idx and
 *                n_tgt = *n_kept builds the compacted cache), when idx (the
 *                match index, [n_tok]) is given;
 *   sel_rows[i]  the row of sel_pos[i] in the compacted cache (-1 for a
 *                position outside [0, n_tok)).  A layer's recomputed tokens
 *                attend over its compacted cache when semshare_qkv_rope_tabled
 *                (RoPE table of their positions sel_pos) and
 *                semshare_prefill_attention take sel_rows as their positions
 *                and *n_kept as n_tok: every kept token before a recomputed
 *                one sits at a lower row, every later one at a higher row.
 *   rank   [n_tok] int32 (a permutation of 0 .. n_tok-1; entries outside
 *          [0, n_tok) count as not ranked).   sel_pos [n_sel] int32 strictly
 *          ascending.   kept_pos, src_idx [n_tok] int32, sel_rows [n_sel]
 *          int32, n_kept [1] int32 (outputs, device; src_idx and idx are
 *          both NULL or both set).   n_tok <= 2^20.  0 <= n_retain.
 */
semshare_status_t semshare_retention_layer(const int32_t* rank, int32_t n_tok, int32_t n_retain,
                                           const int32_t* sel_pos, int32_t n_sel, const int32_t* idx,
                                           int32_t* kept_pos, int32_t* src_idx, int32_t* sel_rows, int32_t* n_kept,
                                           void* stream);

/*
 * Dynamic recompute set (Section 4.3.3 with the Attention Recovery equation
 * of Section 3): the tokens sorted by mass (descending; the lower position
 * first on ties); AR = the smallest count k >= 1 whose top-k mass reaches
 * thres of the total (the paper uses 55%), compared in fp64 on sums taken in
 * 2^-40 fixed point of the masses clamped to [0, 1]; those AR tokens are
 * hot, the rest cold.  Recomputed are floor(w_hot AR + 1/2) hot and
 * floor(w_cold (n_tok - AR) + 1/2) cold tokens (the paper: w_h = 0.5,
 * w_c = 0.1), in each group those with the largest sigma (lower position
 * first on ties), written to sel_pos in ascending position order.
 *   mass, sigma  [n_tok] float32 (sigma >= 0, as deviation_out gives)
 *   sel_pos      [n_tok] int32 (output; the first counts[1] are written)
 *   counts       [3] int32 (output, device): AR, number selected, of them hot
 *   n_tok <= 65536, else SEMSHARE_E_UNSUPPORTED (up to 8192 one workgroup
 *   sorts the keys; beyond, ranks are counted by many workgroups, with the
 *   same keys and the same results).
 *   thres, w_hot, w_cold in [0, 1].
 */
semshare_status_t semshare_dynamic_recompute(const float* mass, const float* sigma, int32_t n_tok, double thres,
                                             double w_hot, double w_cold, int32_t* sel_pos, int32_t* counts,
                                             void* stream);

/*
 * Reference retrieval over a bank of prompts (Appendix A.3 similarity
 * score; Section 5 applies reuse when it exceeds 0.8).  The bank holds
 * n_prompts reference prompts, prompt b being the codes
 * [ref_offsets[b], ref_offsets[b+1]) of ref.  For each prompt the target's
 * tokens are matched against that prompt alone (top-1 Hamming distance, as
 * semshare_match); dist_sum[b] is the sum of those distances and
 * similarity[b] = clip(1 - (dist_sum[b]/n_tgt - dmin) / (dmax - dmin), 0, 1)
 * in fp64 (the paper's min and max are 0 and 30).  A prompt with no tokens
 * counts every target token at the largest distance, 64 * n_words; with
 * n_tgt == 0 every score is 0.
 *   tgt          [n_tgt][n_words] u64 codes.   ref [n_ref][n_words] u64.
 *   ref_offsets  [n_prompts + 1] int64, device, ascending in [0, n_ref]
 *                (the caller's contract; entries outside are clamped).
 *   dist_sum     [n_prompts] int64, similarity [n_prompts] float64 (outputs).
 *   n_words in 1..4; n_prompts <= 65535; dmax > dmin.
 *   workspace    at least semshare_bank_similarity_workspace() bytes, 8-byte
 *                aligned (per target tile partial sums; may be NULL when 0).
 * The sums are exact integers and the scores do not depend on the schedule.
 */
size_t semshare_bank_similarity_workspace(int64_t n_tgt, int32_t n_prompts);
semshare_status_t semshare_bank_similarity(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
                                           const int64_t* ref_offsets, int32_t n_prompts, int32_t n_words,
                                           double dmin, double dmax, int64_t* dist_sum, double* similarity,
                                           void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SEMSHARE_H */
