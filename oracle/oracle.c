/*
 * CPU oracle for the SemShareKV hot path (fuzzy token matching + KV reuse).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * statement of what the GPU path must compute.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg load it; the product
 * library never links, calls or falls back to it, and the two share no code.
 *
 * Conventions
 *  - All arithmetic is fp64.  Inputs arrive as fp64 arrays holding the exact
 *    values of the storage-dtype inputs (bf16 or fp32).
 *  - Values the product path *stores* in a storage dtype (the RoPE'd
 *    embeddings, the recomputed K/V cache rows, the attention operand q and
 *    the attention output) are rounded here to that dtype, round-to-nearest
 *    even, at the same points.  ORC_F64 means "no rounding" and exists for
 *    the pins.
 *  - Loops over independent rows may run on several OpenMP threads; each
 *    output element is computed by exactly one thread in a fixed order, so
 *    results do not depend on the thread count.
 *
 * Parity status: every function below is pinned by the CPU test suite
 * (closed forms, invariants, brute force, library special cases).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F64 = 2 };

/* ---------------------------------------------------------------- rounding */

/* Nearest bf16 value of v (8 significant bits, fp32 exponent range), ties to
 * even, computed directly from the fp64 value (no detour through fp32). */
static double orc_round_bf16(double v) {
    if (v == 0.0 || !isfinite(v)) return v;
    int e;
    (void)frexp(v, &e);          /* v = m * 2^e, 0.5 <= |m| < 1 */
    int sh = e - 8;              /* spacing of bf16 values in [2^(e-1), 2^e) */
    if (sh < -133) sh = -133;    /* subnormal range: fixed spacing 2^-133 */
    double q = ldexp(v, -sh);    /* exact scaling by a power of two */
    double r = nearbyint(q);     /* default rounding mode: ties to even */
    double out = ldexp(r, sh);
    if (fabs(out) > 0x1.FEp127) out = copysign(INFINITY, v);
    return out;
}

static double orc_round(double v, int dt) {
    switch (dt) {
    case ORC_F32: return (double)(float)v;
    case ORC_BF16: return orc_round_bf16(v);
    default: return v;
    }
}

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void orc_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

void orc_round_array(const double* x, double* y, int64_t n, int dt) {
    for (int64_t i = 0; i < n; ++i) y[i] = orc_round(x[i], dt);
}

/* ------------------------------------------------------------ RoPE (a1) */

/* Rotary position embedding of token embeddings, Appendix A.1 Eq. (1), read
 * as standard RoPE (the RoFormer rotation the paper cites in Section 4.3.1):
 * the pair (x_2k, x_2k+1) of the row at position m is rotated by the angle
 * m * theta_k, theta_k = base^(-2k/d), d = the row width.  Row r has
 * position pos0 + r. */
void orc_rope_embed(const double* x, double* y, int64_t n_tok, int32_t dim, int64_t pos0,
                    double base, int dt) {
    const int32_t half = dim / 2;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < n_tok; ++r) {
        const double m = (double)(pos0 + r);
        const double* xr = x + r * (int64_t)dim;
        double* yr = y + r * (int64_t)dim;
        for (int32_t k = 0; k < half; ++k) {
            const double theta = pow(base, -2.0 * (double)k / (double)dim);
            const double a = m * theta;
            const double c = cos(a), s = sin(a);
            const double x0 = xr[2 * k], x1 = xr[2 * k + 1];
            yr[2 * k] = orc_round(c * x0 - s * x1, dt);
            yr[2 * k + 1] = orc_round(s * x0 + c * x1, dt);
        }
    }
}

/* ------------------------------------------------------------- LSH (a2) */

/* Projections p[t][j] = <x_t, r_j> of each row on each random hyperplane
 * (Appendix A.2 hashes x through x . r; the sign-bit form drops b and w). */
void orc_lsh_project(const double* x, const double* planes, double* proj, int64_t n_tok,
                     int32_t dim, int32_t n_bits) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_tok; ++t) {
        const double* xt = x + t * (int64_t)dim;
        for (int32_t j = 0; j < n_bits; ++j) {
            const double* rj = planes + (int64_t)j * dim;
            double p = 0.0;
            for (int32_t i = 0; i < dim; ++i) p += xt[i] * rj[i];
            proj[t * (int64_t)n_bits + j] = p;
        }
    }
}

/* Random-hyperplane LSH code: bit j is 1 iff <x, r_j> > 0 (0 when the
 * projection is exactly zero); bit j lives at bit (j mod 64) of word j/64. */
void orc_lsh_encode(const double* x, const double* planes, uint64_t* codes, int64_t n_tok,
                    int32_t dim, int32_t n_bits) {
    const int32_t n_words = n_bits / 64;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_tok; ++t) {
        const double* xt = x + t * (int64_t)dim;
        uint64_t* ct = codes + t * (int64_t)n_words;
        for (int32_t w = 0; w < n_words; ++w) ct[w] = 0;
        for (int32_t j = 0; j < n_bits; ++j) {
            const double* rj = planes + (int64_t)j * dim;
            double p = 0.0;
            for (int32_t i = 0; i < dim; ++i) p += xt[i] * rj[i];
            if (p > 0.0) ct[j / 64] |= (uint64_t)1 << (j % 64);
        }
    }
}

/* ----------------------------------------------------------- match (a3) */

static int orc_popcount64(uint64_t v) {
    int n = 0;
    while (v) { v &= v - 1; ++n; }
    return n;
}

/* For each target token, the reference token at the smallest Hamming
 * distance between LSH codes (Section 4.2 / 4.3: "the most similar token in
 * the reference prompt"); on equal distance the lowest reference index
 * wins.  Exhaustive scan: exact nearest neighbour in Hamming space. */
void orc_match(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, int64_t n_ref,
               int32_t n_words, int32_t* idx, int32_t* dist) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_tgt; ++t) {
        int best = 1 << 30;
        int64_t best_j = -1;
        for (int64_t j = 0; j < n_ref; ++j) {
            int d = 0;
            for (int32_t w = 0; w < n_words; ++w)
                d += orc_popcount64(tgt[t * n_words + w] ^ ref[j * n_words + w]);
            if (d < best) { best = d; best_j = j; }
        }
        idx[t] = (int32_t)best_j;
        if (dist) dist[t] = best_j < 0 ? -1 : best;
    }
}

/* ---------------------------------------------------------- gather (a4) */

/* Rearrange the reference cache token by token to the target's length
 * (Section 4.3): dst[l][t] = src[l][idx[t]] for every layer l; a row is all
 * heads of one token, copied bit for bit (K is kept post-RoPE and not
 * re-rotated, Section 4.3.2). */
void orc_gather_rows(const uint8_t* src, const int32_t* idx, int64_t n_tgt, int64_t n_ref,
                     uint8_t* dst, int32_t n_layers, int64_t row_bytes) {
    for (int32_t l = 0; l < n_layers; ++l)
        for (int64_t t = 0; t < n_tgt; ++t)
            memcpy(dst + ((int64_t)l * n_tgt + t) * row_bytes,
                   src + ((int64_t)l * n_ref + idx[t]) * row_bytes, (size_t)row_bytes);
}

/* ------------------------------------------------- partial prefill (a5-a7) */

/* Standard RoPE of one head vector (width D) at position p, in place. */
static void orc_rope_head(double* v, int32_t D, double p, double base) {
    for (int32_t k = 0; k < D / 2; ++k) {
        const double theta = pow(base, -2.0 * (double)k / (double)D);
        const double a = p * theta;
        const double c = cos(a), s = sin(a);
        const double x0 = v[2 * k], x1 = v[2 * k + 1];
        v[2 * k] = c * x0 - s * x1;
        v[2 * k + 1] = s * x0 + c * x1;
    }
}

/* y[o] = sum_i x[i] * W[o][i]  (nn.Linear layout W[out][in]). */
static void orc_linear_row(const double* x, const double* W, double* y, int32_t n_out, int32_t n_in) {
    for (int32_t o = 0; o < n_out; ++o) {
        const double* wo = W + (int64_t)o * n_in;
        double acc = 0.0;
        for (int32_t i = 0; i < n_in; ++i) acc += x[i] * wo[i];
        y[o] = acc;
    }
}

/* Step 1 of a partial prefill: recompute q, k, v of the selected tokens.
 * q = RoPE_p(x Wq^T) and k = RoPE_p(x Wk^T) per head, v = x Wv^T, each
 * rounded to the storage dtype.  q_out [n_sel][Hq*D], k_out, v_out
 * [n_sel][Hkv*D]; any of them may be NULL. */
void orc_qkv_rows(const double* x_sel, const int32_t* sel_pos, int64_t n_sel, const double* wq,
                  const double* wk, const double* wv, int32_t hidden, int32_t n_q_heads,
                  int32_t n_kv_heads, int32_t head_dim, double base, double* q_out, double* k_out,
                  double* v_out, int dt) {
    const int32_t nq = n_q_heads * head_dim, nkv = n_kv_heads * head_dim;
#pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < n_sel; ++s) {
        const double* x = x_sel + s * (int64_t)hidden;
        const double p = (double)sel_pos[s];
        if (q_out) {
            double* q = q_out + s * (int64_t)nq;
            orc_linear_row(x, wq, q, nq, hidden);
            for (int32_t h = 0; h < n_q_heads; ++h) orc_rope_head(q + h * head_dim, head_dim, p, base);
            for (int32_t i = 0; i < nq; ++i) q[i] = orc_round(q[i], dt);
        }
        if (k_out) {
            double* k = k_out + s * (int64_t)nkv;
            orc_linear_row(x, wk, k, nkv, hidden);
            for (int32_t h = 0; h < n_kv_heads; ++h) orc_rope_head(k + h * head_dim, head_dim, p, base);
            for (int32_t i = 0; i < nkv; ++i) k[i] = orc_round(k[i], dt);
        }
        if (v_out) {
            double* v = v_out + s * (int64_t)nkv;
            orc_linear_row(x, wv, v, nkv, hidden);
            for (int32_t i = 0; i < nkv; ++i) v[i] = orc_round(v[i], dt);
        }
    }
}

/* KV deviation of Appendix A.4, per token: sigma = ||K_reused - K_recomputed||_2
 * + ||V_reused - V_recomputed||_2 over all kv heads of the token's row. */
void orc_deviation(const double* k_cache, const double* v_cache, const int32_t* sel_pos,
                   int64_t n_sel, const double* k_new, const double* v_new, int32_t row_len,
                   double* sigma) {
    for (int64_t s = 0; s < n_sel; ++s) {
        const double* ko = k_cache + (int64_t)sel_pos[s] * row_len;
        const double* vo = v_cache + (int64_t)sel_pos[s] * row_len;
        const double* kn = k_new + s * (int64_t)row_len;
        const double* vn = v_new + s * (int64_t)row_len;
        double sk = 0.0, sv = 0.0;
        for (int32_t i = 0; i < row_len; ++i) {
            sk += (ko[i] - kn[i]) * (ko[i] - kn[i]);
            sv += (vo[i] - vn[i]) * (vo[i] - vn[i]);
        }
        sigma[s] = sqrt(sk) + sqrt(sv);
    }
}

/* Causal attention of selected rows over the assembled cache: for a query
 * row at position p and head h, scores_j = <q_h, K[j][h/G]> * scale for
 * j <= p, O = sum_j softmax(scores)_j V[j][h/G], G = Hq/Hkv (query heads
 * h = G*g .. G*g+G-1 share kv head g).  O is rounded to the storage dtype.
 * Rows listed in `rows` (indices into the selected set) are computed; rows
 * == NULL means all n_sel rows.  out is [n_sel][Hq*D] (only listed rows are
 * written).  With `keep` (one byte per cache position), only the positions
 * j <= p with keep[j] != 0 are attended: the cache after retention evicted
 * the others (Section 4.3.4); keep == NULL keeps every position. */
void orc_attention_rows(const double* q, const int32_t* sel_pos, int64_t n_sel,
                        const int64_t* rows, int64_t n_rows, const double* k_cache,
                        const double* v_cache, int32_t n_q_heads, int32_t n_kv_heads,
                        int32_t head_dim, double scale, double* out, int dt, const uint8_t* keep) {
    const int32_t G = n_q_heads / n_kv_heads;
    const int32_t nq = n_q_heads * head_dim, nkv = n_kv_heads * head_dim;
    const int64_t count = rows ? n_rows : n_sel;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < count; ++r) {
        const int64_t s = rows ? rows[r] : r;
        const int64_t p = sel_pos[s];
        double* sc = (double*)malloc(sizeof(double) * (size_t)(p + 1));
        double* acc = (double*)malloc(sizeof(double) * (size_t)head_dim);
        for (int32_t h = 0; h < n_q_heads; ++h) {
            const int32_t g = h / G;
            const double* qh = q + s * (int64_t)nq + (int64_t)h * head_dim;
            double mx = -INFINITY;
            for (int64_t j = 0; j <= p; ++j) {
                if (keep && !keep[j]) continue;
                const double* kj = k_cache + j * (int64_t)nkv + (int64_t)g * head_dim;
                double dot = 0.0;
                for (int32_t i = 0; i < head_dim; ++i) dot += qh[i] * kj[i];
                sc[j] = dot * scale;
                if (sc[j] > mx) mx = sc[j];
            }
            double den = 0.0;
            for (int64_t j = 0; j <= p; ++j) {
                if (keep && !keep[j]) { sc[j] = 0.0; continue; }  /* evicted: weight 0 */
                sc[j] = exp(sc[j] - mx);
                den += sc[j];
            }
            /* every output element sums its products in ascending key order */
            double* o = out + s * (int64_t)nq + (int64_t)h * head_dim;
            for (int32_t i = 0; i < head_dim; ++i) acc[i] = 0.0;
            for (int64_t j = 0; j <= p; ++j) {
                const double* vj = v_cache + j * (int64_t)nkv + (int64_t)g * head_dim;
                for (int32_t i = 0; i < head_dim; ++i) acc[i] += sc[j] * vj[i];
            }
            for (int32_t i = 0; i < head_dim; ++i) o[i] = orc_round(acc[i] / den, dt);
        }
        free(sc);
        free(acc);
    }
}

/* Average attention score of every token at a fully computed layer (Section
 * 3, Insight 2): P_h[i][j] is the causal softmax over keys j <= i of
 * <q[i][h], k[j][h/G]> * scale, and mass[j] = sum_h sum_{i >= max(j, row_begin)}
 * P_h[i][j] / (Hq (T - row_begin)).  Two passes: the normaliser
 * (max and sum of exponentials) of every (row, head), then the column sums
 * of the requested keys cols[0 .. n_cols) (all keys when cols == NULL;
 * mass[c] belongs to cols[c]).  q is [T][Hq][D], k is [T][Hkv][D]. */
void orc_attention_mass(const double* q, const double* k, int64_t T, int32_t n_q_heads, int32_t n_kv_heads,
                        int32_t head_dim, double scale, int64_t row_begin, const int64_t* cols, int64_t n_cols,
                        double* mass) {
    const int32_t G = n_q_heads / n_kv_heads;
    double* lse = (double*)malloc(sizeof(double) * (size_t)(T * n_q_heads));
#pragma omp parallel
    {
        double* sc = (double*)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1));
#pragma omp for schedule(dynamic, 16)
        for (int64_t r = 0; r < T * n_q_heads; ++r) {
            const int64_t i = r / n_q_heads;
            const int32_t h = (int32_t)(r % n_q_heads);
            const double* qi = q + (i * n_q_heads + h) * (int64_t)head_dim;
            double mx = -INFINITY, sum = 0.0;
            for (int64_t j = 0; j <= i; ++j) {
                const double* kj = k + (j * n_kv_heads + h / G) * (int64_t)head_dim;
                double dot = 0.0;
                for (int32_t d = 0; d < head_dim; ++d) dot += qi[d] * kj[d];
                sc[j] = dot * scale;
                if (sc[j] > mx) mx = sc[j];
            }
            for (int64_t j = 0; j <= i; ++j) sum += exp(sc[j] - mx);
            lse[r] = mx + log(sum);
        }
        free(sc);
    }
    const int64_t count = cols ? n_cols : T;
    const double norm = (double)n_q_heads * (double)(T - row_begin);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t c = 0; c < count; ++c) {
        const int64_t j = cols ? cols[c] : c;
        double tot = 0.0;
        for (int32_t h = 0; h < n_q_heads; ++h) {
            const double* kj = k + (j * n_kv_heads + h / G) * (int64_t)head_dim;
            for (int64_t i = j > row_begin ? j : row_begin; i < T; ++i) {
                const double* qi = q + (i * n_q_heads + h) * (int64_t)head_dim;
                double dot = 0.0;
                for (int32_t d = 0; d < head_dim; ++d) dot += qi[d] * kj[d];
                tot += exp(dot * scale - lse[i * n_q_heads + h]);
            }
        }
        mass[c] = tot / norm;
    }
    free(lse);
}

/* One layer of partial prefill (Sections 4.2 and 4.3.3): recompute q/k/v of
 * the selected tokens, measure their deviation against the rows currently in
 * the assembled cache (optional), overwrite those cache rows with the
 * recomputed k/v, then attend for every selected token over the updated
 * cache.  out == NULL only rebuilds cache rows (a prompt's own cache).
 * scale <= 0 means 1/sqrt(D). */
void orc_partial_prefill(const double* x_sel, const int32_t* sel_pos, int64_t n_sel,
                         const double* wq, const double* wk, const double* wv, double* k_cache,
                         double* v_cache, int64_t n_tok, int32_t hidden, int32_t n_q_heads,
                         int32_t n_kv_heads, int32_t head_dim, double base, double scale,
                         double* out, double* sigma, int dt) {
    (void)n_tok;
    const int32_t nq = n_q_heads * head_dim, nkv = n_kv_heads * head_dim;
    if (scale <= 0.0) scale = 1.0 / sqrt((double)head_dim);
    double* q = out ? (double*)malloc(sizeof(double) * (size_t)(n_sel * nq)) : NULL;
    double* k = (double*)malloc(sizeof(double) * (size_t)(n_sel * nkv));
    double* v = (double*)malloc(sizeof(double) * (size_t)(n_sel * nkv));
    orc_qkv_rows(x_sel, sel_pos, n_sel, wq, wk, wv, hidden, n_q_heads, n_kv_heads, head_dim, base,
                 q, k, v, dt);
    if (sigma) orc_deviation(k_cache, v_cache, sel_pos, n_sel, k, v, nkv, sigma);
    for (int64_t s = 0; s < n_sel; ++s) {
        memcpy(k_cache + (int64_t)sel_pos[s] * nkv, k + s * nkv, sizeof(double) * (size_t)nkv);
        memcpy(v_cache + (int64_t)sel_pos[s] * nkv, v + s * nkv, sizeof(double) * (size_t)nkv);
    }
    if (out)
        orc_attention_rows(q, sel_pos, n_sel, NULL, 0, k_cache, v_cache, n_q_heads, n_kv_heads,
                           head_dim, scale, out, dt, NULL);
    free(q);
    free(k);
    free(v);
}

/* ------------------------------------------------ HD-token selection (a5) */

static const double* orc_sort_sigma;

static int orc_cmp_desc_sigma(const void* a, const void* b) {
    const int32_t i = *(const int32_t*)a, j = *(const int32_t*)b;
    if (orc_sort_sigma[i] > orc_sort_sigma[j]) return -1;
    if (orc_sort_sigma[i] < orc_sort_sigma[j]) return 1;
    return (i > j) - (i < j);
}

static int orc_cmp_i32(const void* a, const void* b) {
    const int32_t i = *(const int32_t*)a, j = *(const int32_t*)b;
    return (i > j) - (i < j);
}

/* High-deviation tokens (Section 3, Insight 1; Section 4.2): the n_sel
 * positions with the largest deviation (ties: lower position first),
 * returned in ascending position order. */
void orc_select_recompute(const double* sigma, int64_t n_tok, int64_t n_sel, int32_t* sel_pos) {
    int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n_tok > 0 ? n_tok : 1));
    for (int64_t i = 0; i < n_tok; ++i) order[i] = (int32_t)i;
    orc_sort_sigma = sigma;
    qsort(order, (size_t)n_tok, sizeof(int32_t), orc_cmp_desc_sigma);
    memcpy(sel_pos, order, sizeof(int32_t) * (size_t)n_sel);
    qsort(sel_pos, (size_t)n_sel, sizeof(int32_t), orc_cmp_i32);
    free(order);
}

/* ---------------------------------------- prompt-level similarity (A.3) */

/* LSH-distance similarity of Appendix A.3: d_norm = (dist - min)/(max - min)
 * with min = 0 and max = 30, similarity = clip(1 - d_norm, 0, 1).  The
 * paper leaves "LSH_dist" of a prompt pair undefined; it is read here as the
 * mean top-1 Hamming distance of the target tokens. */
double orc_similarity(const int32_t* dist, int64_t n_tgt, double dmin, double dmax) {
    if (n_tgt <= 0) return 0.0;
    double sum = 0.0;
    for (int64_t t = 0; t < n_tgt; ++t) sum += (double)dist[t];
    const double mean = sum / (double)n_tgt;
    const double dn = (mean - dmin) / (dmax - dmin);
    double s = 1.0 - dn;
    if (s < 0.0) s = 0.0;
    if (s > 1.0) s = 1.0;
    return s;
}

/* Reference retrieval over a bank (Appendix A.3 score, Section 5 gate): the
 * bank holds n_prompts reference prompts, prompt b being the codes
 * [offsets[b], offsets[b+1]) of ref.  For each prompt the target's tokens are
 * matched against that prompt alone (orc_match); dist_sum[b] is the sum of
 * their top-1 distances and sim[b] the similarity of those distances
 * (orc_similarity).  A prompt with no tokens counts every target token at the
 * largest possible distance, 64 * n_words. */
void orc_bank_similarity(const uint64_t* tgt, int64_t n_tgt, const uint64_t* ref, const int64_t* offsets,
                         int32_t n_prompts, int32_t n_words, double dmin, double dmax, int64_t* dist_sum,
                         double* sim) {
    int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n_tgt > 0 ? n_tgt : 1));
    int32_t* dist = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n_tgt > 0 ? n_tgt : 1));
    for (int32_t b = 0; b < n_prompts; ++b) {
        const int64_t lo = offsets[b], hi = offsets[b + 1];
        if (hi > lo) {
            orc_match(tgt, n_tgt, ref + lo * n_words, hi - lo, n_words, idx, dist);
        } else {
            for (int64_t t = 0; t < n_tgt; ++t) dist[t] = 64 * n_words;
        }
        int64_t sum = 0;
        for (int64_t t = 0; t < n_tgt; ++t) sum += dist[t];
        dist_sum[b] = sum;
        sim[b] = orc_similarity(dist, n_tgt, dmin, dmax);
    }
    free(idx);
    free(dist);
}

