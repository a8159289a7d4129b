/*
 * CPU oracle for the CMC two-tier decode path.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct statement of what the path computes,
 * in fp64, written from the paper (Sec. 2.5, "Inference with Two-Tier KV
 * Cache Policy").  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load this library; the product path never does.  It
 * shares no code, header, table or constant with the HIP library.
 *
 * Inputs arrive as the exact bits both sides receive (fp32, or bf16 as raw
 * 16-bit patterns); every value is widened losslessly to double and all
 * arithmetic is double.  Readings of points the paper leaves open:
 *   - cosine denominator: max(||m_j||, 1e-8) * max(||q||, 1e-8), so a zero
 *     row or question scores 0;
 *   - exact score ties at the top-k boundary go to the lower index (earlier
 *     document position);
 *   - the Tier-2 window is a ring of capacity W holding the most recent W
 *     tokens; slot (count + t) mod W receives the t-th appended row;
 *   - decode attention is ordinary softmax attention with z = scale * <q,k>
 *     over the explicit key list [pool rows idx[0..k-1]] ++ [ring slots
 *     0..min(count,W)-1]; query head h reads kv head h / (Hq/Hkv); an empty
 *     key list yields a zero output row;
 *   - CME-guided localization works in token offsets; a sequence with no
 *     memory rows falls back to the midpoint floor(|C|/2);
 *   - denoising (Eq. 3): the neighbourhood is the g tokens after i inside
 *     the sequence, so the last token has none and is discarded by Eq. 3;
 *     zero norms are clamped to 1e-8 as in the selection score; the
 *     minimum keep interval m means any m consecutive positions hold a kept
 *     token (a token is kept when the m - 1 positions before it hold none);
 *   - MemoryBridge: Linear -> exact (erf) GELU -> Linear -> LayerNorm (biased
 *     variance, eps inside the square root) -> norm-calibrated tanh cap; the
 *     hidden width F is a parameter (the paper does not state it).
 *
 * Parity pins: tests check this file against exact-rational ranking,
 * list-history attention written without ring arithmetic, a library SDPA
 * special case, closed forms and invariants.
 *
 * Every entry point returns 0 on success and a positive code on an invalid
 * argument (nothing is written then).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_BAD_ARG 1
#define ORACLE_BAD_INDEX 2
#define ORACLE_NO_MEMORY 3

/* bf16 -> double: the bf16 pattern is the top half of an fp32 pattern. */
static double widen_bf16(uint16_t h)
{
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double load_elem(const void *base, int is_bf16, size_t i)
{
    if (is_bf16)
        return widen_bf16(((const uint16_t *)base)[i]);
    return (double)((const float *)base)[i];
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------ */
/* Tier-1 scoring and top-K selection (Sec. 2.5, Tier-1 paragraph and  */
/* its cosine score equation; M is the row-wise concatenation of the   */
/* segments' memory vectors in document order, Sec. 2.3 eq. for M).    */
/* ------------------------------------------------------------------ */

typedef struct {
    double s;
    int j;
} ranked;

/* Descending score; equal scores: ascending index (earlier position). */
static int by_rank(const void *a, const void *b)
{
    const ranked *x = (const ranked *)a, *y = (const ranked *)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->j > y->j) - (x->j < y->j);
}

static int by_value(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/*
 * sel_keys [B][N][D] fp32, or bf16 bit patterns when keys_bf16 is set;
 * q_vec [B][D] fp32.
 * idx_out  [B][k] int32: the K best-scoring rows, written in ascending order
 *          ("re-ordered by original document position").
 * scores_out [B][N] double cosine scores, or NULL.
 * gap_out  [B] double, or NULL: (s_(k) - s_(k+1)) / |s_(k)| for the k-th and
 *          (k+1)-th largest scores; +inf when k == 0 or k == N.
 */
int oracle_select(const void *sel_keys, int keys_bf16, const float *q_vec, int B, int N, int D, int k,
                  int32_t *idx_out, double *scores_out, double *gap_out)
{
    if (B < 0 || N < 0 || D <= 0 || k < 0 || k > N || (B > 0 && (!sel_keys || !q_vec)))
        return ORACLE_BAD_ARG;
    if (B > 0 && k > 0 && !idx_out)
        return ORACLE_BAD_ARG;
    ranked *all = (ranked *)malloc(sizeof(ranked) * (size_t)(N > 0 ? N : 1) * (size_t)(B > 0 ? B : 1));
    if (!all)
        return ORACLE_NO_MEMORY;

#pragma omp parallel for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        const float *q = q_vec + (size_t)b * D;
        double qq = 0.0;
        for (int d = 0; d < D; ++d)
            qq += (double)q[d] * (double)q[d];
        double qn = sqrt(qq);
        ranked *r = all + (size_t)b * N;
        for (int j = 0; j < N; ++j) {
            const size_t row = ((size_t)b * N + j) * D;
            double dot = 0.0, mm = 0.0;
            for (int d = 0; d < D; ++d) {
                const double m = load_elem(sel_keys, keys_bf16, row + d);
                dot += m * (double)q[d];
                mm += m * m;
            }
            double mn = sqrt(mm);
            double s = dot / (fmax(mn, 1e-8) * fmax(qn, 1e-8));
            r[j].s = s;
            r[j].j = j;
            if (scores_out)
                scores_out[(size_t)b * N + j] = s;
        }
        qsort(r, (size_t)N, sizeof(ranked), by_rank);
        int32_t *out = idx_out ? idx_out + (size_t)b * k : NULL;
        for (int i = 0; i < k; ++i)
            out[i] = r[i].j;
        if (k > 0)
            qsort(out, (size_t)k, sizeof(int32_t), by_value);
        if (gap_out) {
            double g;
            if (k == 0 || k == N) {
                g = INFINITY;
            } else {
                double hi = r[k - 1].s, lo = r[k].s;
                double den = fabs(hi);
                g = den > 0.0 ? (hi - lo) / den : (hi > lo ? INFINITY : 0.0);
            }
            gap_out[b] = g;
        }
    }
    free(all);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------ */
/* Tier-2 window (Sec. 2.5, Tier-2 paragraph and its window equation;  */
/* the cache bound K + W + |q| in the KV cache assembly paragraph).    */
/* ------------------------------------------------------------------ */

/* start = max(0, min(|C| - W, alpha - W/2)), W/2 taken as floor(W/2). */
long long oracle_window_start(long long ctx_len, long long W, long long alpha)
{
    long long s = alpha - W / 2;
    long long hi = ctx_len - W;
    if (s > hi) s = hi;
    if (s < 0) s = 0;
    return s;
}

/*
 * Ring append.  win_k/win_v [B][Hkv][W][Dh], new_k/new_v [B][Hkv][T_new][Dh],
 * elements of elem_bytes (2 or 4) bytes, copied verbatim.  For each sequence,
 * row t goes to slot (count + t) mod W, then count += T_new.  W == 0 means
 * there is no Tier-2: nothing is touched.
 */
int oracle_window_append(void *win_k, void *win_v, int elem_bytes, int32_t *win_count,
                         const void *new_k, const void *new_v,
                         int B, int Hkv, int W, int Dh, int T_new)
{
    if (B < 0 || Hkv <= 0 || W < 0 || Dh <= 0 || (elem_bytes != 2 && elem_bytes != 4))
        return ORACLE_BAD_ARG;
    if (W == 0)
        return ORACLE_OK;
    if (T_new < 1 || T_new > W)
        return ORACLE_BAD_ARG;
    size_t row = (size_t)Dh * (size_t)elem_bytes;
    for (int b = 0; b < B; ++b)
        if (win_count[b] < 0)
            return ORACLE_BAD_ARG;
    for (int b = 0; b < B; ++b) {
        int32_t c = win_count[b];
        for (int t = 0; t < T_new; ++t) {
            int slot = (int)(((long long)c + t) % W);
            for (int h = 0; h < Hkv; ++h) {
                size_t dst = (((size_t)b * Hkv + h) * W + slot) * row;
                size_t src = (((size_t)b * Hkv + h) * T_new + t) * row;
                memcpy((char *)win_k + dst, (const char *)new_k + src, row);
                memcpy((char *)win_v + dst, (const char *)new_v + src, row);
            }
        }
        win_count[b] = c + T_new;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------ */
/* MemoryBridge (Sec. 2.3): a two-layer MLP with GELU, LayerNorm on its */
/* output (the appendix's nn.LayerNorm formula), then the norm-         */
/* calibrated tanh cap of the section's equation.                      */
/* ------------------------------------------------------------------ */

/* GELU, the exact (erf) form. */
static double gelu(double x)
{
    return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));
}

/*
 * Hidden layer: hidden[r][f] = GELU(sum_c h[r][c] * w1[f][c] + b1[f]).
 * h [M][Hc] and w1 [F][Hc] are bf16 bit patterns, b1 [F] fp32.
 */
int oracle_bridge_hidden(const uint16_t *h, const uint16_t *w1, const float *b1, int M, int Hc, int F,
                         double *hidden_out)
{
    if (M < 0 || Hc < 1 || F < 1)
        return ORACLE_BAD_ARG;
    #pragma omp parallel for schedule(static)
    for (int r = 0; r < M; ++r) {
        for (int f = 0; f < F; ++f) {
            double u = (double)b1[f];
            for (int c = 0; c < Hc; ++c)
                u += widen_bf16(h[(size_t)r * Hc + c]) * widen_bf16(w1[(size_t)f * Hc + c]);
            hidden_out[(size_t)r * F + f] = gelu(u);
        }
    }
    return ORACLE_OK;
}

/*
 * Output layer, LayerNorm and cap, from given hidden activations [M][F]:
 *   y = hidden . w2^T + b2                        (w2 [Hd][F] bf16, b2 [Hd])
 *   m_hat = gamma * (y - mean) / sqrt(var + eps) + beta   (biased variance)
 *   t = nu * tanh(m_hat)
 *   out = t * min(1, 2 nu / ||t||_2)
 */
int oracle_bridge_out(const double *hidden, const uint16_t *w2, const float *b2, const float *gamma,
                      const float *beta, double nu, double eps, int M, int F, int Hd, double *out)
{
    if (M < 0 || F < 1 || Hd < 1 || !(nu > 0.0) || eps < 0.0)
        return ORACLE_BAD_ARG;
    #pragma omp parallel
    {
        double *y = (double *)malloc(sizeof(double) * (size_t)Hd);
        #pragma omp for schedule(static)
        for (int r = 0; r < M; ++r) {
            double mean = 0.0, var = 0.0, nrm = 0.0;
            for (int j = 0; j < Hd; ++j) {
                double acc = (double)b2[j];
                for (int f = 0; f < F; ++f)
                    acc += hidden[(size_t)r * F + f] * widen_bf16(w2[(size_t)j * F + f]);
                y[j] = acc;
                mean += acc;
            }
            mean /= Hd;
            for (int j = 0; j < Hd; ++j)
                var += (y[j] - mean) * (y[j] - mean);
            var /= Hd;
            double inv = 1.0 / sqrt(var + eps);
            for (int j = 0; j < Hd; ++j) {
                double m_hat = (double)gamma[j] * (y[j] - mean) * inv + (double)beta[j];
                y[j] = nu * tanh(m_hat);
                nrm += y[j] * y[j];
            }
            nrm = sqrt(nrm);
            double c = (nrm > 0.0 && 2.0 * nu / nrm < 1.0) ? 2.0 * nu / nrm : 1.0;
            for (int j = 0; j < Hd; ++j)
                out[(size_t)r * Hd + j] = y[j] * c;
        }
        free(y);
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------ */
/* Graph-based context denoising (Sec. 2.1, Eq. 3; the minimum keep    */
/* interval of the hyper-parameter table and of the appendix on the    */
/* denoising threshold).                                               */
/* ------------------------------------------------------------------ */

/*
 * max_cos_out[b][i] = max over j = i+1 .. min(i+g, n_b-1) of
 *   e_i.e_j / (max(|e_i|, 1e-8) max(|e_j|, 1e-8)),
 * and -inf where that range is empty (the last token of a sequence, and
 * every position at or past n_b).  emb [B][n][H], fp32 or bf16 bits;
 * n_b = n_tokens[b] clamped into [0, n] (all n when n_tokens is NULL).
 */
int oracle_denoise_scores(const void *emb, int is_bf16, const int32_t *n_tokens, int B, int n, int H, int g,
                          double *max_cos_out)
{
    if (B < 0 || n < 0 || H < 1 || g < 1)
        return ORACLE_BAD_ARG;
    for (int b = 0; b < B; ++b) {
        int nb = n_tokens ? n_tokens[b] : n;
        if (nb < 0) nb = 0;
        if (nb > n) nb = n;
        #pragma omp parallel for schedule(static)
        for (int i = 0; i < n; ++i) {
            double best = -INFINITY;
            if (i < nb) {
                size_t ri = ((size_t)b * n + i) * H;
                double ni = 0.0;
                for (int h = 0; h < H; ++h) {
                    double x = load_elem(emb, is_bf16, ri + h);
                    ni += x * x;
                }
                ni = sqrt(ni);
                for (int j = i + 1; j <= i + g && j < nb; ++j) {
                    size_t rj = ((size_t)b * n + j) * H;
                    double dot = 0.0, nj = 0.0;
                    for (int h = 0; h < H; ++h) {
                        double y = load_elem(emb, is_bf16, rj + h);
                        dot += load_elem(emb, is_bf16, ri + h) * y;
                        nj += y * y;
                    }
                    double c = dot / (fmax(ni, 1e-8) * fmax(sqrt(nj), 1e-8));
                    if (c > best) best = c;
                }
            }
            max_cos_out[(size_t)b * n + i] = best;
        }
    }
    return ORACLE_OK;
}

/*
 * Which tokens survive, given max_cos [B][n] (the decision is taken on
 * these values): token i < n_b passes Eq. 3 when max_cos >= tau.  Scanning
 * left to right, a token is kept when it passes, or when keep_min_every > 0
 * and the keep_min_every - 1 positions before it (counting from a virtual
 * kept token at -1) hold no kept token, so that any keep_min_every
 * consecutive positions hold at least one kept token.
 * Outputs: keep_out [B][n] 0/1 (or NULL); kept_idx [B][n] = the kept
 * positions ascending, then -1; kept_count [B]; with chunk_tokens > 0,
 * chunk_offset [B][ceil(n / chunk_tokens)] = the position of the first kept
 * token of each chunk of chunk_tokens kept tokens, then -1, and
 * n_chunks_out [B] = ceil(kept_count / chunk_tokens) (either may be NULL).
 */
int oracle_denoise_select(const double *max_cos, const int32_t *n_tokens, int B, int n, double tau,
                          int keep_min_every, int chunk_tokens, uint8_t *keep_out, int32_t *kept_idx,
                          int32_t *kept_count, int32_t *chunk_offset, int32_t *n_chunks_out)
{
    if (B < 0 || n < 0 || keep_min_every < 0 || chunk_tokens < 0)
        return ORACLE_BAD_ARG;
    int max_chunks = chunk_tokens > 0 ? (n + chunk_tokens - 1) / chunk_tokens : 0;
    for (int b = 0; b < B; ++b) {
        int nb = n_tokens ? n_tokens[b] : n;
        if (nb < 0) nb = 0;
        if (nb > n) nb = n;
        int last = -1, count = 0;
        for (int i = 0; i < n; ++i) {
            int keep = 0;
            if (i < nb) {
                keep = max_cos[(size_t)b * n + i] >= tau;
                if (keep_min_every > 0 && i - last >= keep_min_every)
                    keep = 1;
            }
            if (keep) {
                last = i;
                kept_idx[(size_t)b * n + count] = i;
                ++count;
            }
            if (keep_out)
                keep_out[(size_t)b * n + i] = (uint8_t)keep;
        }
        for (int c = count; c < n; ++c)
            kept_idx[(size_t)b * n + c] = -1;
        kept_count[b] = count;
        if (chunk_tokens > 0) {
            int nc = (count + chunk_tokens - 1) / chunk_tokens;
            for (int c = 0; c < max_chunks; ++c) {
                int v = c < nc ? kept_idx[(size_t)b * n + (size_t)c * chunk_tokens] : -1;
                if (chunk_offset)
                    chunk_offset[(size_t)b * max_chunks + c] = v;
            }
            if (n_chunks_out)
                n_chunks_out[b] = nc;
        }
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------ */
/* CME-guided Tier-2 localization (appendix on Tier-2 window           */
/* localization: alpha is the token offset of the chunk whose CME has */
/* the largest norm; the midpoint heuristic uses alpha = |C|/2).  Each */
/* segment contributes m^(c) consecutive rows, in segment order (the   */
/* concatenation of the segments' CMEs, Sec. 2.2, which the decoder-   */
/* ready rows of Sec. 2.3 keep).                                       */
/* ------------------------------------------------------------------ */

/*
 * norms_out[r] = ||x_r||_2 of the R rows of rows[R][D] (fp32, or bf16 bit
 * patterns when is_bf16 is set).  Localization ranks the norms of the CME
 * vectors h, the encoder's hidden states at the placeholder positions
 * (Sec. 2.2): the decoder-ready rows after Sec. 2.3's cap cannot serve,
 * since the cap sets the norm of every row whose nu tanh(m_hat) exceeds
 * 2 nu to exactly 2 nu.
 */
int oracle_row_norms(const void *rows, int is_bf16, long long R, int D, double *norms_out)
{
    if (R < 0 || D < 1)
        return ORACLE_BAD_ARG;
    #pragma omp parallel for schedule(static)
    for (long long r = 0; r < R; ++r) {
        double s = 0.0;
        for (int d = 0; d < D; ++d) {
            const double x = load_elem(rows, is_bf16, (size_t)r * D + d);
            s += x * x;
        }
        norms_out[r] = sqrt(s);
    }
    return ORACLE_OK;
}

/*
 * Per sequence b (norms [B][N], any non-negative values):
 *   n_b = n_rows[b] clamped into [0, N] (all N rows when n_rows is NULL);
 *   j*  = the row j < n_b with the largest norm, the lowest such j on ties;
 *   the chunk of j* is j* / mems_per_chunk;
 *   alpha = chunk_offset[b][chunk] (chunk * chunk_tokens when chunk_offset is
 *           NULL); a sequence with no rows takes the midpoint floor(|C|/2);
 *   start = max(0, min(|C| - W, alpha - floor(W/2))) with |C| = ctx_len[b].
 * chunk_offset, when given, is [B][n_chunks] with n_chunks * mems_per_chunk
 * >= N.
 */
int oracle_locate(const double *norms, const int32_t *n_rows, int B, int N, int mems_per_chunk,
                  const int32_t *chunk_offset, int n_chunks, int chunk_tokens,
                  const int32_t *ctx_len, int W, int32_t *alpha_out, int32_t *start_out)
{
    if (B < 0 || N < 0 || mems_per_chunk < 1 || W < 0 || chunk_tokens < 0)
        return ORACLE_BAD_ARG;
    if (chunk_offset && (long long)n_chunks * mems_per_chunk < N)
        return ORACLE_BAD_ARG;
    for (int b = 0; b < B; ++b) {
        int nb = n_rows ? n_rows[b] : N;
        if (nb < 0) nb = 0;
        if (nb > N) nb = N;
        long long alpha;
        if (nb == 0) {
            alpha = ctx_len[b] / 2;
        } else {
            int best = 0;
            for (int j = 1; j < nb; ++j)
                if (norms[(size_t)b * N + j] > norms[(size_t)b * N + best])
                    best = j;
            int chunk = best / mems_per_chunk;
            alpha = chunk_offset ? chunk_offset[(size_t)b * n_chunks + chunk]
                                 : (long long)chunk * chunk_tokens;
        }
        alpha_out[b] = (int32_t)alpha;
        start_out[b] = (int32_t)oracle_window_start(ctx_len[b], W, alpha);
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------ */
/* Two-tier decode attention (Sec. 2.5, KV cache assembly: the frozen  */
/* decoder attends over [M* || C_local] (+ question rows, which a      */
/* caller passes as extra pool rows), a cache bounded by K + W + |q|). */
/* ------------------------------------------------------------------ */

/*
 * q       [B][Hq][Dh] fp32
 * cme_k/v [B][Hkv][N][Dh] (bf16 bits or fp32)
 * idx     [B][k] int32 rows of the pool, or NULL for rows 0..k-1
 * win_k/v [B][Hkv][W][Dh] ring, valid slots 0..min(count, W)-1
 * out     [B][Hq][Dh] double
 */
int oracle_two_tier_decode(const float *q, const void *cme_k, const void *cme_v, int kv_is_bf16,
                           const int32_t *idx, int k,
                           const void *win_k, const void *win_v, const int32_t *win_count, int W,
                           int B, int Hq, int Hkv, int Dh, int N, double scale, double *out)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || Dh <= 0 || N < 0 || k < 0 || W < 0)
        return ORACLE_BAD_ARG;
    if (k > N && idx == NULL)
        return ORACLE_BAD_ARG;
    for (int b = 0; b < B; ++b) {
        if (W > 0 && win_count[b] < 0)
            return ORACLE_BAD_ARG;
        for (int i = 0; idx && i < k; ++i)
            if (idx[(size_t)b * k + i] < 0 || idx[(size_t)b * k + i] >= N)
                return ORACLE_BAD_INDEX;
    }
    const int G = Hq / Hkv;
    int status = ORACLE_OK;

#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        for (int h = 0; h < Hq; ++h) {
            const int kv = h / G;
            const int valid = W > 0 ? (win_count[b] < W ? win_count[b] : W) : 0;
            const int n = k + valid;
            const float *qh = q + ((size_t)b * Hq + h) * Dh;
            double *o = out + ((size_t)b * Hq + h) * Dh;
            double *z = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
            size_t *row = (size_t *)malloc(sizeof(size_t) * (size_t)(n > 0 ? n : 1));
            const void **kb = (const void **)malloc(sizeof(void *) * (size_t)(n > 0 ? n : 1));
            const void **vb = (const void **)malloc(sizeof(void *) * (size_t)(n > 0 ? n : 1));
            if (!z || !row || !kb || !vb) {
#pragma omp atomic write
                status = ORACLE_NO_MEMORY;
                free(z); free(row); free(kb); free(vb);
                continue;
            }
            /* The explicit two-tier key list. */
            for (int i = 0; i < k; ++i) {
                int r = idx ? idx[(size_t)b * k + i] : i;
                row[i] = (((size_t)b * Hkv + kv) * N + (size_t)r) * Dh;
                kb[i] = cme_k;
                vb[i] = cme_v;
            }
            for (int s = 0; s < valid; ++s) {
                row[k + s] = (((size_t)b * Hkv + kv) * W + (size_t)s) * Dh;
                kb[k + s] = win_k;
                vb[k + s] = win_v;
            }
            /* Logits and their maximum. */
            double m = -INFINITY;
            for (int i = 0; i < n; ++i) {
                double acc = 0.0;
                for (int d = 0; d < Dh; ++d)
                    acc += (double)qh[d] * load_elem(kb[i], kv_is_bf16, row[i] + d);
                z[i] = scale * acc;
                if (z[i] > m) m = z[i];
            }
            /* Softmax-weighted sum of the values. */
            double den = 0.0;
            for (int i = 0; i < n; ++i) {
                z[i] = exp(z[i] - m);
                den += z[i];
            }
            for (int d = 0; d < Dh; ++d) {
                double acc = 0.0;
                for (int i = 0; i < n; ++i)
                    acc += z[i] * load_elem(vb[i], kv_is_bf16, row[i] + d);
                o[d] = n > 0 ? acc / den : 0.0;
            }
            free(z); free(row); free(kb); free(vb);
        }
    }
    return status;
}
