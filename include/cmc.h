/*
 * cmc.h -- C ABI of the MI355X (gfx950) two-tier KV-cache decode path of CMC
 * ("Compressing Long Context into Answer-Aligned Memory Embeddings for LLM
 * Inference").
 *
 * The paper compresses a long context C into decoder-ready memory rows M
 * (Sec. 2.3, eq. for M) and, at inference, lets the frozen decoder attend to
 * a two-tier cache (Sec. 2.5):
 *   Tier-1  the top-K memory rows by cosine similarity to a mean-pooled
 *           question vector, re-ordered by document position;
 *   Tier-2  a W-token local window of the context at full resolution;
 * with the cache bounded by K + W + |q| at every generation step.  This
 * library implements the per-step hot path of that policy:
 *   cmc_select_cmes      Tier-1 scoring and top-K selection (once per question)
 *   cmc_gather_tier1     copy the selected rows' K/V into one block (once per question)
 *   cmc_window_append    Tier-2 ring-buffer append (every step)
 *   cmc_two_tier_decode  decode attention over [selected rows || window]
 *   cmc_decode_step      append + decode fused into one launch (every step)
 *   *_ragged             the same with per-sequence sizes (ragged batches)
 *   cmc_locate_window    CME-guided Tier-2 window placement (once per question)
 *   cmc_denoise          graph-based context denoising before compression
 *                        (Sec. 2.1, once per context)
 *   cmc_memory_bridge    MemoryBridge projection of CME vectors into selection
 *                        keys (Sec. 2.3, once per context), and the CME norms
 *                        that localization ranks
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers unless stated otherwise; the caller owns
 *     all memory, including workspaces.  The library never allocates, frees,
 *     copies to the host or synchronizes.
 *   - Arrays are dense, row-major, with the shapes given below; every base
 *     pointer must be 16-byte aligned (else CMC_ERR_UNSUPPORTED).
 *   - `stream` is a hipStream_t (NULL = the default stream).  CMC_OK means
 *     the work was enqueued on that stream; device faults surface at the
 *     caller's next synchronization.
 *   - Arguments are validated on the host before anything is enqueued.  On
 *     any non-OK status nothing is enqueued and no output is touched;
 *     cmc_last_error() then returns a description (thread-local).
 *   - Values must be finite.  bf16 tensors are passed as their raw 16-bit
 *     patterns (uint16_t storage).
 *   - Concurrent calls on different streams must not share output buffers,
 *     windows or workspaces.
 */
#ifndef CMC_H
#define CMC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Both enums are int-sized.  In C++ they are declared with int as their
 * underlying type, so that any int a caller passes (an unknown dtype, say)
 * is a valid value the library can reject, rather than undefined behaviour. */
#ifdef __cplusplus
#define CMC_ENUM_INT : int
#else
#define CMC_ENUM_INT
#endif

typedef enum cmc_status CMC_ENUM_INT {
    CMC_OK = 0,
    CMC_ERR_INVALID_ARGUMENT = 1,   /* shape/value out of the documented range   */
    CMC_ERR_UNSUPPORTED = 2,        /* valid but not implemented (dtype, Dh, G, alignment) */
    CMC_ERR_WORKSPACE_TOO_SMALL = 3,
    CMC_ERR_HIP = 4                 /* a HIP runtime call or launch failed        */
} cmc_status;

typedef enum cmc_dtype CMC_ENUM_INT {
    CMC_F32 = 0,
    CMC_BF16 = 1
} cmc_dtype;

/* ------------------------------------------------------------------------ */
/* Tier-1 selection.                                                        */
/* ------------------------------------------------------------------------ */

/* Bytes of workspace cmc_select_cmes needs for these sizes (0 is a valid
 * answer only when B*N == 0): the B*N fp32 scores when scores_out is NULL.
 * The top-k state lives in registers, so k does not enter.  Returns 0 for
 * invalid sizes. */
size_t cmc_select_workspace_bytes(int B, int N);

/*
 * Question-guided top-K selection (Sec. 2.5, Tier-1 paragraph and its score
 * equation; Eq. 2 of the problem statement, M* = TopK(M, q, K)).
 *
 *   sel_keys   [B][N][D]       decoder-ready memory rows m_j of each sequence,
 *                              row j = document position j (Sec. 2.3, eq. M),
 *                              fp32 or bf16 bit patterns as key_dtype says
 *                              (bf16 halves the bytes read; each element is
 *                              widened exactly to fp32)
 *   q_vec      [B][D]    fp32  mean-pooled question embedding q_vec
 *   idx_out    [B][k]    int32 the k rows with the largest
 *                              score_j = m_j.q / (max(|m_j|,1e-8) max(|q|,1e-8)),
 *                              written in ASCENDING order (document order).
 *                              Equal scores at the boundary: lower index wins.
 *   scores_out [B][N]    fp32  the cosine scores, or NULL
 *   workspace  >= cmc_select_workspace_bytes(B, N) bytes, any content
 *
 * Limits: B >= 0, 0 <= k <= N <= 32768, D >= 4 and D % 4 == 0 (fp32 keys)
 * or D % 8 == 0 (bf16 keys), else CMC_ERR_UNSUPPORTED.
 * Arithmetic: fp32 with a fixed reduction order (run-to-run bit-identical).
 */
cmc_status cmc_select_cmes(const void *sel_keys, cmc_dtype key_dtype, const float *q_vec,
                           int B, int N, int D, int k,
                           int32_t *idx_out, float *scores_out,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * Ragged batches: the selection of cmc_select_cmes with a per-sequence
 * candidate count, plus the question rows that the assembled cache keeps
 * beside the selected rows (Sec. 2.5, KV cache assembly: the prefill input is
 * [M* || C_local || q], so the cache holds K + W + |q| rows; the number of
 * memory rows per sequence follows from its context length, Sec. 2.3).
 *
 *   n_rows     [B] int32 (device)  candidates of sequence b: rows [0, n_b) of
 *                                  sel_keys[b] (n_b clamped into [0, N] on the
 *                                  device; rows past it score -inf in
 *                                  scores_out and are never selected)
 *   q_rows     [B] int32 (device)  question rows pinned after the selection, or
 *                                  NULL for none: q_b rows, clamped into
 *                                  [0, idx_stride - k_b]
 *   idx_out    [B][idx_stride] int32  row b = the k_b = min(k, n_b) selected
 *                                  rows ascending (the order and tie rule of
 *                                  cmc_select_cmes), then n_b, n_b+1, ...,
 *                                  n_b+q_b-1 (the question's rows, which the
 *                                  caller stores in the K/V pool right after
 *                                  sequence b's memory rows), then -1 up to
 *                                  idx_stride
 *   k_out      [B] int32           k_b + q_b (the k_len of the ragged decode
 *                                  calls), or NULL
 *   norms_out  [B][N] fp32         |m_j| of every candidate row (0 past n_b),
 *                                  from the same pass over the keys; or NULL.
 *                                  (These are the capped memory rows: not the
 *                                  norms CME-guided localization ranks, see
 *                                  cmc_locate_window.)
 *   sel_keys, key_dtype, q_vec, scores_out, workspace: as cmc_select_cmes (N
 *   is the row stride of sel_keys, scores_out and norms_out)
 *
 * Limits: B >= 0, N >= 0, k >= 0, idx_stride >= k, D >= 4 and D % 4 == 0
 * (fp32 keys) or D % 8 == 0 (bf16 keys), N <= 32768.  k may exceed N (then
 * k_b = n_b).  With n_b = N and no question rows the result equals
 * cmc_select_cmes.
 */
cmc_status cmc_select_cmes_ragged(const void *sel_keys, cmc_dtype key_dtype, const float *q_vec,
                                  const int32_t *n_rows, const int32_t *q_rows,
                                  int B, int N, int D, int k, int idx_stride,
                                  int32_t *idx_out, int32_t *k_out, float *scores_out,
                                  float *norms_out,
                                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * CME-guided Tier-2 localization (appendix on Tier-2 window localization:
 * when the answer offset alpha is not known, alpha is taken as the offset of
 * the chunk whose CME has the largest norm; the window start then follows
 * the Tier-2 window equation of Sec. 2.5).  The CMEs are the encoder's hidden
 * states at the placeholder positions (Sec. 2.2); each chunk (segment)
 * contributes mems_per_chunk consecutive rows (Sec. 2.2, the concatenation
 * H^(c)), so row j belongs to chunk j / mems_per_chunk.  Offsets are in
 * tokens of the context C.
 *
 *   norms        [B][N] fp32   norms of the CME vectors h, e.g. h_norms_out
 *                              of cmc_memory_bridge (B contexts of N rows
 *                              each); the decision is made on these values.
 *                              The capped memory rows m (the bridge output)
 *                              do not rank: Sec. 2.3's cap sets the norm of
 *                              every row whose nu tanh(m_hat) exceeds 2 nu to
 *                              exactly 2 nu, which at decoder widths is every
 *                              row.
 *   n_rows       [B] int32     rows of sequence b (clamped into [0, N]), or
 *                              NULL for all N
 *   ctx_len      [B] int32     |C| of sequence b, in tokens
 *   chunk_offset [B][n_chunks] int32  token offset of each chunk in C, or
 *                              NULL: chunk i starts at i * chunk_tokens
 *   alpha_out    [B] int32     alpha_b, or NULL
 *   start_out    [B] int32     start_b = max(0, min(|C| - W, alpha_b - floor(W/2)))
 *
 * alpha_b is the offset of the chunk of the row with the largest norm among
 * the first n_b rows (the lowest row index on ties).  A sequence with no rows
 * takes the midpoint alpha_b = floor(|C|/2) (the appendix's midpoint
 * heuristic).  Limits: B, N, W, chunk_tokens >= 0, mems_per_chunk >= 1;
 * with chunk_offset, n_chunks * mems_per_chunk >= N.  Results are exact
 * (integer work on the given norms).
 */
cmc_status cmc_locate_window(const float *norms, const int32_t *n_rows, const int32_t *ctx_len,
                             int B, int N, int mems_per_chunk,
                             const int32_t *chunk_offset, int n_chunks, int chunk_tokens,
                             int W, int32_t *alpha_out, int32_t *start_out, void *stream);

/* ------------------------------------------------------------------------ */
/* MemoryBridge.                                                            */
/* ------------------------------------------------------------------------ */

/* Bytes of workspace cmc_memory_bridge needs: the hidden activations,
 * M * F bf16. */
size_t cmc_bridge_workspace_bytes(int M, int F);

/*
 * MemoryBridge projection (Sec. 2.3): each CME vector h (encoder width Hc)
 * becomes a decoder-ready memory row of width Hd,
 *   hidden = GELU(h W1^T + b1)                      (erf form, not the tanh one)
 *   m_hat  = LayerNorm(hidden W2^T + b2)            (gamma, beta, biased variance,
 *                                                    eps inside the square root:
 *                                                    the appendix's nn.LayerNorm)
 *   t      = nu tanh(m_hat)
 *   out    = t * min(1, 2 nu / ||t||_2)             (the section's norm cap:
 *                                                    |out_i| <= nu, ||out|| <= 2 nu)
 * with nu = s * (mean l2 norm of the decoder's token embeddings), computed
 * by the caller.  The rows of out are the selection keys of cmc_select_cmes.
 *
 *   h        [M][Hc] bf16     CME vectors
 *   w1       [F][Hc] bf16     first layer (nn.Linear layout: [out][in]); b1 [F] fp32
 *   w2       [Hd][F] bf16     second layer; b2 [Hd] fp32
 *   ln_gamma, ln_beta [Hd] fp32
 *   out      [M][Hd] fp32
 *   h_norms_out [M] fp32      |h_j|_2 of every input row (bf16 widened exactly,
 *            squares summed in fp32 in a fixed order), the norms that
 *            cmc_locate_window ranks; or NULL
 *   workspace >= cmc_bridge_workspace_bytes(M, F) bytes, any content; after
 *            the call it holds the hidden activations, [M][F] bf16 (rounded
 *            to nearest even from fp32)
 *
 * Limits: M >= 0; Hc % 64 == 0, F % 128 == 0, Hd % 128 == 0 (the GEMM tile);
 * nu > 0 and eps >= 0 finite.  Arithmetic: bf16 operands, fp32 accumulation
 * (MFMA); erf evaluated to within 1.5e-7 absolute (Abramowitz & Stegun
 * 7.1.26), below the bf16 rounding of the hidden activations, which the
 * second layer reads; LayerNorm, tanh and the cap in fp32.
 */
cmc_status cmc_memory_bridge(const void *h, const void *w1, const float *b1,
                             const void *w2, const float *b2,
                             const float *ln_gamma, const float *ln_beta,
                             float nu, float ln_eps, int M, int Hc, int F, int Hd,
                             float *out, float *h_norms_out,
                             void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------ */
/* Context denoising.                                                       */
/* ------------------------------------------------------------------------ */

/* Bytes of workspace cmc_denoise needs (one byte per token); 0 for invalid
 * sizes or B*n == 0. */
size_t cmc_denoise_workspace_bytes(int B, int n);

/*
 * Graph-based context denoising (Sec. 2.1, Eq. 3, with the minimum keep
 * interval of the hyper-parameter table): token i of sequence b is kept when
 *   max over j = i+1 .. min(i+g, n_b-1) of e_i.e_j / (max(|e_i|,1e-8) max(|e_j|,1e-8))
 * is >= tau (the last token has no neighbour and fails), or when
 * keep_min_every = m > 0 and the m-1 positions before it hold no kept token
 * (so any m consecutive positions hold one).  The kept tokens, in order, are
 * the denoised context C', cut into chunks of chunk_tokens tokens.
 *
 *   emb          [B][n][H] fp32 or bf16 (dtype)  token embeddings
 *   n_tokens     [B] int32   tokens of sequence b (clamped into [0, n]), or
 *                            NULL for all n
 *   g, tau       neighbourhood (1..4; the paper uses 3) and threshold (0.05)
 *   keep_min_every  m (0: no floor; the paper uses 16)
 *   max_cos_out  [B][n] fp32  the statistic (-inf where a token has no
 *                            neighbour or lies past n_b), or NULL
 *   keep_out     [B][n] uint8 1 = kept, or NULL
 *   kept_idx     [B][n] int32 kept positions ascending, then -1
 *   kept_count   [B] int32    |C'_b|
 *   chunk_offset [B][ceil(n / chunk_tokens)] int32  position in C of the
 *                            first token of each chunk of C' (the offsets of
 *                            cmc_locate_window), then -1; NULL, or ignored
 *                            when chunk_tokens == 0
 *   n_chunks_out [B] int32    ceil(|C'_b| / chunk_tokens), or NULL
 *   workspace    >= cmc_denoise_workspace_bytes(B, n) bytes, any content
 *
 * Limits: B, n >= 0, H >= 1 with H % 8 == 0 (bf16) or H % 4 == 0 (fp32),
 * 1 <= g <= 4, tau not NaN.  Arithmetic: fp32 with a fixed order; the
 * threshold decision is taken on the fp32 statistic that max_cos_out
 * returns.
 */
cmc_status cmc_denoise(const void *emb, cmc_dtype dtype, const int32_t *n_tokens,
                       int B, int n, int H, int g, float tau, int keep_min_every, int chunk_tokens,
                       float *max_cos_out, uint8_t *keep_out, int32_t *kept_idx, int32_t *kept_count,
                       int32_t *chunk_offset, int32_t *n_chunks_out,
                       void *workspace, size_t workspace_bytes, void *stream);

/*
 * Tier-1 gather (Sec. 2.5, KV cache assembly: the cache holds the selected
 * rows M* as one block): copies, once per question, the K/V rows of the
 * selected memory rows into a contiguous block,
 *   out_k[b][h][j][:] = cme_k[b][h][idx[b][j]][:]  for j < k_b (same for V),
 * so that the per-step decode reads it as a pool with idx == NULL and
 * N = k, streaming whole rows with no index lookups.
 *
 *   cme_k/v    [B][Hkv][N][Dh]   (kv_dtype)
 *   idx        [B][idx_stride] int32, values clamped into [0, N-1] on the
 *              device; NULL copies rows 0..k-1
 *   k_len      [B] int32 (device): k_b = k_len[b] clamped into [0, k], or
 *              NULL for all k; rows j >= k_b of out are left untouched
 *   out_k/v    [B][Hkv][k][Dh]   (kv_dtype)
 *
 * Limits: Hkv >= 1, Dh in {64, 128, 256}, idx_stride >= k when idx is given,
 * k <= N when it is not.  Bit-exact copy.
 */
cmc_status cmc_gather_tier1(const void *cme_k, const void *cme_v, cmc_dtype kv_dtype,
                            const int32_t *idx, const int32_t *k_len, int idx_stride,
                            int B, int Hkv, int N, int k, int Dh,
                            void *out_k, void *out_v, void *stream);

/* ------------------------------------------------------------------------ */
/* Tier-2 window.                                                           */
/* ------------------------------------------------------------------------ */

/*
 * Ring-buffer append keeping the window at its W most recent tokens, which
 * bounds the cache by K + W + |q| during generation (Sec. 2.5, KV cache
 * assembly).
 *
 *   win_k, win_v   [B][Hkv][W][Dh]     ring storage, updated in place
 *   win_count      [B] int32           tokens ever appended (read and advanced);
 *                                      slots 0..min(count,W)-1 are valid
 *   new_k, new_v   [B][Hkv][T_new][Dh] rows to append; row t of sequence b goes
 *                                      to slot (count_b + t) mod W, then
 *                                      count_b += T_new
 *   kv_dtype       element type of the four K/V arrays
 *
 * Limits: Hkv >= 1, Dh in {64, 128, 256}, W >= 0, 1 <= T_new <= W, count_b
 * >= 0 and count_b + T_new < 2^31.  W == 0 (no Tier-2) is a no-op that
 * returns CMC_OK and touches nothing.
 */
cmc_status cmc_window_append(void *win_k, void *win_v, cmc_dtype kv_dtype, int32_t *win_count,
                             const void *new_k, const void *new_v,
                             int B, int Hkv, int W, int Dh, int T_new, void *stream);

/*
 * Host helper (no device work): the Tier-2 window start of Sec. 2.5,
 * start = max(0, min(ctx_len - W, alpha - floor(W/2))), for a caller filling
 * the ring with C[start : start + W] at prefill.
 */
long long cmc_window_start(long long ctx_len, long long W, long long alpha);

/* ------------------------------------------------------------------------ */
/* Two-tier decode attention.                                               */
/* ------------------------------------------------------------------------ */

/* Bytes of workspace cmc_two_tier_decode and cmc_decode_step need for these
 * sizes; 0 for invalid sizes.
 *
 * The decode workspace holds arrival counters (its first 4*(B + B*Hkv)
 * bytes) followed by split-K partials.  It must be ZERO-FILLED before its
 * first use (e.g. allocated zeroed); every call returns the counters to zero,
 * so it can be reused by later calls (also from a captured HIP graph)
 * without clearing.  Do not share one workspace between calls that may run
 * concurrently. */
size_t cmc_decode_workspace_bytes(int B, int Hq, int Hkv, int Dh, int k, int W);

/*
 * One decode step of attention over the two-tier cache (Sec. 2.5, KV cache
 * assembly: the decoder attends over [M* || C_local] (+ question rows), the
 * key set being bounded by K + W + |q|).
 *
 *   q          [B][Hq][Dh] fp32   this step's queries (positional encoding
 *                                 already applied by the caller)
 *   cme_k/v    [B][Hkv][N][Dh]    Tier-1 pool: one K/V row per memory row
 *   idx        [B][k] int32       pool rows to attend to (any order, values in
 *                                 [0, N)), or NULL for rows 0..k-1.  Question
 *                                 rows, when pinned, are extra pool rows here.
 *   win_k/v    [B][Hkv][W][Dh]    Tier-2 ring; slots 0..min(count_b, W)-1 are used
 *   win_count  [B] int32          as maintained by cmc_window_append
 *   scale      logit scale (1/sqrt(Dh) for standard attention)
 *   out        [B][Hq][Dh] fp32   softmax(scale q K^T) V over the key list
 *                                 [pool rows idx] ++ [valid ring slots]; query
 *                                 head h reads kv head h / (Hq/Hkv).  A sequence
 *                                 whose key list is empty gets a zero row.
 *   workspace  >= cmc_decode_workspace_bytes(B, Hq, Hkv, Dh, k, W) bytes,
 *              zero-filled before first use (see cmc_decode_workspace_bytes)
 *
 * Limits: Hq % Hkv == 0 with Hq/Hkv in {1, 2, 4, 8}; Dh in {64, 128, 256};
 * 0 <= k <= N when idx == NULL; k + W >= 1; W >= 0; B, Hkv <= 65535;
 * k + W (+ T_new) <= INT_MAX; with bf16 K/V, N * Dh * 2 and W * Dh * 2 below
 * 4 GiB (one (sequence, kv head)'s pool or ring); else CMC_ERR_UNSUPPORTED,
 * nothing enqueued.  Index values are not
 * checked on the host; the device clamps them into [0, N-1], which keeps
 * memory access in bounds but makes the result meaningless.
 * Arithmetic: fp32 accumulation, fixed reduction order (run-to-run
 * bit-identical).
 */
cmc_status cmc_two_tier_decode(const float *q,
                               const void *cme_k, const void *cme_v,
                               const int32_t *idx, int k,
                               const void *win_k, const void *win_v,
                               const int32_t *win_count, int W,
                               cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh, int N,
                               float scale, float *out,
                               void *workspace, size_t workspace_bytes, void *stream);

/*
 * One whole decode step in a single launch: the ring append of
 * cmc_window_append (new_k/new_v [B][Hkv][T_new][Dh], 1 <= T_new <= W and
 * T_new <= 65535, else CMC_ERR_UNSUPPORTED) followed by cmc_two_tier_decode
 * over the updated cache.  The ring contents and win_count are identical
 * to calling the two in that order, and out is the same attention over the
 * same keys (the appended rows are taken in their own phase, so out may
 * differ from the two calls' in the last bits, within the same accuracy).
 * With W == 0 there is no Tier-2 and new_k/new_v are ignored.
 * Same arguments, limits and workspace as cmc_two_tier_decode otherwise.
 */
cmc_status cmc_decode_step(const float *q,
                           const void *cme_k, const void *cme_v,
                           const int32_t *idx, int k,
                           void *win_k, void *win_v, int32_t *win_count, int W,
                           const void *new_k, const void *new_v, int T_new,
                           cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh, int N,
                           float scale, float *out,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * Ragged batches (Sec. 2.5, KV cache assembly, with per-sequence sizes): as
 * cmc_two_tier_decode and cmc_decode_step, except that sequence b's Tier-1
 * key rows are its first k_b entries of idx, k_b = k_len[b] clamped into
 * [0, k] on the device; k is the row stride of idx.  k_len is typically the
 * k_out of cmc_select_cmes_ragged (selected rows plus pinned question rows).
 * The window fill is per sequence through win_count, as always.  A sequence
 * whose key list is empty gets a zero row.  Same workspace, limits and
 * arithmetic as the uniform calls (the workspace is sized by k and W).
 *
 *   k_len      [B] int32 (device), non-NULL
 */
cmc_status cmc_two_tier_decode_ragged(const float *q,
                                      const void *cme_k, const void *cme_v,
                                      const int32_t *idx, const int32_t *k_len, int k,
                                      const void *win_k, const void *win_v,
                                      const int32_t *win_count, int W,
                                      cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh, int N,
                                      float scale, float *out,
                                      void *workspace, size_t workspace_bytes, void *stream);

cmc_status cmc_decode_step_ragged(const float *q,
                                  const void *cme_k, const void *cme_v,
                                  const int32_t *idx, const int32_t *k_len, int k,
                                  void *win_k, void *win_v, int32_t *win_count, int W,
                                  const void *new_k, const void *new_v, int T_new,
                                  cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh, int N,
                                  float scale, float *out,
                                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * cmc_decode_step without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the arrival counters and split partials live in a
 * fixed 4 MiB array inside the library (one per GPU, held until the process
 * ends).  The call itself allocates nothing; the caller still passes every
 * input and output.  Same arguments as cmc_decode_step minus the workspace,
 * same kernels, results identical to cmc_decode_step.
 *
 * Limits (else CMC_ERR_UNSUPPORTED, nothing enqueued): B + B*Hkv <= 16384
 * arrival counters, and the split partials of the launch plan within the
 * rest of the array (about 4 MiB: e.g. the 8-pair Llama-layer step needs
 * 0.23 MiB; plans with one workgroup per (sequence, kv head) pair need none).
 * The first call on each device looks the array up and zeroes its counters
 * with a small kernel on `stream`; make it outside graph capture.  Every call
 * on one GPU shares that GPU's array: calls that may overlap in time (other
 * streams, other threads, concurrent graph replays) race and must not be
 * made.
 */
cmc_status cmc_decode_step_noalloc(const float *q,
                                   const void *cme_k, const void *cme_v,
                                   const int32_t *idx, int k,
                                   void *win_k, void *win_v, int32_t *win_count, int W,
                                   const void *new_k, const void *new_v, int T_new,
                                   cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh, int N,
                                   float scale, float *out, void *stream);

/* ------------------------------------------------------------------------ */
/* Diagnostics.                                                             */
/* ------------------------------------------------------------------------ */

/* Static name of a status code. */
const char *cmc_status_string(cmc_status s);

/* Thread-local description of the last non-OK return on this thread ("" if
 * none).  Valid until the next call into the library on the same thread. */
const char *cmc_last_error(void);

/* Library version string. */
const char *cmc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CMC_H */
