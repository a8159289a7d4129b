// Host side of the C ABI declared in include/cmc.h: argument validation,
// launch planning and error reporting.  Everything here runs on the host;
// every computation runs in the kernels of decode.hip, select.hip and
// window.hip, enqueued on the caller's stream.
#include <limits.h>
#include <math.h>
#include <algorithm>
#include <mutex>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "cmc.h"
#include "kernels.hpp"

namespace {

thread_local char g_error[512] = "";

cmc_status fail(cmc_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return s;
}

cmc_status ok() {
    g_error[0] = '\0';
    return CMC_OK;
}

cmc_status hip_fail(hipError_t e, const char *what) {
    return fail(CMC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool misaligned(const void *p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u); }

bool supported_dh(int dh) { return dh == 64 || dh == 128 || dh == 256; }

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

// Checks shared by the uniform and ragged selection: the key type and the
// key width it allows (16-byte vectors of 4 fp32 or 8 bf16 elements).
cmc_status check_keys(const char *fn, cmc_dtype key_dtype, int D) {
    if (key_dtype != CMC_F32 && key_dtype != CMC_BF16)
        return fail(CMC_ERR_UNSUPPORTED, "%s: unknown key_dtype %d", fn, (int)key_dtype);
    const int vec = key_dtype == CMC_BF16 ? 8 : 4;
    if (D % vec != 0)
        return fail(CMC_ERR_UNSUPPORTED, "%s: D=%d must be a multiple of %d for %s keys", fn, D, vec,
                    key_dtype == CMC_BF16 ? "bf16" : "fp32");
    return CMC_OK;
}

}  // namespace

// Build-time tuning knob: the number of 4-wave decode workgroups the split
// plan aims for.
#ifndef CMC_DECODE_TARGET_WG
#define CMC_DECODE_TARGET_WG 512
#endif
// Build-time tuning knob: smallest number of keys per split of 4-wave
// workgroups (one 16-key block per wave).
#ifndef CMC_DECODE_GRANULE
#define CMC_DECODE_GRANULE 64
#endif
// Build-time tuning knob: fewest (sequence, kv head) pairs that take one
// 8-wave workgroup each (up to 256 pairs).
#ifndef CMC_DECODE_WIDE_MIN_PAIRS
#define CMC_DECODE_WIDE_MIN_PAIRS 192
#endif

namespace cmc {

// Key-axis split plan.  The decode kernel keeps eight waves resident per CU
// (two per SIMD), so about 2048 waves fill the 256 CUs in one round.
//   - With 192..256 (sequence, kv head) pairs, each pair gets one 8-wave
//     workgroup (S = 1): one round and no cross-workgroup merge.
//   - Otherwise workgroups have 4 waves, two resident per CU, and the plan
//     aims for about kTargetWG of them: a pair is split only when there are
//     fewer pairs than that, never below kGranule keys per split.
// The plan depends only on sizes, so the workspace query and the launch
// always agree.
DecodePlan plan_decode(int B, int Hq, int Hkv, int Dh, int k, int W) {
    constexpr long long kTargetWG = CMC_DECODE_TARGET_WG;
    constexpr long long kGranule = CMC_DECODE_GRANULE;
    constexpr long long kWideMinPairs = CMC_DECODE_WIDE_MIN_PAIRS;
    // The merge stages S*G*2 floats in the kernel's LDS; one split more is
    // reserved for appended rows.
    constexpr long long kMaxSplits = 127;
    DecodePlan pl;
    const long long L = (long long)k + W;
    const long long pairs = (long long)B * Hkv;
    if (L <= 0 || pairs <= 0) return pl;
    long long S, chunk;
    if (pairs >= kWideMinPairs && pairs <= 256 && decode_waves_ok(8, Hq / Hkv, Dh)) {
        pl.waves = 8;
        S = 1;
        chunk = L;
    } else {
        const long long s_target = std::max(1LL, (kTargetWG + pairs - 1) / pairs);
        chunk = (L + s_target - 1) / s_target;
        chunk = std::max(chunk, (L + kMaxSplits - 1) / kMaxSplits);
        chunk = ((chunk + kGranule - 1) / kGranule) * kGranule;
        S = (L + chunk - 1) / chunk;
    }
    const int G = Hq / Hkv;
    pl.S = (int)S;
    pl.chunk = (int)chunk;
    // A split plan merges partials anyway: the rows appended in a call then
    // get a split of their own, so no workgroup handles ring rows and
    // appended rows one after the other.
    const long long Sa = S > 1 && W > 0 ? S + 1 : S;
    pl.S_alloc = (int)Sa;
    pl.counter_bytes = align256((size_t)(B + pairs) * sizeof(unsigned));
    pl.ml_bytes = Sa > 1 ? align256((size_t)(pairs * Sa * G * 2) * sizeof(float)) : 0;
    pl.acc_bytes = Sa > 1 ? align256((size_t)(pairs * Sa * G * Dh) * sizeof(float)) : 0;
    pl.total = pl.counter_bytes + pl.ml_bytes + pl.acc_bytes;
    return pl;
}

}  // namespace cmc

extern "C" {

const char *cmc_version(void) { return "cmc-mi355x 0.1 (gfx950)"; }

const char *cmc_status_string(cmc_status s) {
    switch (s) {
        case CMC_OK: return "CMC_OK";
        case CMC_ERR_INVALID_ARGUMENT: return "CMC_ERR_INVALID_ARGUMENT";
        case CMC_ERR_UNSUPPORTED: return "CMC_ERR_UNSUPPORTED";
        case CMC_ERR_WORKSPACE_TOO_SMALL: return "CMC_ERR_WORKSPACE_TOO_SMALL";
        case CMC_ERR_HIP: return "CMC_ERR_HIP";
    }
    return "CMC_ERR_UNKNOWN";
}

const char *cmc_last_error(void) { return g_error; }

long long cmc_window_start(long long ctx_len, long long W, long long alpha) {
    long long start = alpha - W / 2;
    if (start > ctx_len - W) start = ctx_len - W;
    if (start < 0) start = 0;
    return start;
}

// ------------------------------------------------------------- selection

size_t cmc_select_workspace_bytes(int B, int N) {
    if (B < 0 || N < 0) return 0;
    return align256((size_t)B * (size_t)N * sizeof(float));
}

cmc_status cmc_select_cmes(const void *sel_keys, cmc_dtype key_dtype, const float *q_vec, int B, int N, int D,
                           int k, int32_t *idx_out, float *scores_out, void *workspace, size_t workspace_bytes,
                           void *stream) {
    if (B < 0 || N < 0 || k < 0 || D < 4)
        return fail(CMC_ERR_INVALID_ARGUMENT, "select: need B >= 0, N >= 0, k >= 0, D >= 4 (got B=%d N=%d k=%d D=%d)", B, N, k, D);
    if (k > N) return fail(CMC_ERR_INVALID_ARGUMENT, "select: k=%d exceeds N=%d", k, N);
    if (cmc_status st = check_keys("select", key_dtype, D)) return st;
    if (N > cmc::kSelectMaxN) return fail(CMC_ERR_UNSUPPORTED, "select: N=%d exceeds %d", N, cmc::kSelectMaxN);
    if (B > 65535) return fail(CMC_ERR_UNSUPPORTED, "select: B=%d exceeds 65535", B);
    if ((long long)B * N == 0) return ok();
    if (!sel_keys || !q_vec) return fail(CMC_ERR_INVALID_ARGUMENT, "select: sel_keys and q_vec must be non-null");
    if (k > 0 && !idx_out) return fail(CMC_ERR_INVALID_ARGUMENT, "select: idx_out must be non-null when k > 0");
    if (misaligned(sel_keys) || misaligned(q_vec) || misaligned(idx_out) || misaligned(scores_out) ||
        misaligned(workspace))
        return fail(CMC_ERR_UNSUPPORTED, "select: every pointer must be 16-byte aligned");
    float *scores = scores_out;
    if (!scores) {
        const size_t need = cmc_select_workspace_bytes(B, N);
        if (!workspace || workspace_bytes < need)
            return fail(CMC_ERR_WORKSPACE_TOO_SMALL, "select: workspace of %zu bytes needed, %zu given", need,
                        workspace ? workspace_bytes : (size_t)0);
        scores = static_cast<float *>(workspace);
    }
    cmc::SelectParams p{sel_keys, q_vec, scores, idx_out, B, N, D, k, k, nullptr, nullptr, nullptr, nullptr,
                        key_dtype == CMC_BF16};
    hipError_t e = cmc::launch_select(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "select launch");
    return ok();
}

cmc_status cmc_select_cmes_ragged(const void *sel_keys, cmc_dtype key_dtype, const float *q_vec,
                                  const int32_t *n_rows, const int32_t *q_rows, int B, int N, int D, int k,
                                  int idx_stride, int32_t *idx_out, int32_t *k_out, float *scores_out,
                                  float *norms_out, void *workspace, size_t workspace_bytes, void *stream) {
    if (B < 0 || N < 0 || k < 0 || D < 4)
        return fail(CMC_ERR_INVALID_ARGUMENT, "select_ragged: need B >= 0, N >= 0, k >= 0, D >= 4 (got B=%d N=%d k=%d D=%d)", B, N, k, D);
    if (idx_stride < k)
        return fail(CMC_ERR_INVALID_ARGUMENT, "select_ragged: idx_stride=%d is below k=%d", idx_stride, k);
    if (cmc_status st = check_keys("select_ragged", key_dtype, D)) return st;
    if (N > cmc::kSelectMaxN) return fail(CMC_ERR_UNSUPPORTED, "select_ragged: N=%d exceeds %d", N, cmc::kSelectMaxN);
    if (B > 65535) return fail(CMC_ERR_UNSUPPORTED, "select_ragged: B=%d exceeds 65535", B);
    if (B == 0) return ok();
    if (!n_rows) return fail(CMC_ERR_INVALID_ARGUMENT, "select_ragged: n_rows must be non-null");
    if (N > 0 && (!sel_keys || !q_vec))
        return fail(CMC_ERR_INVALID_ARGUMENT, "select_ragged: sel_keys and q_vec must be non-null");
    if (idx_stride > 0 && !idx_out)
        return fail(CMC_ERR_INVALID_ARGUMENT, "select_ragged: idx_out must be non-null when idx_stride > 0");
    if (misaligned(sel_keys) || misaligned(q_vec) || misaligned(n_rows) || misaligned(q_rows) ||
        misaligned(idx_out) || misaligned(k_out) || misaligned(scores_out) || misaligned(norms_out) ||
        misaligned(workspace))
        return fail(CMC_ERR_UNSUPPORTED, "select_ragged: every pointer must be 16-byte aligned");
    float *scores = scores_out;
    if (!scores && N > 0) {
        const size_t need = cmc_select_workspace_bytes(B, N);
        if (!workspace || workspace_bytes < need)
            return fail(CMC_ERR_WORKSPACE_TOO_SMALL, "select_ragged: workspace of %zu bytes needed, %zu given",
                        need, workspace ? workspace_bytes : (size_t)0);
        scores = static_cast<float *>(workspace);
    }
    cmc::SelectParams p{sel_keys, q_vec, scores, idx_out, B, N, D, k, idx_stride, n_rows, q_rows, k_out,
                        norms_out, key_dtype == CMC_BF16};
    hipError_t e = cmc::launch_select(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "select_ragged launch");
    return ok();
}

cmc_status cmc_locate_window(const float *norms, const int32_t *n_rows, const int32_t *ctx_len, int B, int N,
                             int mems_per_chunk, const int32_t *chunk_offset, int n_chunks, int chunk_tokens,
                             int W, int32_t *alpha_out, int32_t *start_out, void *stream) {
    if (B < 0 || N < 0 || mems_per_chunk < 1 || W < 0 || chunk_tokens < 0 || n_chunks < 0)
        return fail(CMC_ERR_INVALID_ARGUMENT,
                    "locate: need B, N, W, chunk_tokens, n_chunks >= 0 and mems_per_chunk >= 1");
    if (chunk_offset && (long long)n_chunks * mems_per_chunk < N)
        return fail(CMC_ERR_INVALID_ARGUMENT, "locate: n_chunks=%d chunks of %d rows do not cover N=%d", n_chunks,
                    mems_per_chunk, N);
    if (B > 65535) return fail(CMC_ERR_UNSUPPORTED, "locate: B=%d exceeds 65535", B);
    if (B == 0) return ok();
    if (!ctx_len || !start_out || (N > 0 && !norms))
        return fail(CMC_ERR_INVALID_ARGUMENT, "locate: norms, ctx_len and start_out must be non-null");
    if (misaligned(norms) || misaligned(n_rows) || misaligned(ctx_len) || misaligned(chunk_offset) ||
        misaligned(alpha_out) || misaligned(start_out))
        return fail(CMC_ERR_UNSUPPORTED, "locate: every pointer must be 16-byte aligned");
    cmc::LocateParams p{norms, n_rows, chunk_offset, ctx_len, alpha_out, start_out,
                        B, N, mems_per_chunk, n_chunks, chunk_tokens, W};
    hipError_t e = cmc::launch_locate(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "locate launch");
    return ok();
}

// ----------------------------------------------------------- MemoryBridge

size_t cmc_bridge_workspace_bytes(int M, int F) {
    if (M < 0 || F < 0) return 0;
    return align256((size_t)M * (size_t)F * sizeof(uint16_t));
}

cmc_status cmc_memory_bridge(const void *h, const void *w1, const float *b1, const void *w2, const float *b2,
                             const float *ln_gamma, const float *ln_beta, float nu, float ln_eps, int M, int Hc,
                             int F, int Hd, float *out, float *h_norms_out, void *workspace, size_t workspace_bytes,
                             void *stream) {
    if (M < 0 || Hc < 1 || F < 1 || Hd < 1)
        return fail(CMC_ERR_INVALID_ARGUMENT, "bridge: need M >= 0 and Hc, F, Hd >= 1");
    if (!(nu > 0.f) || isinf(nu) || !(ln_eps >= 0.f) || isinf(ln_eps))
        return fail(CMC_ERR_INVALID_ARGUMENT, "bridge: need a finite nu > 0 and a finite eps >= 0");
    if (Hc % cmc::kBridgeK != 0 || F % cmc::kBridgeN != 0 || Hd % cmc::kBridgeN != 0)
        return fail(CMC_ERR_UNSUPPORTED, "bridge: need Hc %% %d == 0 and F, Hd %% %d == 0 (got Hc=%d F=%d Hd=%d)",
                    cmc::kBridgeK, cmc::kBridgeN, Hc, F, Hd);
    if ((long long)((M + 127) / 128) * (F / cmc::kBridgeN) > 0x7fffffffLL ||
        (long long)((M + 127) / 128) * (Hd / cmc::kBridgeN) > 0x7fffffffLL)
        return fail(CMC_ERR_UNSUPPORTED, "bridge: M=%d too large", M);
    if (M == 0) return ok();
    if (!h || !w1 || !b1 || !w2 || !b2 || !ln_gamma || !ln_beta || !out)
        return fail(CMC_ERR_INVALID_ARGUMENT, "bridge: null pointer");
    if (misaligned(h) || misaligned(w1) || misaligned(b1) || misaligned(w2) || misaligned(b2) ||
        misaligned(ln_gamma) || misaligned(ln_beta) || misaligned(out) || misaligned(h_norms_out) ||
        misaligned(workspace))
        return fail(CMC_ERR_UNSUPPORTED, "bridge: every pointer must be 16-byte aligned");
    const size_t need = cmc_bridge_workspace_bytes(M, F);
    if (!workspace || workspace_bytes < need)
        return fail(CMC_ERR_WORKSPACE_TOO_SMALL, "bridge: workspace of %zu bytes needed, %zu given", need,
                    workspace ? workspace_bytes : (size_t)0);
    cmc::BridgeParams p{static_cast<const uint16_t *>(h), static_cast<const uint16_t *>(w1), b1,
                        static_cast<const uint16_t *>(w2), b2, ln_gamma, ln_beta, static_cast<uint16_t *>(workspace),
                        out, h_norms_out, M, Hc, F, Hd, nu, ln_eps};
    hipError_t e = cmc::launch_memory_bridge(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "bridge launch");
    return ok();
}

// ------------------------------------------------------------- denoising

size_t cmc_denoise_workspace_bytes(int B, int n) {
    if (B < 0 || n < 0) return 0;
    return align256((size_t)B * (size_t)n);
}

cmc_status cmc_denoise(const void *emb, cmc_dtype dtype, const int32_t *n_tokens, int B, int n, int H, int g,
                       float tau, int keep_min_every, int chunk_tokens, float *max_cos_out, uint8_t *keep_out,
                       int32_t *kept_idx, int32_t *kept_count, int32_t *chunk_offset, int32_t *n_chunks_out,
                       void *workspace, size_t workspace_bytes, void *stream) {
    if (dtype != CMC_F32 && dtype != CMC_BF16)
        return fail(CMC_ERR_UNSUPPORTED, "denoise: unknown dtype %d", (int)dtype);
    if (B < 0 || n < 0 || H < 1 || g < 1 || keep_min_every < 0 || chunk_tokens < 0)
        return fail(CMC_ERR_INVALID_ARGUMENT,
                    "denoise: need B, n, keep_min_every, chunk_tokens >= 0 and H, g >= 1");
    if (!(tau == tau)) return fail(CMC_ERR_INVALID_ARGUMENT, "denoise: tau is NaN");
    if (g > cmc::kDenoiseMaxG) return fail(CMC_ERR_UNSUPPORTED, "denoise: g=%d exceeds %d", g, cmc::kDenoiseMaxG);
    const int vec = dtype == CMC_BF16 ? 8 : 4;
    if (H % vec != 0) return fail(CMC_ERR_UNSUPPORTED, "denoise: H=%d must be a multiple of %d", H, vec);
    if (B > 65535) return fail(CMC_ERR_UNSUPPORTED, "denoise: B=%d exceeds 65535", B);
    if (B == 0) return ok();
    if ((n > 0 && (!emb || !kept_idx)) || !kept_count)
        return fail(CMC_ERR_INVALID_ARGUMENT, "denoise: emb, kept_idx and kept_count must be non-null");
    if (misaligned(emb) || misaligned(n_tokens) || misaligned(max_cos_out) || misaligned(keep_out) ||
        misaligned(kept_idx) || misaligned(kept_count) || misaligned(chunk_offset) || misaligned(n_chunks_out) ||
        misaligned(workspace))
        return fail(CMC_ERR_UNSUPPORTED, "denoise: every pointer must be 16-byte aligned");
    const size_t need = cmc_denoise_workspace_bytes(B, n);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(CMC_ERR_WORKSPACE_TOO_SMALL, "denoise: workspace of %zu bytes needed, %zu given", need,
                    workspace ? workspace_bytes : (size_t)0);
    cmc::DenoiseParams p{};
    p.emb = emb;
    p.n_tokens = n_tokens;
    p.pass = static_cast<uint8_t *>(workspace);
    p.max_cos = max_cos_out;
    p.keep_out = keep_out;
    p.kept_idx = kept_idx;
    p.kept_count = kept_count;
    p.chunk_offset = chunk_tokens > 0 ? chunk_offset : nullptr;
    p.n_chunks = chunk_tokens > 0 ? n_chunks_out : nullptr;
    p.B = B;
    p.n = n;
    p.H = H;
    p.g = g;
    p.tau = tau;
    p.keep_min_every = keep_min_every;
    p.chunk_tokens = chunk_tokens;
    p.max_chunks = chunk_tokens > 0 ? (n + chunk_tokens - 1) / chunk_tokens : 0;
    hipError_t e = cmc::launch_denoise(p, dtype == CMC_BF16, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "denoise launch");
    return ok();
}

// ---------------------------------------------------------------- window

cmc_status cmc_window_append(void *win_k, void *win_v, cmc_dtype kv_dtype, int32_t *win_count,
                             const void *new_k, const void *new_v, int B, int Hkv, int W, int Dh,
                             int T_new, void *stream) {
    if (kv_dtype != CMC_F32 && kv_dtype != CMC_BF16)
        return fail(CMC_ERR_UNSUPPORTED, "append: unknown kv_dtype %d", (int)kv_dtype);
    if (B < 0 || Hkv < 1 || W < 0)
        return fail(CMC_ERR_INVALID_ARGUMENT, "append: need B >= 0, Hkv >= 1, W >= 0 (got B=%d Hkv=%d W=%d)", B, Hkv, W);
    if (!supported_dh(Dh)) return fail(CMC_ERR_UNSUPPORTED, "append: Dh=%d not in {64,128,256}", Dh);
    if (B > 65535) return fail(CMC_ERR_UNSUPPORTED, "append: B=%d exceeds 65535", B);
    if (W == 0 || B == 0) return ok();
    if (T_new < 1 || T_new > W)
        return fail(CMC_ERR_INVALID_ARGUMENT, "append: need 1 <= T_new <= W (got T_new=%d W=%d)", T_new, W);
    if (!win_k || !win_v || !win_count || !new_k || !new_v)
        return fail(CMC_ERR_INVALID_ARGUMENT, "append: null pointer");
    if (misaligned(win_k) || misaligned(win_v) || misaligned(win_count) || misaligned(new_k) || misaligned(new_v))
        return fail(CMC_ERR_UNSUPPORTED, "append: every pointer must be 16-byte aligned");
    const int elem = kv_dtype == CMC_BF16 ? 2 : 4;
    cmc::AppendParams p{win_k, win_v, win_count, new_k, new_v, B, Hkv, W, T_new, Dh * elem / 16};
    hipError_t e = cmc::launch_window_append(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "append launch");
    return ok();
}

cmc_status cmc_gather_tier1(const void *cme_k, const void *cme_v, cmc_dtype kv_dtype, const int32_t *idx,
                            const int32_t *k_len, int idx_stride, int B, int Hkv, int N, int k, int Dh,
                            void *out_k, void *out_v, void *stream) {
    if (kv_dtype != CMC_F32 && kv_dtype != CMC_BF16)
        return fail(CMC_ERR_UNSUPPORTED, "gather: unknown kv_dtype %d", (int)kv_dtype);
    if (B < 0 || Hkv < 1 || N < 0 || k < 0)
        return fail(CMC_ERR_INVALID_ARGUMENT, "gather: need B, N, k >= 0 and Hkv >= 1");
    if (!supported_dh(Dh)) return fail(CMC_ERR_UNSUPPORTED, "gather: Dh=%d not in {64,128,256}", Dh);
    if (idx && idx_stride < k)
        return fail(CMC_ERR_INVALID_ARGUMENT, "gather: idx_stride=%d is below k=%d", idx_stride, k);
    if (!idx && k > N) return fail(CMC_ERR_INVALID_ARGUMENT, "gather: k=%d exceeds N=%d with idx == NULL", k, N);
    if (k > 0 && N < 1) return fail(CMC_ERR_INVALID_ARGUMENT, "gather: k=%d rows from an empty pool", k);
    if ((long long)B * Hkv * k * Dh > (1LL << 40)) return fail(CMC_ERR_UNSUPPORTED, "gather: too large");
    if ((long long)B * Hkv * k == 0) return ok();
    if (!cme_k || !cme_v || !out_k || !out_v) return fail(CMC_ERR_INVALID_ARGUMENT, "gather: null pointer");
    if (misaligned(cme_k) || misaligned(cme_v) || misaligned(idx) || misaligned(k_len) || misaligned(out_k) ||
        misaligned(out_v))
        return fail(CMC_ERR_UNSUPPORTED, "gather: every pointer must be 16-byte aligned");
    const int elem = kv_dtype == CMC_BF16 ? 2 : 4;
    cmc::GatherParams p{cme_k, cme_v, idx, k_len, out_k, out_v, B, Hkv, N, k, idx ? idx_stride : k,
                        Dh * elem / 16};
    hipError_t e = cmc::launch_gather(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gather launch");
    return ok();
}

// ---------------------------------------------------------------- decode

size_t cmc_decode_workspace_bytes(int B, int Hq, int Hkv, int Dh, int k, int W) {
    if (B < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || k < 0 || W < 0 || !supported_dh(Dh)) return 0;
    return cmc::plan_decode(B, Hq, Hkv, Dh, k, W).total;
}

}  // extern "C"

// ------------------------------------------------- no-allocation scratch
//
// cmc_decode_step_noalloc keeps its arrival counters and split partials in
// this file-scope device array instead of a caller workspace.  Layout:
// [arrival counters, kNoAllocCounterBytes | split partials].  The counter
// region never holds anything else, so it is zero at the start of every
// call: the array is zero when the code object is loaded, the first call on
// a device zeroes the region once more (a fill kernel on its stream), and
// every call re-arms the counters it used before it ends.  Each GPU holds
// its own copy until the process ends; host code reaches it only through
// the address hipGetSymbolAddress returns for the current device.
namespace {
constexpr size_t kNoAllocCounterBytes = size_t(64) << 10;  // up to 16384 counters: B + B*Hkv
constexpr size_t kNoAllocBytes = size_t(4) << 20;
constexpr int kNoAllocMaxDevices = 64;
}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

namespace {

__global__ void zero_words_kernel(uint32_t *p, unsigned n) {
    for (unsigned i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
}

std::mutex g_scratch_mu;
char *g_scratch_ptr[kNoAllocMaxDevices];

// The current device's address of `scratch`, set up on the first call on
// that device (symbol lookup, then the counters zeroed on `stream`).
cmc_status noalloc_scratch(const char *fn, hipStream_t stream, char **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kNoAllocMaxDevices)
        return fail(CMC_ERR_UNSUPPORTED, "%s: device %d beyond the %d supported", fn, dev, kNoAllocMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return fail(CMC_ERR_HIP, "%s: hipGetSymbolAddress returned a null address", fn);
        zero_words_kernel<<<16, 256, 0, stream>>>(static_cast<uint32_t *>(ptr), (unsigned)(kNoAllocCounterBytes / 4));
        e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "zeroing the scratch counters");
        g_scratch_ptr[dev] = static_cast<char *>(ptr);
    }
    *out = g_scratch_ptr[dev];
    return CMC_OK;
}

// The decode calls.  With noalloc, `workspace` is ignored and the counters
// and partials live in `scratch` (sizes beyond it are rejected).
cmc_status decode_impl(const char *fn, const float *q, const void *cme_k, const void *cme_v, const int32_t *idx,
                       const int32_t *k_len, int k, void *win_k, void *win_v, int32_t *win_count, int W, const void *new_k,
                       const void *new_v, int T_new, cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh, int N,
                       float scale, float *out, void *workspace, size_t workspace_bytes, void *stream,
                       bool noalloc = false) {
    if (kv_dtype != CMC_F32 && kv_dtype != CMC_BF16)
        return fail(CMC_ERR_UNSUPPORTED, "%s: unknown kv_dtype %d", fn, (int)kv_dtype);
    if (B < 0 || Hq < 1 || Hkv < 1 || k < 0 || W < 0 || N < 0)
        return fail(CMC_ERR_INVALID_ARGUMENT, "%s: need B >= 0, Hq, Hkv >= 1, k, W, N >= 0", fn);
    if (Hq % Hkv != 0) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: Hq=%d not a multiple of Hkv=%d", fn, Hq, Hkv);
    const int G = Hq / Hkv;
    if (G != 1 && G != 2 && G != 4 && G != 8)
        return fail(CMC_ERR_UNSUPPORTED, "%s: Hq/Hkv=%d not in {1,2,4,8}", fn, G);
    if (!supported_dh(Dh)) return fail(CMC_ERR_UNSUPPORTED, "%s: Dh=%d not in {64,128,256}", fn, Dh);
    if ((long long)k + W < 1) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: empty cache (k + W = 0)", fn);
    if (!idx && k > N) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: k=%d exceeds N=%d with idx == NULL", fn, k, N);
    if (k > 0 && N < 1) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: k=%d rows requested from an empty pool", fn, k);
    if (!(scale == scale) || isinf(scale)) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: scale must be finite", fn);
    if (T_new < 0 || (W > 0 && T_new > W))
        return fail(CMC_ERR_INVALID_ARGUMENT, "%s: need 0 <= T_new <= W (got T_new=%d W=%d)", fn, T_new, W);
    if (T_new > cmc::kMaxAppendRows)
        return fail(CMC_ERR_UNSUPPORTED, "%s: T_new=%d exceeds %d rows per call", fn, T_new, cmc::kMaxAppendRows);
    if (B > 65535 || Hkv > 65535) return fail(CMC_ERR_UNSUPPORTED, "%s: B and Hkv must be <= 65535", fn);
    // The kernel indexes a sequence's key list (k + W + T_new rows) with
    // 32-bit integers, and a bf16 (sequence, kv head) pool or ring with
    // 32-bit byte offsets from its base.
    if ((long long)k + W + T_new > INT_MAX)
        return fail(CMC_ERR_UNSUPPORTED, "%s: k + W + T_new = %lld exceeds %d", fn, (long long)k + W + T_new, INT_MAX);
    if (kv_dtype == CMC_BF16 && ((long long)N * Dh * 2 > 0xFFFFFFFFLL || (long long)W * Dh * 2 > 0xFFFFFFFFLL))
        return fail(CMC_ERR_UNSUPPORTED, "%s: a (sequence, kv head)'s pool (N=%d) or ring (W=%d) of bf16 rows of Dh=%d "
                    "must stay under 4 GiB", fn, N, W, Dh);
    if (W == 0) T_new = 0;  // no Tier-2: appending is a no-op
    if (B == 0) return ok();
    if (!q || !out) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: q and out must be non-null", fn);
    if (k > 0 && (!cme_k || !cme_v)) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: null Tier-1 pool", fn);
    if (W > 0 && (!win_k || !win_v || !win_count))
        return fail(CMC_ERR_INVALID_ARGUMENT, "%s: null Tier-2 window", fn);
    if (T_new > 0 && (!new_k || !new_v)) return fail(CMC_ERR_INVALID_ARGUMENT, "%s: null new rows", fn);
    if (misaligned(q) || misaligned(cme_k) || misaligned(cme_v) || misaligned(idx) || misaligned(k_len) ||
        misaligned(win_k) ||
        misaligned(win_v) || misaligned(win_count) || misaligned(out) || misaligned(workspace) ||
        misaligned(new_k) || misaligned(new_v))
        return fail(CMC_ERR_UNSUPPORTED, "%s: every pointer must be 16-byte aligned", fn);
    const cmc::DecodePlan pl = cmc::plan_decode(B, Hq, Hkv, Dh, k, W);
    char *counters, *partials;
    if (noalloc) {
        const size_t nctr = ((size_t)B + (size_t)B * Hkv) * sizeof(unsigned);
        if (nctr > kNoAllocCounterBytes || pl.ml_bytes + pl.acc_bytes > kNoAllocBytes - kNoAllocCounterBytes)
            return fail(CMC_ERR_UNSUPPORTED,
                        "%s: these sizes need %zu counter bytes (at most %zu) and %zu partial bytes (at most %zu) "
                        "of the library's fixed scratch; use cmc_decode_step with a workspace",
                        fn, nctr, kNoAllocCounterBytes, pl.ml_bytes + pl.acc_bytes,
                        kNoAllocBytes - kNoAllocCounterBytes);
        char *base = nullptr;
        if (cmc_status st = noalloc_scratch(fn, static_cast<hipStream_t>(stream), &base)) return st;
        counters = base;
        partials = base + kNoAllocCounterBytes;
    } else {
        if (!workspace || workspace_bytes < pl.total)
            return fail(CMC_ERR_WORKSPACE_TOO_SMALL, "%s: workspace of %zu bytes needed, %zu given", fn, pl.total,
                        workspace ? workspace_bytes : (size_t)0);
        counters = static_cast<char *>(workspace);
        partials = counters + pl.counter_bytes;
    }
    cmc::DecodeParams p{};
    p.q = q;
    p.cme_k = cme_k;
    p.cme_v = cme_v;
    p.idx = idx;
    p.k_len = k_len;
    p.win_k = W > 0 ? win_k : nullptr;
    p.win_v = W > 0 ? win_v : nullptr;
    p.win_count = W > 0 ? win_count : nullptr;
    p.new_k = T_new > 0 ? new_k : nullptr;
    p.new_v = T_new > 0 ? new_v : nullptr;
    p.out = out;
    p.seq_counter = reinterpret_cast<unsigned *>(counters);
    p.pair_counter = reinterpret_cast<unsigned *>(counters) + B;
    p.part_ml = reinterpret_cast<float *>(partials);
    p.part_acc = reinterpret_cast<float *>(partials + pl.ml_bytes);
    p.k = k;
    p.W = W;
    p.B = B;
    p.Hq = Hq;
    p.Hkv = Hkv;
    p.N = N;
    p.T_new = T_new;
    p.new_split = (pl.S > 1 && T_new > 0) ? 1 : 0;
    p.S = pl.S + p.new_split;
    p.chunk = pl.chunk;
    p.waves = pl.waves;
    p.qscale = cmc::decode_qscale(scale);
    hipError_t e = cmc::launch_two_tier_decode(p, kv_dtype == CMC_BF16, G, Dh, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    return ok();
}

}  // namespace

extern "C" {

cmc_status cmc_two_tier_decode(const float *q, const void *cme_k, const void *cme_v, const int32_t *idx,
                               int k, const void *win_k, const void *win_v, const int32_t *win_count,
                               int W, cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh, int N,
                               float scale, float *out, void *workspace, size_t workspace_bytes,
                               void *stream) {
    // Nothing is appended (T_new = 0), so the window is only read.
    return decode_impl("decode", q, cme_k, cme_v, idx, nullptr, k, const_cast<void *>(win_k), const_cast<void *>(win_v),
                       const_cast<int32_t *>(win_count), W, nullptr, nullptr, 0, kv_dtype, B, Hq, Hkv, Dh, N,
                       scale, out, workspace, workspace_bytes, stream);
}

cmc_status cmc_decode_step(const float *q, const void *cme_k, const void *cme_v, const int32_t *idx, int k,
                           void *win_k, void *win_v, int32_t *win_count, int W, const void *new_k,
                           const void *new_v, int T_new, cmc_dtype kv_dtype, int B, int Hq, int Hkv, int Dh,
                           int N, float scale, float *out, void *workspace, size_t workspace_bytes,
                           void *stream) {
    if (W > 0 && T_new < 1)
        return fail(CMC_ERR_INVALID_ARGUMENT, "decode_step: need 1 <= T_new <= W (got T_new=%d W=%d)", T_new, W);
    return decode_impl("decode_step", q, cme_k, cme_v, idx, nullptr, k, win_k, win_v, win_count, W, new_k, new_v, T_new,
                       kv_dtype, B, Hq, Hkv, Dh, N, scale, out, workspace, workspace_bytes, stream);
}

cmc_status cmc_decode_step_noalloc(const float *q, const void *cme_k, const void *cme_v, const int32_t *idx,
                                   int k, void *win_k, void *win_v, int32_t *win_count, int W, const void *new_k,
                                   const void *new_v, int T_new, cmc_dtype kv_dtype, int B, int Hq, int Hkv,
                                   int Dh, int N, float scale, float *out, void *stream) {
    if (W > 0 && T_new < 1)
        return fail(CMC_ERR_INVALID_ARGUMENT, "decode_step_noalloc: need 1 <= T_new <= W (got T_new=%d W=%d)",
                    T_new, W);
    return decode_impl("decode_step_noalloc", q, cme_k, cme_v, idx, nullptr, k, win_k, win_v, win_count, W, new_k,
                       new_v, T_new, kv_dtype, B, Hq, Hkv, Dh, N, scale, out, nullptr, 0, stream, true);
}

cmc_status cmc_two_tier_decode_ragged(const float *q, const void *cme_k, const void *cme_v, const int32_t *idx,
                                      const int32_t *k_len, int k, const void *win_k, const void *win_v,
                                      const int32_t *win_count, int W, cmc_dtype kv_dtype, int B, int Hq,
                                      int Hkv, int Dh, int N, float scale, float *out, void *workspace,
                                      size_t workspace_bytes, void *stream) {
    if (B > 0 && !k_len) return fail(CMC_ERR_INVALID_ARGUMENT, "decode_ragged: k_len must be non-null");
    return decode_impl("decode_ragged", q, cme_k, cme_v, idx, k_len, k, const_cast<void *>(win_k),
                       const_cast<void *>(win_v), const_cast<int32_t *>(win_count), W, nullptr, nullptr, 0,
                       kv_dtype, B, Hq, Hkv, Dh, N, scale, out, workspace, workspace_bytes, stream);
}

cmc_status cmc_decode_step_ragged(const float *q, const void *cme_k, const void *cme_v, const int32_t *idx,
                                  const int32_t *k_len, int k, void *win_k, void *win_v, int32_t *win_count,
                                  int W, const void *new_k, const void *new_v, int T_new, cmc_dtype kv_dtype,
                                  int B, int Hq, int Hkv, int Dh, int N, float scale, float *out,
                                  void *workspace, size_t workspace_bytes, void *stream) {
    if (B > 0 && !k_len) return fail(CMC_ERR_INVALID_ARGUMENT, "decode_step_ragged: k_len must be non-null");
    if (W > 0 && T_new < 1)
        return fail(CMC_ERR_INVALID_ARGUMENT, "decode_step_ragged: need 1 <= T_new <= W (got T_new=%d W=%d)",
                    T_new, W);
    return decode_impl("decode_step_ragged", q, cme_k, cme_v, idx, k_len, k, win_k, win_v, win_count, W, new_k,
                       new_v, T_new, kv_dtype, B, Hq, Hkv, Dh, N, scale, out, workspace, workspace_bytes, stream);
}

}  // extern "C"
