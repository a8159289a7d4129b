// Internal launch interface between the C ABI (cmc_api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace cmc {

// A decode workgroup has 4 or 8 waves, each streaming its own 16-key blocks;
// the workgroup combines them in LDS.  8 waves (at most 256 VGPRs each) are
// built only for heads whose kernels fit that without spilling: Dh <= 128
// with G <= 4, or one query head per kv head.
constexpr bool decode_waves_ok(int waves, int G, int Dh) {
    return waves == 4 || (waves == 8 && ((Dh <= 128 && G <= 4) || G == 1));
}

struct DecodeParams {
    const float *q;           // [B][Hq][Dh]
    const void *cme_k;        // [B][Hkv][N][Dh]
    const void *cme_v;
    const int32_t *idx;       // [B][k] or nullptr
    const int32_t *k_len;     // [B] pool rows used per sequence (clamped to [0, k]), or nullptr: all k
    void *win_k;              // [B][Hkv][W][Dh]; written only for rows appended this call
    void *win_v;
    int32_t *win_count;       // [B]; advanced by T_new when T_new > 0
    const void *new_k;        // [B][Hkv][T_new][Dh] rows appended by this call, or nullptr
    const void *new_v;
    float *out;               // [B][Hq][Dh]
    float *part_ml;           // [B][Hkv][S][G][2]   (running max in log2 units, denominator)
    float *part_acc;          // [B][Hkv][S][G][Dh]  (unnormalised numerator)
    unsigned *pair_counter;   // [B][Hkv] split arrivals, zero between calls
    unsigned *seq_counter;    // [B] kv-head arrivals, zero between calls
    int k, W, B, Hq, Hkv, N, T_new;
    int S, chunk;             // key-axis splits (launched) and keys per split
    int new_split;            // 1: the last split takes only the T_new appended rows
    int waves;                // waves per workgroup: 4 or 8
    float qscale;             // scale * log2(e)
};

// Rows one decode call may append (the launch packs T_new into 16 bits).
constexpr int kMaxAppendRows = 65535;

// Key-axis split plan; depends only on sizes, so the workspace query and the
// launch agree.  Workspace layout: [sequence counters | pair counters]
// (zero between calls), then the per-split partials.
struct DecodePlan {
    int S = 0, chunk = 0, waves = 4;  // S splits over the k + W rows
    int S_alloc = 0;                  // partials reserved: S, plus one for appended rows when S > 1 and W > 0
    size_t counter_bytes = 0, ml_bytes = 0, acc_bytes = 0, total = 0;
};
DecodePlan plan_decode(int B, int Hq, int Hkv, int Dh, int k, int W);

hipError_t launch_two_tier_decode(const DecodeParams &p, bool bf16, int G, int Dh, hipStream_t stream);
float decode_qscale(float scale);

struct AppendParams {
    void *win_k, *win_v;
    int32_t *win_count;
    const void *new_k, *new_v;
    int B, Hkv, W, T_new;
    int row_vecs;             // 16-byte vectors per row (Dh * elem / 16)
};
hipError_t launch_window_append(const AppendParams &p, hipStream_t stream);

struct GatherParams {
    const void *cme_k, *cme_v;  // [B][Hkv][N][Dh]
    const int32_t *idx;         // [B][idx_stride] or nullptr: rows 0..k-1
    const int32_t *k_len;       // [B] or nullptr: all k
    void *out_k, *out_v;        // [B][Hkv][k][Dh]
    int B, Hkv, N, k, idx_stride;
    int row_vecs;               // 16-byte vectors per row
};
hipError_t launch_gather(const GatherParams &p, hipStream_t stream);

struct SelectParams {
    const void *sel_keys;     // [B][N][D] fp32 or bf16 (keys_bf16)
    const float *q_vec;       // [B][D]
    float *scores;            // [B][N]
    int32_t *idx_out;         // [B][idx_stride]
    int B, N, D, k;
    int idx_stride;           // >= k
    const int32_t *n_rows;    // [B] candidate rows per sequence, or nullptr: all N
    const int32_t *q_rows;    // [B] pinned question rows per sequence, or nullptr: none
    int32_t *k_out;           // [B] entries written per sequence, or nullptr
    float *norms;             // [B][N] row norms |m_j| (0 past n_b), or nullptr
    bool keys_bf16;           // sel_keys holds bf16 bit patterns
};
constexpr int kSelectMaxN = 32768;
hipError_t launch_select(const SelectParams &p, hipStream_t stream);

struct LocateParams {
    const float *norms;         // [B][N]
    const int32_t *n_rows;      // [B] or nullptr: all N
    const int32_t *chunk_offset;  // [B][n_chunks] or nullptr: chunk i at i * chunk_tokens
    const int32_t *ctx_len;     // [B]
    int32_t *alpha_out;         // [B] or nullptr
    int32_t *start_out;         // [B]
    int B, N, mems_per_chunk, n_chunks, chunk_tokens, W;
};
hipError_t launch_locate(const LocateParams &p, hipStream_t stream);

struct DenoiseParams {
    const void *emb;            // [B][n][H] fp32 or bf16
    const int32_t *n_tokens;    // [B] or nullptr: all n
    uint8_t *pass;              // [B][n] Eq. 3 bits (workspace)
    float *max_cos;             // [B][n] or nullptr
    uint8_t *keep_out;          // [B][n] or nullptr
    int32_t *kept_idx;          // [B][n]
    int32_t *kept_count;        // [B]
    int32_t *chunk_offset;      // [B][max_chunks] or nullptr
    int32_t *n_chunks;          // [B] or nullptr
    int B, n, H, g;
    float tau;
    int keep_min_every, chunk_tokens, max_chunks;
};
constexpr int kDenoiseMaxG = 4;

struct BridgeParams {
    const uint16_t *h;          // [M][Hc] bf16 CME vectors
    const uint16_t *w1;         // [F][Hc] bf16
    const float *b1;            // [F]
    const uint16_t *w2;         // [Hd][F] bf16
    const float *b2;            // [Hd]
    const float *ln_gamma;      // [Hd]
    const float *ln_beta;       // [Hd]
    uint16_t *hidden;           // [M][F] bf16 (workspace)
    float *out;                 // [M][Hd]
    float *h_norms;             // [M] |h_j|, or nullptr
    int M, Hc, F, Hd;
    float nu, eps;
};
// Tile multiples of the MemoryBridge GEMMs: Hc (K of the first) a multiple of
// kBridgeK, F and Hd (N of both, K of the second) multiples of kBridgeN.
constexpr int kBridgeK = 64, kBridgeN = 128;
hipError_t launch_memory_bridge(const BridgeParams &p, hipStream_t stream);
hipError_t launch_denoise(const DenoiseParams &p, bool bf16, hipStream_t stream);

}  // namespace cmc
