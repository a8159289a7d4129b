// Graph-based context denoising (Sec. 2.1, Eq. 3): token i of a context is
// kept when its cosine similarity to one of its next g tokens reaches tau;
// the minimum keep interval m (hyper-parameter table; appendix on the
// denoising threshold) makes any m consecutive positions hold a kept token.
// The survivors, in order, form the denoised context C' that is cut into
// chunks of t tokens; the position of each chunk's first token in C is the
// offset CME-guided localization needs.
//
// denoise_score_kernel (fp32 embeddings; bf16 too when the Gram kernel below
// is switched off): one wave per TT consecutive tokens.  Lanes split
// the hidden dimension (16-byte loads, 64 x 16 bytes per pass over a row);
// the wave loads the TT + g rows it needs for P passes at once (one round
// trip covers a 1280-wide bf16 row), keeps the last g rows of a pass in
// registers, and accumulates the TT + g squared norms and the TT x g
// neighbour dot products per lane, then reduces them across the wave.  The
// halo of g rows is the next wave's first rows, so it is mostly served by
// L2.  Output: the fp32 statistic max_cos (-inf where a token has no
// neighbour) and the Eq. 3 bit.
//
// denoise_gram_kernel (bf16): the same statistic from the Gram matrix of 16
// consecutive rows -- 16 - g tokens and their g-row halo -- accumulated by
// v_mfma_f32_16x16x32_bf16 with one fragment as both operands (lane l holds
// 8 elements of row l % 16, so A = X and B = X^T).  The norms are its
// diagonal, the neighbour dots its first g super-diagonals; no cross-lane
// reductions and almost no VALU work, which bounds the VALU variant above.
//
// denoise_select_kernel: one 1024-thread workgroup per sequence scans the
// Eq. 3 bits.  With a(i) the last passing position before i (-1 if none),
// the floor keeps exactly the positions a(i) + m, a(i) + 2m, ... before the
// next passing one, so kept(i) = pass(i) or (i - a(i)) mod m == 0.  a(i) is
// a block-wide max-scan, the output slots a sum-scan; 8 positions per
// thread per round, carried across rounds.
#include <limits.h>

#include "device_common.hpp"
#include "kernels.hpp"

namespace cmc {

namespace {

// Build-time tuning knobs: tokens per wave, row passes loaded at once.
#ifndef CMC_DENOISE_TOKENS
#define CMC_DENOISE_TOKENS 8
#endif
#ifndef CMC_DENOISE_PASSES
#define CMC_DENOISE_PASSES 3
#endif
constexpr int kTokensPerWave = CMC_DENOISE_TOKENS;
constexpr int kPasses = CMC_DENOISE_PASSES;

__device__ __forceinline__ int clamp_tokens(int v, int hi) { return v < 0 ? 0 : (v > hi ? hi : v); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// c + a.lo * b.lo + a.hi * b.hi for two packed bf16 pairs (v_dot2_f32_bf16).
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

template <typename T>
struct Lane16;  // one 16-byte lane load widened to fp32
template <>
struct Lane16<float> {
    static constexpr int N = 4;
    __device__ __forceinline__ static void widen(const uint4 &u, float (&f)[4]) {
        f[0] = __uint_as_float(u.x);
        f[1] = __uint_as_float(u.y);
        f[2] = __uint_as_float(u.z);
        f[3] = __uint_as_float(u.w);
    }
};
template <>
struct Lane16<uint16_t> {
    static constexpr int N = 8;
    __device__ __forceinline__ static void widen(const uint4 &u, float (&f)[8]) {
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __uint_as_float(w[i] << 16);
            f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
};

template <typename T, int G>
__global__ __launch_bounds__(256) void denoise_score_kernel(DenoiseParams p) {
    constexpr int TT = kTokensPerWave, R = TT + G, VEC = Lane16<T>::N, P = kPasses, SPAN = kWave * VEC;
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nb = p.n_tokens ? clamp_tokens(p.n_tokens[b], p.n) : p.n;
    const char *base = static_cast<const char *>(p.emb) + (size_t)b * p.n * p.H * sizeof(T);
    const size_t row_bytes = (size_t)p.H * sizeof(T);
    __shared__ float s_nn[4][R], s_dd[4][TT][G];

    // Each wave walks groups of TT tokens with the grid's stride (no
    // barriers below: the LDS staging is private to the wave).
    for (int i0 = (blockIdx.x * 4 + wave) * TT; i0 < p.n; i0 += gridDim.x * 4 * TT) {
        if (i0 >= nb) {  // wave-uniform: positions past the sequence have no statistic
            const int i = i0 + lane;
            if (lane < TT && i < p.n) {
                const size_t o = (size_t)b * p.n + i;
                if (p.max_cos) p.max_cos[o] = -INFINITY;
                p.pass[o] = 0;
            }
            continue;
        }
        float nn[R], dd[TT][G];
#pragma unroll
        for (int r = 0; r < R; ++r) nn[r] = 0.f;
#pragma unroll
        for (int t = 0; t < TT; ++t)
#pragma unroll
            for (int d = 0; d < G; ++d) dd[t][d] = 0.f;

        for (int eb = 0; eb < p.H; eb += P * SPAN) {
            // All R rows of P passes are loaded up front: rows past the
            // sequence are clamped to its last row and columns past H to the
            // row's last 16 bytes (in bounds), and zeroed after the load, so
            // no load sits behind a branch.
            uint4 raw[P][R];
#pragma unroll
            for (int pp = 0; pp < P; ++pp) {
                const int ec = min(eb + pp * SPAN + lane * VEC, p.H - VEC);
#pragma unroll
                for (int r = 0; r < R; ++r)
                    raw[pp][r] = *reinterpret_cast<const uint4 *>(base + (size_t)min(i0 + r, nb - 1) * row_bytes +
                                                                  (size_t)ec * sizeof(T));
            }
#pragma unroll
            for (int pp = 0; pp < P; ++pp) {
                const bool col_on = eb + pp * SPAN + lane * VEC < p.H;
                if constexpr (sizeof(T) == 2) {
                    // bf16: v_dot2 on packed pairs (two products per op, fp32
                    // accumulation, no widening).
                    uint32_t win[G + 1][4];  // rows r-G .. r (ring by unrolled index)
#pragma unroll
                    for (int r = 0; r < R; ++r) {
                        const bool on = col_on && i0 + r < nb;
                        const uint32_t w[4] = {on ? raw[pp][r].x : 0u, on ? raw[pp][r].y : 0u,
                                               on ? raw[pp][r].z : 0u, on ? raw[pp][r].w : 0u};
#pragma unroll
                        for (int k = 0; k < 4; ++k) nn[r] = dot2_bf16(w[k], w[k], nn[r]);
#pragma unroll
                        for (int d = 1; d <= G; ++d) {
                            if (r - d >= 0 && r - d < TT) {
#pragma unroll
                                for (int k = 0; k < 4; ++k)
                                    dd[r - d][d - 1] = dot2_bf16(win[(r - d) % (G + 1)][k], w[k], dd[r - d][d - 1]);
                            }
                        }
#pragma unroll
                        for (int k = 0; k < 4; ++k) win[r % (G + 1)][k] = w[k];
                    }
                } else {
                    float win[G + 1][VEC];  // rows r-G .. r of this lane slice (ring by unrolled index)
#pragma unroll
                    for (int r = 0; r < R; ++r) {
                        float x[VEC];
                        Lane16<T>::widen(raw[pp][r], x);
                        if (!col_on || i0 + r >= nb) {
#pragma unroll
                            for (int v = 0; v < VEC; ++v) x[v] = 0.f;
                        }
#pragma unroll
                        for (int v = 0; v < VEC; ++v) nn[r] = fmaf(x[v], x[v], nn[r]);
#pragma unroll
                        for (int d = 1; d <= G; ++d) {
                            if (r - d >= 0 && r - d < TT) {
                                const float(&y)[VEC] = win[(r - d) % (G + 1)];
#pragma unroll
                                for (int v = 0; v < VEC; ++v)
                                    dd[r - d][d - 1] = fmaf(y[v], x[v], dd[r - d][d - 1]);
                            }
                        }
#pragma unroll
                        for (int v = 0; v < VEC; ++v) win[r % (G + 1)][v] = x[v];
                    }
                }
            }
        }
        // Wave sums (all reductions first, so their exchange steps interleave),
        // staged in LDS private to the wave so that lane t < TT can finish token
        // i0 + t from its own registers.
#pragma unroll
        for (int r = 0; r < R; ++r) nn[r] = lane_reduce<OpSum, 1, kWave>(nn[r]);
#pragma unroll
        for (int t = 0; t < TT; ++t)
#pragma unroll
            for (int d = 0; d < G; ++d) dd[t][d] = lane_reduce<OpSum, 1, kWave>(dd[t][d]);
        if (lane == 0) {
#pragma unroll
            for (int r = 0; r < R; ++r) s_nn[wave][r] = nn[r];
#pragma unroll
            for (int t = 0; t < TT; ++t)
#pragma unroll
                for (int d = 0; d < G; ++d) s_dd[wave][t][d] = dd[t][d];
        }
        asm volatile("" ::: "memory");  // one wave's LDS accesses execute in order
        const int i = i0 + lane;
        float best = -INFINITY;
        if (lane < TT && i < nb) {
            const float ni = fmaxf(sqrtf(s_nn[wave][lane]), 1e-8f);
#pragma unroll
            for (int d = 1; d <= G; ++d) {
                if (i + d < nb)
                    best = fmaxf(best, s_dd[wave][lane][d - 1] / (ni * fmaxf(sqrtf(s_nn[wave][lane + d]), 1e-8f)));
            }
        }
        if (lane < TT && i < p.n) {
            const size_t o = (size_t)b * p.n + i;
            if (p.max_cos) p.max_cos[o] = best;
            p.pass[o] = (uint8_t)(i < nb && best >= p.tau);
        }
        asm volatile("" ::: "memory");  // this group's LDS reads before the next group's writes
    }
}

// Build-time tuning knob: 32-column k-steps whose loads are issued together
// (a 1280-wide bf16 row in one batch: the wave's whole 40 KB in flight, 218
// VGPRs, two waves per SIMD).  On 64 GPT2-Large-sized contexts (131,392
// tokens) a call took 80.8 us with batches of 8, 78.1 with 10, 72.1 with 20
// and 70.3 with 40.
#ifndef CMC_DENOISE_GRAM_BATCH
#define CMC_DENOISE_GRAM_BATCH 40
#endif

// Gram matrix of the 16 rows a wave owns: every k-step's loads are clamped
// in bounds (row to the sequence's last row, column to the row's last 16
// bytes); with MASK, lanes whose row or column is past the end contribute
// zeros.  k-steps past the row's end in the last batch are skipped
// (uniform branch around the MFMA only).
template <bool MASK>
__device__ __forceinline__ floatx4 gram_tile(const char *row_base, bool row_on, int q4, int H) {
    constexpr int KB = CMC_DENOISE_GRAM_BATCH;
    const int KS = (H + 31) / 32;
    floatx4 c = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < KS; k0 += KB) {
        uint4 v[KB];
#pragma unroll
        for (int j = 0; j < KB; ++j) {
            const int col = min((k0 + j) * 32 + 8 * q4, H - 8);
            v[j] = *reinterpret_cast<const uint4 *>(row_base + (size_t)col * 2);
        }
#pragma unroll
        for (int j = 0; j < KB; ++j) {
            if (k0 + j < KS) {
                uint4 x = v[j];
                if constexpr (MASK) {
                    if (!row_on || (k0 + j) * 32 + 8 * q4 >= H) x = make_uint4(0, 0, 0, 0);
                }
                const bf16x8 f = __builtin_bit_cast(bf16x8, x);
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f, f, c, 0, 0, 0);
            }
        }
    }
    return c;
}

template <int G>
__global__ __launch_bounds__(256) void denoise_gram_kernel(DenoiseParams p) {
    constexpr int TT = 16 - G;  // tokens per wave; rows i0 .. i0 + 15
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, q4 = lane >> 4;
    const int nb = p.n_tokens ? clamp_tokens(p.n_tokens[b], p.n) : p.n;
    const char *base = static_cast<const char *>(p.emb) + (size_t)b * p.n * p.H * 2;
    const size_t row_bytes = (size_t)p.H * 2;
    __shared__ float s_c[4][16][17];

    for (int i0 = (blockIdx.x * 4 + wave) * TT; i0 < p.n; i0 += gridDim.x * 4 * TT) {
        if (i0 >= nb) {  // wave-uniform: positions past the sequence have no statistic
            const int i = i0 + lane;
            if (lane < TT && i < p.n) {
                const size_t o = (size_t)b * p.n + i;
                if (p.max_cos) p.max_cos[o] = -INFINITY;
                p.pass[o] = 0;
            }
            continue;
        }
        const bool row_on = i0 + r16 < nb;
        const char *row_base = base + (size_t)min(i0 + r16, nb - 1) * row_bytes;
        // Unmasked fast path when all 16 rows exist and the row is whole k-steps.
        const floatx4 c = (i0 + 16 <= nb && p.H % 32 == 0) ? gram_tile<false>(row_base, row_on, q4, p.H)
                                                            : gram_tile<true>(row_base, row_on, q4, p.H);
        // C fragment: lane l, element r -> row 4 (l / 16) + r, column l % 16.
#pragma unroll
        for (int r = 0; r < 4; ++r) s_c[wave][4 * q4 + r][r16] = c[r];
        asm volatile("" ::: "memory");  // one wave's LDS accesses execute in order
        const int i = i0 + lane;
        float best = -INFINITY;
        if (lane < TT && i < nb) {
            const float ni = fmaxf(sqrtf(s_c[wave][lane][lane]), 1e-8f);
#pragma unroll
            for (int d = 1; d <= G; ++d) {
                if (i + d < nb)
                    best = fmaxf(best, s_c[wave][lane][lane + d] /
                                           (ni * fmaxf(sqrtf(s_c[wave][lane + d][lane + d]), 1e-8f)));
            }
        }
        if (lane < TT && i < p.n) {
            const size_t o = (size_t)b * p.n + i;
            if (p.max_cos) p.max_cos[o] = best;
            p.pass[o] = (uint8_t)(i < nb && best >= p.tau);
        }
        asm volatile("" ::: "memory");  // this group's LDS reads before the next group's writes
    }
}

// denoise_gram_wg_kernel (bf16): the same statistic with the four waves of a
// workgroup on 64 consecutive rows, 16 each (one batch of whole rows per
// wave, as above), scoring 64 - g tokens: only the last g rows are re-read
// by the next workgroup, so 64 / (64 - g) rows are streamed per token
// instead of 16 / (16 - g).  The dot products that straddle two waves come
// from one more MFMA per k-step, the wave's own fragment against the next
// wave's first g rows, which that wave hands over through LDS (lanes with
// row < g, 16 bytes per k-step).  The norms of those rows are read from the
// next wave's Gram diagonal.  Every barrier sits in control flow that is
// uniform over the workgroup (the loop over groups, the sequence-end test and
// the k batches depend only on the block, the sequence and H).  Two
// workgroups per CU (two waves per SIMD, at most 256 VGPRs each): the
// branch-free batches would otherwise be scheduled into more registers.
template <int G>
__global__ __launch_bounds__(256, 2) void denoise_gram_wg_kernel(DenoiseParams p) {
    constexpr int KB = CMC_DENOISE_GRAM_BATCH;
    constexpr int TT = 64 - G;  // tokens per workgroup; rows i0 .. i0 + 63
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, q4 = lane >> 4;
    const int nb = p.n_tokens ? clamp_tokens(p.n_tokens[b], p.n) : p.n;
    const char *base = static_cast<const char *>(p.emb) + (size_t)b * p.n * p.H * 2;
    const size_t row_bytes = (size_t)p.H * 2;
    const int KS = (p.H + 31) / 32;
    __shared__ uint4 s_slot[4][KB][4][G];  // wave w's rows 0 .. g-1, per k-step and column quarter
    __shared__ float s_c[4][16][17];       // each wave's Gram matrix
    __shared__ float s_x[4][16][G];        // each wave's rows against the next wave's first g rows

    for (int i0 = blockIdx.x * TT; i0 < p.n; i0 += gridDim.x * TT) {  // uniform
        if (i0 >= nb) {  // uniform: positions past the sequence have no statistic
            for (int t = threadIdx.x; t < TT; t += 256) {
                const int i = i0 + t;
                if (i < p.n) {
                    const size_t o = (size_t)b * p.n + i;
                    if (p.max_cos) p.max_cos[o] = -INFINITY;
                    p.pass[o] = 0;
                }
            }
            continue;
        }
        const int row = i0 + 16 * wave + r16;
        const bool on = row < nb;
        const char *rb = base + (size_t)min(row, nb - 1) * row_bytes;
        const bool whole = i0 + 64 <= nb && p.H % 32 == 0;  // uniform: no masking needed
        floatx4 c = {0.f, 0.f, 0.f, 0.f}, x = {0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < KS; k0 += KB) {  // uniform
            uint4 v[KB];
#pragma unroll
            for (int j = 0; j < KB; ++j) {
                const int col = min((k0 + j) * 32 + 8 * q4, p.H - 8);
                v[j] = *reinterpret_cast<const uint4 *>(rb + (size_t)col * 2);
            }
            if (!whole) {
#pragma unroll
                for (int j = 0; j < KB; ++j)
                    if (!on || (k0 + j) * 32 + 8 * q4 >= p.H) v[j] = make_uint4(0, 0, 0, 0);
            }
            if (wave > 0 && r16 < G) {
#pragma unroll
                for (int j = 0; j < KB; ++j) s_slot[wave][j][q4][r16] = v[j];
            }
            __syncthreads();
            // A whole batch (every batch when KB divides H / 32) runs without
            // a branch per k-step, so the scheduler can overlap the straddling
            // operands' LDS reads with the MFMAs; a partial last batch guards
            // each k-step (uniform branches).
#define CMC_DN_MMA(LIVE_)                                                                                      \
    do {                                                                                                       \
        _Pragma("unroll") for (int j = 0; j < KB; ++j) {                                                       \
            if (LIVE_(j)) {                                                                                    \
                const bf16x8 f = __builtin_bit_cast(bf16x8, v[j]);                                             \
                c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f, f, c, 0, 0, 0);                                 \
            }                                                                                                  \
        }                                                                                                      \
        if (wave < 3) { /* wave-uniform */                                                                     \
            /* the next wave's fragments XB k-steps at a time: one LDS round trip per XB straddling MFMAs */  \
            constexpr int XB = 8;                                                                              \
            _Pragma("unroll") for (int j0 = 0; j0 < KB; j0 += XB) {                                            \
                uint4 u[XB];                                                                                   \
                _Pragma("unroll") for (int jj = 0; jj < XB; ++jj)                                              \
                    u[jj] = (j0 + jj < KB && r16 < G) ? s_slot[wave + 1][min(j0 + jj, KB - 1)][q4][r16 % G]    \
                                                      : make_uint4(0, 0, 0, 0);                                \
                _Pragma("unroll") for (int jj = 0; jj < XB; ++jj) {                                            \
                    if (j0 + jj < KB && LIVE_(j0 + jj))                                                        \
                        x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, v[j0 + jj]),    \
                                                                     __builtin_bit_cast(bf16x8, u[jj]), x, 0, 0, 0); \
                }                                                                                              \
            }                                                                                                  \
        }                                                                                                      \
    } while (0)
#define CMC_DN_ALL(j_) true
#define CMC_DN_IN(j_) (k0 + (j_) < KS)
            if (k0 + KB <= KS) CMC_DN_MMA(CMC_DN_ALL);  // uniform
            else CMC_DN_MMA(CMC_DN_IN);
#undef CMC_DN_ALL
#undef CMC_DN_IN
#undef CMC_DN_MMA
            if (k0 + KB < KS) __syncthreads();  // uniform: the slots are read before the next batch writes them
        }
        // C fragment: lane l, element e -> row 4 (l / 16) + e, column l % 16.
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            s_c[wave][4 * q4 + e][r16] = c[e];
            if (r16 < G) s_x[wave][4 * q4 + e][r16] = x[e];
        }
        __syncthreads();
        const int t = 16 * wave + lane;  // token of the workgroup (lanes < 16)
        const int i = i0 + t;
        if (lane < 16 && t < TT) {
            float best = -INFINITY;
            if (i < nb) {
                const float ni = fmaxf(sqrtf(s_c[wave][lane][lane]), 1e-8f);
#pragma unroll
                for (int d = 1; d <= G; ++d) {
                    if (i + d < nb) {
                        const int u = lane + d;  // u >= 16 only below wave 3 (t < TT)
                        const float dot = u < 16 ? s_c[wave][lane][u] : s_x[wave][lane][u - 16];
                        const float nn = u < 16 ? s_c[wave][u][u] : s_c[min(wave + 1, 3)][u - 16][u - 16];
                        best = fmaxf(best, dot / (ni * fmaxf(sqrtf(nn), 1e-8f)));
                    }
                }
            }
            if (i < p.n) {
                const size_t o = (size_t)b * p.n + i;
                if (p.max_cos) p.max_cos[o] = best;
                p.pass[o] = (uint8_t)(i < nb && best >= p.tau);
            }
        }
        __syncthreads();  // the Gram matrices are read before the next group writes them
    }
}

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kPerThread = 8;

// Block-wide exclusive scans over thread order (sum and max), with the
// block total / maximum returned through `total`.
__device__ __forceinline__ int block_excl_sum(int v, int *s_w, int &total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    if (lane == kWave - 1) s_w[wave] = x;
    __syncthreads();
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        base += w < wave ? s_w[w] : 0;
        tot += s_w[w];
    }
    __syncthreads();
    total = tot;
    return base + x - v;
}

__device__ __forceinline__ int block_excl_max(int v, int *s_w, int &total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(x, off);
        if (lane >= off) x = max(x, y);
    }
    const int prev_in_wave = __shfl_up(x, 1);
    if (lane == kWave - 1) s_w[wave] = x;
    __syncthreads();
    int base = INT_MIN, tot = INT_MIN;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        base = w < wave ? max(base, s_w[w]) : base;
        tot = max(tot, s_w[w]);
    }
    __syncthreads();
    total = tot;
    return lane > 0 ? max(base, prev_in_wave) : base;
}

__global__ __launch_bounds__(kSelThreads) void denoise_select_kernel(DenoiseParams p) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int nb = p.n_tokens ? clamp_tokens(p.n_tokens[b], p.n) : p.n;
    const int m = p.keep_min_every;
    const uint8_t *pass = p.pass + (size_t)b * p.n;
    int32_t *idx = p.kept_idx + (size_t)b * p.n;
    __shared__ int s_w[kSelWaves];

    int carry_last = -1, carry_count = 0;
    for (int r0 = 0; r0 < nb; r0 += kSelThreads * kPerThread) {
        const int j0 = r0 + tid * kPerThread;
        uint32_t bits = 0;
        int last = -1;
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int i = j0 + u;
            if (i < nb && pass[i]) {
                bits |= 1u << u;
                last = i;
            }
        }
        int block_last;
        const int before = block_excl_max(last, s_w, block_last);
        int a = max(carry_last, before);
        uint32_t keep = 0;
        int cnt = 0;
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int i = j0 + u;
            if (i < nb) {
                const bool ps = (bits >> u) & 1u;
                const bool k = ps || (m > 0 && (i - a) % m == 0);
                if (ps) a = i;
                if (k) {
                    keep |= 1u << u;
                    ++cnt;
                }
            }
        }
        int block_cnt;
        int o = carry_count + block_excl_sum(cnt, s_w, block_cnt);
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int i = j0 + u;
            if ((keep >> u) & 1u) {
                idx[o] = i;
                if (p.chunk_offset && p.chunk_tokens > 0 && o % p.chunk_tokens == 0)
                    p.chunk_offset[(size_t)b * p.max_chunks + o / p.chunk_tokens] = i;
                ++o;
            }
            if (p.keep_out && i < nb) p.keep_out[(size_t)b * p.n + i] = (uint8_t)((keep >> u) & 1u);
        }
        carry_last = max(carry_last, block_last);
        carry_count += block_cnt;
    }
    const int count = carry_count;
    for (int i = count + tid; i < p.n; i += kSelThreads) idx[i] = -1;
    if (p.keep_out)
        for (int i = nb + tid; i < p.n; i += kSelThreads) p.keep_out[(size_t)b * p.n + i] = 0;
    if (p.chunk_tokens > 0) {
        const int nc = (count + p.chunk_tokens - 1) / p.chunk_tokens;
        if (p.chunk_offset)
            for (int c = nc + tid; c < p.max_chunks; c += kSelThreads)
                p.chunk_offset[(size_t)b * p.max_chunks + c] = -1;
        if (tid == 0 && p.n_chunks) p.n_chunks[b] = nc;
    }
    if (tid == 0) p.kept_count[b] = count;
}

// Build-time tuning knob: workgroups per sequence (0: one per 4 TT tokens;
// otherwise at most this many, each walking its groups with the grid's
// stride).
#ifndef CMC_DENOISE_WG_PER_SEQ
#define CMC_DENOISE_WG_PER_SEQ 0
#endif

// Build-time tuning knob: 1 scores bf16 embeddings with denoise_gram_kernel.
#ifndef CMC_DENOISE_MFMA
#define CMC_DENOISE_MFMA 1
#endif

// Build-time tuning knob: the smallest g that runs denoise_gram_wg_kernel
// (64 rows per workgroup); smaller g run denoise_gram_kernel (16 rows per
// wave).  On 64 GPT2-Large-sized contexts, per call (us), 16-row waves /
// 64-row workgroups: g = 1 63.8-64.2 / 63.3-63.5, g = 2 65.8-65.9 /
// 63.9, g = 3 68.0-68.4 / 65.1-65.2, g = 4 68.7-69.3 (with 16-row waves
// 79.1-79.5) / 65.6-66.0 -- the per-wave kernel grows with the halo.
#ifndef CMC_DENOISE_WG_MIN_G
#define CMC_DENOISE_WG_MIN_G 1
#endif

template <int G>
hipError_t launch_gram(const DenoiseParams &p, hipStream_t stream) {
    constexpr bool kWg = G >= CMC_DENOISE_WG_MIN_G;
    constexpr int per_wg = kWg ? 64 - G : 4 * (16 - G);
    int gx = (p.n + per_wg - 1) / per_wg;
    if (CMC_DENOISE_WG_PER_SEQ > 0 && gx > CMC_DENOISE_WG_PER_SEQ) gx = CMC_DENOISE_WG_PER_SEQ;
    if constexpr (kWg) denoise_gram_wg_kernel<G><<<dim3(gx, p.B), 256, 0, stream>>>(p);
    else denoise_gram_kernel<G><<<dim3(gx, p.B), 256, 0, stream>>>(p);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_scores(const DenoiseParams &p, hipStream_t stream) {
    if (sizeof(T) == 2 && CMC_DENOISE_MFMA) {
        switch (p.g) {
            case 1: return launch_gram<1>(p, stream);
            case 2: return launch_gram<2>(p, stream);
            case 3: return launch_gram<3>(p, stream);
            case 4: return launch_gram<4>(p, stream);
            default: return hipErrorInvalidValue;
        }
    }
    int gx = (p.n + 4 * kTokensPerWave - 1) / (4 * kTokensPerWave);
    if (CMC_DENOISE_WG_PER_SEQ > 0 && gx > CMC_DENOISE_WG_PER_SEQ) gx = CMC_DENOISE_WG_PER_SEQ;
    dim3 grid(gx, p.B);
    switch (p.g) {
        case 1: denoise_score_kernel<T, 1><<<grid, 256, 0, stream>>>(p); break;
        case 2: denoise_score_kernel<T, 2><<<grid, 256, 0, stream>>>(p); break;
        case 3: denoise_score_kernel<T, 3><<<grid, 256, 0, stream>>>(p); break;
        case 4: denoise_score_kernel<T, 4><<<grid, 256, 0, stream>>>(p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_denoise(const DenoiseParams &p, bool bf16, hipStream_t stream) {
    if (p.B == 0) return hipSuccess;
    if (p.n > 0) {
        const hipError_t e = bf16 ? launch_scores<uint16_t>(p, stream) : launch_scores<float>(p, stream);
        if (e != hipSuccess) return e;
    }
    denoise_select_kernel<<<p.B, kSelThreads, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace cmc
