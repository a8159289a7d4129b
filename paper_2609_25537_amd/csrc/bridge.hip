// MemoryBridge (Sec. 2.3): each CME vector h (encoder width Hc) becomes a
// decoder-ready memory row
//   m_hat = LayerNorm(W2 GELU(W1 h + b1) + b2)          (LayerNorm per the appendix)
//   m     = nu tanh(m_hat) * min(1, 2 nu / |nu tanh(m_hat)|)   (the section's cap)
// -- the selection keys of Tier-1.
//
// gemm_nt_kernel: C[M][N] = A[M][K] . B[N][K]^T on MFMA, bf16 operands, fp32
// accumulation.  A workgroup of WGM x WGN waves computes a tile of WGM WTM x
// WGN WTN, each wave WTM x WTN as 16 x 16 v_mfma_f32_16x16x32_bf16 tiles:
// 256 x 256 from eight waves of 128 x 64 where N allows (one workgroup per
// CU), else 128 x 128 from four waves of 64 x 64 (three per CU).  K advances
// BK at a time through two LDS buffers, staged from global memory through
// register sets used in turn (two by default), so a slice's loads have the
// MFMA work of the slices before it to land.  LDS rows are padded by 8 bf16
// (80 or 144 bytes) so that the 16-byte fragment reads of 8 consecutive
// rows hit 8 disjoint groups of 4 banks.  Tiles are handed out so that each
// XCD (workgroups are dealt round-robin to the 8 XCDs) runs a contiguous run
// of them, walked in groups of a few tile rows (see gemm_tile).  The
// epilogue (store_tile) adds the bias and, for the first layer, applies GELU
// and rounds to bf16 (the hidden activations, kept in the workspace); the
// second layer's fp32 result goes to the output.
//
// bridge_norm_kernel: one wave per output row, in place, the row held in
// registers: mean and biased variance (two passes over the registers),
// LayerNorm with gamma/beta, nu tanh, the row norm, and the cap.
//
// cme_norm_kernel (optional): |h_j| of every input row, the norms that
// CME-guided localization ranks (the capped output rows cannot serve: the
// cap pins the norm of every row whose nu tanh(m_hat) exceeds 2 nu at
// exactly 2 nu, which at decoder widths is every row).
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"

namespace cmc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

struct GemmParams {
    const uint16_t *A;  // [M][K]
    const uint16_t *B;  // [N][K]
    const float *bias;  // [N]
    void *C;            // [M][N]: bf16 (epilogue 0) or fp32 (epilogue 1)
    int M, N, K;
};

// GELU(x) = x Phi(x), Phi(x) = (1 + erf(x / sqrt 2)) / 2, with erfc(z) for z =
// |x| / sqrt 2 >= 0 from Abramowitz & Stegun 7.1.26: erfc(z) = t (a1 + t (a2 +
// t (a3 + t (a4 + t a5)))) exp(-z^2), t = 1 / (1 + p z), absolute error at most
// 1.5e-7, below the bf16 rounding the hidden activations then take.  Phi(x) is
// 1 - erfc(z) / 2 for x >= 0 and erfc(z) / 2 below.
__device__ __forceinline__ float gelu_erf(float x) {
    const float z = fabsf(x) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, z, 1.f));
    const float poly =
        t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f), 0.254829592f);
    const float half_erfc = 0.5f * poly * __builtin_amdgcn_exp2f(-1.4426950408889634f * z * z);
    return x * (x >= 0.f ? 1.f - half_erfc : half_erfc);
}

// Build-time tuning knob: 1 evaluates the cap's tanh as below, 0 with the
// library tanhf.
#ifndef CMC_BRIDGE_FAST_TANH
#define CMC_BRIDGE_FAST_TANH 1
#endif

// tanh for the cap, within 4 units of 2^-24 absolute everywhere:
//   |x| <  0.625: x + x^3 P(x^2), P a cubic fitted here by weighted least
//                 squares to (tanh(x)/x - 1)/x^2 (1.35 units in fp32 Horner);
//   |x| >= 0.625: sign(x) (1 - 2 / (e^(2|x|) + 1)) with the hardware 2^y and
//                 reciprocal (3.4 units with a 1-ulp error in each; e = inf
//                 past |x| ~ 44 gives exactly 1; NaN stays NaN).
// About fourteen instructions against about thirty for the library tanhf,
// which made the row kernel VALU-bound.
__device__ __forceinline__ float tanh_cap(float x) {
#if CMC_BRIDGE_FAST_TANH
    const float ax = fabsf(x);
    if (ax < 0.625f) {
        const float s = x * x;
        const float q = fmaf(fmaf(fmaf(0.01489475928246975f, s, -0.05170630291104317f), s, 0.1330212950706482f), s,
                             -0.3333188593387604f);
        return fmaf(x * s, q, x);
    }
    const float e = __builtin_amdgcn_exp2f(ax * 2.8853900817779268f);  // e^(2|x|)
    return copysignf(fmaf(-2.f, __builtin_amdgcn_rcpf(e + 1.f), 1.f), x);
#else
    return tanhf(x);
#endif
}

// Two fp32 values -> packed bf16 (low half first), round to nearest even
// (one v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, bf16x2{(__bf16)lo, (__bf16)hi});
}

// Build-time tuning knob: tile rows per group of the tile order below.
#ifndef CMC_BRIDGE_GROUP_M
#define CMC_BRIDGE_GROUP_M 4
#endif

// Tile order.  Physical workgroup b runs on XCD b % 8, and each XCD takes a
// contiguous run of logical tiles; the run is walked in groups of
// CMC_BRIDGE_GROUP_M tile rows, M fastest inside a group, so the tiles an
// XCD holds at once form a near-square block that shares few A and B
// strips in its L2 (a row-major walk would stream every B strip once per
// tile row).
__device__ __forceinline__ void gemm_tile(int tiles_m, int tiles_n, int &tm, int &tn) {
    const int tiles = gridDim.x, bid = blockIdx.x;
    const int per_xcd = (tiles + 7) / 8;
    int t = (bid % 8) * per_xcd + bid / 8;
    if ((tiles % 8) != 0) t = bid;  // uneven split: plain order
    constexpr int GM = CMC_BRIDGE_GROUP_M;
    const int group = t / (GM * tiles_n);
    const int first = group * GM;
    const int gm = min(GM, tiles_m - first);
    const int local = t - group * GM * tiles_n;
    tm = first + local % gm;
    tn = local / gm;
}

// Epilogue of one wave's accumulators.  The MFMAs compute each 16 x 16 tile
// transposed (B rows as the first operand), so lane l, element r holds tile
// row l % 16, tile column 4 (l / 16) + r: four consecutive columns of one
// row, written with one 8-byte (bf16) or 16-byte (fp32) store.  The stores
// of one row's column tiles are issued back to back, so its cache lines are
// complete when they leave L2 (column tiles outermost wrote 1.4 - 2.4x the
// output bytes to HBM).
//   Epilogue 0 (first layer): + b1, GELU (erf form), rounded to bf16.
//   Epilogue 1 (second layer): + b2, fp32.
template <int EPI, int TM, int TN>
__device__ __forceinline__ void store_tile(const GemmParams &p, const floatx4 (&acc)[TM][TN], int r0, int c0,
                                           int lane) {
    float4 biases[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j)  // 16-byte aligned
        biases[j] = *reinterpret_cast<const float4 *>(p.bias + c0 + j * 16 + 4 * (lane >> 4));
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = c0 + j * 16 + 4 * (lane >> 4);
            const float4 bias = biases[j];
            const int row = r0 + i * 16 + (lane & 15);
            if (row < p.M) {
                const float v0 = acc[i][j][0] + bias.x, v1 = acc[i][j][1] + bias.y;
                const float v2 = acc[i][j][2] + bias.z, v3 = acc[i][j][3] + bias.w;
                if constexpr (EPI == 0) {
                    *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(p.C) + (size_t)row * p.N + col) =
                        make_uint2(pack_bf16x2(gelu_erf(v0), gelu_erf(v1)), pack_bf16x2(gelu_erf(v2), gelu_erf(v3)));
                } else {
                    *reinterpret_cast<float4 *>(static_cast<float *>(p.C) + (size_t)row * p.N + col) =
                        make_float4(v0, v1, v2, v3);
                }
            }
        }
    }
}

// Build-time tuning knob: K slice of the 128 x 128-tile kernel (32, 64 or
// 128; shapes whose K it does not divide use 64).  On the 49152 x 1280 ->
// 4096 -> 4096 projection run on that kernel alone: 32 -> 3.31 ms per call
// (148 VGPRs, 40 KB of LDS: three workgroups per CU), 64 -> 3.48 ms, 128 ->
// 4.84 ms.
#ifndef CMC_BRIDGE_BK
#define CMC_BRIDGE_BK 32
#endif

// Build-time tuning knob: register stages of the 128 x 128-tile kernel's
// global -> LDS staging (1, 2 or 3; see gemm_nt_kernel).  With 32-wide K
// slices three stages need 172 VGPRs (two waves per SIMD instead of three)
// and ran slower (3.50 ms per projection call against 3.25 ms with two).
#ifndef CMC_BRIDGE_REG_STAGES
#define CMC_BRIDGE_REG_STAGES 2
#endif

// WTM x WTN per wave (TM x TN MFMA tiles of 16 x 16), WGM x WGN waves, BK of
// K per LDS slice; the workgroup tile is WGM WTM x WGN WTN.  RS register
// stages: with one,
// slice j + 1 is loaded while slice j feeds the MFMAs and the barrier after
// storing it drains every load; with two, slice j + 2 is loaded while slices
// j and j + 1 are computed (two register sets used in turn, the loop unrolled
// by two) and the barriers wait only for LDS, so each load has two slices of
// MFMA work to land.
template <int EPI, int WTM, int WTN, int WGM, int WGN, int BK, int RS>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_nt_kernel(GemmParams p) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int BM = WGM * WTM, BN = WGN * WTN, LDK = BK + 8, TM = WTM / 16, TN = WTN / 16;
    static_assert(BM == BN, "the A and B slices share one staging map");
    constexpr int kRowChunks = BK / 8;                  // 16-byte chunks per tile row
    constexpr int kChunks = BM * kRowChunks / NT;       // per thread per matrix per slice
    constexpr int kRowsPerPass = NT / kRowChunks;
    static_assert(kChunks * NT == BM * kRowChunks, "whole chunks per thread");
    __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDK];
    __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * LDK];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;

    int tm, tn;
    gemm_tile((p.M + BM - 1) / BM, p.N / BN, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    // Global -> register -> LDS staging: chunk c = tid + NT i is row
    // c / kRowChunks, 16-byte column group c % kRowChunks of the BM x BK slice.
    const int crow0 = tid / kRowChunks, ccol = (tid % kRowChunks) * 8;
    const uint16_t *Ag = p.A + (size_t)ccol, *Bg = p.B + (size_t)n0 * p.K + (size_t)ccol;
#define CMC_GLOAD(RA_, RB_, K0_)                                                                         \
    do {                                                                                                 \
        _Pragma("unroll") for (int i = 0; i < kChunks; ++i) {                                            \
            const int ar = min(m0 + crow0 + kRowsPerPass * i, p.M - 1); /* past M: clamped, discarded */ \
            RA_[i] = *reinterpret_cast<const uint4 *>(Ag + (size_t)ar * p.K + (K0_));                   \
            RB_[i] = *reinterpret_cast<const uint4 *>(Bg + (size_t)(crow0 + kRowsPerPass * i) * p.K + (K0_)); \
        }                                                                                                \
    } while (0)
#define CMC_SSTORE(RA_, RB_, BUF_)                                                                       \
    do {                                                                                                 \
        _Pragma("unroll") for (int i = 0; i < kChunks; ++i) {                                            \
            *reinterpret_cast<uint4 *>(&sA[BUF_][(crow0 + kRowsPerPass * i) * LDK + ccol]) = RA_[i];    \
            *reinterpret_cast<uint4 *>(&sB[BUF_][(crow0 + kRowsPerPass * i) * LDK + ccol]) = RB_[i];    \
        }                                                                                                \
    } while (0)

    floatx4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int KT = p.K / BK;
    const int fr = lane & 15, fk = 8 * (lane >> 4);
#define CMC_MMA(BUF_)                                                                                    \
    do {                                                                                                 \
        _Pragma("unroll") for (int kk = 0; kk < BK; kk += 32) {                                          \
            bf16x8 a[TM], b[TN];                                                                         \
            _Pragma("unroll") for (int i = 0; i < TM; ++i)                                               \
                a[i] = *reinterpret_cast<const bf16x8 *>(&sA[BUF_][(wm * WTM + i * 16 + fr) * LDK + kk + fk]); \
            _Pragma("unroll") for (int jj = 0; jj < TN; ++jj)                                            \
                b[jj] = *reinterpret_cast<const bf16x8 *>(&sB[BUF_][(wn * WTN + jj * 16 + fr) * LDK + kk + fk]); \
            _Pragma("unroll") for (int i = 0; i < TM; ++i)                                               \
                _Pragma("unroll") for (int jj = 0; jj < TN; ++jj)                                        \
                    acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[jj], a[i], acc[i][jj], 0, 0, 0); \
        }                                                                                                \
    } while (0)
    // Past the last slice the loads reload it: no load sits behind a branch
    // (a conditional load here made the compiler keep the staging registers in
    // scratch memory); such copies are never computed on.
    if constexpr (RS == 1) {
        uint4 ra[kChunks], rb[kChunks];
        CMC_GLOAD(ra, rb, 0);
        CMC_SSTORE(ra, rb, 0);
        __syncthreads();
        for (int j = 0; j < KT; ++j) {
            const int buf = j & 1;
            CMC_GLOAD(ra, rb, min(j + 1, KT - 1) * BK);
            CMC_MMA(buf);
            CMC_SSTORE(ra, rb, buf ^ 1);
            __syncthreads();
        }
    } else {
        static_assert(RS == 2 || RS == 3, "one, two or three register stages");
        // Barrier after LDS stores that waits for LDS only (s_waitcnt
        // lgkmcnt(0), vmcnt and expcnt at their maxima): the fences of
        // __syncthreads would drain the loads in flight.
#define CMC_LDS_SYNC()                                             \
    do {                                                           \
        __builtin_amdgcn_s_waitcnt(0xC07F);                        \
        __builtin_amdgcn_s_barrier();                              \
    } while (0)
        // Each register set is one vector value (arrays carried across the
        // loop were kept in scratch memory).
        typedef uint32_t stage_t __attribute__((ext_vector_type(4 * kChunks)));
        stage_t ra0, rb0, ra1, rb1, ra2, rb2;
#define CMC_VLOAD(RA_, RB_, K0_)                                                                         \
    do {                                                                                                 \
        _Pragma("unroll") for (int i = 0; i < kChunks; ++i) {                                            \
            const int ar = min(m0 + crow0 + kRowsPerPass * i, p.M - 1); /* past M: clamped, discarded */ \
            const uint4 ta = *reinterpret_cast<const uint4 *>(Ag + (size_t)ar * p.K + (K0_));           \
            const uint4 tb = *reinterpret_cast<const uint4 *>(Bg + (size_t)(crow0 + kRowsPerPass * i) * p.K + (K0_)); \
            RA_[4 * i] = ta.x; RA_[4 * i + 1] = ta.y; RA_[4 * i + 2] = ta.z; RA_[4 * i + 3] = ta.w;     \
            RB_[4 * i] = tb.x; RB_[4 * i + 1] = tb.y; RB_[4 * i + 2] = tb.z; RB_[4 * i + 3] = tb.w;     \
        }                                                                                                \
    } while (0)
#define CMC_VSTORE(RA_, RB_, BUF_)                                                                       \
    do {                                                                                                 \
        _Pragma("unroll") for (int i = 0; i < kChunks; ++i) {                                            \
            *reinterpret_cast<uint4 *>(&sA[BUF_][(crow0 + kRowsPerPass * i) * LDK + ccol]) =            \
                make_uint4(RA_[4 * i], RA_[4 * i + 1], RA_[4 * i + 2], RA_[4 * i + 3]);                  \
            *reinterpret_cast<uint4 *>(&sB[BUF_][(crow0 + kRowsPerPass * i) * LDK + ccol]) =            \
                make_uint4(RB_[4 * i], RB_[4 * i + 1], RB_[4 * i + 2], RB_[4 * i + 3]);                  \
        }                                                                                                \
    } while (0)
        if constexpr (RS == 2) {
            CMC_VLOAD(ra0, rb0, 0);
            CMC_VSTORE(ra0, rb0, 0);
            CMC_VLOAD(ra1, rb1, min(1, KT - 1) * BK);
            CMC_LDS_SYNC();
            for (int j = 0; j < KT; j += 2) {
                // LDS buffer 0 holds slice j; set 1 is bringing slice j + 1.
                CMC_VLOAD(ra0, rb0, min(j + 2, KT - 1) * BK);
                CMC_MMA(0);
                CMC_VSTORE(ra1, rb1, 1);  // buffer 1 was last read before the previous barrier
                CMC_LDS_SYNC();
                CMC_VLOAD(ra1, rb1, min(j + 3, KT - 1) * BK);
                if (j + 1 < KT) CMC_MMA(1);  // uniform
                CMC_VSTORE(ra0, rb0, 0);      // every wave read buffer 0 before the barrier above
                CMC_LDS_SYNC();
            }
        } else {
            // Three sets: slice s + 3 is loaded while slices s .. s + 2 are
            // computed; LDS buffer s % 2 holds slice s at sub-step s.
            CMC_VLOAD(ra0, rb0, 0);
            CMC_VSTORE(ra0, rb0, 0);
            CMC_VLOAD(ra1, rb1, min(1, KT - 1) * BK);
            CMC_VLOAD(ra2, rb2, min(2, KT - 1) * BK);
            CMC_LDS_SYNC();
#define CMC_SUBSTEP(S_, RL_, RBL_, RN_, RBN_)                                                \
    do {                                                                                     \
        CMC_VLOAD(RL_, RBL_, min((S_) + 3, KT - 1) * BK);                                    \
        if ((S_) < KT) CMC_MMA((S_) & 1); /* uniform */                                      \
        CMC_VSTORE(RN_, RBN_, ((S_) + 1) & 1); /* buffer last read before the last barrier */ \
        CMC_LDS_SYNC();                                                                      \
    } while (0)
            for (int j = 0; j < KT; j += 3) {
                CMC_SUBSTEP(j, ra0, rb0, ra1, rb1);
                CMC_SUBSTEP(j + 1, ra1, rb1, ra2, rb2);
                CMC_SUBSTEP(j + 2, ra2, rb2, ra0, rb0);
            }
#undef CMC_SUBSTEP
        }
        __builtin_amdgcn_s_waitcnt(0);  // drain the reloads past the end before the workgroup exits
#undef CMC_LDS_SYNC
#undef CMC_VLOAD
#undef CMC_VSTORE
    }
#undef CMC_GLOAD
#undef CMC_SSTORE
#undef CMC_MMA

    store_tile<EPI, TM, TN>(p, acc, m0 + wm * WTM, n0 + wn * WTN, lane);
}

// One wave per row; the row stays in registers (NV float4 per lane, Hd <=
// 256 NV): one read and one write of the row.
template <int NV>
__global__ __launch_bounds__(256) void bridge_norm_kernel(BridgeParams p) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= p.M) return;  // wave-uniform; no barriers
    float4 *y4 = reinterpret_cast<float4 *>(p.out + (size_t)row * p.Hd);
    const float4 *g4 = reinterpret_cast<const float4 *>(p.ln_gamma);
    const float4 *b4 = reinterpret_cast<const float4 *>(p.ln_beta);
    const int n4 = p.Hd / 4;
    float4 v[NV];
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
        const int c = lane + u * kWave;
        v[u] = c < n4 ? y4[c] : float4{0.f, 0.f, 0.f, 0.f};
        s += (v[u].x + v[u].y) + (v[u].z + v[u].w);
    }
    const float mean = lane_reduce<OpSum, 1, kWave>(s) / (float)p.Hd;
    float q = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
        if (lane + u * kWave < n4) {
            const float a = v[u].x - mean, b = v[u].y - mean, d = v[u].z - mean, e = v[u].w - mean;
            q = fmaf(a, a, q);
            q = fmaf(b, b, q);
            q = fmaf(d, d, q);
            q = fmaf(e, e, q);
        }
    }
    const float var = lane_reduce<OpSum, 1, kWave>(q) / (float)p.Hd;
    const float inv = 1.f / sqrtf(var + p.eps);
    float nn = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
        const int c = lane + u * kWave;
        if (c < n4) {
            const float4 g = g4[c], b = b4[c];
            v[u] = float4{p.nu * tanh_cap(fmaf(g.x * (v[u].x - mean), inv, b.x)),
                          p.nu * tanh_cap(fmaf(g.y * (v[u].y - mean), inv, b.y)),
                          p.nu * tanh_cap(fmaf(g.z * (v[u].z - mean), inv, b.z)),
                          p.nu * tanh_cap(fmaf(g.w * (v[u].w - mean), inv, b.w))};
            nn = fmaf(v[u].x, v[u].x, nn);
            nn = fmaf(v[u].y, v[u].y, nn);
            nn = fmaf(v[u].z, v[u].z, nn);
            nn = fmaf(v[u].w, v[u].w, nn);
        }
    }
    const float nrm = sqrtf(lane_reduce<OpSum, 1, kWave>(nn));
    const float scale = (nrm > 0.f && 2.f * p.nu < nrm) ? 2.f * p.nu / nrm : 1.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
        const int c = lane + u * kWave;
        if (c < n4) y4[c] = float4{v[u].x * scale, v[u].y * scale, v[u].z * scale, v[u].w * scale};
    }
}

// Rows wider than 256 * 16: the same steps re-reading the row from cache.
__global__ __launch_bounds__(256) void bridge_norm_wide_kernel(BridgeParams p) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= p.M) return;  // wave-uniform; no barriers
    float *y = p.out + (size_t)row * p.Hd;
    const int n4 = p.Hd / 4;
    const float4 *y4 = reinterpret_cast<const float4 *>(y);
    const float4 *g4 = reinterpret_cast<const float4 *>(p.ln_gamma);
    const float4 *b4 = reinterpret_cast<const float4 *>(p.ln_beta);
    float s = 0.f;
    for (int c = lane; c < n4; c += kWave) {
        const float4 v = y4[c];
        s += (v.x + v.y) + (v.z + v.w);
    }
    const float mean = lane_reduce<OpSum, 1, kWave>(s) / (float)p.Hd;
    float q = 0.f;
    for (int c = lane; c < n4; c += kWave) {
        const float4 v = y4[c];
        const float a = v.x - mean, b = v.y - mean, d = v.z - mean, e = v.w - mean;
        q = fmaf(a, a, q);
        q = fmaf(b, b, q);
        q = fmaf(d, d, q);
        q = fmaf(e, e, q);
    }
    const float var = lane_reduce<OpSum, 1, kWave>(q) / (float)p.Hd;
    const float inv = 1.f / sqrtf(var + p.eps);
    auto capped = [&](int c) {
        const float4 v = y4[c], g = g4[c], b = b4[c];
        return float4{p.nu * tanh_cap(fmaf(g.x * (v.x - mean), inv, b.x)),
                      p.nu * tanh_cap(fmaf(g.y * (v.y - mean), inv, b.y)),
                      p.nu * tanh_cap(fmaf(g.z * (v.z - mean), inv, b.z)),
                      p.nu * tanh_cap(fmaf(g.w * (v.w - mean), inv, b.w))};
    };
    float nn = 0.f;
    for (int c = lane; c < n4; c += kWave) {
        const float4 t = capped(c);
        nn = fmaf(t.x, t.x, nn);
        nn = fmaf(t.y, t.y, nn);
        nn = fmaf(t.z, t.z, nn);
        nn = fmaf(t.w, t.w, nn);
    }
    const float nrm = sqrtf(lane_reduce<OpSum, 1, kWave>(nn));
    const float scale = (nrm > 0.f && 2.f * p.nu < nrm) ? 2.f * p.nu / nrm : 1.f;
    // Each lane rewrites only the elements it reads.
    for (int c = lane; c < n4; c += kWave) {
        const float4 t = capped(c);
        reinterpret_cast<float4 *>(y)[c] = float4{t.x * scale, t.y * scale, t.z * scale, t.w * scale};
    }
}

// Norms of the CME vectors h themselves (the encoder's hidden states at the
// placeholder positions), for CME-guided window localization: one wave per
// row, 16-byte loads of 8 bf16 elements widened exactly, squares summed in
// fp32 in a fixed per-lane order, then the DPP/permlane butterfly.  Runs
// before the first GEMM, so that GEMM then finds h in the last-level cache.
__global__ __launch_bounds__(256) void cme_norm_kernel(const uint16_t *h, int M, int Hc, float *norms) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= M) return;  // wave-uniform; no barriers
    const uint4 *h4 = reinterpret_cast<const uint4 *>(h + (size_t)row * Hc);
    // Lane l sums the squares of 16-byte chunks l, l + 64, ... in that order
    // (one fma chain); up to kGroup chunks are requested before any is used,
    // so a row of up to 4096 elements costs one memory round trip.
    constexpr int kGroup = 8;
    const int chunks = Hc / 8;
    float s = 0.f;
    for (int c0 = 0; c0 < chunks; c0 += kGroup * kWave) {
        uint4 v[kGroup];
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
            const int c = c0 + lane + i * kWave;
            v[i] = c < chunks ? h4[c] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
            if (c0 + lane + i * kWave < chunks) {
                float x[8];
                Vec16<uint16_t>::widen(v[i], x);
#pragma unroll
                for (int e = 0; e < 8; ++e) s = fmaf(x[e], x[e], s);
            }
        }
    }
    s = lane_reduce<OpSum, 1, kWave>(s);
    if (lane == 0) norms[row] = sqrtf(s);
}

hipError_t launch_norm(const BridgeParams &p, hipStream_t stream) {
    const unsigned grid = (unsigned)((p.M + 3) / 4);
    if (p.Hd <= 256 * 4)
        bridge_norm_kernel<4><<<grid, 256, 0, stream>>>(p);
    else if (p.Hd <= 256 * 8)
        bridge_norm_kernel<8><<<grid, 256, 0, stream>>>(p);
    else if (p.Hd <= 256 * 16)
        bridge_norm_kernel<16><<<grid, 256, 0, stream>>>(p);
    else
        bridge_norm_wide_kernel<<<grid, 256, 0, stream>>>(p);
    return hipGetLastError();
}

template <int WTM, int WTN, int WGM, int WGN, int BK, int RS>
hipError_t launch_gemm_t(int epi, const GemmParams &g, hipStream_t stream) {
    constexpr int BM = WGM * WTM, BN = WGN * WTN, NT = 64 * WGM * WGN;
    if (g.N % BN != 0 || g.K % BK != 0) return hipErrorInvalidValue;
    const long long tiles = (long long)((g.M + BM - 1) / BM) * (g.N / BN);
    if (tiles == 0) return hipSuccess;
    if (epi == 0)
        gemm_nt_kernel<0, WTM, WTN, WGM, WGN, BK, RS><<<(unsigned)tiles, NT, 0, stream>>>(g);
    else
        gemm_nt_kernel<1, WTM, WTN, WGM, WGN, BK, RS><<<(unsigned)tiles, NT, 0, stream>>>(g);
    return hipGetLastError();
}

// Build-time tuning knob: 1 runs N % 256 == 0 shapes on 256 x 256 tiles of
// eight waves, 128 x 64 each (one workgroup per CU), with K slices of
// CMC_BRIDGE_BIG_BK and CMC_BRIDGE_BIG_STAGES register stages; other shapes
// (and 0) use 128 x 128 tiles of four 64 x 64 waves.  On the 49152 x 1280 ->
// 4096 -> 4096 projection: 128 x 128 tiles 3.22 ms per call; 256 x 256 tiles
// with 32-wide slices 3.14 ms (two stages) and 2.99 ms (three), with 64-wide
// slices 3.05 ms (one stage) and 2.94 ms (two); the same with the transposed
// accumulators' vector stores 2.79 ms, GELU by A&S 7.1.26 2.73 ms, each
// row's stores back to back 2.51 ms.  A direct-to-LDS variant of the
// 256 x 256 tile (four or five LDS stages, fragment reads interleaved with
// the MFMAs) measured 2.95 - 3.06 ms.
#ifndef CMC_BRIDGE_BIG
#define CMC_BRIDGE_BIG 1
#endif
#ifndef CMC_BRIDGE_BIG_BK
#define CMC_BRIDGE_BIG_BK 64
#endif
#ifndef CMC_BRIDGE_BIG_STAGES
#define CMC_BRIDGE_BIG_STAGES 2
#endif

hipError_t launch_gemm(int epi, const GemmParams &g, hipStream_t stream) {
    if constexpr (CMC_BRIDGE_BIG) {
        if (g.N % 256 == 0 && g.K % CMC_BRIDGE_BIG_BK == 0)
            return launch_gemm_t<128, 64, 2, 4, CMC_BRIDGE_BIG_BK, CMC_BRIDGE_BIG_STAGES>(epi, g, stream);
    }
    constexpr int RS = CMC_BRIDGE_REG_STAGES;
    if (CMC_BRIDGE_BK != 64 && g.K % CMC_BRIDGE_BK == 0)
        return launch_gemm_t<64, 64, 2, 2, CMC_BRIDGE_BK, RS>(epi, g, stream);
    return launch_gemm_t<64, 64, 2, 2, 64, RS>(epi, g, stream);
}

}  // namespace

hipError_t launch_memory_bridge(const BridgeParams &p, hipStream_t stream) {
    if (p.M == 0) return hipSuccess;
    hipError_t e;
    if (p.h_norms) {
        cme_norm_kernel<<<(unsigned)((p.M + 3) / 4), 256, 0, stream>>>(p.h, p.M, p.Hc, p.h_norms);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    GemmParams g1{p.h, p.w1, p.b1, p.hidden, p.M, p.F, p.Hc};
    e = launch_gemm(0, g1, stream);
    if (e != hipSuccess) return e;
    GemmParams g2{p.hidden, p.w2, p.b2, p.out, p.M, p.Hd, p.F};
    e = launch_gemm(1, g2, stream);
    if (e != hipSuccess) return e;
    return launch_norm(p, stream);
}

}  // namespace cmc
