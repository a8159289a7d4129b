// MemoryBridge (Sec. 2.2): each CME vector h (encoder width Hc) becomes a
// decoder-ready memory row
//   m_hat = LayerNorm(W2 GELU(W1 h + b1) + b2)          (LayerNorm per the appendix)
//   m     = nu tanh(m_hat) * min(1, 2 nu / |nu tanh(m_hat)|)   (the section's cap)
// -- the selection keys of Tier-1.
//
// gemm_nt_kernel: C[M][N] = A[M][K] . B[N][K]^T on MFMA, bf16 operands, fp32
// accumulation.  A 256-thread workgroup of 2 x 2 waves computes a 2WT x 2WT
// tile, each wave WT x WT as (WT/16)^2 v_mfma_f32_16x16x32_bf16 tiles (WT =
// 64 by default; WT = 128 halves the LDS reads per MFMA flop but leaves one
// workgroup per CU, and measured no faster).  K advances BK (32 by default)
// at a time through two LDS buffers, staged from global memory through
// register sets used in turn (two by default), so a slice's loads have the
// MFMA work of the slices before it to land.  LDS rows are padded by 8 bf16
// (80 or 144 bytes) so that the 16-byte fragment reads of 8 consecutive
// rows hit 8 disjoint groups of 4 banks.  Tiles are handed out so that each
// XCD (workgroups are dealt round-robin to the 8 XCDs) runs a contiguous run
// of them, walked in groups of a few tile rows (see gemm_tile).
//   Epilogue 0 (first layer): + b1, exact GELU, rounded to bf16 (the hidden
//   activations, kept in the workspace).  Epilogue 1 (second layer): + b2,
//   fp32 into the output.
//
// gemm_deep_kernel: the same product with direct-to-LDS loads and 3 or more LDS
// stages (a build-time alternative; measured slower here).
//
// bridge_norm_kernel: one wave per output row, in place, the row held in
// registers: mean and biased variance (two passes over the registers),
// LayerNorm with gamma/beta, nu tanh, the row norm, and the cap.
#include "device_common.hpp"
#include "kernels.hpp"

namespace cmc {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kGemmThreads = 256;  // 2 x 2 waves

struct GemmParams {
    const uint16_t *A;  // [M][K]
    const uint16_t *B;  // [N][K]
    const float *bias;  // [N]
    void *C;            // [M][N]: bf16 (epilogue 0) or fp32 (epilogue 1)
    int M, N, K;
};

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

__device__ __forceinline__ uint16_t to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
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

// Build-time tuning knob: K slice of the 64 x 64-per-wave kernel (32, 64 or
// 128; shapes whose K it does not divide use 64).  On the 49152 x 1280 ->
// 4096 -> 4096 projection: 32 -> 3.31 ms per call (148 VGPRs, 40 KB of LDS:
// three workgroups per CU), 64 -> 3.48 ms, 128 -> 4.84 ms.
#ifndef CMC_BRIDGE_BK
#define CMC_BRIDGE_BK 32
#endif

// Build-time tuning knob: register stages of the global -> LDS staging (1, 2
// or 3; see gemm_nt_kernel).  With 32-wide K slices three stages need 172
// VGPRs (two waves per SIMD instead of three) and ran slower (3.50 ms per
// projection call against 3.25 ms with two).
#ifndef CMC_BRIDGE_REG_STAGES
#define CMC_BRIDGE_REG_STAGES 2
#endif

// WT x WT per wave (4 x 4 or 8 x 8 MFMA tiles of 16 x 16), BK of K per LDS
// slice; the workgroup tile is 2 WT x 2 WT.  RS register stages: with one,
// slice j + 1 is loaded while slice j feeds the MFMAs and the barrier after
// storing it drains every load; with two, slice j + 2 is loaded while slices
// j and j + 1 are computed (two register sets used in turn, the loop unrolled
// by two) and the barriers wait only for LDS, so each load has two slices of
// MFMA work to land.
template <int EPI, int WT, int BK, int RS>
__global__ __launch_bounds__(kGemmThreads) void gemm_nt_kernel(GemmParams p) {
    constexpr int BM = 2 * WT, BN = 2 * WT, LDK = BK + 8, T = WT / 16;
    constexpr int kRowChunks = BK / 8;                            // 16-byte chunks per tile row
    constexpr int kChunks = BM * kRowChunks / kGemmThreads;       // per thread per matrix per slice
    constexpr int kRowsPerPass = kGemmThreads / kRowChunks;
    __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDK];
    __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * LDK];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    int tm, tn;
    gemm_tile((p.M + BM - 1) / BM, p.N / BN, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    // Global -> register -> LDS staging: chunk c = tid + 256 i is row
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

    floatx4 acc[T][T];
#pragma unroll
    for (int i = 0; i < T; ++i)
#pragma unroll
        for (int j = 0; j < T; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int KT = p.K / BK;
    const int fr = lane & 15, fk = 8 * (lane >> 4);
#define CMC_MMA(BUF_)                                                                                    \
    do {                                                                                                 \
        _Pragma("unroll") for (int kk = 0; kk < BK; kk += 32) {                                          \
            bf16x8 a[T], b[T];                                                                           \
            _Pragma("unroll") for (int i = 0; i < T; ++i)                                                \
                a[i] = *reinterpret_cast<const bf16x8 *>(&sA[BUF_][(wm * WT + i * 16 + fr) * LDK + kk + fk]); \
            _Pragma("unroll") for (int jj = 0; jj < T; ++jj)                                             \
                b[jj] = *reinterpret_cast<const bf16x8 *>(&sB[BUF_][(wn * WT + jj * 16 + fr) * LDK + kk + fk]); \
            _Pragma("unroll") for (int i = 0; i < T; ++i)                                                \
                _Pragma("unroll") for (int jj = 0; jj < T; ++jj)                                         \
                    acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[jj], acc[i][jj], 0, 0, 0); \
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

    // C fragment: lane l, element r -> row 4 (l / 16) + r, column l % 16.
#pragma unroll
    for (int j = 0; j < T; ++j) {
        const int col = n0 + wn * WT + j * 16 + fr;
        const float bias = p.bias[col];
#pragma unroll
        for (int i = 0; i < T; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = m0 + wm * WT + i * 16 + 4 * (lane >> 4) + r;
                if (row < p.M) {
                    const float v = acc[i][j][r] + bias;
                    if constexpr (EPI == 0)
                        static_cast<uint16_t *>(p.C)[(size_t)row * p.N + col] = to_bf16_rne(gelu_erf(v));
                    else
                        static_cast<float *>(p.C)[(size_t)row * p.N + col] = v;
                }
            }
        }
    }
}

// Deep-pipelined variant: 256 x 256 workgroup tile (128 x 128 per wave),
// K in slices of 32 staged through NS LDS stages by direct-to-LDS loads
// (global_load_lds, 16 bytes per lane), so NS - 1 slices are in flight with
// no registers held for them.  Each 16-row x 32-k block of a slice occupies
// 1 KB of LDS in MFMA fragment order -- lane l's 16 bytes at offset 16 l are
// row l % 16, k 8 (l / 16) .. +7, exactly the A/B operand of
// v_mfma_f32_16x16x32_bf16 -- so the global load of a block and the
// fragment read of it use the same lane mapping and the read is one
// contiguous, bank-conflict-free ds_read_b128.  Waves 0-1 load the A
// blocks of a slice, waves 2-3 the B blocks (WT / 16 blocks per wave).
// WT x WT per wave, 2 WT x 2 WT per workgroup: WT = 128 holds 256
// accumulators per lane (one wave per SIMD), WT = 64 keeps two workgroups
// per CU.
#ifndef CMC_BRIDGE_DEEP_STAGES
#define CMC_BRIDGE_DEEP_STAGES 4
#endif
#ifndef CMC_BRIDGE_DEEP_WT
#define CMC_BRIDGE_DEEP_WT 128
#endif
constexpr int kDeepStages = CMC_BRIDGE_DEEP_STAGES;

template <int EPI, int WT>
__global__ __launch_bounds__(kGemmThreads) void gemm_deep_kernel(GemmParams p) {
    constexpr int BM = 2 * WT, BN = 2 * WT, BK = 32, T = WT / 16, NS = kDeepStages;
    constexpr int kBlk = 1024;                          // bytes per 16 x 32 block
    constexpr int kStage = (BM / 16 + BN / 16) * kBlk;  // WT / 4 KB
    constexpr int LPW = T;                              // blocks (loads) per wave per slice
    static_assert(NS >= 3 && NS * kStage <= 160 * 1024, "the stages must fit the 160 KB of LDS");
    __shared__ __attribute__((aligned(1024))) char smem[NS * kStage];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    int tm, tn;
    gemm_tile((p.M + BM - 1) / BM, p.N / BN, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    // This lane's source rows for the LPW blocks its wave loads per slice.
    const bool loads_a = wave < 2;
    const int blk0 = (wave & 1) * LPW;               // first block (of 2 LPW) of this wave's matrix
    const int fr = lane & 15, fk = 8 * (lane >> 4);
    const uint16_t *src[LPW];
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
        const int r = (blk0 + i) * 16 + fr;
        src[i] = loads_a ? p.A + (size_t)min(m0 + r, p.M - 1) * p.K + fk : p.B + (size_t)(n0 + r) * p.K + fk;
    }
    const int ldsw = (loads_a ? 0 : (BM / 16) * kBlk) + blk0 * kBlk;  // this wave's blocks, in a stage
    auto issue = [&](int slice) {
        const int st = slice % NS;
        char *dst = smem + st * kStage + ldsw;
#pragma unroll
        for (int i = 0; i < LPW; ++i)
            __builtin_amdgcn_global_load_lds((const void *)(src[i] + (size_t)slice * BK),
                                             (__attribute__((address_space(3))) void *)(dst + i * kBlk), 16, 0, 0);
    };

    floatx4 acc[T][T];
#pragma unroll
    for (int i = 0; i < T; ++i)
#pragma unroll
        for (int j = 0; j < T; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int KT = p.K / BK;
    // Prologue: slices 0 .. NS-2 in flight.  Past the end the last slice is
    // loaded again (identical bytes into its own stage), which keeps LPW
    // loads per wave per iteration so that the counted wait below stays exact.
#pragma unroll
    for (int sl = 0; sl < NS - 1; ++sl) issue(min(sl, KT - 1));
    for (int j = 0; j < KT; ++j) {
        // Wait for this wave's loads of slice j (the NS - 2 later slices may
        // stay in flight: LPW loads each), then for every wave's.  A bare
        // s_barrier: the fences of __syncthreads would drain every load.
        // s_waitcnt encoding: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt
        // at their maxima (not waited).
        constexpr int kVm = LPW * (NS - 2);
        static_assert(kVm < 64, "vmcnt field is 6 bits");
        __builtin_amdgcn_s_waitcnt((kVm & 15) | ((kVm >> 4) << 14) | (7 << 4) | (15 << 8));
        __builtin_amdgcn_s_barrier();
        // Stage (j - 1) % NS was read by every wave before the barrier: refill it.
        issue(min(j + NS - 1, KT - 1));
        const char *stg = smem + (j % NS) * kStage;
        bf16x8 a[T], b[T];
#pragma unroll
        for (int i = 0; i < T; ++i)
            a[i] = *reinterpret_cast<const bf16x8 *>(stg + (wm * T + i) * kBlk + lane * 16);
#pragma unroll
        for (int jj = 0; jj < T; ++jj)
            b[jj] = *reinterpret_cast<const bf16x8 *>(stg + (BM / 16 + wn * T + jj) * kBlk + lane * 16);
#pragma unroll
        for (int i = 0; i < T; ++i)
#pragma unroll
            for (int jj = 0; jj < T; ++jj)
                acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[jj], acc[i][jj], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);  // drain the reloads past the end before the workgroup exits

#pragma unroll
    for (int j = 0; j < T; ++j) {
        const int col = n0 + wn * WT + j * 16 + fr;
        const float bias = p.bias[col];
#pragma unroll
        for (int i = 0; i < T; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = m0 + wm * WT + i * 16 + 4 * (lane >> 4) + r;
                if (row < p.M) {
                    const float v = acc[i][j][r] + bias;
                    if constexpr (EPI == 0)
                        static_cast<uint16_t *>(p.C)[(size_t)row * p.N + col] = to_bf16_rne(gelu_erf(v));
                    else
                        static_cast<float *>(p.C)[(size_t)row * p.N + col] = v;
                }
            }
        }
    }
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
            v[u] = float4{p.nu * tanhf(fmaf(g.x * (v[u].x - mean), inv, b.x)),
                          p.nu * tanhf(fmaf(g.y * (v[u].y - mean), inv, b.y)),
                          p.nu * tanhf(fmaf(g.z * (v[u].z - mean), inv, b.z)),
                          p.nu * tanhf(fmaf(g.w * (v[u].w - mean), inv, b.w))};
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
        return float4{p.nu * tanhf(fmaf(g.x * (v.x - mean), inv, b.x)),
                      p.nu * tanhf(fmaf(g.y * (v.y - mean), inv, b.y)),
                      p.nu * tanhf(fmaf(g.z * (v.z - mean), inv, b.z)),
                      p.nu * tanhf(fmaf(g.w * (v.w - mean), inv, b.w))};
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

// Build-time tuning knob: wave tile of the bridge GEMMs, 64 (128 x 128 per
// workgroup, two workgroups per CU) or 128 (256 x 256, one per CU; for N a
// multiple of 256).  Measured on the 49152 x 1280 -> 4096 -> 4096 workload:
// 64 is slightly faster; both are held back by global-load latency with one
// slice in flight.
#ifndef CMC_BRIDGE_WAVE_TILE
#define CMC_BRIDGE_WAVE_TILE 64
#endif

template <int WT, int BK>
hipError_t launch_gemm_t(int epi, const GemmParams &g, hipStream_t stream) {
    constexpr int BM = 2 * WT, BN = 2 * WT;
    if (g.N % BN != 0 || g.K % BK != 0) return hipErrorInvalidValue;
    const long long tiles = (long long)((g.M + BM - 1) / BM) * (g.N / BN);
    if (tiles == 0) return hipSuccess;
    constexpr int RS = WT == 128 ? 1 : CMC_BRIDGE_REG_STAGES;  // two sets of 128-wide tiles spill
    if (epi == 0)
        gemm_nt_kernel<0, WT, BK, RS><<<(unsigned)tiles, kGemmThreads, 0, stream>>>(g);
    else
        gemm_nt_kernel<1, WT, BK, RS><<<(unsigned)tiles, kGemmThreads, 0, stream>>>(g);
    return hipGetLastError();
}

// Build-time tuning knob: 1 runs the deep-pipelined direct-to-LDS kernel for
// the shapes it takes (N % (2 CMC_BRIDGE_DEEP_WT) == 0, K % 32 == 0).  On the
// 49152 x 1280 -> 4096 -> 4096 projection it measured 4.05 ms per call with
// 256 x 256 tiles and 4 stages (4.02 with 5), 4.35 - 4.66 ms with 128 x 128
// tiles and 3 - 5 stages, against 3.66 ms for the register-staged kernels,
// so those are the default.
#ifndef CMC_BRIDGE_DEEP
#define CMC_BRIDGE_DEEP 0
#endif

hipError_t launch_gemm(int epi, const GemmParams &g, hipStream_t stream) {
    constexpr int DB = 2 * CMC_BRIDGE_DEEP_WT;
    if (CMC_BRIDGE_DEEP && g.N % DB == 0 && g.K % 32 == 0) {
        const long long tiles = (long long)((g.M + DB - 1) / DB) * (g.N / DB);
        if (tiles == 0) return hipSuccess;
        if (epi == 0)
            gemm_deep_kernel<0, CMC_BRIDGE_DEEP_WT><<<(unsigned)tiles, kGemmThreads, 0, stream>>>(g);
        else
            gemm_deep_kernel<1, CMC_BRIDGE_DEEP_WT><<<(unsigned)tiles, kGemmThreads, 0, stream>>>(g);
        return hipGetLastError();
    }
    if (CMC_BRIDGE_WAVE_TILE == 128 && g.N % 256 == 0) return launch_gemm_t<128, 32>(epi, g, stream);
    if (CMC_BRIDGE_BK != 64 && g.K % CMC_BRIDGE_BK == 0) return launch_gemm_t<64, CMC_BRIDGE_BK>(epi, g, stream);
    return launch_gemm_t<64, 64>(epi, g, stream);
}

}  // namespace

hipError_t launch_memory_bridge(const BridgeParams &p, hipStream_t stream) {
    if (p.M == 0) return hipSuccess;
    GemmParams g1{p.h, p.w1, p.b1, p.hidden, p.M, p.F, p.Hc};
    hipError_t e = launch_gemm(0, g1, stream);
    if (e != hipSuccess) return e;
    GemmParams g2{p.hidden, p.w2, p.b2, p.out, p.M, p.Hd, p.F};
    e = launch_gemm(1, g2, stream);
    if (e != hipSuccess) return e;
    return launch_norm(p, stream);
}

}  // namespace cmc
