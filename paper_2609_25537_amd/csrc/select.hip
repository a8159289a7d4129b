// Tier-1 question-guided selection (Sec. 2.5, Tier-1 paragraph and its score
// equation): score_j = m_j.q / (|m_j| |q|), keep the K best, emit them in
// document order.
//
// score_kernel: one wave per memory row (R rows per wave).  The dot product
// and |m_j|^2 come out of ONE pass over the row (16-byte loads of fp32 or
// bf16 keys, bf16 widened exactly, fp32 FMA in a fixed per-lane order, then a
// DPP/permlane butterfly), |q|^2 from the same loop over q (fp32).  Zero
// norms are clamped to 1e-8, so a zero row scores 0.
//
// topk_kernel: one 1024-thread workgroup per sequence.  Scores become
// order-preserving uint32 keys (kept in registers, ceil(N / 1024) per thread
// rounded up to a power of two, at most 32, so N <= 32768).  The k-th largest key T is found bit by bit from the top: T is the
// largest value with count(key >= T) >= k, one block-wide count per bit.
// Then every key > T is taken, plus the first (k - count(key > T)) keys equal
// to T in index order (ties go to the earlier document position).  Two
// block-wide exclusive scans over the threads' contiguous index ranges give
// each selected row its output slot, so idx comes out ascending.
//
// Ragged batches: sequence b has its own candidate count n_b (rows past it
// score -inf and are never selected), keeps k_b = min(k, n_b) rows, and may
// pin q_b question rows after them (pool rows n_b .. n_b + q_b - 1, the
// question's place in the assembled cache [M* || C_local || q]).
#include <limits.h>

#include "device_common.hpp"
#include "kernels.hpp"

namespace cmc {

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int clamp_count(int v, int hi) { return v < 0 ? 0 : (v > hi ? hi : v); }

// One row's dot product with q and its squared norm, accumulated per lane
// over 16-byte vectors of the row (4 fp32 or 8 bf16 elements, widened
// exactly); |q|^2 from the same loop over q.
template <int R, bool BF16>
__device__ __forceinline__ void score_rows(const SelectParams &p, int b, int j0, int nb, int lane, float (&dot)[R],
                                           float (&nn)[R], float &qq) {
    const float4 *q4 = reinterpret_cast<const float4 *>(p.q_vec + (size_t)b * p.D);
    const char *rows[R];
    constexpr int EB = BF16 ? 2 : 4;  // bytes per key element
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = min(j0 + r, nb - 1);
        rows[r] = static_cast<const char *>(p.sel_keys) + ((size_t)b * p.N + j) * p.D * EB;
    }
    constexpr int E = 16 / EB;  // elements per 16-byte vector
    const int DV = p.D / E;
#pragma unroll 2
    for (int c = lane; c < DV; c += kWave) {
        float qv[E];
#pragma unroll
        for (int i = 0; i < E / 4; ++i) {
            const float4 t = q4[c * (E / 4) + i];
            qv[4 * i + 0] = t.x;
            qv[4 * i + 1] = t.y;
            qv[4 * i + 2] = t.z;
            qv[4 * i + 3] = t.w;
        }
#pragma unroll
        for (int e = 0; e < E; ++e) qq = fmaf(qv[e], qv[e], qq);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            // Non-temporal: each key row is read once (0.81 -> 0.74 ms on the
            // 64 x 4096 x 4096 fp32 Mistral-shaped batch).
            const f32x4 mw = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(rows[r] + (size_t)c * 16));
            float mv[E];
            if constexpr (BF16) {
                const uint4 u = make_uint4(__float_as_uint(mw.x), __float_as_uint(mw.y), __float_as_uint(mw.z),
                                           __float_as_uint(mw.w));
                Vec16<uint16_t>::widen(u, mv);
            } else {
                mv[0] = mw.x;
                mv[1] = mw.y;
                mv[2] = mw.z;
                mv[3] = mw.w;
            }
#pragma unroll
            for (int e = 0; e < E; ++e) dot[r] = fmaf(mv[e], qv[e], dot[r]);
#pragma unroll
            for (int e = 0; e < E; ++e) nn[r] = fmaf(mv[e], mv[e], nn[r]);
        }
    }
}

template <int R, bool BF16>
__global__ __launch_bounds__(256) void score_kernel(SelectParams p) {
    const int b = blockIdx.y;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int j0 = (blockIdx.x * 4 + wave) * R;
    if (j0 >= p.N) return;  // wave-uniform; no barriers below
    // Rows past this sequence's count are not candidates: they score -inf
    // and are not read.
    const int nb = p.n_rows ? clamp_count(p.n_rows[b], p.N) : p.N;
    if (j0 >= nb) {
        if (lane < R && j0 + lane < p.N) {
            p.scores[(size_t)b * p.N + j0 + lane] = -INFINITY;
            if (p.norms) p.norms[(size_t)b * p.N + j0 + lane] = 0.f;
        }
        return;
    }

    float dot[R], nn[R], qq = 0.f;
#pragma unroll
    for (int r = 0; r < R; ++r) dot[r] = nn[r] = 0.f;
    score_rows<R, BF16>(p, b, j0, nb, lane, dot, nn, qq);
    qq = lane_reduce<OpSum, 1, kWave>(qq);
    const float qn = fmaxf(sqrtf(qq), 1e-8f);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float d = lane_reduce<OpSum, 1, kWave>(dot[r]);
        const float n2 = lane_reduce<OpSum, 1, kWave>(nn[r]);
        const int j = j0 + r;
        if (lane == 0 && j < p.N) {
            const float mn = sqrtf(n2);
            p.scores[(size_t)b * p.N + j] = j < nb ? d / (fmaxf(mn, 1e-8f) * qn) : -INFINITY;
            if (p.norms) p.norms[(size_t)b * p.N + j] = j < nb ? mn : 0.f;
        }
    }
}

__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;  // -0 ranks as +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / kWave;
constexpr int kMaxPerThread = kSelectMaxN / kTopkThreads;  // 32

// Block-wide sum of an integer count (< 2^24, exact in fp32); every thread
// gets the same total.  `slot` alternates between two LDS rows so one barrier
// per call suffices.
__device__ __forceinline__ int block_count(int v, float (*s_part)[kTopkWaves], int &slot) {
    const float w = lane_reduce<OpSum, 1, kWave>((float)v);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) s_part[slot][wave] = w;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < kTopkWaves; ++i) t += s_part[slot][i];
    slot ^= 1;
    return (int)t;
}

// Block-wide exclusive prefix sum of v over thread order.
__device__ __forceinline__ int block_exclusive_scan(int v, int *s_wave) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(x, off);
        if (lane >= off) x += y;
    }
    if (lane == kWave - 1) s_wave[wave] = x;
    __syncthreads();
    int base = 0;
    for (int i = 0; i < wave; ++i) base += s_wave[i];
    __syncthreads();  // s_wave may be reused by the next scan
    return base + x - v;
}

// PER keys per thread (a power of two, PER * 1024 >= N): the per-thread
// loops run over PER registers only, so a batch of N = 4096 rows does an
// eighth of the compares of the largest instantiation.
template <int PER>
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(SelectParams p) {
    constexpr int kPerThread = PER;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int N = p.N;
    const int nb = p.n_rows ? clamp_count(p.n_rows[b], N) : N;  // candidates: rows [0, nb)
    const int k = min(p.k, nb);
    const int per = (N + kTopkThreads - 1) / kTopkThreads;  // <= PER
    const int j0 = tid * per;
    const int cnt = max(0, min(per, nb - j0));

    __shared__ float s_part[2][kTopkWaves];
    __shared__ int s_wave[kTopkWaves];
    int slot = 0;

    uint32_t key[kPerThread];
    const float *sc = p.scores + (size_t)b * N;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) key[i] = i < cnt ? order_key(sc[j0 + i]) : 0u;

    // T = largest value with count(key >= T) >= k.
    uint32_t T = 0;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t cand = T | (1u << bit);
        int c = 0;
#pragma unroll
        for (int i = 0; i < kPerThread; ++i) c += (i < cnt && key[i] >= cand) ? 1 : 0;
        if (block_count(c, s_part, slot) >= k) T = cand;
    }

    int gt = 0, eq = 0;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
        gt += (i < cnt && key[i] > T) ? 1 : 0;
        eq += (i < cnt && key[i] == T) ? 1 : 0;
    }
    const int need_eq = k - block_count(gt, s_part, slot);
    int eq_seen = block_exclusive_scan(eq, s_wave);

    int take = 0;
    uint32_t mask = 0;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
        bool sel = false;
        if (i < cnt) {
            if (key[i] > T) {
                sel = true;
            } else if (key[i] == T) {
                sel = eq_seen < need_eq;
                ++eq_seen;
            }
        }
        if (sel) {
            mask |= 1u << i;
            ++take;
        }
    }
    int pos = block_exclusive_scan(take, s_wave);
    int32_t *out = p.idx_out + (size_t)b * p.idx_stride;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i)
        if (mask & (1u << i)) out[pos++] = j0 + i;
    // Pinned question rows (pool rows nb, nb+1, ...) follow the selection,
    // then -1 up to the row stride.
    const int qb = p.q_rows ? clamp_count(p.q_rows[b], p.idx_stride - k) : 0;
    for (int t = tid; t < p.idx_stride - k; t += kTopkThreads) out[k + t] = t < qb ? nb + t : -1;
    if (tid == 0 && p.k_out) p.k_out[b] = k + qb;
}

// CME-guided Tier-2 localization: one 256-thread workgroup per sequence
// finds the row with the largest norm among its n_b rows (lowest index on
// ties), maps it to its chunk and the chunk's token offset alpha, and
// applies the window equation.  A sequence without rows takes the midpoint.
__global__ __launch_bounds__(256) void locate_kernel(LocateParams p) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nb = p.n_rows ? clamp_count(p.n_rows[b], p.N) : p.N;
    const float *nr = p.norms + (size_t)b * p.N;
    float best = -INFINITY;
    int bj = INT_MAX;
    for (int j = tid; j < nb; j += 256) {
        const float v = nr[j];
        if (v > best) {  // strided ascending scan: the first maximum is kept
            best = v;
            bj = j;
        }
    }
    // (max value, then min index) across the wave, then across the 4 waves
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float ov = __shfl_xor(best, off);
        const int oj = __shfl_xor(bj, off);
        if (ov > best || (ov == best && oj < bj)) {
            best = ov;
            bj = oj;
        }
    }
    __shared__ float s_v[4];
    __shared__ int s_j[4];
    if (lane == 0) {
        s_v[wave] = best;
        s_j[wave] = bj;
    }
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < 4; ++w) {
            if (s_v[w] > best || (s_v[w] == best && s_j[w] < bj)) {
                best = s_v[w];
                bj = s_j[w];
            }
        }
        const long long ctx = p.ctx_len[b];
        long long alpha;
        if (nb == 0) {
            alpha = ctx / 2;
        } else {
            if (bj >= nb) bj = 0;  // no comparable value (NaN norms): keeps the read in bounds
            const int chunk = bj / p.mems_per_chunk;
            alpha = p.chunk_offset ? (long long)p.chunk_offset[(size_t)b * p.n_chunks + chunk]
                                   : (long long)chunk * p.chunk_tokens;
        }
        long long start = alpha - p.W / 2;
        if (start > ctx - p.W) start = ctx - p.W;
        if (start < 0) start = 0;
        if (p.alpha_out) p.alpha_out[b] = (int32_t)alpha;
        p.start_out[b] = (int32_t)start;
    }
}

}  // namespace

hipError_t launch_locate(const LocateParams &p, hipStream_t stream) {
    if (p.B == 0) return hipSuccess;
    locate_kernel<<<p.B, 256, 0, stream>>>(p);
    return hipGetLastError();
}

hipError_t launch_select(const SelectParams &p, hipStream_t stream) {
    if (p.B == 0) return hipSuccess;
    hipError_t e = hipSuccess;
    if (p.N > 0) {
        const long long rows = (long long)p.B * p.N;
        if (rows >= 65536) {
            dim3 grid((p.N + 15) / 16, p.B);
            if (p.keys_bf16) score_kernel<4, true><<<grid, 256, 0, stream>>>(p);
            else score_kernel<4, false><<<grid, 256, 0, stream>>>(p);
        } else {
            dim3 grid((p.N + 3) / 4, p.B);
            if (p.keys_bf16) score_kernel<1, true><<<grid, 256, 0, stream>>>(p);
            else score_kernel<1, false><<<grid, 256, 0, stream>>>(p);
        }
        e = hipGetLastError();
    }
    if (e != hipSuccess || (p.idx_stride == 0 && !p.k_out)) return e;
    const int per = (p.N + kTopkThreads - 1) / kTopkThreads;
    if (per <= 1) topk_kernel<1><<<p.B, kTopkThreads, 0, stream>>>(p);
    else if (per <= 2) topk_kernel<2><<<p.B, kTopkThreads, 0, stream>>>(p);
    else if (per <= 4) topk_kernel<4><<<p.B, kTopkThreads, 0, stream>>>(p);
    else if (per <= 8) topk_kernel<8><<<p.B, kTopkThreads, 0, stream>>>(p);
    else if (per <= 16) topk_kernel<16><<<p.B, kTopkThreads, 0, stream>>>(p);
    else if (per <= kMaxPerThread) topk_kernel<kMaxPerThread><<<p.B, kTopkThreads, 0, stream>>>(p);
    else return hipErrorInvalidValue;  // N > kSelectMaxN is rejected by the host checks
    return hipGetLastError();
}

}  // namespace cmc
