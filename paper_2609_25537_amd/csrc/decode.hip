// Two-tier decode attention (Sec. 2.5, KV cache assembly): one decode step of
// softmax attention over the key list [Tier-1 pool rows idx[0..k-1]] ++
// [Tier-2 ring slots 0..min(count,W)-1], split over the key axis.
//
// Pass 1 (decode_split_kernel): grid (S, Hkv, B), 256 threads.  Workgroup s
// owns keys [s*chunk, (s+1)*chunk) of the virtual list of sequence b and all
// G = Hq/Hkv query heads that share kv head h, so every K/V byte is read
// from HBM once per step and reused G times from registers.  Each 16-byte
// lane load covers Vec16<T>::N elements of one row; LPR lanes cover a row
// (a 256-byte bf16 row of Dh = 128 is 16 lanes, four rows per wave load).
// Scores use the lane's slice of q (pre-scaled by scale*log2 e) and a DPP
// butterfly over the row's lanes; softmax is online per wave (a running
// max per head, rescaled once per block of U row-loads); the four waves are
// combined through LDS and the workgroup writes one (m, l, acc[Dh]) partial
// per head.
//
// Pass 2 (decode_merge_kernel): grid (Hkv, B); combines the S partials of
// each head in fixed split order: M = max m_s, out = sum 2^(m_s-M) acc_s /
// sum 2^(m_s-M) l_s.  A head whose key list is empty gets zeros.
#include "device_common.hpp"
#include "kernels.hpp"

namespace cmc {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

template <typename T, int DH, int G, int U>
__global__ __launch_bounds__(256) void decode_split_kernel(DecodeParams p) {
    constexpr int VEC = Vec16<T>::N;
    constexpr int LPR = DH / VEC;      // lanes per row
    constexpr int RPW = kWave / LPR;   // rows per wave load
    constexpr int WAVES = 4;
    static_assert(LPR >= 1 && LPR <= kWave && (kWave % LPR) == 0, "row layout");

    const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int grp = lane / LPR, e = lane % LPR;

    int valid = 0;
    if (p.W > 0) {
        valid = p.win_count[b];
        valid = valid < 0 ? 0 : (valid > p.W ? p.W : valid);
    }
    const int L = p.k + valid;
    const int c0 = s * p.chunk;
    const int c1 = min(c0 + p.chunk, L);

    // This lane's slice of the G query rows, pre-scaled for exp2.
    float qf[G][VEC];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const float4 *qp = reinterpret_cast<const float4 *>(
            p.q + ((size_t)b * p.Hq + (size_t)kvh * G + g) * DH + e * VEC);
#pragma unroll
        for (int i = 0; i < VEC / 4; ++i) {
            float4 t = qp[i];
            qf[g][4 * i + 0] = t.x * p.qscale;
            qf[g][4 * i + 1] = t.y * p.qscale;
            qf[g][4 * i + 2] = t.z * p.qscale;
            qf[g][4 * i + 3] = t.w * p.qscale;
        }
    }

    const size_t head = (size_t)b * p.Hkv + kvh;
    const T *poolK = static_cast<const T *>(p.cme_k) + head * (size_t)p.N * DH + e * VEC;
    const T *poolV = static_cast<const T *>(p.cme_v) + head * (size_t)p.N * DH + e * VEC;
    const T *winK = p.W > 0 ? static_cast<const T *>(p.win_k) + head * (size_t)p.W * DH + e * VEC : nullptr;
    const T *winV = p.W > 0 ? static_cast<const T *>(p.win_v) + head * (size_t)p.W * DH + e * VEC : nullptr;
    const int32_t *idxb = p.idx ? p.idx + (size_t)b * p.k : nullptr;
    const int nmax = p.N > 0 ? p.N - 1 : 0;

    float m[G], l[G], acc[G][VEC];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        m[g] = -INFINITY;
        l[g] = 0.f;
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[g][i] = 0.f;
    }

    constexpr int STRIDE = WAVES * RPW;  // rows between a wave's consecutive loads
    for (int r0 = c0 + wave * RPW; r0 < c1; r0 += STRIDE * U) {
        uint4 kr[U], vr[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int row = r0 + u * STRIDE + grp;
            ok[u] = row < c1;
            kr[u] = make_uint4(0, 0, 0, 0);
            vr[u] = make_uint4(0, 0, 0, 0);
            if (ok[u]) {
                const T *kp, *vp;
                if (row < p.k) {
                    int r = idxb ? idxb[row] : row;
                    r = r < 0 ? 0 : (r > nmax ? nmax : r);
                    kp = poolK + (size_t)r * DH;
                    vp = poolV + (size_t)r * DH;
                } else {
                    const int slot = row - p.k;
                    kp = winK + (size_t)slot * DH;
                    vp = winV + (size_t)slot * DH;
                }
                kr[u] = *reinterpret_cast<const uint4 *>(kp);
                vr[u] = *reinterpret_cast<const uint4 *>(vp);
            }
        }

        float sc[U][G];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float kf[VEC];
            Vec16<T>::widen(kr[u], kf);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                float d = 0.f;
#pragma unroll
                for (int i = 0; i < VEC; ++i) d = fmaf(qf[g][i], kf[i], d);
                d = lane_reduce<OpSum, 1, LPR>(d);
                sc[u][g] = ok[u] ? d : -INFINITY;
            }
        }

        float vf[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) Vec16<T>::widen(vr[u], vf[u]);

#pragma unroll
        for (int g = 0; g < G; ++g) {
            float mb = sc[0][g];
#pragma unroll
            for (int u = 1; u < U; ++u) mb = fmaxf(mb, sc[u][g]);
            mb = lane_reduce<OpMax, LPR, kWave>(mb);    // max over the wave's rows
            const float mn = fmaxf(m[g], mb);            // finite: row r0 is valid
            const float alpha = exp2f(m[g] - mn);
            l[g] *= alpha;
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[g][i] *= alpha;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float pu = exp2f(sc[u][g] - mn);
                l[g] += pu;
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[g][i] = fmaf(pu, vf[u][i], acc[g][i]);
            }
            m[g] = mn;
        }
    }

    // Sum the row groups of each wave (m is already wave-uniform).
#pragma unroll
    for (int g = 0; g < G; ++g) {
        l[g] = lane_reduce<OpSum, LPR, kWave>(l[g]);
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[g][i] = lane_reduce<OpSum, LPR, kWave>(acc[g][i]);
    }

    // Combine the four waves through LDS.
    __shared__ float s_acc[WAVES][G][DH];
    __shared__ float s_m[WAVES][G], s_l[WAVES][G];
    if (grp == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) s_acc[wave][g][e * VEC + i] = acc[g][i];
            if (e == 0) {
                s_m[wave][g] = m[g];
                s_l[wave][g] = l[g];
            }
        }
    }
    __syncthreads();

    const size_t part = (head * p.S + s) * G;
    for (int t = threadIdx.x; t < G * DH; t += 256) {
        const int g = t / DH, d = t % DH;
        float M = s_m[0][g];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) M = fmaxf(M, s_m[w][g]);
        float num = 0.f, den = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < WAVES; ++w) {
                const float f = exp2f(s_m[w][g] - M);
                num = fmaf(f, s_acc[w][g][d], num);
                den = fmaf(f, s_l[w][g], den);
            }
        }
        p.part_acc[(part + g) * DH + d] = num;
        if (d == 0) {
            p.part_ml[(part + g) * 2 + 0] = M;
            p.part_ml[(part + g) * 2 + 1] = den;
        }
    }
}

template <int DH, int G>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeParams p) {
    const int kvh = blockIdx.x, b = blockIdx.y;
    const size_t head = (size_t)b * p.Hkv + kvh;
    for (int t = threadIdx.x; t < G * DH; t += 256) {
        const int g = t / DH, d = t % DH;
        const float *ml = p.part_ml + head * p.S * G * 2;
        const float *ac = p.part_acc + head * p.S * G * DH;
        float M = -INFINITY;
        for (int s = 0; s < p.S; ++s) M = fmaxf(M, ml[(s * G + g) * 2]);
        float o = 0.f;
        if (M != -INFINITY) {
            float num = 0.f, den = 0.f;
            for (int s = 0; s < p.S; ++s) {
                const float f = exp2f(ml[(s * G + g) * 2] - M);
                den = fmaf(f, ml[(s * G + g) * 2 + 1], den);
                num = fmaf(f, ac[(s * G + g) * DH + d], num);
            }
            o = num / den;
        }
        p.out[((size_t)b * p.Hq + (size_t)kvh * G + g) * DH + d] = o;
    }
}

template <typename T, int DH, int G>
hipError_t launch_typed(const DecodeParams &p, hipStream_t stream) {
    constexpr int U = (sizeof(T) == 2 && DH >= 128) ? 4 : 2;
    dim3 g1(p.S, p.Hkv, p.B);
    decode_split_kernel<T, DH, G, U><<<g1, 256, 0, stream>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2(p.Hkv, p.B);
    decode_merge_kernel<DH, G><<<g2, 256, 0, stream>>>(p);
    return hipGetLastError();
}

template <typename T, int DH>
hipError_t launch_g(const DecodeParams &p, int G, hipStream_t stream) {
    switch (G) {
        case 1: return launch_typed<T, DH, 1>(p, stream);
        case 2: return launch_typed<T, DH, 2>(p, stream);
        case 4: return launch_typed<T, DH, 4>(p, stream);
        case 8: return launch_typed<T, DH, 8>(p, stream);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_dh(const DecodeParams &p, int G, int Dh, hipStream_t stream) {
    switch (Dh) {
        case 64: return launch_g<T, 64>(p, G, stream);
        case 128: return launch_g<T, 128>(p, G, stream);
        case 256: return launch_g<T, 256>(p, G, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_two_tier_decode(const DecodeParams &p, bool bf16, int G, int Dh, hipStream_t stream) {
    if (p.B == 0) return hipSuccess;
    return bf16 ? launch_dh<uint16_t>(p, G, Dh, stream) : launch_dh<float>(p, G, Dh, stream);
}

float decode_qscale(float scale) { return scale * kLog2e; }

}  // namespace cmc
