// Tier-2 ring append (Sec. 2.5: the window keeps the W most recent tokens so
// the cache stays bounded by K + W + |q| while generating), and the Tier-1
// gather that copies the selected memory rows' K/V into a contiguous block
// once per question.
//
// One workgroup per sequence: row t of kv head h goes to slot
// (count + t) mod W, then count += T_new.  Every thread reads count before
// the barrier and only thread 0 writes it after, so the workgroup owns
// count[b] and no atomics are needed.  Rows move as 16-byte vectors.
#include "device_common.hpp"
#include "kernels.hpp"

namespace cmc {

namespace {

__global__ __launch_bounds__(256) void window_append_kernel(AppendParams p) {
    const int b = blockIdx.x;
    const int count = p.win_count[b] < 0 ? 0 : p.win_count[b];  // count >= 0 is a precondition
    const int per_row = p.row_vecs;
    const int total = p.Hkv * p.T_new * per_row;
    uint4 *wk = static_cast<uint4 *>(p.win_k);
    uint4 *wv = static_cast<uint4 *>(p.win_v);
    const uint4 *nk = static_cast<const uint4 *>(p.new_k);
    const uint4 *nv = static_cast<const uint4 *>(p.new_v);
    for (int i = threadIdx.x; i < total; i += blockDim.x) {
        const int v = i % per_row;
        const int t = (i / per_row) % p.T_new;
        const int h = i / (per_row * p.T_new);
        const int slot = (int)(((long long)count + t) % p.W);
        const size_t dst = (((size_t)b * p.Hkv + h) * p.W + slot) * per_row + v;
        const size_t src = (((size_t)b * p.Hkv + h) * p.T_new + t) * per_row + v;
        wk[dst] = nk[src];
        wv[dst] = nv[src];
    }
    __syncthreads();
    if (threadIdx.x == 0) p.win_count[b] = count + p.T_new;
}

// Tier-1 gather: out[b][h][j] = pool[b][h][idx[b][j]] (clamped into the
// pool) for j < k_b, 16-byte vectors, one thread per vector: consecutive
// threads copy consecutive vectors of a row, so every row moves as whole
// 64-byte segments.  Rows j >= k_b are left untouched.
__global__ __launch_bounds__(256) void gather_kernel(GatherParams p) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t per_seq = (size_t)p.Hkv * p.k * p.row_vecs;
    const int b = (int)(i / per_seq);
    if (b >= p.B) return;
    const size_t r = i % per_seq;
    const int v = (int)(r % p.row_vecs);
    const int j = (int)((r / p.row_vecs) % p.k);
    const int h = (int)(r / ((size_t)p.row_vecs * p.k));
    int kb = p.k;
    if (p.k_len) {
        const int x = p.k_len[b];
        kb = x < 0 ? 0 : (x > p.k ? p.k : x);
    }
    if (j >= kb) return;
    int src = p.idx ? p.idx[(size_t)b * p.idx_stride + j] : j;
    src = src < 0 ? 0 : (src > p.N - 1 ? p.N - 1 : src);
    const size_t head = (size_t)b * p.Hkv + h;
    const size_t s_off = (head * p.N + src) * p.row_vecs + v;
    const size_t d_off = (head * p.k + j) * p.row_vecs + v;
    static_cast<uint4 *>(p.out_k)[d_off] = static_cast<const uint4 *>(p.cme_k)[s_off];
    static_cast<uint4 *>(p.out_v)[d_off] = static_cast<const uint4 *>(p.cme_v)[s_off];
}

}  // namespace

hipError_t launch_gather(const GatherParams &p, hipStream_t stream) {
    const size_t total = (size_t)p.B * p.Hkv * p.k * p.row_vecs;
    if (total == 0) return hipSuccess;
    gather_kernel<<<(unsigned)((total + 255) / 256), 256, 0, stream>>>(p);
    return hipGetLastError();
}

hipError_t launch_window_append(const AppendParams &p, hipStream_t stream) {
    if (p.B == 0 || p.W == 0) return hipSuccess;
    window_append_kernel<<<p.B, 256, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace cmc
