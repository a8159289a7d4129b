// Tier-2 ring append (Sec. 2.5: the window keeps the W most recent tokens so
// the cache stays bounded by K + W + |q| while generating).
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

}  // namespace

hipError_t launch_window_append(const AppendParams &p, hipStream_t stream) {
    if (p.B == 0 || p.W == 0) return hipSuccess;
    window_append_kernel<<<p.B, 256, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace cmc
