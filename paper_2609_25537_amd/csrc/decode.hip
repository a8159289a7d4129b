// Two-tier decode attention (Sec. 2.5, KV cache assembly): one decode step of
// softmax attention over the key list [Tier-1 pool rows idx[0..k-1]] ++
// [Tier-2 ring slots 0..min(count,W)-1], optionally fused with the ring append
// of this step's new rows, in ONE launch.
//
// Grid (S, Hkv, B), 4 or 8 waves per workgroup (chosen by the split plan).  Workgroup s owns keys
// [s*chunk, (s+1)*chunk) of sequence b's virtual key list and all G = Hq/Hkv
// query heads sharing kv head h, so each K/V byte is read from HBM once per
// step and reused G times on chip.
//
// Fused append: with T_new > 0, the rows appended this step go to slots
// (count + t) mod W.  The workgroup owning such a slot reads the row from
// new_k/new_v instead of the ring and writes it into the ring; count is
// advanced once every (sequence, kv head) pair has been completed, i.e.
// after every workgroup of the sequence has read it.  The result equals
// cmc_window_append followed by the decode.
//
// Main loop, two variants:
//   MFMA (bf16 K/V, G <= 4): a wave takes 16 keys per block.  S = Q K^T is one
//     v_mfma_f32_16x16x32_bf16 chain per Dh/32 slice, with the 16 A-rows
//     holding the G query heads repeated (row m = head m % G), so every lane
//     ends with all G scores of key (lane % 16).  q is split into bf16
//     hi + lo parts (two MFMAs per slice), which keeps the logit error at the
//     level of fp32 accumulation.  P V runs on the VALU in fp32 in four
//     quarters of 4 keys: lane l owns key (l & 3) of each quarter and Dh/16
//     dims; the p values reach that layout through 16 x G floats of LDS
//     private to the wave.  V rows are loaded non-temporally, K rows with
//     ordinary loads (see ld16).
//   VALU (fp32 K/V, or G = 8): 16-byte lane loads, LPR lanes per row, dot
//     products reduced by a DPP butterfly.
// Both keep an online softmax per wave (running max in log2 units, q
// pre-scaled by scale*log2 e), then combine the waves through LDS.
//
// Latency (one launch of a single layer at batch 1 is a chain of memory round
// trips, not a stream): the first K/V loads depend only on kernel arguments
// that arrive preloaded in SGPRs.  The ring count is fetched with a vector
// load and read where the masks need it, q is loaded and split after the
// first K/V loads are issued, and when the key list is split anyway the rows
// appended in this call get a split of their own, so no workgroup runs two
// dependent phases.  Measured, the step is bound by that chain and by memory:
// with P V taken out entirely a step got only 2-3% faster.
//
// Split merge, inside the same launch: with S == 1 the workgroup writes the
// output directly.  With S > 1 every workgroup publishes (m, l, acc[Dh]) per
// head to the workspace and arrives on a per-(b, kv head) counter; the last
// to arrive merges the S partials in fixed split order (so results are
// bit-identical run to run), writes the output and re-arms the counter.
// Publication uses agent-coherent relaxed atomics plus a store-completion
// wait instead of device-scope fences (see coherent_store2).  A head whose key
// list is empty gets zeros.
#include <limits.h>

#include "device_common.hpp"
#include "kernels.hpp"

namespace cmc {

namespace {

// Build-time tuning knob: smallest query-group size that takes the MFMA path
// (smaller groups use the VALU path).
#ifndef CMC_MFMA_MIN_G
#define CMC_MFMA_MIN_G 1
#endif
// Build-time tuning knob: widest head that double-buffers its K/V rows.
#ifndef CMC_DOUBLE_BUFFER_MAX_DH
#define CMC_DOUBLE_BUFFER_MAX_DH 128
#endif

constexpr float kLog2e = 1.4426950408889634f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// K/V row pointers of one key; rk/rv are set (to the ring slot the row must
// be written to) only for a row appended in this call.
template <typename T>
struct RowPtrs {
    const T *k, *v;
    T *rk, *rv;
};

// Where the rows of sequence b's key list live, for one kv head (the
// layout of the MFMA path's phases, below): rows [0, k) are pool rows
// idx[row] (clamped into the pool), rows [k, k + W) ring slots row - k
// (masked as in RingRows), rows [k + W, k + W + T_new) the appended rows,
// written to ring slots (slot0 + t) mod W.
template <typename T>
struct RowMap {
    int stride;               // elements per row (Dh)
    const T *poolK, *poolV;   // pool of this (b, kv head)
    T *winK, *winV;           // ring of this (b, kv head)
    const T *newK, *newV;     // appended rows of this (b, kv head)
    const int32_t *idx;       // this sequence's index list, or nullptr
    int k, W, nmax, slot0, T_new, nvalid;
};

// Row lookup on values already in registers (free functions over scalars:
// selecting between fields of a struct in memory would keep it on the
// stack).  fetch_row() issues the only memory access of a lookup -- the
// index-list entry of a pool row -- so callers can prefetch it one block
// ahead; row_ptrs() is pure arithmetic on its result.
__device__ __forceinline__ int fetch_row(int row, const int32_t *idx, int k) {
    return (row < k && idx) ? idx[row] : row;
}

template <typename T>
__device__ __forceinline__ RowPtrs<T> row_ptrs(int row, int r, const T *poolK, const T *poolV, T *winK,
                                               T *winV, const T *newK, const T *newV, int k, int W, int nmax,
                                               int slot0, int T_new, int stride) {
    const bool in_pool = row < k;
    r = r < 0 ? 0 : (r > nmax ? nmax : r);
    const int slot = row - k;
    const bool is_new = !in_pool && slot >= W;
    const int t = slot - W;  // appended row, when is_new
    int ws = slot0 + t;      // its ring slot
    ws -= ws >= W ? W : 0;
    const size_t op = (size_t)r * stride, ow = (size_t)slot * stride, on = (size_t)t * stride,
                 oa = (size_t)ws * stride;
    RowPtrs<T> o;
    o.k = in_pool ? poolK + op : (is_new ? newK + on : winK + ow);
    o.v = in_pool ? poolV + op : (is_new ? newV + on : winV + ow);
    o.rk = is_new ? winK + oa : nullptr;
    o.rv = is_new ? winV + oa : nullptr;
    return o;
}

// Whether key-list row `row` holds a key of this step (only ring slots can
// be masked).
__device__ __forceinline__ bool row_valid(int row, int k, int W, int slot0, int T_new, int nvalid) {
    const int s = row - k;
    if (s < 0 || s >= W) return true;
    int d = s - slot0;
    d += d < 0 ? W : 0;
    return s < nvalid && d >= T_new;
}

// Unpacks a RowMap into locals and defines LOCATE(row) over them.
#define CMC_UNPACK_ROWMAP(rm)                                                            \
    const auto poolK_ = (rm).poolK;                                                      \
    const auto poolV_ = (rm).poolV;                                                      \
    const auto winK_ = (rm).winK;                                                        \
    const auto winV_ = (rm).winV;                                                        \
    const auto newK_ = (rm).newK;                                                        \
    const auto newV_ = (rm).newV;                                                        \
    const int32_t *idx_ = (rm).idx;                                                      \
    const int k_ = (rm).k, W_ = (rm).W, nmax_ = (rm).nmax, slot0_ = (rm).slot0,          \
              tnew_ = (rm).T_new, stride_ = (rm).stride, nvalid_ = (rm).nvalid
#define FETCH(row) fetch_row(row, idx_, k_)
#define PTRS(row, r) \
    row_ptrs(row, r, poolK_, poolV_, winK_, winV_, newK_, newV_, k_, W_, nmax_, slot0_, tnew_, stride_)
#define LOCATE(row) PTRS(row, FETCH(row))
#define VALID(row) row_valid(row, k_, W_, slot0_, tnew_, nvalid_)

template <typename T>
__device__ __forceinline__ RowMap<T> make_rowmap(const DecodeParams &p, int b, int kvh, int DH, int kb,
                                                 int slot0, int nvalid) {
    RowMap<T> m;
    const size_t head = (size_t)b * p.Hkv + kvh;
    m.poolK = static_cast<const T *>(p.cme_k) + head * (size_t)p.N * DH;
    m.poolV = static_cast<const T *>(p.cme_v) + head * (size_t)p.N * DH;
    m.winK = p.W > 0 ? static_cast<T *>(p.win_k) + head * (size_t)p.W * DH : nullptr;
    m.winV = p.W > 0 ? static_cast<T *>(p.win_v) + head * (size_t)p.W * DH : nullptr;
    m.newK = p.T_new > 0 ? static_cast<const T *>(p.new_k) + head * (size_t)p.T_new * DH : nullptr;
    m.newV = p.T_new > 0 ? static_cast<const T *>(p.new_v) + head * (size_t)p.T_new * DH : nullptr;
    m.idx = p.idx ? p.idx + (size_t)b * p.k : nullptr;
    m.k = kb;
    m.W = p.W;
    m.nmax = p.N > 0 ? p.N - 1 : 0;
    m.slot0 = slot0;
    m.T_new = p.T_new;
    m.nvalid = nvalid;
    m.stride = DH;
    return m;
}

// Orders this wave's LDS writes before its following LDS reads (and reads
// before later writes).  LDS operations of one wave execute in order, so only
// the compiler must be kept from moving memory accesses across this point; a
// fence would also wait for every outstanding global load, including the
// next block's prefetch.
__device__ __forceinline__ void wave_lds_sync() { asm volatile("" ::: "memory"); }

// 2^x with the hardware instruction alone (no denormal-result fix-up; a
// softmax weight below 2^-126 contributes nothing at fp32 precision anyway).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 16-byte load; NT marks it non-temporal.  The MFMA path loads its V rows
// that way and its K rows with ordinary loads.  Launch times, with the
// Mistral-shaped batch rotated over 8 copies so that nothing is reused from
// the last-level cache (ordinary / V non-temporal / K and V / K only):
// 74.7 / 66.1 / 66.7 / 70.1 us; the 32-layer stack 38.4 / 36.3 / 36.3 /
// 36.7 us; the Dh = 256 layer 136.5 / 128.4 / 139.6 / 127.8 us.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
template <bool NT = false>
__device__ __forceinline__ uint4 ld16(const void *p) {
    if constexpr (NT) {
        const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
        return make_uint4(v.x, v.y, v.z, v.w);
    } else {
        return *reinterpret_cast<const uint4 *>(p);
    }
}
__device__ __forceinline__ void st16(void *p, const uint4 &v) { *reinterpret_cast<uint4 *>(p) = v; }

// Per-wave online-softmax state for G heads and VEC output dims per lane.
template <int G, int VEC>
struct WaveState {
    float m[G], l[G], acc[G][VEC];
    __device__ __forceinline__ void init() {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            m[g] = -INFINITY;
            l[g] = 0.f;
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[g][i] = 0.f;
        }
    }
};

// The ring count, fetched by a wave with a vector load issued after its
// first K/V loads (nothing waits for it before they are in flight) and read
// where a mask or a ring slot needs it, and at the end of the walk (stored
// into LDS before the arrival).
struct RingCount {
    int raw;
    bool loaded;  // wave-uniform
    __device__ __forceinline__ void load(const int32_t *win_count, int b) {
        if (!loaded) {
            raw = win_count ? __hip_atomic_load(win_count + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
            loaded = true;
        }
    }
    __device__ __forceinline__ int value() const {  // clamped at 0, wave-uniform
        const int c = __builtin_amdgcn_readfirstlane(raw);
        return c < 0 ? 0 : c;
    }
};

// One arrival on a counter (relaxed, agent scope) that returns the previous
// value.  The address goes through a VGPR so that the compiler keeps it a
// single returning atomic: its atomic optimizer would otherwise turn it into
// a wave-wide scan that reads the result at once, and since loads and atomics
// complete in order, that wait would also cover every load issued before.
// As it is, the result is waited for only where it is used.
__device__ __forceinline__ unsigned arrive_once(unsigned *ctrs, int i, unsigned one) {
    int iv;
    asm volatile("v_mov_b32 %0, %1" : "=v"(iv) : "s"(i));
    return __hip_atomic_fetch_add(ctrs + iv, one, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// --------------------------------------------------------------- MFMA loop
//
// The key list is walked in three phases, each a contiguous run of rows
// addressed from one uniform base with 32-bit offsets:
//   pool  rows [0, kb):          pool row idx[row] (clamped into the pool);
//   ring  rows [kb, kb + W):     ring slot row - kb, masked unless it holds a
//                                token that survives this call's append
//                                (slot < min(count, W), not one of the slots
//                                (count + t) mod W, t < T_new);
//   new   rows [kb + W, L):      the T_new rows appended in this call, read
//                                from new_k/new_v and written to ring slots
//                                (count + t) mod W.
// That is the same key set as [pool rows] ++ [ring slots after the append];
// softmax attention does not depend on key order.  No address and no phase
// boundary depends on the ring count, so the first K/V loads are issued
// without waiting for it; the count only enters the masks and the slots the
// new rows are written to.  (A masked slot that is being overwritten in the
// same launch may be read before or after the write: its value is unused.)

// IX: rows through the index list (else the pool is the gathered block and
// row r is pool row r; the list pointer is then never read).
template <bool IX>
struct PoolRows {
    const int32_t *idx;  // index list base (IX)
    size_t off;          // this sequence's first entry
    int nmax;
    static constexpr bool kMasked = false;
    __device__ __forceinline__ int key(int row) const {
        if constexpr (IX) return idx[off + row];
        else return row;
    }
    __device__ __forceinline__ int slot(int, int key) const { return key < 0 ? 0 : (key > nmax ? nmax : key); }
    __device__ __forceinline__ bool valid(int) const { return true; }
    __device__ __forceinline__ bool all_valid(int, int) const { return true; }
    __device__ __forceinline__ void resolve(const RingCount &) {}
    __device__ __forceinline__ int limit(int r1) const { return r1; }
};
// The ring in physical slot order: row `first` is slot 0.  Addresses do not
// depend on the count; a slot holds a key of this step when it is filled
// (slot < min(count, W)) and not overwritten by this step's append (slots
// (count + t) mod W, t < T_new) -- a mask applied at compute time.
struct RingRows {
    int first, T_new, W;
    int nvalid = 0, cnt_mod = 0;  // set by resolve(), before the first mask
    static constexpr bool kMasked = true;
    __device__ __forceinline__ void resolve(const RingCount &cnt) {
        const int c = cnt.value();
        nvalid = min(c, W);
        cnt_mod = c % W;
    }
    // Slots past the filled ones hold no key: once the count is known the
    // phase ends there (a ring that has not wrapped yet is not read whole).
    __device__ __forceinline__ int limit(int r1) const { return min(r1, first + nvalid); }
    __device__ __forceinline__ int key(int row) const { return row; }
    __device__ __forceinline__ int slot(int row, int) const { return row - first; }
    __device__ __forceinline__ bool valid(int row) const {
        const int s = row - first;
        int d = s - cnt_mod;
        d += d < 0 ? W : 0;
        return s < nvalid && d >= T_new;
    }
    // Whether every row of [r0, r1) is valid (wave-uniform; in steady state
    // only the T_new slots being overwritten are masked).
    __device__ __forceinline__ bool all_valid(int r0, int r1) const {
        const int s0 = r0 - first, s1 = r1 - first;
        if (s1 > nvalid) return false;
        for (int t = 0; t < T_new; ++t) {
            int sl = cnt_mod + t;
            sl -= sl >= W ? W : 0;
            if (sl >= s0 && sl < s1) return false;
        }
        return true;
    }
};
struct NewRows {
    int first, W;  // row `first` is appended row 0, bound for ring slot count mod W
    int slot0 = 0;  // set by resolve()
    static constexpr bool kMasked = false;
    __device__ __forceinline__ void resolve(const RingCount &cnt) { slot0 = cnt.value() % W; }
    __device__ __forceinline__ int limit(int r1) const { return r1; }
    __device__ __forceinline__ int key(int row) const { return row; }
    __device__ __forceinline__ int slot(int row, int) const { return row - first; }
    __device__ __forceinline__ bool valid(int) const { return true; }
    __device__ __forceinline__ bool all_valid(int, int) const { return true; }
    __device__ __forceinline__ int ring_slot(int row) const {
        const int sl = slot0 + (row - first);
        return sl >= W ? sl - W : sl;
    }
};

// q's A operand: this lane's slice of query head (lane % 16) % G, pre-scaled,
// as bf16 hi + lo parts.
template <int DH, int G>
__device__ __forceinline__ void load_q_operand(const DecodeParams &p, int b, int kvh, bf16x8 (&qa_hi)[DH / 32],
                                               bf16x8 (&qa_lo)[DH / 32]) {
    const int lane = threadIdx.x & 63;
    const int r16 = lane & 15, q4 = lane >> 4;
    const float *qp = p.q + ((size_t)b * p.Hq + (size_t)kvh * G + (r16 % G)) * DH + 8 * q4;
#pragma unroll
    for (int i = 0; i < DH / 32; ++i) {
        const float4 x0 = *reinterpret_cast<const float4 *>(qp + 32 * i);
        const float4 x1 = *reinterpret_cast<const float4 *>(qp + 32 * i + 4);
        const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float v = xs[e] * p.qscale;
            const __bf16 h = (__bf16)v;
            qa_hi[i][e] = h;
            qa_lo[i][e] = (__bf16)(v - (float)h);
        }
    }
}

// q's A operand, filled by the first phase that has a block for the wave,
// after that block's K/V loads are issued (both round trips overlap).
template <int DH>
struct QOperand {
    bf16x8 hi[DH / 32], lo[DH / 32];
    bool ready;
};

// One phase: rows [r0, r1) from bases kbase/vbase (bytes).  A wave takes 16
// rows per block.  K: the lane's row blk + (lane % 16) in the MFMA B layout
// (dims 32i + 8*(lane/16) .. +7).  V: four quarters of 4 rows; in quarter qq
// the lane owns row blk + 4qq + (lane % 4) and dims (DH/16)*(lane/4) ..
// +DH/16-1, so each lane accumulates DH/16 output dims per head.  The p
// values travel from the score layout (lane r holds key r's G weights) to
// the V layout through a 16 x G slot of LDS private to the wave.  Keys
// (index-list entries) are fetched one block ahead of the K/V rows, and the
// K/V rows one block ahead of their use.
template <int NW, int DH, int G, class Rows, bool RING_WRITE>
__device__ __forceinline__ void mfma_phase(const DecodeParams &p, int b, int kvh, int r0, int r1, Rows rows,
                                           const char *kbase, const char *vbase, char *ringK, char *ringV,
                                           QOperand<DH> &qo, RingCount &cnt, float *s_p,
                                           WaveState<G, DH / 16> &st) {
    constexpr int SL = DH / 32, VD = DH / 16, RB = DH * 2;
    constexpr int VB = VD * 2;                 // bytes of V per lane per quarter: 8, 16 or 32
    constexpr int VW = VB >= 16 ? VB / 16 : 1; // 16-byte words (or one 8-byte word)
    constexpr int BSTRIDE = NW * 16;
    constexpr bool kDoubleBuffer = DH <= CMC_DOUBLE_BUFFER_MAX_DH;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, q4 = lane >> 4, kq = lane & 3, dg = lane >> 2;
    const uint32_t koff = 16u * q4;        // + 64 * i for slice i
    const uint32_t voff = (uint32_t)VB * dg;

    int blk = r0 + wave * 16;
    if (blk >= r1) return;  // wave-uniform

    // Rows past the phase end are clamped to its last row and loaded anyway
    // (branch-free loads keep the compiler's wait counts exact, so a block's
    // prefetch is never waited for early); their scores are masked to -inf,
    // so they contribute p = 0.
#define CMC_KEYS(B0_, K_, V_)                                               \
    do {                                                                   \
        K_ = rows.key(min((B0_) + r16, r1 - 1));                           \
        _Pragma("unroll") for (int qq = 0; qq < 4; ++qq)                   \
            V_[qq] = rows.key(min((B0_) + 4 * qq + kq, r1 - 1));           \
    } while (0)
#define CMC_LOAD(B0_, K_, V_, KR_, VR_)                                                                \
    do {                                                                                             \
        {                                                                                            \
            const uint32_t o = (uint32_t)rows.slot(min((B0_) + r16, r1 - 1), K_) * RB + koff;       \
            _Pragma("unroll") for (int i = 0; i < SL; ++i) KR_[i] = ld16(kbase + o + 64 * i);        \
        }                                                                                            \
        _Pragma("unroll") for (int qq = 0; qq < 4; ++qq) {                                           \
            const uint32_t o = (uint32_t)rows.slot(min((B0_) + 4 * qq + kq, r1 - 1), V_[qq]) * RB + voff; \
            if constexpr (VB >= 16) {                                                                \
                _Pragma("unroll") for (int j = 0; j < VW; ++j) VR_[qq][j] = ld16<true>(vbase + o + 16 * j);  \
            } else {                                                                                 \
                const uint2 t = *reinterpret_cast<const uint2 *>(vbase + o);                         \
                VR_[qq][0] = make_uint4(t.x, t.y, 0, 0);                                             \
            }                                                                                        \
        }                                                                                            \
    } while (0)
    // S = Q K^T by MFMA; online softmax rescaling the accumulators only when
    // a head's running max grows (wave-uniform: every lane row holds the same
    // scores); P V on the VALU.
#define CMC_COMPUTE(B0_, KR_, VR_)                                                                     \
    do {                                                                                             \
        /* uniform; a block reaching past r1 is never "full": its rows past the */                    \
        /* phase end may have been loaded before r1 was limited by the count */                     \
        const bool bfull = (B0_) + 16 <= r1 && rows.all_valid((B0_), (B0_) + 16);                   \
        const bool kval = (B0_) + r16 < r1 && (bfull || rows.valid((B0_) + r16));                    \
        floatx4 c = {0.f, 0.f, 0.f, 0.f};                                                            \
        _Pragma("unroll") for (int i = 0; i < SL; ++i) {                                             \
            const bf16x8 kbf = __builtin_bit_cast(bf16x8, KR_[i]);                                   \
            c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qo.hi[i], kbf, c, 0, 0, 0);                 \
            c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qo.lo[i], kbf, c, 0, 0, 0);                 \
        }                                                                                            \
        float pk[G], mbs[G];                                                                         \
        /* the G heads' maxima first, in straight-line code, so their chains interleave */            \
        _Pragma("unroll") for (int g = 0; g < G; ++g) mbs[g] = lane_max16(kval ? c[g] : -INFINITY);      \
        _Pragma("unroll") for (int g = 0; g < G; ++g) {                                              \
            const float sc = kval ? c[g] : -INFINITY;                                                \
            const float mb = mbs[g];                                                                 \
            if (mb > st.m[g]) {                                                                      \
                if (st.m[g] != -INFINITY) { /* before the first valid key l and acc are 0 */         \
                    const float alpha = fast_exp2(st.m[g] - mb);                                     \
                    st.l[g] *= alpha;                                                                \
                    _Pragma("unroll") for (int i = 0; i < VD; ++i) st.acc[g][i] *= alpha;            \
                }                                                                                    \
                st.m[g] = mb;                                                                        \
            }                                                                                        \
            /* a masked key weighs 0 (also before any valid key: m is -inf) */                       \
            pk[g] = kval ? fast_exp2(sc - st.m[g]) : 0.f;                                            \
            st.l[g] += pk[g];                                                                        \
        }                                                                                            \
        if (q4 == 0) {                                                                               \
            _Pragma("unroll") for (int g = 0; g < G; ++g) s_p[r16 * G + g] = pk[g];                 \
        }                                                                                            \
        wave_lds_sync();                                                                             \
        _Pragma("unroll") for (int qq = 0; qq < 4; ++qq) {                                           \
            if constexpr (Rows::kMasked) {                                                           \
                /* masked ring slots (and unfilled slots past r1) may hold anything, */              \
                /* NaN included: zero their values, since 0 * NaN is NaN (p is 0) */                  \
                const int vrow = (B0_) + 4 * qq + kq;                                                \
                if (!bfull && !(vrow < r1 && rows.valid(vrow))) {                                    \
                    _Pragma("unroll") for (int j = 0; j < VW; ++j) VR_[qq][j] = make_uint4(0, 0, 0, 0); \
                }                                                                                    \
            }                                                                                        \
            float pv[G];                                                                             \
            _Pragma("unroll") for (int g = 0; g < G; ++g) pv[g] = s_p[(4 * qq + kq) * G + g];         \
            _Pragma("unroll") for (int j = 0; j < VW; ++j) {                                         \
                float vf[8];                                                                         \
                Vec16<uint16_t>::widen(VR_[qq][j], vf);                                              \
                _Pragma("unroll") for (int g = 0; g < G; ++g)                                        \
                    _Pragma("unroll") for (int e = 0; e < (VD < 8 ? VD : 8); ++e)                    \
                        st.acc[g][8 * j + e] = fmaf(pv[g], vf[e], st.acc[g][8 * j + e]);             \
            }                                                                                        \
        }                                                                                            \
        wave_lds_sync();                                                                             \
        if constexpr (RING_WRITE) {                                                                  \
            if ((B0_) + r16 < r1) {                                                                  \
                const uint32_t o = (uint32_t)rows.ring_slot((B0_) + r16) * RB + koff;                \
                _Pragma("unroll") for (int i = 0; i < SL; ++i) st16(ringK + o + 64 * i, KR_[i]);     \
            }                                                                                        \
            _Pragma("unroll") for (int qq = 0; qq < 4; ++qq) {                                       \
                const int vrow = (B0_) + 4 * qq + kq;                                                \
                if (vrow < r1) {                                                                     \
                    const uint32_t o = (uint32_t)rows.ring_slot(vrow) * RB + voff;                   \
                    if constexpr (VB >= 16) {                                                        \
                        _Pragma("unroll") for (int j = 0; j < VW; ++j) st16(ringV + o + 16 * j, VR_[qq][j]); \
                    } else {                                                                         \
                        *reinterpret_cast<uint2 *>(ringV + o) = make_uint2(VR_[qq][0].x, VR_[qq][0].y); \
                    }                                                                                \
                }                                                                                    \
            }                                                                                        \
        }                                                                                            \
    } while (0)

    // Once the wave's first K/V loads are in flight: fetch the ring count
    // and q, split q (both round trips overlap the K/V loads'), then read the
    // count into the masks and end the phase at the last filled ring slot
    // (a phase without masks does not wait for the count).
#define CMC_AFTER_FIRST_LOAD()                    \
    do {                                          \
        if (!qo.ready) {                          \
            cnt.load(p.win_count, b);             \
            load_q_operand<DH, G>(p, b, kvh, qo.hi, qo.lo); \
            qo.ready = true;                      \
        }                                         \
        rows.resolve(cnt);                        \
        r1 = rows.limit(r1);                      \
    } while (0)

    // Two register sets used in turn: the next block's K/V loads are in
    // flight while this block computes (the loop is unrolled by two so no
    // registers are copied).  Index-list entries are fetched two blocks
    // ahead and issued before the next block's K/V loads: loads retire in
    // issue order, so waiting for the entries then never waits for the
    // prefetched K/V rows.  The wave's last block prefetches nothing (loads
    // past the end would be drained by the barrier after the loop).
    int kc, kvc[4], kn, kvn[4];
    if constexpr (!kDoubleBuffer) {
        // Wide heads: one register set (two would cost an extra wave per SIMD
        // of occupancy); the index entries are still fetched a block ahead.
        uint4 kr[SL], vr[4][VW];
        CMC_KEYS(blk, kc, kvc);
#pragma unroll 1
        for (; blk < r1; blk += BSTRIDE) {
            CMC_LOAD(blk, kc, kvc, kr, vr);
            CMC_AFTER_FIRST_LOAD();
            CMC_KEYS(blk + BSTRIDE, kc, kvc);
            CMC_COMPUTE(blk, kr, vr);
        }
        return;
    }
    uint4 kA[SL], vA[4][VW], kB[SL], vB[4][VW];
    CMC_KEYS(blk, kc, kvc);
    CMC_LOAD(blk, kc, kvc, kA, vA);
    CMC_AFTER_FIRST_LOAD();
    CMC_KEYS(blk + BSTRIDE, kc, kvc);
#pragma unroll 1
    while (true) {
        int nb = blk + BSTRIDE;
        if (nb >= r1) {  // wave-uniform
            CMC_COMPUTE(blk, kA, vA);
            break;
        }
        CMC_KEYS(nb + BSTRIDE, kn, kvn);
        CMC_LOAD(nb, kc, kvc, kB, vB);
        kc = kn;
#pragma unroll
        for (int i = 0; i < 4; ++i) kvc[i] = kvn[i];
        __builtin_amdgcn_sched_barrier(0);  // keep the prefetch above this block's compute
        CMC_COMPUTE(blk, kA, vA);
        blk = nb;
        nb = blk + BSTRIDE;
        if (nb >= r1) {
            CMC_COMPUTE(blk, kB, vB);
            break;
        }
        CMC_KEYS(nb + BSTRIDE, kn, kvn);
        CMC_LOAD(nb, kc, kvc, kA, vA);
        kc = kn;
#pragma unroll
        for (int i = 0; i < 4; ++i) kvc[i] = kvn[i];
        __builtin_amdgcn_sched_barrier(0);
        CMC_COMPUTE(blk, kB, vB);
        blk = nb;
    }
#undef CMC_KEYS
#undef CMC_LOAD
#undef CMC_COMPUTE
#undef CMC_AFTER_FIRST_LOAD
}

template <int NW, int DH, int G, bool IX>
__device__ __forceinline__ void mfma_loop(const DecodeParams &p, int b, int kvh, int kb, int c0, int c1,
                                          RingCount &cnt, float *s_p, WaveState<G, DH / 16> &st) {
    QOperand<DH> qo;
    qo.ready = false;
    const size_t head = (size_t)b * p.Hkv + kvh;
    const int T_new = p.W > 0 ? p.T_new : 0;
    const int pool_end = kb, ring_end = kb + p.W;

    // pool rows
    {
        const PoolRows<IX> rows{p.idx, (size_t)b * p.k, p.N > 0 ? p.N - 1 : 0};
        const char *kb = static_cast<const char *>(p.cme_k) + head * (size_t)p.N * DH * 2;
        const char *vb = static_cast<const char *>(p.cme_v) + head * (size_t)p.N * DH * 2;
        mfma_phase<NW, DH, G, PoolRows<IX>, false>(p, b, kvh, c0, min(c1, pool_end), rows, kb, vb, nullptr, nullptr, qo,
                                               cnt, s_p, st);
    }
    if (p.W > 0) {
        char *wk = static_cast<char *>(p.win_k) + head * (size_t)p.W * DH * 2;
        char *wv = static_cast<char *>(p.win_v) + head * (size_t)p.W * DH * 2;
        // the W ring slots in physical order, masked by the count
        const RingRows rr{pool_end, T_new, p.W};
        mfma_phase<NW, DH, G, RingRows, false>(p, b, kvh, max(c0, pool_end), min(c1, ring_end), rr, wk, wv, nullptr,
                                               nullptr, qo, cnt, s_p, st);
        // rows appended in this call
        if (T_new > 0) {
            const NewRows nr{ring_end, p.W};
            const char *nk = static_cast<const char *>(p.new_k) + head * (size_t)T_new * DH * 2;
            const char *nv = static_cast<const char *>(p.new_v) + head * (size_t)T_new * DH * 2;
            mfma_phase<NW, DH, G, NewRows, true>(p, b, kvh, max(c0, ring_end), c1, nr, nk, nv, wk, wv, qo, cnt, s_p,
                                                 st);
        }
    }
    // Wave totals: l over the 16 keys of one lane row (rows hold copies),
    // acc over the 4 keys sharing a dim group.
#pragma unroll
    for (int g = 0; g < G; ++g) {
        st.l[g] = lane_reduce<OpSum, 1, 16>(st.l[g]);
#pragma unroll
        for (int i = 0; i < DH / 16; ++i) st.acc[g][i] = lane_reduce<OpSum, 1, 4>(st.acc[g][i]);
    }
}

// --------------------------------------------------------------- VALU loop

template <int NW, typename T, int DH, int G, int U>
__device__ __forceinline__ void valu_loop(const DecodeParams &p, const RowMap<T> &rm, int b, int kvh, int c0,
                                          int c1, WaveState<G, Vec16<T>::N> &st) {
    constexpr int VEC = Vec16<T>::N;
    constexpr int LPR = DH / VEC;
    constexpr int RPW = kWave / LPR;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int grp = lane / LPR, e = lane % LPR;
    CMC_UNPACK_ROWMAP(rm);

    float qf[G][VEC];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const float4 *qp = reinterpret_cast<const float4 *>(
            p.q + ((size_t)b * p.Hq + (size_t)kvh * G + g) * DH + e * VEC);
#pragma unroll
        for (int i = 0; i < VEC / 4; ++i) {
            const float4 t = qp[i];
            qf[g][4 * i + 0] = t.x * p.qscale;
            qf[g][4 * i + 1] = t.y * p.qscale;
            qf[g][4 * i + 2] = t.z * p.qscale;
            qf[g][4 * i + 3] = t.w * p.qscale;
        }
    }

    constexpr int STRIDE = NW * RPW;
    for (int r0 = c0 + wave * RPW; r0 < c1; r0 += STRIDE * U) {
        uint4 kr[U], vr[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int row = r0 + u * STRIDE + grp;
            ok[u] = row < c1 && VALID(row);
            kr[u] = vr[u] = make_uint4(0, 0, 0, 0);
            if (ok[u]) {
                const RowPtrs<T> rp = LOCATE(row);
                kr[u] = ld16(rp.k + e * VEC);
                vr[u] = ld16(rp.v + e * VEC);
                if (rp.rk) {
                    st16(rp.rk + e * VEC, kr[u]);
                    st16(rp.rv + e * VEC, vr[u]);
                }
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
            mb = lane_reduce<OpMax, LPR, kWave>(mb);
            const float mn = fmaxf(st.m[g], mb);
            const float alpha = mn == -INFINITY ? 1.f : exp2f(st.m[g] - mn);  // nothing valid yet: keep
            st.l[g] *= alpha;
#pragma unroll
            for (int i = 0; i < VEC; ++i) st.acc[g][i] *= alpha;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float pu = ok[u] ? exp2f(sc[u][g] - mn) : 0.f;
                st.l[g] += pu;
#pragma unroll
                for (int i = 0; i < VEC; ++i) st.acc[g][i] = fmaf(pu, vf[u][i], st.acc[g][i]);
            }
            st.m[g] = mn;
        }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
        st.l[g] = lane_reduce<OpSum, LPR, kWave>(st.l[g]);
#pragma unroll
        for (int i = 0; i < VEC; ++i) st.acc[g][i] = lane_reduce<OpSum, LPR, kWave>(st.acc[g][i]);
    }
}

// ------------------------------------------------------------------ kernel

// Cross-workgroup publication without device-scope fences.  The partials are
// written and read with relaxed agent-scope atomic accesses (coherent across
// the XCDs' L2 caches, unlike plain accesses), the writer waits until its
// stores have completed (s_waitcnt) before arriving on the counter, and the
// reader issues its loads only after the arrival count has returned.  An
// agent-scope fence would instead write back and invalidate the whole L2 of
// the XCD for every workgroup, which costs microseconds each.
// Two adjacent floats (8-byte aligned) as one 64-bit coherent access.
__device__ __forceinline__ void coherent_store2(float *p, float a, float b) {
    const uint64_t v = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
    __hip_atomic_store(reinterpret_cast<uint64_t *>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 coherent_load2(const float *p) {
    const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t *>(p), __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
    return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}

// Combine the waves' (m, l, acc) of head g, dim d; returns the joint max.
template <int NW, int G, int DH>
__device__ __forceinline__ float combine_waves(const float (&sm)[NW][G], const float (&sl)[NW][G],
                                               const float (&sa)[NW][G][DH], int g, int d, float &num,
                                               float &den) {
    // Every LDS read issued before the first wait, and no branch on M: with
    // no valid key in any wave (M = -inf) every weight is exp2(-inf) = 0
    // against finite accumulators (zeros), so num = den = 0.
    float mw[NW], lw[NW], aw[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        mw[w] = sm[w][g];
        lw[w] = sl[w][g];
        aw[w] = sa[w][g][d];
    }
    float M = mw[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, mw[w]);
    const float Mc = M == -INFINITY ? 0.f : M;
    num = 0.f;
    den = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const float f = fast_exp2(mw[w] - Mc);
        num = fmaf(f, aw[w], num);
        den = fmaf(f, lw[w], den);
    }
    return M;
}

// The leading arguments are the fields the first K/V loads need (info packs
// S, new_split, whether k_len is given, and T_new); they arrive in
// SGPRs at wave launch (kernel-argument preloading, 14 dwords), so those
// loads never wait for the kernel-argument segment.  The rest of the
// parameters come from `pm`.
template <int NW, typename T, int DH, int G, bool MF, bool IX>
__global__ __launch_bounds__(NW * kWave) void decode_kernel(const void *cme_k, const void *cme_v, void *win_k,
                                                            void *win_v, int k, int W, int N, int Hkv, int chunk,
                                                            int info, DecodeParams pm) {
    DecodeParams p = pm;
    p.cme_k = cme_k;
    p.cme_v = cme_v;
    p.win_k = win_k;
    p.win_v = win_v;
    p.k = k;
    p.W = W;
    p.N = N;
    p.Hkv = Hkv;
    p.chunk = chunk;
    p.S = info & 0xFF;
    p.new_split = (info >> 8) & 1;
    const bool has_klen = (info >> 10) & 1;
    p.T_new = (int)((unsigned)info >> 16);
    constexpr int kThreads = NW * kWave;
    constexpr int VEC = MF ? DH / 16 : Vec16<T>::N;  // output dims a lane accumulates
    const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

    // Ring count.  MFMA path: fetched by each wave after its first K/V loads
    // (RingCount), so they never wait for it.  VALU path: read up front (its
    // row map resolves ring slots before the loads).
    RingCount cnt{0, false};
    int cnt0 = 0, slot0 = 0;
    if (p.W > 0) {
        if constexpr (!MF) {
            cnt.raw = p.win_count[b];
            cnt.loaded = true;
            cnt0 = cnt.raw < 0 ? 0 : cnt.raw;
            slot0 = cnt0 % p.W;
        }
    }
    int kb = p.k;  // pool rows of this sequence
    if (has_klen) {
        const int v = p.k_len[b];
        kb = v < 0 ? 0 : (v > p.k ? p.k : v);
    }
    // Key list: kb pool rows, the W ring slots, the T_new appended rows (see
    // the phases above); its length does not depend on the ring count.  The
    // split plan covers k + W rows in chunks; the appended rows go to the last
    // split, or to a split of their own (the last) when p.new_split is set.
    const int Lkw = kb + p.W;
    const int L = kb + (p.W > 0 ? p.W + p.T_new : 0);
    int c0, c1;
    if (p.new_split) {
        const bool own = s == p.S - 1;
        c0 = own ? Lkw : s * p.chunk;
        c1 = own ? L : (s == p.S - 2 ? Lkw : min(c0 + p.chunk, Lkw));
    } else {
        c0 = s * p.chunk;
        c1 = s == p.S - 1 ? L : min(c0 + p.chunk, L);
    }
    const RowMap<T> rm = make_rowmap<T>(p, b, kvh, DH, kb, slot0, min(cnt0, p.W));

    // Ring count.  It may be advanced only after every wave of the
    // sequence's workgroups has read it.  Each wave stores the count it read
    // into LDS before the barrier that ends its walk (a store of the loaded
    // value, so the read has returned by then); after that barrier one
    // arrival per (sequence, kv head) pair goes to the sequence's counter:
    //   S == 1: thread 0 of the workgroup, right after the barrier;
    //   S > 1: each split arrives on its pair counter after that barrier, and
    //     the merging workgroup (the last split of the pair) then arrives for
    //     the pair, overlapping its merge loads.
    // The last of the Hkv arrivals writes the advanced count and re-arms the
    // counter, at its workgroup's end (the arrival's value is waited for only
    // there).  No data is published through the counter, so no fence is
    // needed.
    const bool bump = p.T_new > 0 && p.W > 0;
    unsigned prev = ~0u;  // the sequence counter before this workgroup's arrival (one lane)

    WaveState<G, VEC> st;
    st.init();
    if constexpr (MF) {
        __shared__ float s_pw[NW][16 * G];
        mfma_loop<NW, DH, G, IX>(p, b, kvh, kb, c0, c1, cnt, s_pw[threadIdx.x >> 6], st);
    } else {
        constexpr int U = (sizeof(T) == 2 && DH >= 128) ? 4 : 2;
        valu_loop<NW, T, DH, G, U>(p, rm, b, kvh, c0, c1, st);
    }
    if (p.W > 0) cnt.load(p.win_count, b);  // a wave without K/V rows
    const int cnt_now = MF ? cnt.value() : cnt0;
#define CMC_BUMP()                                                                         \
    do {                                                                                 \
        if (bump && prev == (unsigned)(p.Hkv - 1)) { /* one lane per sequence */       \
            p.win_count[b] = cnt_now + p.T_new;                                          \
            __hip_atomic_store(&p.seq_counter[b], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); \
        }                                                                                \
    } while (0)

    // Lanes holding each dim group after the wave reduction.
    constexpr int LPR = MF ? 4 : DH / Vec16<T>::N;         // lanes per dim group stride
    const bool holder = MF ? ((lane & 3) == 0) : (lane < LPR);
    const int dbase = MF ? (lane >> 2) * VEC : lane * VEC;

    __shared__ float s_acc[NW][G][DH];
    __shared__ float s_m[NW][G], s_l[NW][G];
    if (holder) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int i = 0; i < VEC; ++i) s_acc[wave][g][dbase + i] = st.acc[g][i];
    }
    if (lane == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            s_m[wave][g] = st.m[g];
            s_l[wave][g] = st.l[g];
        }
    }
    __shared__ int s_cnt[NW];
    if (bump && lane == 0) s_cnt[wave] = cnt.raw;  // stored once the wave's count read has returned
    __syncthreads();

    const size_t head = (size_t)b * p.Hkv + kvh;
    float *outp = p.out + ((size_t)b * p.Hq + (size_t)kvh * G) * DH;
    __shared__ int s_last;
    if (p.S == 1) {
        // every wave's count read returned before the barrier above
        if (bump && threadIdx.x == 0) prev = arrive_once(p.seq_counter, b, (unsigned)(s_cnt[NW - 1] != INT_MIN));
        for (int t = threadIdx.x; t < G * DH; t += kThreads) {
            const int g = t / DH, d = t % DH;
            float num, den;
            combine_waves<NW, G, DH>(s_m, s_l, s_acc, g, d, num, den);
            outp[t] = den > 0.f ? num * __builtin_amdgcn_rcpf(den) : 0.f;
        }
        CMC_BUMP();
    } else {
        // Publish this split's partial with agent-coherent 64-bit stores (two
        // dims per thread), wait for them to complete, then arrive on the
        // (b, kv head) counter.
        const size_t part = (head * p.S + s) * G;
        for (int t = threadIdx.x; t < G * DH / 2; t += kThreads) {
            const int g = (2 * t) / DH, d = (2 * t) % DH;
            float n0, n1, den;
            const float M = combine_waves<NW, G, DH>(s_m, s_l, s_acc, g, d, n0, den);
            combine_waves<NW, G, DH>(s_m, s_l, s_acc, g, d + 1, n1, den);
            coherent_store2(&p.part_acc[(part + g) * DH + d], n0, n1);
            if (d == 0) coherent_store2(&p.part_ml[(part + g) * 2], M, den);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0) {
            const unsigned prev = __hip_atomic_fetch_add(&p.pair_counter[head], 1u, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT);
            s_last = prev == (unsigned)(p.S - 1);
        }
        __syncthreads();
        if (!s_last) return;  // workgroup-uniform
        // The last split merges all S partials in fixed split order.  Its
        // first batch of acc partials (up to kMB splits per dim pair) and all
        // (m, l) pairs are requested together, so the merge costs one round
        // trip when S <= kMB; the (m, l) pairs are staged in LDS.  The
        // batch's loads are issued unconditionally (splits past S - 1 reload
        // split S - 1 and are never used): as atomic loads they cannot be
        // speculated, and a branch around each cost about a dozen
        // instructions between the arrival and the merge's data.
        constexpr int kPairs = (G * DH / 2 + kThreads - 1) / kThreads;  // dim pairs per thread
        constexpr int kMB = kPairs >= 4 ? 8 : 16;
        const float *ml = p.part_ml + head * p.S * G * 2;
        const float *ac = p.part_acc + head * p.S * G * DH;
        float *s_ml = &s_acc[0][0][0];  // reuse: S*G*2 <= NW*G*DH floats (S <= 2*DH)
        // The (m, l) pairs are requested first (loads complete in issue
        // order, and the max and the weights need only them), and the barrier
        // that publishes them in LDS waits for LDS alone: the acc partials
        // may still be in flight while the weights are computed, and their
        // first use waits for them.
        const bool ml_first = threadIdx.x < p.S * G;  // the first kThreads pairs
        float2 mlv = make_float2(0.f, 0.f);
        if (ml_first) mlv = coherent_load2(&ml[2 * threadIdx.x]);
        float2 a[kPairs][kMB];
#pragma unroll
        for (int pr = 0; pr < kPairs; ++pr) {
            const int t = threadIdx.x + pr * kThreads;
            const int g = (2 * min(t, G * DH / 2 - 1)) / DH, d = (2 * min(t, G * DH / 2 - 1)) % DH;
#pragma unroll
            for (int j = 0; j < kMB; ++j) a[pr][j] = coherent_load2(&ac[(min(j, p.S - 1) * G + g) * DH + d]);
        }
        if (ml_first) {
            s_ml[2 * threadIdx.x] = mlv.x;
            s_ml[2 * threadIdx.x + 1] = mlv.y;
        }
        for (int t = threadIdx.x + kThreads; t < p.S * G; t += kThreads) {
            const float2 v = coherent_load2(&ml[2 * t]);
            s_ml[2 * t] = v.x;
            s_ml[2 * t + 1] = v.y;
        }
        // this workgroup completes the pair; the arrival overlaps the merge loads
        if (bump && threadIdx.x == 0) prev = arrive_once(p.seq_counter, b, (unsigned)(s_cnt[NW - 1] != INT_MIN));
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0) only: vmcnt and expcnt at their maxima
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
#pragma unroll
        for (int pr = 0; pr < kPairs; ++pr) {
            const int t = threadIdx.x + pr * kThreads;
            if (t >= G * DH / 2) continue;
            const int g = (2 * t) / DH, d = (2 * t) % DH;
            // The first batch's (m, l) pairs read together (splits past S - 1
            // read split S - 1 again), and its terms masked by selects rather
            // than branches: no LDS round trip waits for another.  The max
            // is unchanged by the repeats, and the sums take the splits in
            // order as before.
            float mj[kMB], lj[kMB];
#pragma unroll
            for (int j = 0; j < kMB; ++j) {
                const float2 v = *reinterpret_cast<const float2 *>(&s_ml[(min(j, p.S - 1) * G + g) * 2]);
                mj[j] = v.x;
                lj[j] = v.y;
            }
            float M = -INFINITY;
#pragma unroll
            for (int j = 0; j < kMB; ++j) M = fmaxf(M, mj[j]);
            for (int q = kMB; q < p.S; ++q) M = fmaxf(M, s_ml[(q * G + g) * 2]);
            float n0 = 0.f, n1 = 0.f, den = 0.f;
            if (M != -INFINITY) {
#pragma unroll
                for (int j = 0; j < kMB; ++j) {
                    const bool in = j < p.S;
                    const float f = fast_exp2(mj[j] - M);
                    den = in ? fmaf(f, lj[j], den) : den;
                    n0 = in ? fmaf(f, a[pr][j].x, n0) : n0;
                    n1 = in ? fmaf(f, a[pr][j].y, n1) : n1;
                }
                for (int q0 = kMB; q0 < p.S; q0 += kMB) {
                    float2 x[kMB];
#pragma unroll
                    for (int j = 0; j < kMB; ++j)
                        x[j] = q0 + j < p.S ? coherent_load2(&ac[((q0 + j) * G + g) * DH + d])
                                            : make_float2(0.f, 0.f);
#pragma unroll
                    for (int j = 0; j < kMB; ++j) {
                        if (q0 + j < p.S) {
                            const int q = q0 + j;
                            const float f = fast_exp2(s_ml[(q * G + g) * 2] - M);
                            den = fmaf(f, s_ml[(q * G + g) * 2 + 1], den);
                            n0 = fmaf(f, x[j].x, n0);
                            n1 = fmaf(f, x[j].y, n1);
                        }
                    }
                }
            }
            const float inv = den > 0.f ? __builtin_amdgcn_rcpf(den) : 0.f;  // within 1 ulp
            *reinterpret_cast<float2 *>(&outp[g * DH + d]) = make_float2(n0 * inv, n1 * inv);
        }
        if (threadIdx.x == 0)
            __hip_atomic_store(&p.pair_counter[head], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        CMC_BUMP();
    }
#undef CMC_BUMP

}

template <typename T, int DH, int G>
hipError_t launch3(const DecodeParams &p, hipStream_t stream) {
    dim3 grid(p.S, p.Hkv, p.B);
    constexpr bool kMf = sizeof(T) == 2 && G >= CMC_MFMA_MIN_G && G <= 4;
    if (p.S < 1 || p.S > 0xFF || p.T_new < 0 || p.T_new > kMaxAppendRows) return hipErrorInvalidValue;
    const int info = p.S | (p.new_split << 8) | ((p.k_len != nullptr) << 10) | (p.T_new << 16);
    const bool ix = kMf && p.idx != nullptr;
#define CMC_LAUNCH(NW_, IX_)                                                                                     \
    decode_kernel<NW_, T, DH, G, kMf, IX_><<<grid, NW_ * kWave, 0, stream>>>(p.cme_k, p.cme_v, p.win_k, p.win_v, \
                                                                             p.k, p.W, p.N, p.Hkv, p.chunk, info, p)
    if (p.waves == 4) {
        if (ix) CMC_LAUNCH(4, kMf);
        else CMC_LAUNCH(4, false);
    } else if constexpr (decode_waves_ok(8, G, DH)) {
        if (p.waves != 8) return hipErrorInvalidValue;
        if (ix) CMC_LAUNCH(8, kMf);
        else CMC_LAUNCH(8, false);
    } else {
        return hipErrorInvalidValue;
    }
#undef CMC_LAUNCH
    return hipGetLastError();
}

template <typename T, int DH>
hipError_t launch_g(const DecodeParams &p, int G, hipStream_t stream) {
    switch (G) {
        case 1: return launch3<T, DH, 1>(p, stream);
        case 2: return launch3<T, DH, 2>(p, stream);
        case 4: return launch3<T, DH, 4>(p, stream);
        case 8: return launch3<T, DH, 8>(p, stream);
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
