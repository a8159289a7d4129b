"""Seeded synthetic workloads for the two-tier decode path.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic (no scoring, no selection, no attention). Both the HIP
path and the CPU oracle are fed from it, so it imports neither.

Every tensor comes from its own counter-keyed stream,
``numpy.random.default_rng([seed, role, layer, ...])``, so any slice
(a sequence, a head, a decode step) can be regenerated on its own without
drawing the rest.  bf16 tensors are produced by drawing fp32 values and
rounding them to bf16 with round-to-nearest-even; they are returned as the
raw 16-bit patterns (``numpy.uint16``).

The shapes follow the Llama/Mistral-class decoders the paper evaluates
(Sec. 3, efficiency study; App. A.5 geometry n_h, d_h, n_l), with Tier-1
size k and window W as in Sec. 2.5.  The paper's own efficiency runs use
SQuAD, which is not available here; these synthetic inputs stand in for it.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional, Sequence

import numpy as np

# Stream roles: part of the seed key of every draw.
ROLE = {
    "sel_keys": 1,   # decoder-ready memory rows M (selection keys)
    "q_vec": 2,      # mean-pooled question vector
    "cme_k": 3,      # Tier-1 pool keys, one row per CME
    "cme_v": 4,      # Tier-1 pool values
    "win_k": 5,      # initial Tier-2 window keys (prefilled C_local)
    "win_v": 6,      # initial Tier-2 window values
    "q": 7,          # per-step decoder queries
    "new_k": 8,      # per-step appended key row
    "new_v": 9,      # per-step appended value row
    "chan": 10,      # log-normal per-channel scale
    "full_k": 11,    # uncompressed-cache baseline keys
    "full_v": 12,    # uncompressed-cache baseline values
    "ragged": 13,    # per-sequence sizes of a ragged batch
    "emb": 14,       # token embeddings of the denoising workloads
}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic decode workload.

    B batch, Hq/Hkv query/key-value heads, Dh head dim, N CMEs per
    sequence, D selection-key dim, k Tier-1 size, W window capacity,
    steps decode steps, layers decoder layers sharing one index list.
    ``kv_dtype`` is "f32" or "bf16"; selection keys, q_vec and decoder
    queries are always fp32.  ``kv_std`` is the standard deviation of the
    K/V/query draws before any channel scale; ``chan_sigma`` > 0 multiplies
    K and V by exp(N(0, chan_sigma^2)) per (kv head, channel).
    ``full_ctx`` > 0 describes an uncompressed-cache baseline of that many
    prefilled tokens.

    Ragged batches (``ragged``): sequence b has a context of ctx_b tokens,
    drawn log-uniform in [ctx_min, ctx_max]; it has n_b = ceil(ctx_b /
    ratio) memory rows (N is the largest), keeps k_b = min(k, n_b) of them,
    pins q_b question rows (uniform in [q_min, q_max]) stored in its pool
    right after its memory rows, and starts with min(W, ctx_b) tokens in its
    window.
    """

    name: str
    B: int
    Hq: int
    Hkv: int
    Dh: int
    N: int
    D: int
    k: int
    W: int
    steps: int
    kv_dtype: str
    kv_std: float
    seed: int
    layers: int = 1
    chan_sigma: float = 0.0
    full_ctx: int = 0
    gap_min: float = 1e-3
    ragged: bool = False
    ctx_min: int = 0
    ctx_max: int = 0
    ratio: int = 4
    q_min: int = 0
    q_max: int = 0

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.Dh)

    @property
    def kv_bytes(self) -> int:
        return 2 if self.kv_dtype == "bf16" else 4

    @property
    def pool_rows(self) -> int:
        """Rows of each (sequence, kv head) pool: the memory rows plus room
        for the pinned question rows."""
        return self.N + self.q_max

    @property
    def idx_stride(self) -> int:
        """Entries per index-list row: the selection plus the question rows."""
        return self.k + self.q_max

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    # Tiny fp32 single layer: the correctness case.
    "tiny_fp32": Workload("tiny_fp32", B=1, Hq=4, Hkv=4, Dh=64, N=64, D=256, k=16,
                          W=128, steps=16, kv_dtype="f32", kv_std=1.0, seed=101),
    # One Llama-3-8B-shaped layer: 8192-token context at ratio 4 -> 2048 CMEs.
    "llama3_8b_layer": Workload("llama3_8b_layer", B=1, Hq=32, Hkv=8, Dh=128, N=2048,
                                D=4096, k=256, W=512, steps=3000, kv_dtype="bf16",
                                kv_std=1.0 / math.sqrt(128.0), seed=202),
    # Mistral-7B-shaped batched decode, per-sequence pools and index lists.
    "mistral7b_batch64": Workload("mistral7b_batch64", B=64, Hq=32, Hkv=8, Dh=128,
                                  N=4096, D=4096, k=512, W=1024, steps=3000,
                                  kv_dtype="bf16", kv_std=1.0 / math.sqrt(128.0),
                                  seed=303),
    # Long-context wide-head layer: 131072 tokens at ratio 8 -> 16384 CMEs.
    "long_wide_d256": Workload("long_wide_d256", B=16, Hq=16, Hkv=16, Dh=256, N=16384,
                               D=3072, k=1024, W=2048, steps=3000, kv_dtype="bf16",
                               kv_std=1.0, seed=404, chan_sigma=1.0),
    # Ragged Mistral-7B-shaped batch: contexts of 512..16384 tokens at ratio 4
    # (128..4096 memory rows, some below k), 8..48 pinned question rows.
    "ragged_batch64": Workload("ragged_batch64", B=64, Hq=32, Hkv=8, Dh=128, N=4096,
                               D=4096, k=512, W=1024, steps=3000, kv_dtype="bf16",
                               kv_std=1.0 / math.sqrt(128.0), seed=606, ragged=True,
                               ctx_min=512, ctx_max=16384, ratio=4, q_min=8, q_max=48),
    # The paper's own cache sizes (batch 8, K = 40 memory rows, W = 130 window
    # tokens, contexts of up to 3072 tokens at ratio 4 -> 768 CMEs) with Llama
    # heads: latency context next to the larger configurations.
    "paper_scale_b8": Workload("paper_scale_b8", B=8, Hq=32, Hkv=8, Dh=128, N=768, D=4096, k=40,
                               W=130, steps=3000, kv_dtype="bf16", kv_std=1.0 / math.sqrt(128.0),
                               seed=909),
    # 32-layer Llama-shaped decode stack; baseline is a 32768-token full cache.
    "llama_stack32": Workload("llama_stack32", B=32, Hq=32, Hkv=8, Dh=128, N=8192,
                              D=4096, k=512, W=1024, steps=3000, kv_dtype="bf16",
                              kv_std=1.0 / math.sqrt(128.0), seed=505, layers=32,
                              full_ctx=32768),
    # The Mistral-shaped batch over 8 copies of its layer (3.2 GB of K/V):
    # consecutive launches reuse nothing from the 256 MB last-level cache.
    "mistral7b_batch64_x8": Workload("mistral7b_batch64_x8", B=64, Hq=32, Hkv=8, Dh=128,
                                     N=4096, D=4096, k=512, W=1024, steps=3000,
                                     kv_dtype="bf16", kv_std=1.0 / math.sqrt(128.0),
                                     seed=303, layers=8),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


# ---------------------------------------------------------------- streams

def _rng(seed: int, role: str, *ids: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), ROLE[role], *[int(i) for i in ids]])


def normal_f32(seed: int, role: str, ids: Sequence[int], shape, std: float = 1.0) -> np.ndarray:
    """fp32 N(0, std^2) draws from the stream keyed by (seed, role, *ids)."""
    x = _rng(seed, role, *ids).standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


# ------------------------------------------------------------------ bf16

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); return the bits.

    Inputs are finite draws, so NaN handling is not needed here.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _kv_cast(w: Workload, x: np.ndarray) -> np.ndarray:
    return f32_to_bf16_bits(x) if w.kv_dtype == "bf16" else x


# ------------------------------------------------------------- selection

def sel_keys(w: Workload, b: Optional[int] = None) -> np.ndarray:
    """Selection keys M, fp32 N(0,1): [B][N][D], or [N][D] for one sequence."""
    if b is not None:
        return normal_f32(w.seed, "sel_keys", (b,), (w.N, w.D))
    return np.stack([sel_keys(w, i) for i in range(w.B)])


def q_vec(w: Workload, b: int, attempt: int = 0) -> np.ndarray:
    """Question vector for sequence b, fp32 N(0,1) [D]; ``attempt`` picks a
    fresh draw (used by tests that reject draws with a narrow score gap)."""
    return normal_f32(w.seed, "q_vec", (b, attempt), (w.D,))


def q_vecs(w: Workload, attempts: Optional[Sequence[int]] = None) -> np.ndarray:
    att = attempts if attempts is not None else [0] * w.B
    return np.stack([q_vec(w, b, att[b]) for b in range(w.B)])


# ------------------------------------------------------------- KV caches

def chan_scale(w: Workload, layer: int = 0) -> Optional[np.ndarray]:
    """Per (kv head, channel) log-normal scale [Hkv][Dh], or None."""
    if w.chan_sigma <= 0:
        return None
    z = normal_f32(w.seed, "chan", (layer,), (w.Hkv, w.Dh))
    return np.exp(np.float32(w.chan_sigma) * z).astype(np.float32)


def _kv_rows(w: Workload, role: str, layer: int, b: int, h: int, rows: int,
             scale: Optional[np.ndarray], extra: Sequence[int] = ()) -> np.ndarray:
    x = normal_f32(w.seed, role, (layer, b, h, *extra), (rows, w.Dh), w.kv_std)
    if scale is not None:
        x *= scale[h][None, :]
    return x


def ragged_sizes(w: Workload) -> Dict[str, np.ndarray]:
    """Per-sequence sizes of a ragged batch (int32 [B] each): ctx (context
    tokens), n_rows (memory rows), q_rows (pinned question rows), fill
    (initial window tokens).  A uniform workload gets ctx = N * ratio,
    n_rows = N, q_rows = 0 and fill = W."""
    if not w.ragged:
        return {"ctx": np.full(w.B, w.N * w.ratio, np.int32), "n_rows": np.full(w.B, w.N, np.int32),
                "q_rows": np.zeros(w.B, np.int32), "fill": np.full(w.B, w.W, np.int32)}
    r = _rng(w.seed, "ragged")
    u = r.random(w.B)
    ctx = np.exp(math.log(w.ctx_min) + u * (math.log(w.ctx_max) - math.log(w.ctx_min)))
    ctx = np.clip(np.round(ctx), w.ctx_min, w.ctx_max).astype(np.int64)
    n_rows = np.minimum((ctx + w.ratio - 1) // w.ratio, w.N)
    q_rows = r.integers(w.q_min, w.q_max + 1, size=w.B)
    fill = np.minimum(ctx, w.W)
    return {"ctx": ctx.astype(np.int32), "n_rows": n_rows.astype(np.int32),
            "q_rows": q_rows.astype(np.int32), "fill": fill.astype(np.int32)}


def pool_kv(w: Workload, layer: int = 0, b: Optional[int] = None,
            h: Optional[int] = None, rows: Optional[int] = None):
    """Tier-1 pool K and V, [B][Hkv][pool_rows][Dh] (or one sequence / one
    head): memory rows, then (ragged workloads) room for question rows, all
    drawn from one stream per (sequence, head), so the first N rows do not
    depend on the room added after them.

    ``rows`` overrides that (the uncompressed baseline uses the same layout
    with ``full_ctx`` rows and its own roles).
    """
    n = w.pool_rows if rows is None else rows
    rk, rv = ("cme_k", "cme_v") if rows is None else ("full_k", "full_v")
    s = chan_scale(w, layer)
    bs = range(w.B) if b is None else [b]
    hs = range(w.Hkv) if h is None else [h]
    K = np.stack([np.stack([_kv_rows(w, rk, layer, bb, hh, n, s) for hh in hs]) for bb in bs])
    V = np.stack([np.stack([_kv_rows(w, rv, layer, bb, hh, n, s) for hh in hs]) for bb in bs])
    if h is not None:
        K, V = K[:, 0], V[:, 0]
    if b is not None:
        K, V = K[0], V[0]
    return _kv_cast(w, K), _kv_cast(w, V)


def window_kv(w: Workload, layer: int = 0, fill=None):
    """Initial Tier-2 ring [B][Hkv][W][Dh] and its count [B] (int32).

    Sequence b's ring starts holding fill_b prefilled tokens in slots
    0..fill_b-1 (unused slots are zero).  ``fill`` is one count for every
    sequence or one per sequence; by default the ring is full (W), or, for
    a ragged workload, holds min(W, ctx_b) tokens.
    """
    if fill is None:
        fills = ragged_sizes(w)["fill"]
    else:
        fills = np.broadcast_to(np.asarray(fill, np.int32), (w.B,))
    s = chan_scale(w, layer)
    K = np.zeros((w.B, w.Hkv, w.W, w.Dh), np.float32)
    V = np.zeros((w.B, w.Hkv, w.W, w.Dh), np.float32)
    for b in range(w.B):
        f = int(fills[b])
        for h in range(w.Hkv):
            if f:
                K[b, h, :f] = _kv_rows(w, "win_k", layer, b, h, f, s)
                V[b, h, :f] = _kv_rows(w, "win_v", layer, b, h, f, s)
    count = np.array(fills, np.int32)
    return _kv_cast(w, K), _kv_cast(w, V), count


# ------------------------------------------------------------ decode steps

def step_q(w: Workload, step: int, layer: int = 0) -> np.ndarray:
    """Decoder queries for one step: fp32 [B][Hq][Dh], N(0, kv_std^2)."""
    return normal_f32(w.seed, "q", (layer, step), (w.B, w.Hq, w.Dh), w.kv_std)


def step_new_kv(w: Workload, step: int, layer: int = 0, t_new: int = 1):
    """Rows appended at one step: [B][Hkv][t_new][Dh] each (K, V)."""
    s = chan_scale(w, layer)
    K = normal_f32(w.seed, "new_k", (layer, step), (w.B, w.Hkv, t_new, w.Dh), w.kv_std)
    V = normal_f32(w.seed, "new_v", (layer, step), (w.B, w.Hkv, t_new, w.Dh), w.kv_std)
    if s is not None:
        K *= s[None, :, None, :]
        V *= s[None, :, None, :]
    return _kv_cast(w, K), _kv_cast(w, V)


def kv_to_f32(w: Workload, x: np.ndarray) -> np.ndarray:
    """K/V tensor as exact fp32 values (bf16 widened)."""
    return bf16_bits_to_f32(x) if w.kv_dtype == "bf16" else np.asarray(x, np.float32)


# ------------------------------------------------- device-side generation
#
# The 32-layer stack (tens of GB of K/V) is drawn directly on the GPU with
# torch's counter-based generator, one stream per (seed, role, ids) as above.
# These draws are not bit-identical to the numpy ones; they feed timing
# runs only (parity for that shape runs one layer from the numpy
# streams).

def _device_seed(seed: int, role: str, ids: Sequence[int]) -> int:
    ss = np.random.SeedSequence([int(seed), ROLE[role], *[int(i) for i in ids]])
    return int(ss.generate_state(1, np.uint64)[0] & np.uint64((1 << 63) - 1))


def device_normal(seed: int, role: str, ids: Sequence[int], shape, std: float, device, dtype):
    """N(0, std^2) draws generated on `device`, returned in `dtype`."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(_device_seed(seed, role, ids))
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


# ------------------------------------------------------------- denoising

@dataclasses.dataclass(frozen=True)
class DenoiseWorkload:
    """Token embeddings for graph-based context denoising (Sec. 2.1, Eq. 3).

    B contexts of up to n tokens (lengths uniform in [n_min, n]) with
    hidden size H.  Token i links to token i-1 with probability p_link:
    e_i = 0.6 e_{i-1} + 0.8 z_i, else e_i = z_i, z ~ N(0, I).  Linked runs
    stand in for coherent phrases (neighbour cosine about 0.6, 0.36, ...),
    unlinked tokens for isolated ones (cosine about N(0, 1/H)); p_link is
    set so that about 14% of the tokens survive tau = 0.05 with g = 3 and
    the keep-every-16 floor, the retention the paper reports.
    """

    name: str
    B: int
    n: int
    H: int
    dtype: str
    seed: int
    n_min: int = 0
    p_link: float = 0.02
    g: int = 3
    tau: float = 0.05
    keep_min_every: int = 16
    chunk_tokens: int = 256

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def replace(self, **kw) -> "DenoiseWorkload":
        return dataclasses.replace(self, **kw)


DENOISE_WORKLOADS: Dict[str, DenoiseWorkload] = {
    # GPT2-Large-sized encoder inputs at the paper's maximum input length.
    "denoise_gpt2l_batch64": DenoiseWorkload("denoise_gpt2l_batch64", B=64, n=3072, H=1280, dtype="bf16",
                                             seed=707, n_min=1024),
}


def denoise_tokens(w: DenoiseWorkload) -> np.ndarray:
    """Context lengths [B] int32."""
    if w.n_min >= w.n:
        return np.full(w.B, w.n, np.int32)
    return _rng(w.seed, "ragged", 1).integers(w.n_min, w.n + 1, size=w.B).astype(np.int32)


def denoise_emb(w: DenoiseWorkload, b: Optional[int] = None) -> np.ndarray:
    """Embeddings [B][n][H] (or [n][H] for one context): fp32, or bf16 bits."""
    if b is None:
        return np.stack([denoise_emb(w, i) for i in range(w.B)])
    r = _rng(w.seed, "emb", b)
    z = r.standard_normal(size=(w.n, w.H), dtype=np.float32)
    link = r.random(w.n) < w.p_link
    e = np.empty_like(z)
    e[0] = z[0]
    for i in range(1, w.n):
        e[i] = np.float32(0.6) * e[i - 1] + np.float32(0.8) * z[i] if link[i] else z[i]
    return f32_to_bf16_bits(e) if w.dtype == "bf16" else e


# ----------------------------------------------------------- MemoryBridge

@dataclasses.dataclass(frozen=True)
class BridgeWorkload:
    """MemoryBridge inputs (Sec. 2.3): M CME vectors of the encoder width Hc
    projected through hidden width F to the decoder width Hd.  Weights are
    nn.Linear-scaled draws (N(0, 1/fan_in)), biases N(0, 0.02^2), LayerNorm
    gamma 1 + N(0, 0.1^2) and beta N(0, 0.1^2), all rounded to bf16 where
    the kernel reads bf16; nu = s * nu_bar."""

    name: str
    M: int
    Hc: int
    F: int
    Hd: int
    seed: int
    nu: float = 1.0
    eps: float = 1e-5

    def replace(self, **kw) -> "BridgeWorkload":
        return dataclasses.replace(self, **kw)


BRIDGE_WORKLOADS: Dict[str, BridgeWorkload] = {
    # 64 GPT2-Large contexts of 3072 tokens: 12 chunks of 256 tokens at ratio 4
    # -> 64 CMEs per chunk, 768 per context; projected into Llama-3-8B's width.
    "bridge_gpt2l_llama3_batch64": BridgeWorkload("bridge_gpt2l_llama3_batch64", M=64 * 768, Hc=1280, F=4096,
                                                  Hd=4096, seed=808),
}


def bridge_params(w: BridgeWorkload) -> Dict[str, np.ndarray]:
    """Weights: w1 [F][Hc], w2 [Hd][F] (bf16 bits), b1 [F], b2, gamma, beta [Hd] (fp32)."""
    return {
        "w1": f32_to_bf16_bits(normal_f32(w.seed, "cme_k", (1,), (w.F, w.Hc), 1.0 / math.sqrt(w.Hc))),
        "w2": f32_to_bf16_bits(normal_f32(w.seed, "cme_v", (1,), (w.Hd, w.F), 1.0 / math.sqrt(w.F))),
        "b1": normal_f32(w.seed, "cme_k", (2,), (w.F,), 0.02),
        "b2": normal_f32(w.seed, "cme_v", (2,), (w.Hd,), 0.02),
        "gamma": (1.0 + normal_f32(w.seed, "chan", (1,), (w.Hd,), 0.1)).astype(np.float32),
        "beta": normal_f32(w.seed, "chan", (2,), (w.Hd,), 0.1),
    }


def bridge_h(w: BridgeWorkload, rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """CME vectors [M][Hc] (bf16 bits), N(0, 1), drawn in blocks of 1024 rows
    so that any row can be regenerated alone (rows=None: all)."""
    blk = 1024
    if rows is None:
        out = np.empty((w.M, w.Hc), np.uint16)
        for b0 in range(0, w.M, blk):
            n = min(blk, w.M - b0)
            out[b0:b0 + n] = f32_to_bf16_bits(normal_f32(w.seed, "emb", (b0 // blk,), (blk, w.Hc))[:n])
        return out
    out = np.empty((len(rows), w.Hc), np.uint16)
    for i, r in enumerate(rows):
        out[i] = f32_to_bf16_bits(normal_f32(w.seed, "emb", (r // blk,), (blk, w.Hc))[r % blk])
    return out
