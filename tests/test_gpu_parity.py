"""HIP path vs the CPU oracle, through the C ABI, on identical input bits.

Selection: index sets bit-exact.  Attention: max-abs 1e-5 (fp32 K/V) or
2e-3 (bf16 K/V) against the fp64 oracle.  Ring state: bit-exact."""
import math

import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, max_abs, say, to_dev, to_host, tol_for
from tests.inputs import accepted_attempts

pytestmark = pytest.mark.gpu


def _bf16(x):
    return wl.f32_to_bf16_bits(x)


# ------------------------------------------------------------------ select

def _check_select(orc, keys, qv, k, what):
    say(f"select {what}: B={keys.shape[0]} N={keys.shape[1]} D={keys.shape[2]} k={k}")
    ref_idx, ref_s, _ = orc.select(keys, qv, k)
    scores = torch.empty(keys.shape[:2], dtype=torch.float32, device=DEV)
    idx = cmc.cmc_select_cmes(to_dev(keys), to_dev(qv), k, scores_out=scores)
    torch.cuda.synchronize()
    got = to_host(idx)
    assert (got == ref_idx).all(), f"{what}: index sets differ"
    assert max_abs(to_host(scores), ref_s) < 1e-6
    # the workspace variant (scores not returned) gives the same indices
    idx2 = cmc.cmc_select_cmes(to_dev(keys), to_dev(qv), k)
    torch.cuda.synchronize()
    assert (to_host(idx2) == got).all()


def test_select_tiny(orc):
    w = wl.get("tiny_fp32")
    att = accepted_attempts(w, orc)
    _check_select(orc, wl.sel_keys(w), wl.q_vecs(w, att), w.k, "tiny")


def _separated(B, N, D, seed, dup_every=0):
    """Keys whose cosine scores are distinct and well separated (in fp32),
    with optional exact duplicates that tie exactly."""
    rng = np.random.default_rng(seed)
    keys = rng.standard_normal((B, N, D)).astype(np.float32) * np.float32(1e-3)
    qv = np.zeros((B, D), np.float32)
    qv[:, 0] = 1.0
    for b in range(B):
        a = (rng.permutation(N).astype(np.float64) / max(N, 1) * 10.0 - 5.0).astype(np.float32)
        keys[b, :, 0] = a
        keys[b, :, 1] = 1.0
        keys[b, :, 2:] = 0.0
        if dup_every:
            for j in range(dup_every, N, dup_every):
                keys[b, j] = keys[b, j - dup_every // 2]
    return keys, qv


@pytest.mark.parametrize("B,N,D,k", [
    (1, 1, 4, 1), (1, 7, 8, 0), (1, 7, 8, 7), (3, 33, 12, 5), (2, 1000, 64, 999),
    (4, 4096, 16, 512), (1, 32768, 8, 1024), (2, 32768, 8, 32768), (5, 2047, 260, 1),
    (65535, 6, 8, 2),  # the largest batch the host accepts (one grid row per sequence)
    # the top-k keeps ceil(N / 1024) keys per thread rounded up to a power of two:
    # the first size of each instantiation (1, 2, 4, 8, 16, 32 keys per thread)
    (2, 1024, 8, 100), (2, 1025, 8, 100), (2, 2049, 8, 300), (2, 4097, 16, 300), (2, 8193, 8, 2000),
    (1, 16385, 8, 64),
])
def test_select_sizes(orc, B, N, D, k):
    keys, qv = _separated(B, N, D, seed=N + k)
    _check_select(orc, keys, qv, k, f"sizes")


@pytest.mark.parametrize("seed", range(12))
def test_select_random_configs(orc, seed):
    """Seeded random batch, pool size, key width and k (well-separated scores,
    some with exact duplicate rows)."""
    r = np.random.default_rng(4000 + seed)
    B, N = int(r.integers(1, 9)), int(r.integers(1, 20000))
    D, k = 4 * int(r.integers(1, 80)), int(r.integers(0, N + 1))
    keys, qv = _separated(B, N, D, seed=5000 + seed, dup_every=int(r.choice([0, 0, 6])))
    _check_select(orc, keys, qv, k, f"random {seed}")


@pytest.mark.parametrize("N,k", [(64, 16), (1000, 100), (20000, 700)])
def test_select_exact_ties(orc, N, k):
    keys, qv = _separated(2, N, 8, seed=7, dup_every=4)
    _check_select(orc, keys, qv, k, "ties")


@pytest.mark.parametrize("B,N,D,k,dup", [
    (1, 7, 8, 3, 0), (3, 33, 16, 5, 0), (4, 4096, 64, 512, 6), (1, 32768, 8, 1024, 0), (2, 2047, 264, 1, 4),
    (3, 30001, 64, 700, 5),  # >= 65536 rows: the large-batch launch (four rows per wave), ragged last block
])
def test_select_bf16_keys(orc, B, N, D, k, dup):
    """bf16 selection keys (key_dtype = CMC_BF16) against the oracle on the
    same bits.  Rounding the separated keys to bf16 merges close ones into
    exact duplicates, which tie exactly on both sides (lower index wins)."""
    keys, qv = _separated(B, N, D, seed=N + k + 1, dup_every=dup)
    kb = _bf16(keys)
    say(f"select bf16 keys: B={B} N={N} D={D} k={k}")
    ref_idx, ref_s, _ = orc.select(kb, qv, k)
    scores = torch.empty((B, N), dtype=torch.float32, device=DEV)
    idx = cmc.cmc_select_cmes(to_dev(kb), to_dev(qv), k, scores_out=scores)
    torch.cuda.synchronize()
    assert (to_host(idx) == ref_idx).all(), "index sets differ"
    assert max_abs(to_host(scores), ref_s) < 1e-6


def _accepted_bf16(w, orc, keys_bf16):
    """Per sequence, the first question draw whose top-k gap on the bf16
    keys clears the workload's rule."""
    att = []
    for b in range(w.B):
        a = 0
        while orc.select(keys_bf16[b:b + 1], wl.q_vec(w, b, a)[None], w.k)[2][0] < w.gap_min:
            a += 1
            assert a < 2000
        att.append(a)
    return att


def test_select_bf16_keys_llama_layer_full_size(orc):
    """The Llama-layer selection (N = 2048, D = 4096) with its keys rounded
    to bf16, which halves the bytes the scoring pass reads."""
    w = wl.get("llama3_8b_layer")
    kb = _bf16(wl.sel_keys(w))
    qv = wl.q_vecs(w, _accepted_bf16(w, orc, kb))
    say("select bf16 keys: llama3_8b_layer")
    ref_idx, _, gap = orc.select(kb, qv, w.k)
    assert (gap >= w.gap_min).all()
    idx = cmc.cmc_select_cmes(to_dev(kb), to_dev(qv), w.k)
    torch.cuda.synchronize()
    assert (to_host(idx) == ref_idx).all()


def test_select_zero_rows_and_question(orc):
    keys, qv = _separated(2, 100, 8, seed=3)
    keys[0, 10] = 0.0
    keys[0, 50] = 0.0
    qv[1] = 0.0               # every score 0: the first k rows win
    _check_select(orc, keys, qv, 30, "zeros")


def test_select_llama_layer_full_size(orc):
    w = wl.get("llama3_8b_layer")
    att = accepted_attempts(w, orc)
    _check_select(orc, wl.sel_keys(w), wl.q_vecs(w, att), w.k, "llama3_8b_layer")


# ------------------------------------------------------------------ append

@pytest.mark.parametrize("dtype,Dh,W,T", [("f32", 64, 8, 1), ("bf16", 128, 5, 2), ("bf16", 256, 3, 3),
                                          ("f32", 128, 1, 1)])
def test_window_append_ring(orc, dtype, Dh, W, T):
    rng = np.random.default_rng(W * 10 + T)
    B, Hkv = 3, 2
    mk = (lambda *s: _bf16(rng.standard_normal(s).astype(np.float32))) if dtype == "bf16" else \
        (lambda *s: rng.standard_normal(s).astype(np.float32))
    wk, wv = mk(B, Hkv, W, Dh), mk(B, Hkv, W, Dh)
    cnt = np.array([0, min(2, W - 1), W + 3], np.int32)
    dk, dv, dc = to_dev(wk), to_dev(wv), to_dev(cnt)
    for step in range(2 * W + 1):
        say(f"append {dtype} Dh={Dh} W={W} T={T} step {step}")
        nk, nv = mk(B, Hkv, T, Dh), mk(B, Hkv, T, Dh)
        orc.window_append(wk, wv, cnt, nk, nv)
        cmc.cmc_window_append(dk, dv, dc, to_dev(nk), to_dev(nv))
    torch.cuda.synchronize()
    assert (to_host(dk) == wk).all() and (to_host(dv) == wv).all()
    assert (to_host(dc) == cnt).all()


# ------------------------------------------------------------------ gather

@pytest.mark.parametrize("dtype,Dh,idx_mode,k_len", [
    ("bf16", 128, "idx", None), ("f32", 64, "idx", [5, 0, 9]), ("bf16", 256, "none", None),
    ("bf16", 128, "clamp", [9, 9, 3]),
])
def test_gather_tier1(dtype, Dh, idx_mode, k_len):
    """Bit-exact copy of the selected rows (numpy indexing as the
    reference); rows past k_b stay untouched; out-of-range entries clamp."""
    rng = np.random.default_rng(Dh + len(idx_mode))
    B, Hkv, N, k, stride = 3, 2, 40, 9, 12
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    cv = _bf16 if dtype == "bf16" else (lambda x: x)
    pk, pv = cv(f(B, Hkv, N, Dh)), cv(f(B, Hkv, N, Dh))
    idx = rng.integers(0, N, size=(B, stride)).astype(np.int32)
    if idx_mode == "clamp":
        idx[:, 0], idx[:, 1] = -7, N + 100
    say(f"gather {dtype} Dh={Dh} {idx_mode} k_len={k_len}")
    fill = np.full((B, Hkv, k, Dh), 7, dtype=pk.dtype)
    ok, ov = to_dev(fill), to_dev(fill)
    cmc.cmc_gather_tier1(to_dev(pk), to_dev(pv), None if idx_mode == "none" else to_dev(idx), k,
                         k_len=None if k_len is None else to_dev(np.array(k_len, np.int32)), out_k=ok, out_v=ov)
    torch.cuda.synchronize()
    src = np.arange(k)[None].repeat(B, 0) if idx_mode == "none" else np.clip(idx[:, :k], 0, N - 1)
    kb = [k] * B if k_len is None else [min(max(x, 0), k) for x in k_len]
    gk, gv = to_host(ok), to_host(ov)
    for b in range(B):
        assert (gk[b, :, :kb[b]] == pk[b][:, src[b, :kb[b]]]).all() and (gv[b, :, :kb[b]] == pv[b][:, src[b, :kb[b]]]).all()
        assert (gk[b, :, kb[b]:] == 7).all() and (gv[b, :, kb[b]:] == 7).all()


# ------------------------------------------------------------------ decode

def _logit_bound_tol(q, keys_f64, scale, vmax, Dh):
    """Bound on the fp32 output error when the logits are large: each fp32
    logit is off by at most gamma_Dh * scale * sum_d |q_d k_d| (gamma_n =
    n u / (1 - n u), u = 2^-24), which moves the softmax weights by at most
    that amount relatively, so |out error| <= 2 * max dz * max |v| (+ the
    fp32 rounding of the weighted sum itself)."""
    u = 2.0 ** -24
    gamma = Dh * u / (1 - Dh * u)
    dz = gamma * abs(scale) * float(np.max(np.abs(q.astype(np.float64)) @ np.abs(keys_f64).T))
    return 2.0 * dz * vmax + 1e-5


def _same_bits(a, b) -> bool:
    """Bitwise equality (NaN patterns included)."""
    a, b = np.ascontiguousarray(a), np.ascontiguousarray(b)
    u = {2: np.uint16, 4: np.uint32}[a.dtype.itemsize]
    return a.shape == b.shape and a.dtype == b.dtype and bool((a.view(u) == b.view(u)).all())


def _nan_like(x):
    """A NaN of x's element type (bf16 bits are uint16)."""
    return np.uint16(0x7FC0) if x.dtype == np.uint16 else np.float32("nan")


def _decode_case(orc, B, Hq, Hkv, Dh, N, k, W, fill, dtype, seed, steps=3, idx_none=False, scale=None,
                 kv_std=1.0, derived_tol=False, fused=False, t_new=1, unused_nan=False):
    rng = np.random.default_rng(seed)
    f = lambda *s: (rng.standard_normal(s) * kv_std).astype(np.float32)
    cv = _bf16 if dtype == "bf16" else (lambda x: x)
    pk, pv = cv(f(B, Hkv, N, Dh)), cv(f(B, Hkv, N, Dh))
    if idx_none:
        idx = None
    else:
        idx = np.stack([np.sort(rng.choice(N, size=k, replace=False)) for _ in range(B)]).astype(np.int32)
    wk = np.zeros((B, Hkv, W, Dh), np.float32)
    wv = np.zeros((B, Hkv, W, Dh), np.float32)
    if fill:
        wk[:, :, :fill] = f(B, Hkv, fill, Dh)
        wv[:, :, :fill] = f(B, Hkv, fill, Dh)
    wk, wv = cv(wk), cv(wv)
    if unused_nan:  # slots never filled hold NaN: they must not reach the output
        wk[:, :, fill:] = _nan_like(wk)
        wv[:, :, fill:] = _nan_like(wv)
    cnt = np.full((B,), fill, np.int32)
    scale = 1.0 / math.sqrt(Dh) if scale is None else scale
    d = dict(pk=to_dev(pk), pv=to_dev(pv), idx=None if idx is None else to_dev(idx),
             wk=to_dev(wk) if W else None, wv=to_dev(wv) if W else None, wc=to_dev(cnt) if W else None)
    ws = cmc.decode_workspace(B, Hq, Hkv, Dh, k, W, DEV)
    worst = 0.0
    for step in range(steps):
        say(f"decode {dtype} B={B} Hq={Hq} Hkv={Hkv} Dh={Dh} N={N} k={k} W={W} fill={fill} "
            f"fused={fused} t_new={t_new} step={step}")
        nk = nv = None
        if W:
            nk, nv = cv(f(B, Hkv, t_new, Dh)), cv(f(B, Hkv, t_new, Dh))
            orc.window_append(wk, wv, cnt, nk, nv)
            if not fused:
                cmc.cmc_window_append(d["wk"], d["wv"], d["wc"], to_dev(nk), to_dev(nv))
        q = f(B, Hq, Dh)
        ref = orc.two_tier_decode(q, pk, pv, idx, k, wk, wv, cnt, W, scale)
        if fused:
            out = cmc.cmc_decode_step(to_dev(q), d["pk"], d["pv"], d["idx"], k, d["wk"], d["wv"], d["wc"],
                                      None if nk is None else to_dev(nk), None if nv is None else to_dev(nv),
                                      scale, W=W, workspace=ws)
        else:
            out = cmc.cmc_two_tier_decode(to_dev(q), d["pk"], d["pv"], d["idx"], k, d["wk"], d["wv"], d["wc"],
                                          scale, W=W, workspace=ws)
        torch.cuda.synchronize()
        assert not ws[:4 * (B + B * Hkv)].any(), "arrival counters must return to zero"
        if W:
            assert _same_bits(to_host(d["wk"]), wk) and _same_bits(to_host(d["wv"]), wv), "ring contents"
            assert (to_host(d["wc"]) == cnt).all(), "ring count"
        err = max_abs(to_host(out), ref)
        worst = max(worst, err)
        tol = tol_for(dtype)
        if derived_tol:
            allk = np.concatenate([pk.reshape(-1, Dh), wk.reshape(-1, Dh)]).astype(np.float64)
            vmax = float(max(np.abs(pv).max(), np.abs(wv).max()))
            tol = max(tol, _logit_bound_tol(q.reshape(-1, Dh), allk, scale, vmax, Dh))
        assert np.isfinite(to_host(out)).all()
        assert err <= tol, f"step {step}: max abs err {err:.3e} > {tol:.3e}"
    return worst


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Dh", [64, 128, 256])
@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_decode_head_shapes(orc, dtype, Dh, G):
    _decode_case(orc, B=2, Hq=2 * G, Hkv=2, Dh=Dh, N=97, k=37, W=19, fill=11, dtype=dtype, seed=Dh + G)


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("k,W,fill", [(1, 0, 0), (0, 5, 2), (0, 64, 64), (300, 0, 0), (5, 1, 0),
                                      (2000, 3000, 2999), (513, 700, 0)])
def test_decode_key_counts(orc, k, W, fill, fused):
    _decode_case(orc, B=2, Hq=8, Hkv=2, Dh=128, N=max(k, 1) + 50, k=k, W=W, fill=fill, dtype="bf16",
                 seed=k * 7 + W, fused=fused)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Dh,G", [(64, 4), (128, 4), (128, 1), (256, 1), (128, 8), (64, 2)])
@pytest.mark.parametrize("t_new,W,fill", [(1, 7, 0), (2, 9, 9), (3, 300, 100), (5, 5, 3)])
def test_decode_step_fused(orc, dtype, Dh, G, t_new, W, fill):
    """Append fused into the decode launch equals append then decode, and
    the ring contents/count match the oracle's after every step."""
    _decode_case(orc, B=3, Hq=2 * G, Hkv=2, Dh=Dh, N=300, k=120, W=W, fill=fill, dtype=dtype,
                 seed=Dh * G + t_new + W, steps=4, fused=True, t_new=t_new)


@pytest.mark.parametrize("B,Hkv,G,Dh,dtype,N,k,W,fill", [
    (48, 4, 4, 128, "bf16", 64, 37, 75, 75),      # 192 pairs: one 8-wave workgroup each
    (32, 8, 4, 128, "bf16", 400, 300, 500, 500),  # 256 pairs, several blocks per wave, ragged tail
    (32, 8, 4, 128, "bf16", 20, 0, 16, 3),        # 256 pairs, fewer keys than waves
    (64, 4, 8, 64, "bf16", 40, 20, 33, 10),       # VALU path (G = 8), ring not yet full
    (32, 8, 1, 256, "bf16", 100, 64, 128, 128),   # wide head, G = 1
    (32, 8, 2, 256, "bf16", 40, 30, 50, 50),      # wide head, G = 2: stays on 4 waves
    (40, 5, 2, 128, "f32", 50, 45, 60, 60),       # 200 pairs, fp32
    (64, 4, 1, 64, "f32", 30, 10, 0, 0),          # 256 pairs, no window
])
def test_decode_wide_workgroups(orc, B, Hkv, G, Dh, dtype, N, k, W, fill):
    """Batches with 192..256 (sequence, kv head) pairs run one 8-wave
    workgroup per pair; results match the oracle like every other plan."""
    _decode_case(orc, B=B, Hq=G * Hkv, Hkv=Hkv, Dh=Dh, N=N, k=k, W=W, fill=fill, dtype=dtype,
                 seed=B * Hkv + G + Dh, steps=3, fused=W > 0)


def _random_decode_config(seed):
    """A seeded random decode configuration within the ABI's limits."""
    r = np.random.default_rng(seed)
    Dh = int(r.choice([64, 128, 256]))
    G = int(r.choice([1, 2, 4, 8]))
    Hkv = int(r.choice([1, 2, 3, 4]))
    B = int(r.integers(1, 7))
    N = int(r.integers(1, 700))
    k = int(r.integers(0, N + 1))
    W = int(r.choice([0, int(r.integers(1, 9)), int(r.integers(9, 400))]))
    if k + W == 0:
        k = 1
    fill = int(r.integers(0, W + 1)) if W else 0
    return dict(B=B, Hq=G * Hkv, Hkv=Hkv, Dh=Dh, N=N, k=k, W=W, fill=fill,
                dtype=str(r.choice(["f32", "bf16"])), fused=bool(W and r.integers(0, 2)),
                t_new=int(r.integers(1, max(2, min(W, 6)))) if W else 1, idx_none=bool(r.integers(0, 4) == 0))


@pytest.mark.parametrize("seed", range(24))
def test_decode_random_configs(orc, seed):
    """Seeded random shapes (head size, group size, batch, pool, k, ring size and
    fill, dtype, fused append with several rows, identity index) against the
    oracle, two steps each."""
    c = _random_decode_config(1000 + seed)
    if c["idx_none"]:
        c["N"] = max(c["N"], c["k"])
    t_new = c["t_new"] if c["fused"] else 1
    _decode_case(orc, c["B"], c["Hq"], c["Hkv"], c["Dh"], c["N"], c["k"], c["W"], c["fill"], c["dtype"],
                 seed=2000 + seed, steps=2, idx_none=c["idx_none"], fused=c["fused"], t_new=t_new)


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("B,Hkv,G,Dh,dtype,N,k,W,fill", [
    (1, 8, 4, 128, "bf16", 300, 256, 512, 100),   # Llama-layer shape, split plan, ring a fifth full
    (1, 8, 4, 128, "bf16", 300, 0, 512, 1),       # one filled slot
    (2, 2, 1, 64, "bf16", 90, 40, 700, 333),      # G = 1, many splits
    (32, 8, 4, 128, "bf16", 64, 32, 300, 45),     # 256 pairs: one 8-wave workgroup each (S = 1)
    (3, 2, 2, 256, "bf16", 50, 20, 200, 17),      # wide head, single-buffered loop
    (2, 2, 8, 128, "bf16", 50, 20, 200, 17),      # G = 8: VALU path
    (2, 2, 4, 128, "f32", 50, 20, 200, 17),       # fp32: VALU path
])
def test_decode_unfilled_slots_hold_nan(orc, fused, B, Hkv, G, Dh, dtype, N, k, W, fill):
    """Ring slots that were never filled may hold anything, NaN included:
    the output must equal the oracle's (which never reads them) and stay
    finite, with a ring that is not full and (where the plan splits) splits
    that start past the filled slots."""
    _decode_case(orc, B=B, Hq=G * Hkv, Hkv=Hkv, Dh=Dh, N=N, k=k, W=W, fill=fill, dtype=dtype,
                 seed=B + W + fill + G, steps=3, fused=fused, unused_nan=True)


def test_decode_empty_window_zero_output(orc):
    """k = 0 and an empty ring: zeros, like the oracle."""
    _decode_case(orc, B=1, Hq=4, Hkv=4, Dh=64, N=10, k=0, W=4, fill=0, dtype="f32", seed=1, steps=1)


def test_decode_identity_index(orc):
    _decode_case(orc, B=3, Hq=8, Hkv=8, Dh=64, N=40, k=40, W=0, fill=0, dtype="f32", seed=5, idx_none=True)


def test_decode_large_logits(orc):
    """Logits around +-3e2: online max subtraction must keep it finite; the
    tolerance is the fp32 logit-error bound, since 1e-5 absolute is below
    what any fp32 evaluation of logits this large can guarantee."""
    _decode_case(orc, B=2, Hq=4, Hkv=2, Dh=128, N=60, k=30, W=16, fill=16, dtype="f32", seed=9,
                 scale=1.0, kv_std=3.0, derived_tol=True)


def test_decode_bit_identical_runs():
    rng = np.random.default_rng(0)
    B, Hq, Hkv, Dh, N, k, W = 4, 32, 8, 128, 512, 128, 256
    q = to_dev(rng.standard_normal((B, Hq, Dh)).astype(np.float32))
    pk = to_dev(_bf16(rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)))
    pv = to_dev(_bf16(rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)))
    wk = to_dev(_bf16(rng.standard_normal((B, Hkv, W, Dh)).astype(np.float32)))
    wv = to_dev(_bf16(rng.standard_normal((B, Hkv, W, Dh)).astype(np.float32)))
    wc = to_dev(np.array([W, 7, 0, 1000], np.int32))
    idx = to_dev(np.sort(rng.choice(N, size=(B, k)), axis=1).astype(np.int32))
    say("decode bit-identical runs")
    a = cmc.cmc_two_tier_decode(q, pk, pv, idx, k, wk, wv, wc, 0.088)
    b = cmc.cmc_two_tier_decode(q, pk, pv, idx, k, wk, wv, wc, 0.088)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_tiny_workload_end_to_end(orc):
    """The tiny fp32 workload: select, then 16 steps of append + decode."""
    w = wl.get("tiny_fp32")
    att = accepted_attempts(w, orc)
    keys, qv = wl.sel_keys(w), wl.q_vecs(w, att)
    ref_idx, _, _ = orc.select(keys, qv, w.k)
    say("tiny e2e: select")
    idx = cmc.cmc_select_cmes(to_dev(keys), to_dev(qv), w.k)
    pk, pv = wl.pool_kv(w)
    wk, wv, cnt = wl.window_kv(w)
    d_pk, d_pv, d_wk, d_wv, d_wc = map(to_dev, (pk, pv, wk, wv, cnt))
    torch.cuda.synchronize()
    assert (to_host(idx) == ref_idx).all()
    for t in range(w.steps):
        say(f"tiny e2e: step {t}")
        nk, nv = wl.step_new_kv(w, t)
        q = wl.step_q(w, t)
        orc.window_append(wk, wv, cnt, nk, nv)
        ref = orc.two_tier_decode(q, pk, pv, ref_idx, w.k, wk, wv, cnt, w.W, w.scale)
        cmc.cmc_window_append(d_wk, d_wv, d_wc, to_dev(nk), to_dev(nv))
        out = cmc.cmc_two_tier_decode(to_dev(q), d_pk, d_pv, idx, w.k, d_wk, d_wv, d_wc, w.scale)
        torch.cuda.synchronize()
        assert max_abs(to_host(out), ref) <= 1e-5, t
    assert (to_host(d_wk) == wk).all() and (to_host(d_wc) == cnt).all()


@pytest.mark.timeout(300)
@pytest.mark.parametrize("B,Hq,Hkv,dtype", [(65535, 2, 1, "bf16"), (1, 65535, 65535, "f32")])
def test_decode_grid_limits(orc, B, Hq, Hkv, dtype):
    """The largest batch and the largest kv-head count the host accepts
    (65535 each: one grid dimension per sequence / kv head), fused append
    and decode, every output checked."""
    _decode_case(orc, B=B, Hq=Hq, Hkv=Hkv, Dh=64, N=3, k=2, W=3, fill=2, dtype=dtype, seed=B + Hkv, steps=2,
                 fused=True)
