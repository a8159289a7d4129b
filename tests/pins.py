"""Pins for the CPU oracle: checks against things other than the oracle.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises AssertionError when
the oracle disagrees with what the paper and the mathematics fix:
hand-derived closed forms (tests/golden/closed_forms.json), exact-rational
brute force, list-history attention without ring arithmetic, a library
special case (fp64 SDPA / argsort), and invariants.  They are plain
functions so that ``test_oracle_mutants`` can run them against deliberately
broken builds of the oracle and show that each plausible mistake fails at
least one of them.

Run as ``python -m tests.pins <liboracle.so>``: exit 0 iff every pin holds.
"""
from __future__ import annotations

import json
import math
import os
import sys

import numpy as np

from tests import brute

_GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "closed_forms.json")


def _golden():
    with open(_GOLDEN) as f:
        return json.load(f)


def _close(a, b, tol, what):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs err {err:.3e} > {tol:.1e}"


def _bf16(x):
    u = np.ascontiguousarray(x, np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> 16) & 1)) >> 16).astype(np.uint16)


# ------------------------------------------------------------ selection

def pin_golden_selection(orc):
    """Closed-form cosine scores and top-k sets (incl. an exact tie)."""
    for case in _golden()["selection"]:
        keys = np.array([case["sel_keys"]], np.float32)
        q = np.array([case["q_vec"]], np.float32)
        for c in case["cases"]:
            idx, scores, _ = orc.select(keys, q, c["k"])
            assert idx[0].tolist() == c["idx"], (case["derivation"], c, idx)
            _close(scores[0], case["scores"], 1e-15, "golden scores")


def pin_select_exact_rational(orc):
    """Random small problems, with duplicated rows creating exact ties."""
    rng = np.random.default_rng(7)
    for trial in range(24):
        N = int(rng.integers(1, 24))
        D = int(rng.integers(1, 12))
        keys = rng.standard_normal((N, D)).astype(np.float32)
        if N >= 4 and trial % 2 == 0:
            keys[N - 1] = keys[1]          # exact tie, later index must lose
            keys[N - 2] = keys[0] * 4      # positive rescale: same score, exact
        q = rng.standard_normal(D).astype(np.float32)
        for k in sorted({0, 1, N // 2, max(0, N - 1), N}):
            idx, _, _ = orc.select(keys[None], q[None], k)
            assert idx[0].tolist() == brute.exact_topk(keys, q, k), (trial, N, D, k)


def pin_select_library(orc):
    """Scores match fp64 torch cosine_similarity; the set matches a stable
    numpy argsort of them (a library special case of the definition)."""
    import torch
    rng = np.random.default_rng(11)
    B, N, D, k = 3, 200, 64, 37
    keys = rng.standard_normal((B, N, D)).astype(np.float32)
    q = rng.standard_normal((B, D)).astype(np.float32)
    idx, scores, gap = orc.select(keys, q, k)
    ref = torch.nn.functional.cosine_similarity(
        torch.from_numpy(keys).double(), torch.from_numpy(q).double()[:, None, :], dim=-1).numpy()
    _close(scores, ref, 1e-13, "cosine vs torch")
    for b in range(B):
        order = np.argsort(-ref[b], kind="stable")
        assert idx[b].tolist() == sorted(order[:k].tolist())
        s = np.sort(ref[b])[::-1]
        assert abs(gap[b] - (s[k - 1] - s[k]) / abs(s[k - 1])) < 1e-9


def pin_select_rescale_invariance(orc):
    """Scaling one row or the question by a positive power of two leaves
    the ranking (and every score) unchanged: catches a missing row norm."""
    rng = np.random.default_rng(5)
    B, N, D, k = 2, 40, 16, 10
    keys = rng.standard_normal((B, N, D)).astype(np.float32)
    q = rng.standard_normal((B, D)).astype(np.float32)
    idx, s0, _ = orc.select(keys, q, k)
    k2 = keys.copy()
    for b in range(B):
        out = [j for j in range(N) if j not in set(idx[b].tolist())]
        k2[b, out[0]] *= np.float32(1024.0)
        k2[b, idx[b][0]] *= np.float32(1.0 / 1024.0)
    idx2, s2, _ = orc.select(k2, q * np.float32(64.0), k)
    assert (idx == idx2).all()
    _close(s0, s2, 0.0, "rescaled scores")


def pin_select_zero_norm(orc):
    """A zero row and a zero question score 0 (cosine denominator clamp);
    with a zero question every score ties and the first k rows win."""
    keys = np.array([[[0, 0, 0], [1, 2, 3], [-1, 0, -1], [0, 0, 0]]], np.float32)
    q = np.array([[0, 0, 1]], np.float32)
    idx, s, _ = orc.select(keys, q, 3)
    assert idx[0].tolist() == [0, 1, 3], idx
    assert s[0, 0] == 0.0 and s[0, 3] == 0.0
    idx, s, _ = orc.select(keys, np.zeros((1, 3), np.float32), 2)
    assert idx[0].tolist() == [0, 1] and not s.any()


# --------------------------------------------------------------- window

def pin_golden_window_start(orc):
    for c in _golden()["window_start"]["cases"]:
        assert orc.window_start(c["ctx_len"], c["W"], c["alpha"]) == c["start"], c


def pin_golden_ring(orc):
    g = _golden()["ring"]
    W, T = g["W"], g["tokens"]
    wk = np.zeros((1, 1, W, 1), np.float32)
    wv = np.zeros((1, 1, W, 1), np.float32)
    cnt = np.zeros((1,), np.int32)
    for t in range(T):
        tok = np.full((1, 1, 1, 1), t, np.float32)
        orc.window_append(wk, wv, cnt, tok, -tok)
    assert wk[0, 0, :, 0].tolist() == g["slots_after"]
    assert (-wv[0, 0, :, 0]).tolist() == g["slots_after"]
    assert int(cnt[0]) == g["count_after"]


def pin_ring_multiset(orc):
    """After any append schedule the ring holds exactly the last
    min(W, count) tokens, and multi-row appends equal single-row ones."""
    rng = np.random.default_rng(3)
    for W in (1, 2, 5, 8):
        B, H, Dh = 2, 2, 3
        wk = np.zeros((B, H, W, Dh), np.float32)
        wv = np.zeros_like(wk)
        cnt = np.zeros((B,), np.int32)
        hist = []
        for step in range(13):
            T = int(rng.integers(1, W + 1))
            nk = rng.standard_normal((B, H, T, Dh)).astype(np.float32)
            orc.window_append(wk, wv, cnt, nk, nk * 2)
            hist.extend(nk[:, :, t] for t in range(T))
            last = hist[-W:]
            for b in range(B):
                for h in range(H):
                    got = sorted(map(tuple, wk[b, h, :min(W, len(hist))].tolist()))
                    want = sorted(tuple(x[b, h].tolist()) for x in last)
                    assert got == want, (W, step)
            assert (cnt == len(hist)).all()
            _close(wv, 2 * wk, 0.0, "values follow keys")


# ------------------------------------------------------------- attention

def pin_golden_attention(orc):
    for c in _golden()["attention"]:
        W = c.get("W", 2)
        q = np.array(c["q"], np.float32)
        pk = np.array(c["pool_k"], np.float32)
        pv = np.array(c["pool_v"], np.float32)
        idx = np.array(c["idx"], np.int32)
        wk = None if c["win_k"] is None else np.array(c["win_k"], np.float32)
        wv = None if c["win_v"] is None else np.array(c["win_v"], np.float32)
        wc = np.array(c["win_count"], np.int32)
        out = orc.two_tier_decode(q, pk, pv, idx, idx.shape[1], wk, wv, wc, W, c["scale"])
        _close(out, c["out"], c["tol"], c["derivation"])


def _history_run(orc, B, Hq, Hkv, Dh, N, k, W, fill, steps, t_new, dtype, seed):
    """Drive the oracle's append+decode and compare every step with the
    list-history brute force."""
    rng = np.random.default_rng(seed)
    f32 = lambda *s: rng.standard_normal(s).astype(np.float32)
    pk, pv = f32(B, Hkv, N, Dh), f32(B, Hkv, N, Dh)
    idx = np.stack([np.sort(rng.choice(N, size=k, replace=False)) for _ in range(B)]).astype(np.int32)
    wk = np.zeros((B, Hkv, max(W, 1), Dh), np.float32)[:, :, :W].copy()
    wv = wk.copy()
    wk[:, :, :fill] = f32(B, Hkv, fill, Dh)
    wv[:, :, :fill] = f32(B, Hkv, fill, Dh)
    cnt = np.full((B,), fill, np.int32)
    hist_k = [[[wk[b, h, s] for s in range(fill)] for h in range(Hkv)] for b in range(B)]
    hist_v = [[[wv[b, h, s] for s in range(fill)] for h in range(Hkv)] for b in range(B)]
    conv = (lambda x: x) if dtype == "f32" else _bf16
    widen = (lambda x: x) if dtype == "f32" else (
        lambda h: (h.astype(np.uint32) << 16).view(np.float32))
    pk_d, pv_d = conv(pk), conv(pv)
    wk_d, wv_d = conv(wk), conv(wv)
    pk_f, pv_f = widen(pk_d), widen(pv_d)
    if dtype != "f32":
        hist_k = [[[widen(conv(r)) for r in hh] for hh in hb] for hb in hist_k]
        hist_v = [[[widen(conv(r)) for r in hh] for hh in hb] for hb in hist_v]
    scale = 1.0 / math.sqrt(Dh)
    for step in range(steps):
        nk, nv = conv(f32(B, Hkv, t_new, Dh)), conv(f32(B, Hkv, t_new, Dh))
        if W > 0:
            orc.window_append(wk_d, wv_d, cnt, nk, nv)
        for b in range(B):
            for h in range(Hkv):
                for t in range(t_new):
                    hist_k[b][h].append(widen(nk[b, h, t]))
                    hist_v[b][h].append(widen(nv[b, h, t]))
        q = f32(B, Hq, Dh)
        out = orc.two_tier_decode(q, pk_d, pv_d, idx, k, wk_d, wv_d, cnt, W, scale)
        for b in range(B):
            ref = brute.history_attention(q[b], pk_f[b], pv_f[b], idx[b].tolist(),
                                          hist_k[b], hist_v[b], W, scale)
            _close(out[b], ref, 1e-12, f"history step {step} b {b}")


def pin_decode_history(orc):
    """Append+decode over several steps vs list-history attention: partial
    fill, wrap-around, GQA, multi-row appends, bf16 bits."""
    _history_run(orc, B=2, Hq=4, Hkv=2, Dh=8, N=12, k=5, W=4, fill=1, steps=7, t_new=1,
                 dtype="f32", seed=1)
    _history_run(orc, B=1, Hq=6, Hkv=3, Dh=4, N=9, k=9, W=3, fill=0, steps=5, t_new=2,
                 dtype="bf16", seed=2)
    _history_run(orc, B=2, Hq=2, Hkv=2, Dh=5, N=7, k=0, W=5, fill=5, steps=4, t_new=1,
                 dtype="f32", seed=3)
    _history_run(orc, B=1, Hq=4, Hkv=1, Dh=6, N=10, k=4, W=0, fill=0, steps=2, t_new=1,
                 dtype="f32", seed=4)


def _sdpa(q, K, V, scale):
    """fp64 library attention; q [Hq][Dh], K/V [Hkv][L][Dh]."""
    import torch
    Hq = q.shape[0]
    G = Hq // K.shape[0]
    Kt = torch.from_numpy(np.repeat(K, G, axis=0)).double()
    Vt = torch.from_numpy(np.repeat(V, G, axis=0)).double()
    qt = torch.from_numpy(q).double()[:, None, :]
    o = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, scale=scale)
    return o[:, 0, :].numpy()


def pin_full_attention_library(orc):
    """I-1: k = N with W = 0 is full attention over every memory row;
    I-8: k = N with a ring that never wrapped is full attention over the
    memory rows followed by every token."""
    rng = np.random.default_rng(9)
    B, Hq, Hkv, Dh, N = 2, 8, 2, 16, 33
    q = rng.standard_normal((B, Hq, Dh)).astype(np.float32)
    pk = rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)
    pv = rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)
    out = orc.two_tier_decode(q, pk, pv, None, N, None, None, None, 0, 0.3)
    for b in range(B):
        _close(out[b], _sdpa(q[b], pk[b], pv[b], 0.3), 1e-12, "I-1")
    W, T = 20, 11
    wk = np.zeros((B, Hkv, W, Dh), np.float32)
    wv = np.zeros_like(wk)
    cnt = np.zeros((B,), np.int32)
    toks_k = rng.standard_normal((B, Hkv, T, Dh)).astype(np.float32)
    toks_v = rng.standard_normal((B, Hkv, T, Dh)).astype(np.float32)
    orc.window_append(wk, wv, cnt, toks_k, toks_v)
    ident = np.tile(np.arange(N, dtype=np.int32), (B, 1))
    out = orc.two_tier_decode(q, pk, pv, ident, N, wk, wv, cnt, W, 0.3)
    for b in range(B):
        K = np.concatenate([pk[b], toks_k[b]], axis=1)
        V = np.concatenate([pv[b], toks_v[b]], axis=1)
        _close(out[b], _sdpa(q[b], K, V, 0.3), 1e-12, "I-8")


def pin_identical_keys_mean(orc):
    """I-2: identical keys give the plain mean of the values."""
    rng = np.random.default_rng(4)
    B, Hq, Hkv, Dh, N, k, W = 1, 4, 2, 8, 10, 6, 5
    q = rng.standard_normal((B, Hq, Dh)).astype(np.float32)
    row = rng.standard_normal(Dh).astype(np.float32)
    pk = np.broadcast_to(row, (B, Hkv, N, Dh)).copy()
    pv = rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)
    wk = np.broadcast_to(row, (B, Hkv, W, Dh)).copy()
    wv = rng.standard_normal((B, Hkv, W, Dh)).astype(np.float32)
    cnt = np.array([3], np.int32)
    idx = np.array([[0, 2, 3, 5, 8, 9]], np.int32)
    out = orc.two_tier_decode(q, pk, pv, idx, k, wk, wv, cnt, W, 0.7)
    for h in range(Hq):
        kv = h // (Hq // Hkv)
        mean = np.concatenate([pv[0, kv, idx[0]], wv[0, kv, :3]]).astype(np.float64).mean(0)
        _close(out[0, h], mean, 1e-14, "I-2")


def pin_order_invariance(orc):
    """I-3: permuting the memory rows (selection keys and pool together)
    permutes the selected indices and leaves the output unchanged."""
    rng = np.random.default_rng(12)
    B, Hq, Hkv, Dh, N, D, k, W = 2, 4, 2, 8, 30, 12, 9, 6
    keys = rng.standard_normal((B, N, D)).astype(np.float32)
    qv = rng.standard_normal((B, D)).astype(np.float32)
    pk = rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)
    pv = rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)
    wk = rng.standard_normal((B, Hkv, W, Dh)).astype(np.float32)
    wv = rng.standard_normal((B, Hkv, W, Dh)).astype(np.float32)
    cnt = np.array([W, 2], np.int32)
    q = rng.standard_normal((B, Hq, Dh)).astype(np.float32)
    idx, _, _ = orc.select(keys, qv, k)
    out = orc.two_tier_decode(q, pk, pv, idx, k, wk, wv, cnt, W, 0.25)
    perm = rng.permutation(N)                  # new row perm[j] holds old row j
    keys2 = np.empty_like(keys)
    keys2[:, perm] = keys
    pk2 = np.empty_like(pk)
    pk2[:, :, perm] = pk
    pv2 = np.empty_like(pv)
    pv2[:, :, perm] = pv
    idx2, _, _ = orc.select(keys2, qv, k)
    for b in range(B):
        assert idx2[b].tolist() == sorted(perm[idx[b]].tolist())
    out2 = orc.two_tier_decode(q, pk2, pv2, idx2, k, wk, wv, cnt, W, 0.25)
    _close(out, out2, 1e-13, "I-3")


def pin_softmax_shift(orc):
    """I-5: adding one vector c to every key shifts each head's logits by a
    constant and leaves the output unchanged, even with logits near 1e3
    (dyadic values keep every sum exact)."""
    rng = np.random.default_rng(8)
    B, Hq, Hkv, Dh, N, W = 1, 2, 1, 4, 6, 4
    dy = lambda *s: (rng.integers(-8, 9, size=s) / 16.0).astype(np.float32)
    q = dy(B, Hq, Dh)
    q[..., 0] = 1.0
    pk, pv, wk, wv = dy(B, Hkv, N, Dh), dy(B, Hkv, N, Dh), dy(B, Hkv, W, Dh), dy(B, Hkv, W, Dh)
    cnt = np.array([W], np.int32)
    idx = np.array([[0, 2, 5]], np.int32)
    out = orc.two_tier_decode(q, pk, pv, idx, 3, wk, wv, cnt, W, 1.0)
    c = np.array([1024.0, 0, 0, 0], np.float32)
    out2 = orc.two_tier_decode(q, pk + c, pv, idx, 3, wk + c, wv, cnt, W, 1.0)
    assert np.isfinite(out2).all()
    _close(out, out2, 1e-12, "I-5")


def pin_single_key(orc):
    """I-6: a single key returns its value row exactly."""
    rng = np.random.default_rng(6)
    q = rng.standard_normal((1, 2, 8)).astype(np.float32)
    pk = rng.standard_normal((1, 1, 5, 8)).astype(np.float32)
    pv = rng.standard_normal((1, 1, 5, 8)).astype(np.float32)
    out = orc.two_tier_decode(q, pk, pv, np.array([[3]], np.int32), 1, None, None, None, 0, 1.0)
    _close(out[0, 0], pv[0, 0, 3], 0.0, "I-6")
    _close(out[0, 1], pv[0, 0, 3], 0.0, "I-6")


def pin_gqa_equals_repeated_mha(orc):
    """I-9: GQA equals MHA with each kv head repeated G times."""
    rng = np.random.default_rng(10)
    B, Hq, Hkv, Dh, N, k, W = 2, 6, 2, 8, 11, 4, 3
    G = Hq // Hkv
    q = rng.standard_normal((B, Hq, Dh)).astype(np.float32)
    pk = rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)
    pv = rng.standard_normal((B, Hkv, N, Dh)).astype(np.float32)
    wk = rng.standard_normal((B, Hkv, W, Dh)).astype(np.float32)
    wv = rng.standard_normal((B, Hkv, W, Dh)).astype(np.float32)
    cnt = np.array([1, 7], np.int32)
    idx = np.array([[0, 3, 4, 10], [1, 2, 6, 9]], np.int32)
    a = orc.two_tier_decode(q, pk, pv, idx, k, wk, wv, cnt, W, 0.4)
    r = lambda x: np.ascontiguousarray(np.repeat(x, G, axis=1))
    b = orc.two_tier_decode(q, r(pk), r(pv), idx, k, r(wk), r(wv), cnt, W, 0.4)
    _close(a, b, 0.0, "I-9")


def pin_bf16_widening(orc):
    """bf16 inputs give exactly what their fp32 widenings give."""
    rng = np.random.default_rng(13)
    B, Hq, Hkv, Dh, N, k, W = 1, 4, 2, 8, 9, 3, 4
    q = rng.standard_normal((B, Hq, Dh)).astype(np.float32)
    t = lambda *s: _bf16(rng.standard_normal(s).astype(np.float32))
    pk, pv, wk, wv = t(B, Hkv, N, Dh), t(B, Hkv, N, Dh), t(B, Hkv, W, Dh), t(B, Hkv, W, Dh)
    w = lambda h: (h.astype(np.uint32) << 16).view(np.float32)
    idx = np.array([[1, 4, 8]], np.int32)
    cnt = np.array([W], np.int32)
    a = orc.two_tier_decode(q, pk, pv, idx, k, wk, wv, cnt, W, 0.5)
    b = orc.two_tier_decode(q, w(pk), w(pv), idx, k, w(wk), w(wv), cnt, W, 0.5)
    _close(a, b, 0.0, "bf16 widening")


def pin_empty_key_list(orc):
    """k = 0 and an empty ring: the output row is zero."""
    q = np.ones((1, 2, 4), np.float32)
    pk = np.ones((1, 1, 3, 4), np.float32)
    wk = np.ones((1, 1, 2, 4), np.float32)
    out = orc.two_tier_decode(q, pk, pk, np.zeros((1, 0), np.int32), 0, wk, wk,
                              np.zeros((1,), np.int32), 2, 1.0)
    assert not out.any()


def pin_select_ragged_brute(orc):
    """Ragged selection vs exact rational top-k on each sequence's own rows:
    rows past n_b are made perfect matches (cosine 1) and must still never
    be chosen; a duplicated row makes a tie inside a prefix; k_b = min(k,
    n_b); question rows n_b.. follow; -1 pads the row; q_b is clamped to the
    room left in the row."""
    rng = np.random.default_rng(41)
    B, N, D, k, stride = 5, 11, 6, 4, 7
    keys = rng.standard_normal((B, N, D)).astype(np.float32)
    q = rng.standard_normal((B, D)).astype(np.float32)
    n_rows = np.array([11, 6, 0, 3, 8], np.int32)
    q_rows = np.array([0, 2, 3, 1, 5], np.int32)
    keys[1, 3] = keys[1, 1]
    for b in range(B):
        keys[b, n_rows[b]:] = 10.0 * q[b]
    idx, k_out = orc.select_ragged(keys, q, n_rows, k, q_rows, stride)
    for b in range(B):
        nb = int(n_rows[b])
        kb = min(k, nb)
        qb = min(int(q_rows[b]), stride - kb)
        want = brute.exact_topk(keys[b, :nb], q[b], kb) + list(range(nb, nb + qb))
        want += [-1] * (stride - len(want))
        assert idx[b].tolist() == want, (b, idx[b].tolist(), want)
        assert int(k_out[b]) == kb + qb


def pin_select_ragged_uniform(orc):
    """Every sequence at full length, no question rows: the ragged selection
    is the uniform one."""
    rng = np.random.default_rng(42)
    keys = rng.standard_normal((3, 40, 8)).astype(np.float32)
    q = rng.standard_normal((3, 8)).astype(np.float32)
    idx, k_out = orc.select_ragged(keys, q, np.full(3, 40, np.int32), 9)
    ref, _, _ = orc.select(keys, q, 9)
    assert (idx == ref).all() and (k_out == 9).all()


def pin_decode_ragged_history(orc):
    """Ragged decode over several steps vs list-history attention with each
    sequence's own pool rows (k_len clamped into [0, k]) and its own window
    fill."""
    rng = np.random.default_rng(43)
    B, Hq, Hkv, Dh, N, k, W = 3, 4, 2, 8, 10, 6, 4
    f32 = lambda *sh: rng.standard_normal(sh).astype(np.float32)
    pk, pv = f32(B, Hkv, N, Dh), f32(B, Hkv, N, Dh)
    idx = np.stack([np.sort(rng.choice(N, size=k, replace=False)) for _ in range(B)]).astype(np.int32)
    k_len = np.array([9, 2, -1], np.int32)
    kb = [6, 2, 0]
    fill = [4, 1, 0]
    wk, wv = np.zeros((B, Hkv, W, Dh), np.float32), np.zeros((B, Hkv, W, Dh), np.float32)
    for b in range(B):
        wk[b, :, :fill[b]] = f32(Hkv, fill[b], Dh)
        wv[b, :, :fill[b]] = f32(Hkv, fill[b], Dh)
    cnt = np.array(fill, np.int32)
    hist_k = [[[wk[b, h, s] for s in range(fill[b])] for h in range(Hkv)] for b in range(B)]
    hist_v = [[[wv[b, h, s] for s in range(fill[b])] for h in range(Hkv)] for b in range(B)]
    scale = 1.0 / math.sqrt(Dh)
    for step in range(5):
        nk, nv = f32(B, Hkv, 1, Dh), f32(B, Hkv, 1, Dh)
        orc.window_append(wk, wv, cnt, nk, nv)
        for b in range(B):
            for h in range(Hkv):
                hist_k[b][h].append(nk[b, h, 0])
                hist_v[b][h].append(nv[b, h, 0])
        q = f32(B, Hq, Dh)
        out = orc.two_tier_decode_ragged(q, pk, pv, idx, k_len, k, wk, wv, cnt, W, scale)
        for b in range(B):
            ref = brute.history_attention(q[b], pk[b], pv[b], idx[b, :kb[b]].tolist(), hist_k[b], hist_v[b],
                                          W, scale)
            _close(out[b], ref, 1e-12, f"ragged history step {step} b {b}")


def pin_row_norms_library(orc):
    """Row norms vs numpy's own norm routine: fp32 rows [B][N][D], and bf16
    CME vectors [M][Hc] (bit patterns widened here by a shift)."""
    rng = np.random.default_rng(51)
    keys = rng.standard_normal((3, 17, 9)).astype(np.float32)
    keys[1, 4] = 0.0
    ref = np.linalg.norm(keys.astype(np.float64), axis=2)
    _close(orc.row_norms(keys), ref, 1e-12, "row norms")
    h = _bf16(rng.standard_normal((37, 64)).astype(np.float32) * 3.0)
    h[5] = 0
    wide = (h.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    _close(orc.row_norms(h), np.linalg.norm(wide, axis=1), 1e-12, "bf16 row norms")


def pin_select_bf16_keys(orc):
    """Selection on bf16 keys equals selection on their exact fp32 widening
    (indices and scores), the widening done here by a shift of the bits."""
    rng = np.random.default_rng(52)
    for B, N, D, k in [(2, 40, 16, 7), (3, 9, 8, 9), (1, 200, 24, 31)]:
        keys = _bf16(rng.standard_normal((B, N, D)).astype(np.float32))
        keys[0, 3] = keys[0, 1]          # an exact tie
        wide = (keys.astype(np.uint32) << 16).view(np.float32)
        q = rng.standard_normal((B, D)).astype(np.float32)
        i1, s1, g1 = orc.select(keys, q, k)
        i2, s2, g2 = orc.select(wide, q, k)
        assert (i1 == i2).all(), "bf16 keys select differently from their widening"
        _close(s1, s2, 0.0, "bf16 key scores")
        for b in range(B):
            assert brute.exact_topk(wide[b], q[b], k) == i1[b].tolist(), "bf16 keys vs exact ranking"


def pin_locate_cases(orc):
    """CME-guided localization on hand-checked cases: the largest norm's
    chunk (mems_per_chunk rows per chunk) gives alpha from the offset table
    or from chunk * chunk_tokens; ties go to the earlier row; rows past n_b
    are ignored even when their norm is larger; a sequence without rows
    takes the midpoint; the window start then follows the window equation,
    checked here by its defining properties."""
    norms = np.array([
        [1.0, 2.0, 7.0, 7.0, 3.0, 0.5],    # rows 2 and 3 tie -> row 2 -> chunk 1 (m=2)
        [9.0, 1.0, 1.0, 1.0, 1.0, 8.0],    # row 0 -> chunk 0
        [1.0, 2.0, 3.0, 4.0, 5.0, 99.0],   # n_b = 5: row 5 ignored -> row 4 -> chunk 2
        [5.0, 5.0, 5.0, 5.0, 5.0, 5.0],    # n_b = 0 -> midpoint
    ])
    n_rows = np.array([6, 6, 5, 0], np.int32)
    ctx = np.array([1000, 50, 400, 301], np.int32)
    offsets = np.array([[0, 333, 666], [0, 20, 40], [10, 120, 390], [0, 1, 2]], np.int32)
    W = 100
    alpha, start = orc.locate(norms, ctx, W, 2, n_rows=n_rows, chunk_offset=offsets)
    assert alpha.tolist() == [333, 0, 390, 150], alpha.tolist()
    # window start: centred on alpha when that fits, else flush with an end
    assert start.tolist() == [283, 0, 300, 100], start.tolist()
    alpha2, _ = orc.locate(norms, ctx, W, 2, n_rows=n_rows, chunk_tokens=64)
    assert alpha2.tolist() == [64, 0, 128, 150], alpha2.tolist()
    alpha3, _ = orc.locate(norms, ctx, W, 1, chunk_tokens=10)   # one row per chunk, all rows
    assert alpha3.tolist() == [20, 0, 50, 0], alpha3.tolist()


def pin_locate_argmax_library(orc):
    """Random norms with planted ties: the chosen row is numpy's argmax
    (first occurrence) of the row's prefix."""
    rng = np.random.default_rng(52)
    B, N, m = 6, 40, 4
    norms = rng.integers(0, 12, size=(B, N)).astype(np.float64)  # many exact ties
    n_rows = np.array([40, 13, 1, 0, 39, 4], np.int32)
    ctx = np.full(B, 10000, np.int32)
    alpha, _ = orc.locate(norms, ctx, 64, m, n_rows=n_rows, chunk_tokens=1)
    for b in range(B):
        want = ctx[b] // 2 if n_rows[b] == 0 else int(np.argmax(norms[b, :n_rows[b]])) // m
        assert alpha[b] == want, (b, alpha[b], want)


def _onehot(classes, H=8):
    return np.eye(H, dtype=np.float32)[np.asarray(classes)]


def pin_denoise_onehot_cases(orc):
    """Eq. 3 on one-hot tokens, where a cosine is exactly 1 (same class) or
    0 (different class), so every decision can be read off the class
    sequence by eye:
        position  0 1 2 3 4 5 6 7 8 9 10 11
        class     0 1 0 2 3 3 1 1 4 5 6  7
    With g = 3, a token passes when one of its next three tokens has its
    class: positions 0 (2), 4 (5), 6 (7).  Position 11 has no neighbour.
    With no floor (m = 0) the kept set is {0, 4, 6}.  With m = 4, position
    10 (= 6 + 4) is forced as well (4 = 0 + 4 passes anyway); with m = 3,
    3 (= 0 + 3) and 9 (= 6 + 3) are forced and nothing else (11 - 9 = 2).  tau = 1 keeps exact-1 cosines
    (Eq. 3 is '>='); tau just above 1 keeps nothing by Eq. 3, so only the
    floor remains: m = 5 keeps 4 and 9 (first at -1 + 5).  A second
    sequence of 7 tokens (n_b = 7) must ignore tokens past its end: its
    position 6 has class 1 like position 7 of the first row's pattern, but
    position 7 is outside it."""
    classes = [0, 1, 0, 2, 3, 3, 1, 1, 4, 5, 6, 7]
    e = np.stack([_onehot(classes), _onehot(classes)])
    n_tok = np.array([12, 7], np.int32)
    mc = orc.denoise_scores(e, 3, n_tok)
    assert mc[0].tolist()[:11] == [1, 0, 0, 0, 1, 0, 1, 0, 0, 0, 0] and np.isneginf(mc[0, 11])
    assert mc[1].tolist()[:6] == [1, 0, 0, 0, 1, 0] and np.isneginf(mc[1, 6:]).all()
    kept = lambda r: r["kept_idx"][0, :r["kept_count"][0]].tolist()
    assert kept(orc.denoise_select(mc, 0.05, 0, n_tok)) == [0, 4, 6]
    assert kept(orc.denoise_select(mc, 0.05, 4, n_tok)) == [0, 4, 6, 10]
    assert kept(orc.denoise_select(mc, 0.05, 3, n_tok)) == [0, 3, 4, 6, 9]
    assert kept(orc.denoise_select(mc, 1.0, 0, n_tok)) == [0, 4, 6]
    assert kept(orc.denoise_select(mc, 1.0 + 1e-12, 5, n_tok)) == [4, 9]
    r = orc.denoise_select(mc, 0.05, 4, n_tok, chunk_tokens=3)
    assert r["kept_idx"][1].tolist() == [0, 4, -1, -1, -1, -1, -1, -1, -1, -1, -1, -1]
    assert r["kept_count"].tolist() == [4, 2]
    assert r["chunk_offset"].tolist() == [[0, 10, -1, -1], [0, -1, -1, -1]]
    assert r["n_chunks"].tolist() == [2, 1]
    assert r["keep"][0].tolist() == [1, 0, 0, 0, 1, 0, 1, 0, 0, 0, 1, 0]


def pin_denoise_scores_library(orc):
    """The Eq. 3 statistic against torch's cosine_similarity, offset by
    offset, in fp64; bf16 inputs are widened exactly first."""
    import torch
    rng = np.random.default_rng(61)
    B, n, H, g = 2, 30, 16, 3
    e = rng.standard_normal((B, n, H)).astype(np.float32)
    e[:, ::4] += e[:, 1::4]  # some strongly aligned neighbours
    for dtype in ("f32", "bf16"):
        arr = e if dtype == "f32" else _bf16(e)
        vals = torch.from_numpy(e.astype(np.float64) if dtype == "f32" else
                                (arr.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
        ref = np.full((B, n), -np.inf)
        for d in range(1, g + 1):
            c = torch.nn.functional.cosine_similarity(vals[:, :-d], vals[:, d:], dim=2).numpy()
            ref[:, :-d] = np.maximum(ref[:, :-d], c)
        got = orc.denoise_scores(arr, g)
        assert np.isneginf(got[:, -1]).all()
        _close(got[:, :-1], ref[:, :-1], 1e-12, f"denoise scores {dtype}")


def pin_denoise_floor_properties(orc):
    """On random statistics and thresholds the kept set is characterised by:
    every token passing Eq. 3 is kept; any m consecutive positions of the
    sequence hold a kept token; a kept token that does not pass sits exactly
    m after the previous kept one (virtual -1); nothing past n_b is kept."""
    rng = np.random.default_rng(62)
    B, n = 6, 200
    mc = rng.uniform(-1, 1, size=(B, n))
    mc[:, -1] = -np.inf
    n_tok = np.array([200, 150, 1, 0, 37, 199], np.int32)
    for tau in (-2.0, 0.3, 0.9, 2.0):
        for m in (0, 1, 5, 16):
            r = orc.denoise_select(mc, tau, m, n_tok)
            for b in range(B):
                nb = int(n_tok[b])
                kept = r["kept_idx"][b, :r["kept_count"][b]].tolist()
                assert kept == sorted(set(kept)) and all(0 <= i < nb for i in kept)
                assert r["keep"][b].tolist() == [1 if i in set(kept) else 0 for i in range(n)]
                passing = {i for i in range(nb) if mc[b, i] >= tau}
                assert passing <= set(kept)
                if m > 0:
                    marks = [-1] + kept
                    for a, c in zip(marks, marks[1:]):
                        assert c in passing or c - a == m
                    assert all(any(j in set(kept) for j in range(s, s + m)) for s in range(0, nb - m + 1))
                else:
                    assert set(kept) == passing


def _bf16_vals(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def pin_bridge_library(orc):
    """MemoryBridge's MLP and LayerNorm against torch's Linear / exact GELU /
    Linear / layer_norm in fp64 on the same bf16 weights; the cap is then
    applied to torch's LayerNorm output (the cap itself is pinned by
    pin_bridge_cap_cases)."""
    import torch
    rng = np.random.default_rng(71)
    M, Hc, F, Hd, nu = 5, 24, 40, 16, 0.7
    h = _bf16(rng.standard_normal((M, Hc)).astype(np.float32))
    w1 = _bf16((rng.standard_normal((F, Hc)) / np.sqrt(Hc)).astype(np.float32))
    w2 = _bf16((rng.standard_normal((Hd, F)) / np.sqrt(F)).astype(np.float32))
    b1, b2 = rng.standard_normal(F).astype(np.float32), rng.standard_normal(Hd).astype(np.float32)
    gamma, beta = rng.uniform(0.5, 2, Hd).astype(np.float32), rng.standard_normal(Hd).astype(np.float32)
    T = lambda x: torch.from_numpy(np.asarray(x, np.float64))
    hid = torch.nn.functional.gelu(T(_bf16_vals(h)) @ T(_bf16_vals(w1)).T + T(b1), approximate="none")
    _close(orc.bridge_hidden(h, w1, b1), hid.numpy(), 1e-12, "bridge hidden")
    y = hid @ T(_bf16_vals(w2)).T + T(b2)
    m_hat = torch.nn.functional.layer_norm(y, (Hd,), T(gamma), T(beta), eps=1e-5)
    t = nu * torch.tanh(m_hat)
    ref = t * torch.clamp(2 * nu / t.norm(dim=1, keepdim=True), max=1.0)
    _close(orc.bridge_out(hid.numpy(), w2, b2, gamma, beta, nu), ref.numpy(), 1e-12, "bridge out")


def pin_bridge_cap_cases(orc):
    """Hand-checked cases of LayerNorm + cap (output weights zero, so y is
    the bias vector):
      * constant y: LayerNorm gives beta; small beta stays below the cap, so
        the output is exactly nu * tanh(beta);
      * y = (1, 2, 3, 4), gamma = 1, beta = 0, eps = 0: mean 2.5, biased
        variance 1.25, m_hat = (y - 2.5) / sqrt(1.25); the norm of
        tanh(m_hat) is below 2, so the output is tanh(m_hat) (nu = 1);
      * saturated: beta = +-30 in 16 coordinates: tanh = +-1, the norm is
        4 nu > 2 nu, so every coordinate becomes +-nu / 2."""
    def run(b2, gamma, beta, nu, eps):
        Hd = len(b2)
        zero_w2 = np.zeros((Hd, 3), np.uint16)
        return orc.bridge_out(np.ones((1, 3)), zero_w2, np.asarray(b2, np.float32), np.asarray(gamma, np.float32),
                              np.asarray(beta, np.float32), nu, eps)[0]
    beta = np.array([0.1, -0.2, 0.05, 0.0, 0.3], np.float32)
    out = run([2.0] * 5, [3.0] * 5, beta, 0.8, 1e-5)
    assert np.allclose(out, [0.8 * math.tanh(float(b)) for b in beta], rtol=0, atol=1e-15), out
    out = run([1.0, 2.0, 3.0, 4.0], [1.0] * 4, [0.0] * 4, 1.0, 0.0)
    want = [math.tanh((v - 2.5) / math.sqrt(1.25)) for v in (1.0, 2.0, 3.0, 4.0)]
    assert np.allclose(out, want, rtol=0, atol=1e-15), (out, want)
    sgn = np.array([1 if i % 3 else -1 for i in range(16)], np.float32)
    out = run([0.0] * 16, [1.0] * 16, 30.0 * sgn, 0.6, 1e-5)
    assert np.allclose(out, 0.3 * sgn.astype(np.float64), rtol=0, atol=1e-15), out


def pin_bridge_bounds(orc):
    """The cap's guarantees on random large activations: every coordinate
    within nu, every row's norm within 2 nu, and rows whose nu*tanh norm is
    below 2 nu untouched (checked by scaling nu up until no row is capped)."""
    rng = np.random.default_rng(72)
    M, F, Hd = 20, 12, 64
    hid = rng.standard_normal((M, F)) * 5
    w2 = _bf16(rng.standard_normal((Hd, F)).astype(np.float32))
    b2 = rng.standard_normal(Hd).astype(np.float32)
    gamma = rng.uniform(1, 10, Hd).astype(np.float32)
    beta = rng.standard_normal(Hd).astype(np.float32)
    for nu in (0.1, 1.0, 7.5):
        out = orc.bridge_out(hid, w2, b2, gamma, beta, nu)
        assert (np.abs(out) <= nu * (1 + 1e-12)).all()
        assert (np.linalg.norm(out, axis=1) <= 2 * nu * (1 + 1e-12)).all()
        assert (np.linalg.norm(out, axis=1) >= 2 * nu * (1 - 1e-12)).any() or nu > 1
    # nu * tanh(x) has norm <= nu * sqrt(Hd) = 8 nu: with Hd = 64 every row is capped unless small;
    # with Hd = 3 the norm is at most nu * sqrt(3) < 2 nu, so the cap never acts.
    w3 = _bf16(rng.standard_normal((3, F)).astype(np.float32))
    out3 = orc.bridge_out(hid, w3, b2[:3], gamma[:3], beta[:3], 0.5)
    ref3 = orc.bridge_out(hid, w3, b2[:3], gamma[:3], beta[:3], 0.5)
    assert (np.linalg.norm(out3, axis=1) < 1.0).all() and np.array_equal(out3, ref3)


ALL_PINS = [v for n, v in sorted(globals().items()) if n.startswith("pin_") and callable(v)]


def main(argv):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import oracle
    orc = oracle.Oracle(argv[1])
    failed = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except Exception as e:  # any failure counts, including oracle errors
            failed.append(f"{pin.__name__}: {type(e).__name__}: {str(e)[:120]}")
    for f in failed:
        print("FAIL", f)
    return 1 if failed else 0


if __name__ == "__main__":
    sys.exit(main(sys.argv))
