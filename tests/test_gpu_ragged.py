"""Ragged batches on the GPU vs the oracle, through the C ABI: per-sequence
candidate counts, selection sizes, pinned question rows, pool-row counts and
window fills.  Index lists and counts bit-exact; attention within 1e-5
(fp32 K/V) or 2e-3 (bf16 K/V); ring state bit-exact."""
import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, max_abs, say, to_dev, to_host, tol_for
from tests.inputs import accepted_attempts
from tests.test_gpu_parity import _separated

pytestmark = pytest.mark.gpu


def _check_select_ragged(orc, keys, qv, n_rows, k, q_rows, stride, what):
    say(f"select_ragged {what}: B={keys.shape[0]} N={keys.shape[1]} D={keys.shape[2]} k={k} stride={stride}")
    ref_idx, ref_k = orc.select_ragged(keys, qv, n_rows, k, q_rows, stride)
    scores = torch.empty(keys.shape[:2], dtype=torch.float32, device=DEV)
    idx, k_out = cmc.cmc_select_cmes_ragged(to_dev(keys), to_dev(qv), to_dev(n_rows), k,
                                            q_rows=None if q_rows is None else to_dev(q_rows),
                                            idx_stride=stride, scores_out=scores)
    torch.cuda.synchronize()
    assert (to_host(idx) == ref_idx).all(), f"{what}: index lists differ"
    assert (to_host(k_out) == ref_k).all(), f"{what}: k_out differs"
    s = to_host(scores)
    for b in range(keys.shape[0]):
        nb = min(max(int(n_rows[b]), 0), keys.shape[1])
        if nb:
            _, ref_s, _ = orc.select(keys[b:b + 1, :nb], qv[b:b + 1], 0)
            assert max_abs(s[b, :nb], ref_s[0]) < 1e-6
        assert np.isneginf(s[b, nb:]).all(), "rows past n_b must score -inf"
    # workspace variant, no scores returned
    idx2, _ = cmc.cmc_select_cmes_ragged(to_dev(keys), to_dev(qv), to_dev(n_rows), k,
                                         q_rows=None if q_rows is None else to_dev(q_rows), idx_stride=stride)
    torch.cuda.synchronize()
    assert (to_host(idx2) == ref_idx).all()


@pytest.mark.parametrize("B,N,D,k,stride,n_list,q_list", [
    (4, 100, 8, 10, 16, [100, 37, 5, 0], [0, 3, 6, 16]),                 # n_b < k, n_b = 0, q clamps
    (3, 2048, 64, 256, 300, [2048, 300, 255], [44, 0, 1]),
    (2, 32768, 8, 1024, 1100, [32768, 20000], [76, 80]),                  # largest N; q clamps to 76
    (5, 333, 12, 0, 4, [333, 1, 0, 7, 100], [4, 2, 0, 9, -3]),            # k = 0: question rows only
    (2, 50, 4, 80, 80, [50, 20], None),                                   # k > N
    (3, 64, 16, 8, 8, [-5, 64, 99], None),                                # n_b clamped into [0, N]
])
def test_select_ragged_sizes(orc, B, N, D, k, stride, n_list, q_list):
    keys, qv = _separated(B, N, D, seed=N + k + stride)
    n_rows = np.array(n_list, np.int32)
    q_rows = None if q_list is None else np.array(q_list, np.int32)
    _check_select_ragged(orc, keys, qv, n_rows, k, q_rows, stride, "sizes")


@pytest.mark.parametrize("B,N,D,k,stride,n_list,q_list", [
    (4, 100, 8, 10, 16, [100, 37, 5, 0], [0, 3, 6, 16]),
    (3, 4096, 64, 512, 560, [4096, 1000, 511], [48, 8, 20]),
    # >= 65536 rows (the large-batch launch): counts ending inside a wave's rows
    (3, 25003, 32, 400, 420, [25003, 12345, 7], [0, 20, 5]),
])
def test_select_ragged_bf16_keys(orc, B, N, D, k, stride, n_list, q_list):
    """bf16 selection keys through the ragged call (same bits on both sides;
    rounding merges close keys into exact ties, resolved to the lower row)."""
    keys, qv = _separated(B, N, D, seed=N + k + stride + 1)
    _check_select_ragged(orc, wl.f32_to_bf16_bits(keys), qv, np.array(n_list, np.int32), k,
                         np.array(q_list, np.int32), stride, "bf16 keys")


def test_select_ragged_ties(orc):
    keys, qv = _separated(3, 1000, 8, seed=11, dup_every=4)
    _check_select_ragged(orc, keys, qv, np.array([1000, 401, 77], np.int32), 100,
                         np.array([5, 5, 5], np.int32), 110, "ties")


def test_select_ragged_full_length_equals_uniform(orc):
    keys, qv = _separated(3, 500, 16, seed=12)
    idx, k_out = cmc.cmc_select_cmes_ragged(to_dev(keys), to_dev(qv), to_dev(np.full(3, 500, np.int32)), 40)
    ref = cmc.cmc_select_cmes(to_dev(keys), to_dev(qv), 40)
    torch.cuda.synchronize()
    assert (to_host(idx) == to_host(ref)).all() and (to_host(k_out) == 40).all()


def _ragged_decode_case(orc, B, Hq, Hkv, Dh, N, k, W, k_len, fills, dtype, seed, steps=3, fused=True,
                        idx_none=False):
    rng = np.random.default_rng(seed)
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    cv = wl.f32_to_bf16_bits if dtype == "bf16" else (lambda x: x)
    pk, pv = cv(f(B, Hkv, N, Dh)), cv(f(B, Hkv, N, Dh))
    idx = None if idx_none else np.stack(
        [np.concatenate([np.sort(rng.choice(N, size=k, replace=False))]) for _ in range(B)]).astype(np.int32)
    wk = np.zeros((B, Hkv, W, Dh), np.float32)
    wv = np.zeros((B, Hkv, W, Dh), np.float32)
    for b in range(B):
        wk[b, :, :fills[b]] = f(Hkv, fills[b], Dh)
        wv[b, :, :fills[b]] = f(Hkv, fills[b], Dh)
    wk, wv = cv(wk), cv(wv)
    cnt = np.array(fills, np.int32)
    kl = np.array(k_len, np.int32)
    scale = 1.0 / np.sqrt(Dh)
    d = dict(pk=to_dev(pk), pv=to_dev(pv), idx=None if idx is None else to_dev(idx), kl=to_dev(kl),
             wk=to_dev(wk) if W else None, wv=to_dev(wv) if W else None, wc=to_dev(cnt) if W else None)
    ws = cmc.decode_workspace(B, Hq, Hkv, Dh, k, W, DEV)
    for step in range(steps):
        say(f"decode_ragged {dtype} B={B} Hq={Hq} Hkv={Hkv} Dh={Dh} N={N} k={k} W={W} step={step}")
        nk = nv = None
        if W:
            nk, nv = cv(f(B, Hkv, 1, Dh)), cv(f(B, Hkv, 1, Dh))
            orc.window_append(wk, wv, cnt, nk, nv)
            if not fused:
                cmc.cmc_window_append(d["wk"], d["wv"], d["wc"], to_dev(nk), to_dev(nv))
        q = f(B, Hq, Dh)
        ref = orc.two_tier_decode_ragged(q, pk, pv, idx, kl, k, wk, wv, cnt, W, scale)
        if fused:
            out = cmc.cmc_decode_step_ragged(to_dev(q), d["pk"], d["pv"], d["idx"], d["kl"], k, d["wk"], d["wv"],
                                             d["wc"], None if nk is None else to_dev(nk),
                                             None if nv is None else to_dev(nv), scale, W=W, workspace=ws)
        else:
            out = cmc.cmc_two_tier_decode_ragged(to_dev(q), d["pk"], d["pv"], d["idx"], d["kl"], k, d["wk"],
                                                 d["wv"], d["wc"], scale, W=W, workspace=ws)
        torch.cuda.synchronize()
        assert not ws[:4 * (B + B * Hkv)].any(), "arrival counters must return to zero"
        if W:
            assert (to_host(d["wk"]) == wk).all() and (to_host(d["wv"]) == wv).all(), "ring contents"
            assert (to_host(d["wc"]) == cnt).all(), "ring count"
        err = max_abs(to_host(out), ref)
        assert np.isfinite(to_host(out)).all()
        assert err <= tol_for(dtype), f"step {step}: max abs err {err:.3e}"


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("dtype,Dh,G", [("bf16", 128, 4), ("bf16", 64, 8), ("f32", 128, 2), ("bf16", 256, 1)])
def test_decode_ragged_small(orc, fused, dtype, Dh, G):
    """Four sequences: all k rows, a few, none (empty list: the window
    alone), more than k (clamped); fills full, partial, empty."""
    _ragged_decode_case(orc, B=4, Hq=2 * G, Hkv=2, Dh=Dh, N=90, k=40, W=24, k_len=[40, 7, 0, 99],
                        fills=[24, 5, 0, 13], dtype=dtype, seed=Dh + G, fused=fused)


def test_decode_ragged_empty_sequence_zero(orc):
    """k_len 0 and an empty ring: that sequence's output is zero."""
    _ragged_decode_case(orc, B=2, Hq=4, Hkv=4, Dh=64, N=10, k=6, W=3, k_len=[0, 6], fills=[0, 0],
                        dtype="f32", seed=3, steps=1, fused=False)


@pytest.mark.parametrize("B,Hkv,k,W", [(64, 4, 300, 200), (16, 8, 1500, 700), (3, 2, 2500, 0)])
def test_decode_ragged_plans(orc, B, Hkv, k, W):
    """Batches that take the 8-wave plan (256 pairs), key splits with a
    merge (few pairs, long lists) and no window."""
    rng = np.random.default_rng(B + k)
    k_len = rng.integers(-2, k + 3, size=B).tolist()
    fills = rng.integers(0, W + 1, size=B).tolist() if W else [0] * B
    _ragged_decode_case(orc, B=B, Hq=4 * Hkv, Hkv=Hkv, Dh=128, N=k + 50, k=k, W=W, k_len=k_len, fills=fills,
                        dtype="bf16", seed=B * k, steps=2, fused=W > 0)


def test_decode_ragged_identity_index(orc):
    _ragged_decode_case(orc, B=3, Hq=8, Hkv=8, Dh=64, N=40, k=40, W=0, k_len=[40, 13, 1], fills=[0, 0, 0],
                        dtype="f32", seed=5, steps=1, fused=False, idx_none=True)


def _ragged_end_to_end(orc, w, steps, samples):
    """Selection with pinned question rows, then fused decode steps with
    k_len = k_out, against the oracle's chain."""
    att = accepted_attempts(w, orc)
    rs = wl.ragged_sizes(w)
    keys, qv = wl.sel_keys(w), wl.q_vecs(w, att)
    ref_idx, ref_k = orc.select_ragged(keys, qv, rs["n_rows"], w.k, rs["q_rows"], w.idx_stride)
    say(f"{w.name}: select_ragged on GPU")
    idx, k_out = cmc.cmc_select_cmes_ragged(to_dev(keys), to_dev(qv), to_dev(rs["n_rows"]), w.k,
                                            q_rows=to_dev(rs["q_rows"]), idx_stride=w.idx_stride)
    torch.cuda.synchronize()
    assert (to_host(idx) == ref_idx).all() and (to_host(k_out) == ref_k).all()
    del keys
    pk, pv = wl.pool_kv(w)
    wk, wv, cnt = wl.window_kv(w)
    d_pk, d_pv, d_wk, d_wv, d_wc = map(to_dev, (pk, pv, wk, wv, cnt))
    # the benchmark's configuration: gathered once, decoded with idx == NULL
    d_pk, d_pv = cmc.cmc_gather_tier1(d_pk, d_pv, idx, w.idx_stride, k_len=k_out)
    ws = cmc.decode_workspace(w.B, w.Hq, w.Hkv, w.Dh, w.idx_stride, w.W, DEV)
    out = torch.empty((w.B, w.Hq, w.Dh), dtype=torch.float32, device=DEV)
    worst = 0.0
    for t in range(steps):
        nk, nv = wl.step_new_kv(w, t)
        orc.window_append(wk, wv, cnt, nk, nv)
        sampled = t in samples
        q = wl.step_q(w, t) if sampled else None
        d_q = to_dev(q) if sampled else to_dev(np.zeros((w.B, w.Hq, w.Dh), np.float32))
        cmc.cmc_decode_step_ragged(d_q, d_pk, d_pv, None, k_out, w.idx_stride, d_wk, d_wv, d_wc, to_dev(nk),
                                   to_dev(nv), w.scale, out=out, workspace=ws)
        if sampled:
            say(f"{w.name}: step {t}")
            ref = orc.two_tier_decode_ragged(q, pk, pv, ref_idx, ref_k, w.idx_stride, wk, wv, cnt, w.W, w.scale)
            torch.cuda.synchronize()
            err = max_abs(to_host(out), ref)
            worst = max(worst, err)
            assert err <= tol_for(w.kv_dtype), f"step {t}: max abs err {err:.3e}"
    torch.cuda.synchronize()
    assert (to_host(d_wc) == cnt).all()
    assert (to_host(d_wk) == wk).all() and (to_host(d_wv) == wv).all()
    say(f"{w.name}: worst max-abs error {worst:.3e}")


def test_ragged_small_end_to_end(orc):
    w = wl.get("ragged_batch64").replace(name="ragged_small", B=6, N=300, D=64, k=40, W=64, steps=80,
                                         ctx_min=40, ctx_max=1200, q_min=1, q_max=9)
    _ragged_end_to_end(orc, w, w.steps, samples={0, 1, 30, 63, 64, 79})


@pytest.mark.timeout(900)
def test_full_ragged_batch64(orc):
    """The benchmark's ragged workload at full size, in its launch
    configuration: every sequence's selection, all 3000 steps with the
    oracle's ring advanced every step, attention at sampled steps."""
    w = wl.get("ragged_batch64")
    _ragged_end_to_end(orc, w, w.steps, samples={0, 1, 500, 1023, 1024, 1025, w.steps - 1})
