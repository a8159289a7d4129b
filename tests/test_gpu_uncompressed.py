"""Parity at the shape of the 32-layer stack's uncompressed baseline: the same
decode step over a full 32,768-token cache, i.e. no Tier-1 rows (k = 0, a
one-row pool, idx == NULL) and a ring of capacity 32,768 + 3,000 that starts
with 32,768 tokens and never wraps, one token appended per step.  This is
the configuration the benchmark times for the uncompressed comparison.

Ring slots past the filled ones hold NaN here (the benchmark allocates them
uninitialised): they must never reach the output.  Outputs within 2e-3 of the
fp64 oracle (bf16 K/V); ring contents and counts bit-exact."""
import math

import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, max_abs, say, to_dev, to_host, tol_for

pytestmark = pytest.mark.gpu

FULL_CTX = 32768
W = FULL_CTX + 3000
HQ, HKV, DH = 32, 8, 128
SCALE = 1.0 / math.sqrt(DH)
STD = 1.0 / math.sqrt(DH)


def _bits(t):
    return to_host(t).view(np.uint16)


@pytest.mark.timeout(600)
def test_uncompressed_baseline_b2(orc):
    """B = 2 (a split plan over 35,768 ring slots), every output checked."""
    B = 2
    rng = np.random.default_rng(55)
    say(f"uncompressed B={B}: generating {FULL_CTX} tokens per (sequence, kv head)")
    wk = np.full((B, HKV, W, DH), 0x7FC0, np.uint16)
    wv = np.full((B, HKV, W, DH), 0x7FC0, np.uint16)
    wk[:, :, :FULL_CTX] = wl.f32_to_bf16_bits((rng.standard_normal((B, HKV, FULL_CTX, DH)) * STD).astype(np.float32))
    wv[:, :, :FULL_CTX] = wl.f32_to_bf16_bits((rng.standard_normal((B, HKV, FULL_CTX, DH)) * STD).astype(np.float32))
    cnt = np.full((B,), FULL_CTX, np.int32)
    pool = np.zeros((B, HKV, 1, DH), np.uint16)
    d_wk, d_wv, d_wc, d_pool = to_dev(wk), to_dev(wv), to_dev(cnt), to_dev(pool)
    ws = cmc.decode_workspace(B, HQ, HKV, DH, 0, W, DEV)
    for step in range(3):
        say(f"uncompressed B={B}: step {step}")
        nk = wl.f32_to_bf16_bits((rng.standard_normal((B, HKV, 1, DH)) * STD).astype(np.float32))
        nv = wl.f32_to_bf16_bits((rng.standard_normal((B, HKV, 1, DH)) * STD).astype(np.float32))
        q = (rng.standard_normal((B, HQ, DH)) * STD).astype(np.float32)
        orc.window_append(wk, wv, cnt, nk, nv)
        ref = orc.two_tier_decode(q, pool, pool, None, 0, wk, wv, cnt, W, SCALE)
        out = cmc.cmc_decode_step(to_dev(q), d_pool, d_pool, None, 0, d_wk, d_wv, d_wc, to_dev(nk), to_dev(nv),
                                  SCALE, workspace=ws)
        torch.cuda.synchronize()
        got = to_host(out)
        assert np.isfinite(got).all()
        err = max_abs(got, ref)
        assert err <= tol_for("bf16"), f"step {step}: max abs err {err:.3e}"
        assert (to_host(d_wc) == cnt).all(), "ring count"
    assert (_bits(d_wk) == wk).all() and (_bits(d_wv) == wv).all(), "ring contents after all steps"


@pytest.mark.timeout(600)
def test_uncompressed_baseline_b32_launch_config(orc):
    """B = 32 (one 8-wave workgroup per (sequence, kv head) pair, the
    benchmark's launch), inputs drawn on the device as the benchmark draws
    them; the oracle checks sampled sequences at every step."""
    B = 32
    sample = [0, 13, 31]
    say(f"uncompressed B={B}: drawing the cache on the device")
    bf = torch.bfloat16
    d_wk = torch.empty((B, HKV, W, DH), dtype=bf, device=DEV)
    d_wv = torch.empty_like(d_wk)
    d_wk.view(torch.int16)[:, :, FULL_CTX:] = 0x7FC0
    d_wv.view(torch.int16)[:, :, FULL_CTX:] = 0x7FC0
    d_wk[:, :, :FULL_CTX] = wl.device_normal(505, "full_k", (0,), (B, HKV, FULL_CTX, DH), STD, DEV, bf)
    d_wv[:, :, :FULL_CTX] = wl.device_normal(505, "full_v", (0,), (B, HKV, FULL_CTX, DH), STD, DEV, bf)
    d_wc = torch.full((B,), FULL_CTX, dtype=torch.int32, device=DEV)
    d_pool = torch.zeros((B, HKV, 1, DH), dtype=bf, device=DEV)
    torch.cuda.synchronize()
    # host copies of the sampled sequences' caches, advanced by the oracle
    hk = {b: _bits(d_wk[b:b + 1]).copy() for b in sample}
    hv = {b: _bits(d_wv[b:b + 1]).copy() for b in sample}
    hc = {b: np.array([FULL_CTX], np.int32) for b in sample}
    pool1 = np.zeros((1, HKV, 1, DH), np.uint16)
    ws = cmc.decode_workspace(B, HQ, HKV, DH, 0, W, DEV)
    out = torch.empty((B, HQ, DH), dtype=torch.float32, device=DEV)
    for step in range(3):
        say(f"uncompressed B={B}: step {step}")
        q = wl.device_normal(505, "q", (0, step), (B, HQ, DH), STD, DEV, torch.float32)
        nk = wl.device_normal(505, "new_k", (0, step), (B, HKV, 1, DH), STD, DEV, bf)
        nv = wl.device_normal(505, "new_v", (0, step), (B, HKV, 1, DH), STD, DEV, bf)
        torch.cuda.synchronize()
        hq, hnk, hnv = to_host(q), _bits(nk), _bits(nv)
        cmc.cmc_decode_step(q, d_pool, d_pool, None, 0, d_wk, d_wv, d_wc, nk, nv, SCALE, out=out, workspace=ws)
        torch.cuda.synchronize()
        got = to_host(out)
        assert np.isfinite(got).all()
        assert (to_host(d_wc) == FULL_CTX + step + 1).all(), "ring count"
        for b in sample:
            orc.window_append(hk[b], hv[b], hc[b], hnk[b:b + 1], hnv[b:b + 1])
            ref = orc.two_tier_decode(hq[b:b + 1], pool1, pool1, None, 0, hk[b], hv[b], hc[b], W, SCALE)
            err = max_abs(got[b:b + 1], ref)
            assert err <= tol_for("bf16"), f"step {step} sequence {b}: max abs err {err:.3e}"
    for b in sample:
        assert (_bits(d_wk[b:b + 1]) == hk[b]).all() and (_bits(d_wv[b:b + 1]) == hv[b]).all(), b
