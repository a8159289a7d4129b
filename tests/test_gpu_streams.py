"""Independent calls on different streams share no state.

Two decode problems -- one on a split plan (a single sequence, its key list
cut across workgroups that merge through their workspace) and one on an
unsplit 8-wave plan -- and a selection run on three streams of default
priority, each with its own workspace, their launches interleaved with no
synchronisation between the streams.  Every output is checked against the
oracle afterwards (bf16 K/V within 2e-3, ring contents and counts bit-exact,
index sets bit-exact), and the workspaces' arrival counters are back at zero."""
import math

import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, max_abs, say, to_dev, to_host, tol_for

pytestmark = pytest.mark.gpu

STEPS = 4


class _Problem:
    """One decode problem: pool, ring, per-step inputs and the oracle's outputs."""

    def __init__(self, orc, seed, B, Hq, Hkv, Dh, N, k, W, fill):
        rng = np.random.default_rng(seed)
        std = 1.0 / math.sqrt(Dh)
        f = lambda *s: wl.f32_to_bf16_bits((rng.standard_normal(s) * std).astype(np.float32))
        self.B, self.Hq, self.Hkv, self.Dh, self.k, self.W = B, Hq, Hkv, Dh, k, W
        self.scale = 1.0 / math.sqrt(Dh)
        pk, pv = f(B, Hkv, N, Dh), f(B, Hkv, N, Dh)
        idx = np.stack([np.sort(rng.choice(N, size=k, replace=False)) for _ in range(B)]).astype(np.int32)
        wk = np.zeros((B, Hkv, W, Dh), np.uint16)
        wv = np.zeros((B, Hkv, W, Dh), np.uint16)
        wk[:, :, :fill], wv[:, :, :fill] = f(B, Hkv, fill, Dh), f(B, Hkv, fill, Dh)
        cnt = np.full((B,), fill, np.int32)
        self.d = dict(pk=to_dev(pk), pv=to_dev(pv), idx=to_dev(idx), wk=to_dev(wk), wv=to_dev(wv), wc=to_dev(cnt))
        self.ws = cmc.decode_workspace(B, Hq, Hkv, Dh, k, W, DEV)
        self.q, self.nk, self.nv, self.out, self.ref = [], [], [], [], []
        for _ in range(STEPS):
            q = (rng.standard_normal((B, Hq, Dh)) * std).astype(np.float32)
            nk, nv = f(B, Hkv, 1, Dh), f(B, Hkv, 1, Dh)
            orc.window_append(wk, wv, cnt, nk, nv)
            self.ref.append(orc.two_tier_decode(q, pk, pv, idx, k, wk, wv, cnt, W, self.scale))
            self.q.append(to_dev(q))
            self.nk.append(to_dev(nk))
            self.nv.append(to_dev(nv))
            self.out.append(torch.empty((B, Hq, Dh), dtype=torch.float32, device=DEV))
        self.wk_ref, self.wv_ref, self.cnt_ref = wk, wv, cnt

    def step(self, t):
        d = self.d
        cmc.cmc_decode_step(self.q[t], d["pk"], d["pv"], d["idx"], self.k, d["wk"], d["wv"], d["wc"], self.nk[t],
                            self.nv[t], self.scale, out=self.out[t], workspace=self.ws)

    def check(self):
        for t in range(STEPS):
            err = max_abs(to_host(self.out[t]), self.ref[t])
            assert err <= tol_for("bf16"), f"step {t}: max abs err {err:.3e}"
        assert (to_host(self.d["wk"]) == self.wk_ref).all() and (to_host(self.d["wv"]) == self.wv_ref).all()
        assert (to_host(self.d["wc"]) == self.cnt_ref).all()
        assert not self.ws[:4 * (self.B + self.B * self.Hkv)].any(), "arrival counters must return to zero"


def test_streams_interleaved(orc):
    split = _Problem(orc, 11, B=1, Hq=32, Hkv=8, Dh=128, N=600, k=256, W=512, fill=512)
    wide = _Problem(orc, 12, B=32, Hq=32, Hkv=8, Dh=128, N=200, k=64, W=128, fill=100)
    # a selection running beside them
    rng = np.random.default_rng(13)
    keys = rng.standard_normal((4, 3000, 64)).astype(np.float32)
    qv = np.zeros((4, 64), np.float32)
    for b in range(4):
        while True:
            q = rng.standard_normal(64).astype(np.float32)
            if orc.select(keys[b:b + 1], q[None], 100)[2][0] >= 1e-3:
                break
        qv[b] = q
    ref_idx = orc.select(keys, qv, 100)[0]
    d_keys, d_qv = to_dev(keys), to_dev(qv)
    idx = torch.empty((4, 100), dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()

    s1, s2, s3 = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    say("streams: interleaving a split-plan decode, an 8-wave decode and a selection")
    for t in range(STEPS):
        with torch.cuda.stream(s1):
            split.step(t)
        with torch.cuda.stream(s2):
            wide.step(t)
        if t == 1:
            with torch.cuda.stream(s3):
                cmc.cmc_select_cmes(d_keys, d_qv, 100, idx_out=idx)
    torch.cuda.synchronize()
    split.check()
    wide.check()
    assert (to_host(idx) == ref_idx).all()
