"""HIP-graph replay of the paths bench.py times equals eager execution.

bench.py captures a whole pass (selection, gather, decode steps with the
fused ring append) and the denoising and MemoryBridge calls in HIP graphs and
replays them.  Here each graph is replayed several times, with eager work and
synchronisations between the replays, and every replay is compared bit for
bit with the same calls run eagerly from the same starting state (the kernels
are deterministic).  The decode pass changes the ring on every replay, so
each replay is checked against its own eager run.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, say, to_dev

pytestmark = pytest.mark.gpu

REPLAYS = 4


def _eager_noise():
    """Unrelated eager work on the same stream between replays."""
    a = torch.randn(256, 256, device=DEV)
    (a @ a).sum().item()
    torch.cuda.synchronize()


def _capture(fn):
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


class _Pass:
    """Device state of one decode pass: selection keys and pool, the ring,
    per-step queries and appended rows, outputs and workspaces."""

    def __init__(self, rng, B, Hq, Hkv, Dh, N, D, k, W, fill, steps):
        self.B, self.Hq, self.Hkv, self.Dh, self.k, self.W, self.steps = B, Hq, Hkv, Dh, k, W, steps
        f = lambda *s: rng.standard_normal(s).astype(np.float32)
        bf = lambda x: to_dev(wl.f32_to_bf16_bits(x))
        self.keys, self.qv = to_dev(f(B, N, D)), to_dev(f(B, D))
        self.pk, self.pv = bf(f(B, Hkv, N, Dh) / 8), bf(f(B, Hkv, N, Dh) / 8)
        wk, wv = np.zeros((B, Hkv, W, Dh), np.float32), np.zeros((B, Hkv, W, Dh), np.float32)
        wk[:, :, :fill], wv[:, :, :fill] = f(B, Hkv, fill, Dh) / 8, f(B, Hkv, fill, Dh) / 8
        self.wk, self.wv = bf(wk), bf(wv)
        self.wc = to_dev(np.full((B,), fill, np.int32))
        self.q = [to_dev(f(B, Hq, Dh)) for _ in range(steps)]
        self.nk = [bf(f(B, Hkv, 1, Dh) / 8) for _ in range(steps)]
        self.nv = [bf(f(B, Hkv, 1, Dh) / 8) for _ in range(steps)]
        self._outputs()

    def _outputs(self):
        B, Hkv, Dh, k = self.B, self.Hkv, self.Dh, self.k
        self.idx = torch.empty((B, k), dtype=torch.int32, device=DEV)
        self.gk = torch.empty((B, Hkv, k, Dh), dtype=torch.bfloat16, device=DEV)
        self.gv = torch.empty_like(self.gk)
        self.out = [torch.empty((B, self.Hq, Dh), dtype=torch.float32, device=DEV) for _ in range(self.steps)]
        N = self.keys.shape[1]
        self.sel_ws = torch.empty(max(1, cmc.cmc_select_workspace_bytes(B, N)), dtype=torch.uint8, device=DEV)
        self.dec_ws = cmc.decode_workspace(B, self.Hq, Hkv, Dh, k, self.W, DEV)

    def fork(self):
        """Same inputs and ring state, own ring copies, outputs and workspaces."""
        o = object.__new__(_Pass)
        o.__dict__.update(self.__dict__)
        o.wk, o.wv, o.wc = self.wk.clone(), self.wv.clone(), self.wc.clone()
        o._outputs()
        return o

    def run(self):
        scale = 1.0 / math.sqrt(self.Dh)
        cmc.cmc_select_cmes(self.keys, self.qv, self.k, idx_out=self.idx, workspace=self.sel_ws)
        cmc.cmc_gather_tier1(self.pk, self.pv, self.idx, self.k, out_k=self.gk, out_v=self.gv)
        for j in range(self.steps):
            cmc.cmc_decode_step(self.q[j], self.gk, self.gv, None, self.k, self.wk, self.wv, self.wc,
                                self.nk[j], self.nv[j], scale, out=self.out[j], workspace=self.dec_ws)


@pytest.mark.parametrize("B,Hq,Hkv,Dh,N,D,k,W,fill", [
    (2, 8, 2, 128, 300, 256, 64, 48, 40),     # split plan: a few pairs, ring wraps during the replays
    (48, 16, 4, 128, 200, 128, 32, 40, 40),   # 192 pairs: one 8-wave workgroup per pair
])
def test_decode_pass_graph(B, Hq, Hkv, Dh, N, D, k, W, fill):
    say(f"graph decode pass B={B} Hq={Hq} Hkv={Hkv} Dh={Dh} N={N} k={k} W={W}")
    live = _Pass(np.random.default_rng(B * 1000 + W), B, Hq, Hkv, Dh, N, D, k, W, fill, steps=3)
    g = _capture(live.run)  # capture runs nothing: the state is still the initial one
    for r in range(REPLAYS):
        ref = live.fork()
        ref.run()
        torch.cuda.synchronize()
        _eager_noise()
        g.replay()
        torch.cuda.synchronize()
        say(f"  replay {r}")
        assert torch.equal(live.idx, ref.idx), f"replay {r}: selected rows"
        assert torch.equal(live.gk, ref.gk) and torch.equal(live.gv, ref.gv), f"replay {r}: gathered rows"
        for j in range(live.steps):
            assert torch.equal(live.out[j], ref.out[j]), f"replay {r}, step {j}: decode output"
        assert torch.equal(live.wk, ref.wk) and torch.equal(live.wv, ref.wv), f"replay {r}: ring contents"
        assert torch.equal(live.wc, ref.wc), f"replay {r}: ring count"
        assert int(live.wc[0]) == fill + 3 * (r + 1)
        assert not live.dec_ws[:4 * (B + B * Hkv)].any(), f"replay {r}: arrival counters re-armed"


def test_bridge_graph():
    say("graph memory bridge")
    rng = np.random.default_rng(11)
    M, Hc, F, Hd = 600, 128, 512, 256  # 256 x 256 tiles for both layers
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    bf = lambda x: to_dev(wl.f32_to_bf16_bits(x))
    h, w1, w2 = bf(f(M, Hc)), bf(f(F, Hc) / math.sqrt(Hc)), bf(f(Hd, F) / math.sqrt(F))
    b1, b2 = to_dev(f(F) * 0.1), to_dev(f(Hd) * 0.1)
    gamma, beta = to_dev(1 + 0.1 * f(Hd)), to_dev(0.1 * f(Hd))
    out = torch.empty((M, Hd), dtype=torch.float32, device=DEV)
    ws = torch.empty(cmc.cmc_bridge_workspace_bytes(M, F), dtype=torch.uint8, device=DEV)
    call = lambda o, w: cmc.cmc_memory_bridge(h, w1, b1, w2, b2, gamma, beta, nu=0.9, out=o, workspace=w)
    ref = torch.empty_like(out)
    ref_ws = torch.empty_like(ws)
    call(ref, ref_ws)
    torch.cuda.synchronize()
    g = _capture(lambda: call(out, ws))
    for r in range(REPLAYS):
        out.fill_(float("nan"))
        _eager_noise()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {r}: output"
        assert torch.equal(ws, ref_ws), f"replay {r}: hidden activations"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_denoise_graph(dtype):
    say(f"graph denoise {dtype}")
    rng = np.random.default_rng(12)
    B, n, H = 3, 700, 256
    x = rng.standard_normal((B, n, H)).astype(np.float32)
    x[:, 1::2] = x[:, 0:-1:2] + 0.1 * x[:, 1::2]  # neighbours that pass the threshold
    emb = to_dev(wl.f32_to_bf16_bits(x)) if dtype == "bf16" else to_dev(x)
    n_tok = to_dev(np.array([700, 517, 3], np.int32))

    def outputs():
        return dict(max_cos_out=torch.empty((B, n), dtype=torch.float32, device=DEV),
                    keep_out=torch.empty((B, n), dtype=torch.uint8, device=DEV),
                    kept_idx=torch.empty((B, n), dtype=torch.int32, device=DEV),
                    kept_count=torch.empty((B,), dtype=torch.int32, device=DEV),
                    chunk_offset=torch.empty((B, -(-n // 64)), dtype=torch.int32, device=DEV),
                    n_chunks_out=torch.empty((B,), dtype=torch.int32, device=DEV),
                    workspace=torch.empty(max(1, cmc.cmc_denoise_workspace_bytes(B, n)), dtype=torch.uint8,
                                          device=DEV))

    call = lambda o: cmc.cmc_denoise(emb, g=3, tau=0.5, keep_min_every=16, n_tokens=n_tok, chunk_tokens=64, **o)
    ref, live = outputs(), outputs()
    call(ref)
    torch.cuda.synchronize()
    g = _capture(lambda: call(live))
    for r in range(REPLAYS):
        for t in live.values():
            t.zero_()
        _eager_noise()
        g.replay()
        torch.cuda.synchronize()
        for name in ("max_cos_out", "keep_out", "kept_idx", "kept_count", "chunk_offset", "n_chunks_out"):
            a, b = live[name], ref[name]
            if name == "kept_idx":  # entries past each sequence's count are unspecified
                for s in range(B):
                    c = int(ref["kept_count"][s])
                    assert torch.equal(a[s, :c], b[s, :c]), f"replay {r}: kept_idx[{s}]"
            elif name == "chunk_offset":
                for s in range(B):
                    c = int(ref["n_chunks_out"][s])
                    assert torch.equal(a[s, :c], b[s, :c]), f"replay {r}: chunk_offset[{s}]"
            else:
                assert torch.equal(a, b), f"replay {r}: {name}"
