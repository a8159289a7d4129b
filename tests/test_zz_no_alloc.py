"""cmc_decode_step_noalloc (the decode step whose counters and split partials
live in the library's fixed scratch array) against cmc_decode_step with a
workspace, through the C ABI: two calls in a row, the second on a smaller
input, then the first shape again; outputs, ring contents and counts must be
bit-identical to the workspace path's (same kernels and plan), and within the
bf16 bar of the oracle."""
import math

import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, max_abs, say, to_dev, to_host, tol_for

pytestmark = pytest.mark.gpu


def _case(seed, B, Hq, Hkv, Dh, N, k, W, fill):
    rng = np.random.default_rng(seed)
    f = lambda *s: wl.f32_to_bf16_bits((rng.standard_normal(s) / math.sqrt(Dh)).astype(np.float32))
    wk = np.zeros((B, Hkv, W, Dh), np.uint16)
    wv = np.zeros((B, Hkv, W, Dh), np.uint16)
    wk[:, :, :fill], wv[:, :, :fill] = f(B, Hkv, fill, Dh), f(B, Hkv, fill, Dh)
    return dict(q=(rng.standard_normal((B, Hq, Dh)) / math.sqrt(Dh)).astype(np.float32),
                pk=f(B, Hkv, N, Dh), pv=f(B, Hkv, N, Dh),
                idx=np.stack([np.sort(rng.choice(N, size=k, replace=False)) for _ in range(B)]).astype(np.int32),
                wk=wk, wv=wv, cnt=np.full((B,), fill, np.int32), nk=f(B, Hkv, 1, Dh), nv=f(B, Hkv, 1, Dh),
                k=k, W=W, scale=1.0 / math.sqrt(Dh))


def _both(orc, c, what):
    say(f"noalloc {what}: q {c['q'].shape} k={c['k']} W={c['W']}")
    dev = {n: to_dev(c[n]) for n in ("q", "pk", "pv", "idx", "nk", "nv")}
    ring_a = [to_dev(c["wk"]), to_dev(c["wv"]), to_dev(c["cnt"])]
    ring_b = [to_dev(c["wk"]), to_dev(c["wv"]), to_dev(c["cnt"])]
    out_a = cmc.cmc_decode_step(dev["q"], dev["pk"], dev["pv"], dev["idx"], c["k"], *ring_a, dev["nk"], dev["nv"],
                                c["scale"])
    out_b = torch.empty_like(out_a)
    cmc.cmc_decode_step_noalloc(dev["q"], dev["pk"], dev["pv"], dev["idx"], c["k"], *ring_b, dev["nk"], dev["nv"],
                                c["scale"], out=out_b)
    torch.cuda.synchronize()
    wk, wv, cnt = c["wk"].copy(), c["wv"].copy(), c["cnt"].copy()
    orc.window_append(wk, wv, cnt, c["nk"], c["nv"])
    ref = orc.two_tier_decode(c["q"], c["pk"], c["pv"], c["idx"], c["k"], wk, wv, cnt, c["W"], c["scale"])
    assert torch.equal(out_a, out_b), f"{what}: outputs differ from the workspace path"
    assert max_abs(to_host(out_b), ref) <= tol_for("bf16"), what
    for x, y in zip(ring_a, ring_b):
        assert torch.equal(x, y), f"{what}: ring state differs"
    assert (to_host(ring_b[2]) == cnt).all() and (to_host(ring_b[0]) == wk).all()


def test_noalloc_matches_workspace_path(orc):
    # the Llama-layer shape (13 splits + the appended rows' split: partials in the scratch), then a smaller
    # input (fewer pairs, a shorter key list), then the first shape again
    big = _case(1, B=1, Hq=32, Hkv=8, Dh=128, N=2048, k=256, W=512, fill=512)
    small = _case(2, B=2, Hq=8, Hkv=2, Dh=128, N=100, k=40, W=60, fill=33)
    _both(orc, big, "first call, Llama-layer shape")
    _both(orc, small, "second call, smaller input")
    _both(orc, big, "third call, first shape again")


def test_noalloc_under_graph_capture(orc):
    """The callers it is for: three fused decode steps captured into a HIP
    graph (after one set-up call outside capture), the graph replayed four
    times with eager work in between; after every replay the outputs and the
    ring equal the same three steps run eagerly through cmc_decode_step with
    a workspace from the same state."""
    c = _case(3, B=1, Hq=32, Hkv=8, Dh=128, N=2048, k=256, W=512, fill=300)  # split plan: partials in the array
    rng = np.random.default_rng(33)
    steps = 3
    qs = [to_dev((rng.standard_normal(c["q"].shape) / 11.3).astype(np.float32)) for _ in range(steps)]
    nks = [to_dev(wl.f32_to_bf16_bits((rng.standard_normal(c["nk"].shape) / 11.3).astype(np.float32)))
           for _ in range(steps)]
    nvs = [to_dev(wl.f32_to_bf16_bits((rng.standard_normal(c["nv"].shape) / 11.3).astype(np.float32)))
           for _ in range(steps)]
    pk, pv, idx = to_dev(c["pk"]), to_dev(c["pv"]), to_dev(c["idx"])
    ring_g = [to_dev(c["wk"]), to_dev(c["wv"]), to_dev(c["cnt"])]
    ring_e = [t.clone() for t in ring_g]
    outs_g = [torch.empty((1, 32, 128), dtype=torch.float32, device=DEV) for _ in range(steps)]
    outs_e = [torch.empty_like(o) for o in outs_g]
    # set-up call outside capture (its result is discarded; the rings are re-copied below)
    scratch_ring = [t.clone() for t in ring_g]
    cmc.cmc_decode_step_noalloc(qs[0], pk, pv, idx, c["k"], *scratch_ring, nks[0], nvs[0], c["scale"],
                                out=outs_g[0])
    torch.cuda.synchronize()
    say("noalloc graph: capturing")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for t in range(steps):
            cmc.cmc_decode_step_noalloc(qs[t], pk, pv, idx, c["k"], *ring_g, nks[t], nvs[t], c["scale"],
                                        out=outs_g[t])
    torch.cuda.synchronize()
    ws = cmc.decode_workspace(1, 32, 8, 128, c["k"], c["W"], DEV)
    for r in range(4):
        say(f"noalloc graph: replay {r}")
        g.replay()
        for t in range(steps):
            cmc.cmc_decode_step(qs[t], pk, pv, idx, c["k"], *ring_e, nks[t], nvs[t], c["scale"], out=outs_e[t],
                                workspace=ws)
        torch.cuda.synchronize()
        for t in range(steps):
            assert torch.equal(outs_g[t], outs_e[t]), f"replay {r} step {t}: output"
        for x, y in zip(ring_g, ring_e):
            assert torch.equal(x, y), f"replay {r}: ring state"
        a = torch.randn(256, 256, device=DEV)
        (a @ a).sum().item()

