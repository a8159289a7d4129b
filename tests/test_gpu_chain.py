"""The MemoryBridge and Tier-1 selection composed on the GPU, against the
oracle's own chain.

The bridge turns each context's CME vectors into decoder-ready memory rows
(Sec. 2.3); those rows are the keys Tier-1 selection scores against the
question embedding (Sec. 2.5, Tier-1 paragraph and its score equation).  The
GPU chain is cmc_memory_bridge -> cmc_select_cmes on its fp32 output; the
oracle chain is its fp64 hidden layer rounded to bf16 (the reading that the
hidden activations are held as bf16) -> its fp64 output layer, LayerNorm and
cap -> its selection on those rows.  Each sequence's question vector is drawn
until the oracle chain's k-th and (k+1)-th scores are at least 1e-3 apart
(relative), the rule every selection parity case uses; the index sets must
then be bit-exact, and the scores agree to well within that gap.  Nothing is
staged through the other side's intermediate values."""
import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, say, to_dev, to_host

pytestmark = pytest.mark.gpu

GAP_MIN = 1e-3


def _params(rng, Hc, F, Hd):
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    return {"w1": wl.f32_to_bf16_bits(f(F, Hc) / np.float32(np.sqrt(Hc))),
            "w2": wl.f32_to_bf16_bits(f(Hd, F) / np.float32(np.sqrt(F))),
            "b1": f(F) * np.float32(0.02), "b2": f(Hd) * np.float32(0.02),
            "gamma": (1 + 0.1 * f(Hd)).astype(np.float32),
            "beta": f(Hd) * np.float32(0.1)}


@pytest.mark.parametrize("B,N,Hc,F,Hd,k,nu", [
    (4, 512, 256, 512, 1024, 64, 1.0),
    (3, 1000, 128, 256, 512, 100, 0.7),
    (2, 2048, 64, 384, 256, 256, 1.5),
])
def test_bridge_then_select(orc, B, N, Hc, F, Hd, k, nu):
    rng = np.random.default_rng(B * 1000 + N + Hd)
    M = B * N
    h = wl.f32_to_bf16_bits(rng.standard_normal((M, Hc)).astype(np.float32))
    p = _params(rng, Hc, F, Hd)
    say(f"bridge -> select: B={B} N={N} Hc={Hc} F={F} Hd={Hd} k={k}")

    # oracle chain
    hid = orc.bridge_hidden(h, p["w1"], p["b1"])
    hid_bf16 = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(hid.astype(np.float32))).astype(np.float64)
    rows = orc.bridge_out(hid_bf16, p["w2"], p["b2"], p["gamma"], p["beta"], nu)
    keys_ref = rows.astype(np.float32).reshape(B, N, Hd)
    qv = np.zeros((B, Hd), np.float32)
    for b in range(B):
        for attempt in range(500):
            q = rng.standard_normal(Hd).astype(np.float32)
            if orc.select(keys_ref[b:b + 1], q[None], k)[2][0] >= GAP_MIN:
                break
        else:
            pytest.fail(f"sequence {b}: no question vector with a clear k-th gap")
        qv[b] = q
    ref_idx, ref_scores, gap = orc.select(keys_ref, qv, k)
    assert (gap >= GAP_MIN).all()

    # GPU chain
    bf = lambda a: to_dev(np.ascontiguousarray(a))
    ws = torch.empty(cmc.cmc_bridge_workspace_bytes(M, F), dtype=torch.uint8, device=DEV)
    out = cmc.cmc_memory_bridge(bf(h), bf(p["w1"]), to_dev(p["b1"]), bf(p["w2"]), to_dev(p["b2"]),
                                to_dev(p["gamma"]), to_dev(p["beta"]), nu, workspace=ws)
    scores = torch.empty((B, N), dtype=torch.float32, device=DEV)
    idx = cmc.cmc_select_cmes(out.view(B, N, Hd), to_dev(qv), k, scores_out=scores)
    torch.cuda.synchronize()

    got_idx = to_host(idx)
    got_scores = to_host(scores).astype(np.float64)
    score_err = float(np.max(np.abs(got_scores - ref_scores)))
    say(f"bridge -> select: max score difference {score_err:.2e}, smallest gap {gap.min():.2e}")
    assert (got_idx == ref_idx).all(), "selected index sets differ"
    # the chain's score error stays under half the k-th gap the index sets rely on
    top = -np.sort(-ref_scores, axis=1)
    abs_gap = top[:, k - 1] - top[:, k]
    assert (np.abs(got_scores - ref_scores).max(axis=1) < 0.5 * abs_gap).all()
