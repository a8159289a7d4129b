"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times (selection, the selected rows gathered once, one
cmc_decode_step per step reading them with idx == NULL, the library's own
split plan): selection bit-exact for every sequence, then all decode steps run on
the GPU while the oracle advances its own ring every step and recomputes the
attention at sampled steps -- the first ones, those around the ring wrap,
and the last."""
import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, max_abs, say, to_dev, to_host, tol_for
from tests.inputs import accepted_attempts

pytestmark = pytest.mark.gpu


def _run_full(orc, name, sample_extra=(), gathered=True):
    w = wl.get(name)
    say(f"{name}: generating inputs")
    att = accepted_attempts(w, orc)
    keys, qv = wl.sel_keys(w), wl.q_vecs(w, att)
    ref_idx, _, gap = orc.select(keys, qv, w.k)
    assert (gap >= w.gap_min).all()
    say(f"{name}: select on GPU")
    idx = cmc.cmc_select_cmes(to_dev(keys), to_dev(qv), w.k)
    torch.cuda.synchronize()
    assert (to_host(idx) == ref_idx).all(), "selected index sets differ"
    del keys
    pk, pv = wl.pool_kv(w)
    wk, wv, cnt = wl.window_kv(w)
    d_pk, d_pv, d_wk, d_wv, d_wc = map(to_dev, (pk, pv, wk, wv, cnt))
    if gathered:
        # The benchmark's configuration: the selected rows gathered once into
        # contiguous blocks, the decode reading them with idx == NULL.
        d_pk, d_pv = cmc.cmc_gather_tier1(d_pk, d_pv, idx, w.k)
        dec_idx = None
    else:
        dec_idx = idx
    ws = cmc.decode_workspace(w.B, w.Hq, w.Hkv, w.Dh, w.k, w.W, DEV)
    out = torch.empty((w.B, w.Hq, w.Dh), dtype=torch.float32, device=DEV)
    samples = sorted({0, 1, w.W - 1, w.W, w.W + 1, w.steps - 1, *sample_extra})
    worst = 0.0
    for t in range(w.steps):
        nk, nv = wl.step_new_kv(w, t)
        orc.window_append(wk, wv, cnt, nk, nv)
        sampled = t in samples
        q = wl.step_q(w, t) if sampled else None
        d_q = to_dev(q) if sampled else to_dev(np.zeros((w.B, w.Hq, w.Dh), np.float32))
        cmc.cmc_decode_step(d_q, d_pk, d_pv, dec_idx, w.k, d_wk, d_wv, d_wc, to_dev(nk), to_dev(nv), w.scale,
                            out=out, workspace=ws)
        if sampled:
            say(f"{name}: step {t}")
            ref = orc.two_tier_decode(q, pk, pv, ref_idx, w.k, wk, wv, cnt, w.W, w.scale)
            torch.cuda.synchronize()
            err = max_abs(to_host(out), ref)
            worst = max(worst, err)
            assert err <= tol_for(w.kv_dtype), f"step {t}: max abs err {err:.3e}"
    torch.cuda.synchronize()
    assert (to_host(d_wc) == cnt).all()
    assert (to_host(d_wk) == wk).all() and (to_host(d_wv) == wv).all(), "ring contents after all steps"
    say(f"{name}: worst max-abs error {worst:.3e}")


@pytest.mark.timeout(300)
def test_full_llama3_8b_layer(orc):
    _run_full(orc, "llama3_8b_layer", sample_extra=(2, 100, 1500))


@pytest.mark.timeout(300)
def test_full_llama3_8b_layer_index_list(orc):
    """The same workload decoding straight from the pool through idx."""
    _run_full(orc, "llama3_8b_layer", gathered=False)


@pytest.mark.timeout(600)
def test_full_mistral7b_batch64(orc):
    _run_full(orc, "mistral7b_batch64")


@pytest.mark.timeout(900)
def test_full_long_wide_d256(orc):
    _run_full(orc, "long_wide_d256")


@pytest.mark.timeout(900)
def test_full_paper_scale_b8(orc):
    """The paper's own cache sizes (B = 8, K = 40, W = 130, N = 768) with
    Llama heads: k and W not multiples of the 16-row block, a split plan."""
    _run_full(orc, "paper_scale_b8")


@pytest.mark.timeout(900)
def test_full_llama_stack32_layer(orc):
    """One layer of the 32-layer stack's shape (B=32, 256 (sequence, kv
    head) pairs: one 8-wave workgroup each) from the numpy streams; the
    stack benchmark draws its 32 layers on the device instead."""
    _run_full(orc, "llama_stack32")
