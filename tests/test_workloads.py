"""The seeded generator: determinism, slicing, bf16 rounding."""
import numpy as np
import torch

from paper_2609_25537_amd import workloads as wl
from tests.inputs import accepted_attempts


def test_bf16_round_to_nearest_even_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10 ** rng.uniform(-6, 6),
                        np.array([1.0, -1.0, 0.0, -0.0, 1.00390625, 1.005859375], np.float32)])
    x = x.astype(np.float32)
    ours = wl.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (ours == ref).all()
    back = wl.bf16_bits_to_f32(ours)
    assert (torch.from_numpy(back) == torch.from_numpy(x).to(torch.bfloat16).float()).all()


def test_deterministic_and_sliceable():
    w = wl.get("tiny_fp32").replace(B=2, Hkv=2, Hq=4)
    K1, V1 = wl.pool_kv(w)
    K2, V2 = wl.pool_kv(w)
    assert (K1 == K2).all() and (V1 == V2).all()
    kb, vb = wl.pool_kv(w, b=1, h=1)
    assert (kb == K1[1, 1]).all() and (vb == V1[1, 1]).all()
    assert (wl.sel_keys(w, 1) == wl.sel_keys(w)[1]).all()
    assert not (wl.q_vec(w, 0, 0) == wl.q_vec(w, 0, 1)).all()
    q0 = wl.step_q(w, 3)
    assert q0.shape == (2, 4, 64) and (q0 == wl.step_q(w, 3)).all()


def test_window_fill_and_bf16_shapes():
    w = wl.get("tiny_fp32").replace(kv_dtype="bf16", W=8)
    wk, wv, cnt = wl.window_kv(w, fill=3)
    assert wk.dtype == np.uint16 and wk.shape == (1, 4, 8, 64)
    assert (cnt == 3).all() and not wk[:, :, 3:].any()
    nk, nv = wl.step_new_kv(w, 0, t_new=2)
    assert nk.shape == (1, 4, 2, 64) and nk.dtype == np.uint16


def test_lognormal_channel_scale():
    w = wl.get("long_wide_d256").replace(B=1, Hq=2, Hkv=2, N=64)
    s = wl.chan_scale(w)
    assert s.shape == (2, 256) and (s > 0).all()
    K, _ = wl.pool_kv(w)
    Kf = wl.kv_to_f32(w, K)
    # per-channel spread follows the scale
    ratio = Kf[0, 0].std(axis=0) / s[0]
    assert 0.6 < np.median(ratio) < 1.4


def test_tiny_gap_rule(orc):
    w = wl.get("tiny_fp32")
    att = accepted_attempts(w, orc)
    _, _, gap = orc.select(wl.sel_keys(w), wl.q_vecs(w, att), w.k)
    assert (gap >= w.gap_min).all()
