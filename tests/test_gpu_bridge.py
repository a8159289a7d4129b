"""MemoryBridge on the GPU vs the oracle, through the C ABI, in two stages
decided on the same values: the hidden activations the kernel leaves in
its workspace (bf16) against the oracle's fp64 GELU layer, within bf16
rounding plus the fp32 accumulation bound; then the output against the
oracle's second stage run on those same bf16 activations, within a
first-order fp32 error bound carried through the output GEMM, LayerNorm,
tanh and the cap."""
import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, say, to_dev, to_host

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def _gamma(n):
    return n * U / (1 - n * U)


def _vals(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _stage1_tol(h, w1, b1, ref):
    acc = np.abs(_vals(h)) @ np.abs(_vals(w1)).T + np.abs(b1.astype(np.float64))
    return 2.0 ** -8 * np.abs(ref) * (1 + 1e-6) + 1.13 * (_gamma(h.shape[1] + 1) * acc + 4 * U * np.abs(acc)) + 1e-30


def _stage2_tol(hid, w2, b2, gamma, beta, nu, eps):
    """First-order bound on |fp32 result - exact result| per element."""
    W = _vals(w2)
    F, Hd = hid.shape[1], W.shape[0]
    y = hid @ W.T + b2
    e_y = _gamma(F + 1) * (np.abs(hid) @ np.abs(W).T + np.abs(b2))
    mu = y.mean(1, keepdims=True)
    d = y - mu
    e_mu = e_y.mean(1, keepdims=True) + _gamma(Hd) * np.abs(y).mean(1, keepdims=True)
    e_d = e_y + e_mu + U * np.abs(d)
    var = (d * d).mean(1, keepdims=True)
    e_var = (2 * np.abs(d) * e_d + e_d ** 2).mean(1, keepdims=True) + _gamma(Hd + 1) * var
    inv = 1 / np.sqrt(var + eps)
    rel_inv = e_var / (2 * (var + eps)) + 3 * U
    g = np.abs(gamma.astype(np.float64))
    m_hat = gamma * d * inv + beta
    e_m = g * (e_d * inv + np.abs(d) * inv * rel_inv) + 3 * U * (np.abs(m_hat) + np.abs(beta))
    t = nu * np.tanh(m_hat)
    e_t = nu * e_m + nu * 4 * U + U * np.abs(t)
    n = np.linalg.norm(t, axis=1, keepdims=True)
    e_n = np.linalg.norm(e_t, axis=1, keepdims=True) + _gamma(Hd + 1) * n
    c = np.minimum(1.0, 2 * nu / n)
    e_c = np.where(2 * nu / n < 1.0, c * e_n / n + 2 * U * c, 0.0)
    return 2.0 * (e_t * c + np.abs(t) * e_c + U * np.abs(t * c)) + 1e-9 * nu


def _run(orc, h, p, nu, eps=1e-5, rows=None, what=""):
    """Bridge on the GPU; checks the given rows (all by default)."""
    M, Hc = h.shape
    F, Hd = p["w1"].shape[0], p["w2"].shape[0]
    say(f"bridge {what}: M={M} Hc={Hc} F={F} Hd={Hd} nu={nu}")
    bf = lambda a: to_dev(np.ascontiguousarray(a))
    ws = torch.empty(cmc.cmc_bridge_workspace_bytes(M, F), dtype=torch.uint8, device=DEV)
    out = cmc.cmc_memory_bridge(bf(h), bf(p["w1"]), to_dev(p["b1"]), bf(p["w2"]), to_dev(p["b2"]),
                                to_dev(p["gamma"]), to_dev(p["beta"]), nu, eps, workspace=ws)
    torch.cuda.synchronize()
    sel = np.arange(M) if rows is None else np.asarray(rows)
    hid_bits = to_host(ws[:M * F * 2].view(torch.int16)).view(np.uint16).reshape(M, F)[sel]
    got = to_host(out)[sel].astype(np.float64)
    ref_h = orc.bridge_hidden(h[sel], p["w1"], p["b1"])
    err1 = np.abs(_vals(hid_bits) - ref_h)
    tol1 = _stage1_tol(h[sel], p["w1"], p["b1"], ref_h)
    assert (err1 <= tol1).all(), f"hidden: worst excess {np.max(err1 - tol1):.3e}"
    hid = _vals(hid_bits)
    ref = orc.bridge_out(hid, p["w2"], p["b2"], p["gamma"], p["beta"], nu, eps)
    tol2 = _stage2_tol(hid, p["w2"], p["b2"].astype(np.float64), p["gamma"].astype(np.float64),
                       p["beta"].astype(np.float64), nu, eps)
    err2 = np.abs(got - ref)
    assert np.isfinite(got).all()
    assert (err2 <= tol2).all(), f"out: worst excess {np.max(err2 - tol2):.3e} (max err {err2.max():.3e})"
    assert (np.abs(got) <= nu * (1 + 1e-6)).all()
    assert (np.linalg.norm(got, axis=1) <= 2 * nu * (1 + 1e-5)).all()
    return float(err2.max())


def _params(rng, Hc, F, Hd, gamma_scale=1.0):
    f = lambda *s: rng.standard_normal(s).astype(np.float32)
    return {"w1": wl.f32_to_bf16_bits(f(F, Hc) / np.float32(np.sqrt(Hc))),
            "w2": wl.f32_to_bf16_bits(f(Hd, F) / np.float32(np.sqrt(F))),
            "b1": f(F) * np.float32(0.02), "b2": f(Hd) * np.float32(0.02),
            "gamma": (np.float32(gamma_scale) * (1 + 0.1 * f(Hd))).astype(np.float32),
            "beta": f(Hd) * np.float32(0.1 * gamma_scale)}


@pytest.mark.parametrize("M,Hc,F,Hd", [
    (1, 64, 128, 128), (129, 64, 128, 256), (300, 128, 256, 128), (256, 1280, 512, 384), (77, 192, 128, 1024),
    (40, 64, 256, 256), (513, 64, 512, 256), (1000, 192, 768, 512),
])
def test_bridge_shapes(orc, M, Hc, F, Hd):
    """Tile edges: M not a multiple of 128 or 256, several N and K tiles,
    and K of two 32-wide slices (fewer slices than the pipeline's stages)."""
    rng = np.random.default_rng(M + Hc + F + Hd)
    h = wl.f32_to_bf16_bits(rng.standard_normal((M, Hc)).astype(np.float32))
    _run(orc, h, _params(rng, Hc, F, Hd), nu=0.8, what="shapes")


def test_bridge_more_tiles_than_cus(orc):
    """More 256 x 256 tiles than CUs (33 x 8 = 264 for the first layer), so
    workgroups of a persistent grid take several tiles; every row checked."""
    rng = np.random.default_rng(8)
    M, Hc, F, Hd = 8192 + 77, 64, 2048, 512
    h = wl.f32_to_bf16_bits(rng.standard_normal((M, Hc)).astype(np.float32))
    _run(orc, h, _params(rng, Hc, F, Hd), nu=0.8, what="many tiles")


@pytest.mark.parametrize("gamma_scale,nu", [(0.02, 1.0), (0.2, 0.5), (3.0, 2.0)])
def test_bridge_cap_regimes(orc, gamma_scale, nu):
    """Small LayerNorm outputs (cap inactive), rows near the cap, saturated
    tanh (every row capped)."""
    rng = np.random.default_rng(int(gamma_scale * 100))
    h = wl.f32_to_bf16_bits(rng.standard_normal((200, 64)).astype(np.float32))
    _run(orc, h, _params(rng, 64, 128, 128, gamma_scale), nu=nu, what=f"gamma x{gamma_scale}")


def test_bridge_large_inputs(orc):
    """Inputs with a wide dynamic range (rows scaled by 2^-6 .. 2^6)."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((256, 256)).astype(np.float32)
    x *= np.float32(2.0) ** rng.integers(-6, 7, size=(256, 1)).astype(np.float32)
    _run(orc, wl.f32_to_bf16_bits(x), _params(rng, 256, 256, 256), nu=1.5, what="range")


def test_bridge_deterministic():
    rng = np.random.default_rng(6)
    h = to_dev(wl.f32_to_bf16_bits(rng.standard_normal((500, 128)).astype(np.float32)))
    p = _params(rng, 128, 256, 256)
    args = [to_dev(p[k]) for k in ("w1", "b1", "w2", "b2", "gamma", "beta")]
    a = cmc.cmc_memory_bridge(h, *args, nu=1.0)
    b = cmc.cmc_memory_bridge(h, *args, nu=1.0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.timeout(600)
def test_full_bridge_workload(orc):
    """The benchmark's workload at full size (49152 CME vectors, 1280 ->
    4096 -> 4096), in its launch configuration; the oracle checks 64 rows
    (the first and last tiles' edges and random rows)."""
    w = wl.BRIDGE_WORKLOADS["bridge_gpt2l_llama3_batch64"]
    say(f"{w.name}: generating inputs")
    h = wl.bridge_h(w)
    p = wl.bridge_params(w)
    rng = np.random.default_rng(0)
    rows = sorted({0, 1, 127, 128, w.M - 129, w.M - 1, *rng.integers(0, w.M, size=58).tolist()})
    err = _run(orc, h, p, nu=w.nu, eps=w.eps, rows=rows, what=w.name)
    say(f"{w.name}: max abs error {err:.3e} on {len(rows)} rows")
