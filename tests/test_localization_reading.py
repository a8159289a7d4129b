"""Why CME-guided localization ranks the encoder CMEs' norms, shown with the
oracle on the MemoryBridge workload (CPU only).

Sec. 2.3's cap multiplies nu*tanh(m_hat) by min(1, 2 nu / ||nu*tanh(m_hat)||),
so every memory row whose nu*tanh(m_hat) is longer than 2 nu leaves the
bridge with norm exactly 2 nu.  At the decoder width of the workload (4096)
that is every row: the norms of the bridge output tie, and an argmax over them
would be decided by rounding.  The CME vectors h themselves (the encoder's
hidden states at the placeholder positions, Sec. 2.2) have distinct norms.
"""
import numpy as np

from paper_2609_25537_amd import workloads as wl

# 16 CMEs spread over the first context's 12 chunks of the bridge workload
_ROWS = list(range(0, 768, 48))


def _inputs():
    w = wl.BRIDGE_WORKLOADS["bridge_gpt2l_llama3_batch64"]
    return w, wl.bridge_h(w, _ROWS), wl.bridge_params(w)


def test_post_cap_norms_tie_at_two_nu(orc):
    w, h, p = _inputs()
    out = orc.memory_bridge(h, p["w1"], p["b1"], p["w2"], p["b2"], p["gamma"], p["beta"], w.nu, w.eps)
    n_out = np.linalg.norm(out, axis=1)
    assert np.all(np.abs(n_out - 2.0 * w.nu) <= 1e-12 * 2.0 * w.nu), n_out
    # in fp32 (what a kernel would rank) those norms are 2 nu to within a few ulps: no ranking
    n32 = np.linalg.norm(out.astype(np.float32).astype(np.float64), axis=1)
    assert np.all(np.abs(n32 - 2.0 * w.nu) <= 4 * np.finfo(np.float32).eps * 2.0 * w.nu)
    # the encoder CME vectors' norms are spread out and rank the rows
    n_h = orc.row_norms(h)
    assert n_h.max() - n_h.min() > 1.0, n_h
    assert len(np.unique(n_h)) == len(_ROWS)


def test_cap_binds_on_every_row(orc):
    """The cap binds because ||nu*tanh(m_hat)|| is far above 2 nu: a
    LayerNorm output of about unit variance gives E tanh^2 ~ 0.39, so about
    nu*sqrt(0.39*4096) ~ 40 nu.  m_hat is formed here with numpy from the
    oracle's fp64 hidden layer (Linear, then nn.LayerNorm semantics: biased
    variance, eps inside the root), and the oracle's output is that row
    scaled to norm 2 nu."""
    w, h, p = _inputs()
    hidden = orc.bridge_hidden(h, p["w1"], p["b1"])
    w2 = (p["w2"].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    y = hidden @ w2.T + p["b2"].astype(np.float64)
    mu = y.mean(axis=1, keepdims=True)
    var = ((y - mu) ** 2).mean(axis=1, keepdims=True)
    m_hat = p["gamma"].astype(np.float64) * (y - mu) / np.sqrt(var + w.eps) + p["beta"].astype(np.float64)
    t = w.nu * np.tanh(m_hat)
    tn = np.linalg.norm(t, axis=1)
    assert np.all(tn > 20.0 * w.nu), tn
    out = orc.bridge_out(hidden, p["w2"], p["b2"], p["gamma"], p["beta"], w.nu, w.eps)
    assert np.max(np.abs(out - t * (2.0 * w.nu / tn)[:, None])) < 1e-9
