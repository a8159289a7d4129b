"""Graph-based context denoising on the GPU vs the oracle, through the C ABI.

The statistic (largest cosine to the next g tokens) is compared with the
oracle's fp64 values within the fp32 rounding bound of its dot products;
positions without a neighbour must be -inf on both sides.  The decisions
(Eq. 3 threshold, minimum keep interval, compaction, chunk offsets) are
integer work on that statistic, so the oracle is run on the GPU's own fp32
statistic and everything must match bit for bit."""
import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, say, to_dev, to_host

pytestmark = pytest.mark.gpu


def _stat_tol(H):
    """fp32 bound on a cosine from H-term dot products and norms: each of
    the three sums is off by at most gamma_H relative to its absolute sum,
    and |x.y| <= |x||y|, so |error| <= 3 gamma_H (+ the final roundings)."""
    u = 2.0 ** -24
    return 3.0 * H * u / (1 - H * u) + 8 * u


def _check_denoise(orc, emb, g, tau, m, n_tokens=None, chunk_tokens=0, what=""):
    B, n, H = emb.shape
    say(f"denoise {what}: B={B} n={n} H={H} dtype={emb.dtype} g={g} tau={tau} m={m} t={chunk_tokens}")
    d_emb = to_dev(emb)
    mc = torch.empty((B, n), dtype=torch.float32, device=DEV)
    keep = torch.empty((B, n), dtype=torch.uint8, device=DEV)
    nt = None if n_tokens is None else to_dev(np.asarray(n_tokens, np.int32))
    r = cmc.cmc_denoise(d_emb, g=g, tau=tau, keep_min_every=m, n_tokens=nt, chunk_tokens=chunk_tokens,
                        max_cos_out=mc, keep_out=keep)
    torch.cuda.synchronize()
    got_mc = to_host(mc).astype(np.float64)
    ref_mc = orc.denoise_scores(emb, g, n_tokens)
    assert (np.isneginf(got_mc) == np.isneginf(ref_mc)).all(), "positions without a neighbour differ"
    fin = np.isfinite(ref_mc)
    if fin.any():
        err = float(np.max(np.abs(got_mc[fin] - ref_mc[fin])))
        assert err <= _stat_tol(H), f"statistic error {err:.3e}"
    ref = orc.denoise_select(got_mc, float(np.float32(tau)), m, n_tokens, chunk_tokens)
    assert (to_host(r["kept_count"]) == ref["kept_count"]).all(), "kept counts differ"
    assert (to_host(r["kept_idx"]) == ref["kept_idx"]).all(), "kept positions differ"
    assert (to_host(keep) == ref["keep"]).all(), "keep mask differs"
    if chunk_tokens > 0:
        assert (to_host(r["chunk_offset"]) == ref["chunk_offset"]).all(), "chunk offsets differ"
        assert (to_host(r["n_chunks"]) == ref["n_chunks"]).all()
    # the same decisions without the optional outputs
    r2 = cmc.cmc_denoise(d_emb, g=g, tau=tau, keep_min_every=m, n_tokens=nt, chunk_tokens=chunk_tokens)
    torch.cuda.synchronize()
    assert (to_host(r2["kept_idx"]) == ref["kept_idx"]).all()
    return ref


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("g", [1, 2, 3, 4])
def test_denoise_neighbourhoods(orc, dtype, g):
    rng = np.random.default_rng(g)
    e = rng.standard_normal((3, 300, 64)).astype(np.float32)
    e[:, 1:] += 0.3 * e[:, :-1]
    emb = wl.f32_to_bf16_bits(e) if dtype == "bf16" else e
    _check_denoise(orc, emb, g, 0.05, 16, [300, 151, 17], chunk_tokens=7, what="neighbourhoods")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,H,n_tokens", [
    (1, 8, None), (15, 8, [15, 0]), (16, 16, [16, 1]), (17, 128, [17, 2]), (65, 40, [65, 64]),
    (1000, 1280, [1000, 999]), (9000, 16, [9000, 8193]), (200, 1288, [200, 53]),
    (26, 64, [26, 25]), (39, 96, [39, 13]), (52, 160, [52, 51]), (66, 256, [66, 14]),
])
def test_denoise_sizes(orc, dtype, n, H, n_tokens):
    """Tile edges (8 tokens per wave for fp32; 16 - g rows per wave for
    bf16, 13 at g = 3: sequences of exactly 2, 3 and 4 waves, and of 5 and
    one token), row
    widths that are not whole 32-column steps (8, 40, 1288), the last token,
    empty and one-token sequences, and sequences longer than one round of
    the selection scan (8192 positions)."""
    rng = np.random.default_rng(n + H)
    e = rng.standard_normal((2, n, H)).astype(np.float32)
    e[:, 1:] += 0.2 * e[:, :-1]
    emb = wl.f32_to_bf16_bits(e) if dtype == "bf16" else e
    _check_denoise(orc, emb, 3, 0.05, 16, n_tokens, chunk_tokens=256, what="sizes")


@pytest.mark.parametrize("seed", range(12))
def test_denoise_random_configs(orc, seed):
    """Seeded random batch, length, width, neighbourhood, threshold, floor,
    chunk size, dtype and per-sequence lengths against the oracle."""
    r = np.random.default_rng(3000 + seed)
    dtype = str(r.choice(["f32", "bf16"]))
    B, n = int(r.integers(1, 5)), int(r.integers(1, 2500))
    H = int(r.integers(1, 100)) * (8 if dtype == "bf16" else 4)
    g, m = int(r.integers(1, 5)), int(r.choice([0, 1, int(r.integers(2, 40))]))
    tau = float(r.choice([0.0, 0.05, 0.3, 0.8]))
    n_tokens = [int(r.integers(0, n + 1)) for _ in range(B)]
    e = r.standard_normal((B, n, H)).astype(np.float32)
    e[:, 1:] += float(r.uniform(0.0, 1.5)) * e[:, :-1]
    emb = wl.f32_to_bf16_bits(e) if dtype == "bf16" else e
    _check_denoise(orc, emb, g, tau, m, n_tokens, chunk_tokens=int(r.choice([0, 1, 7, 256])), what=f"random {seed}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("tau,m", [(-2.0, 0), (2.0, 16), (2.0, 1), (0.3, 3), (0.05, 0)])
def test_denoise_threshold_and_floor(orc, dtype, tau, m):
    rng = np.random.default_rng(7)
    e = rng.standard_normal((4, 500, 32)).astype(np.float32)
    e[:, 1:] += 0.4 * e[:, :-1]
    emb = wl.f32_to_bf16_bits(e) if dtype == "bf16" else e
    _check_denoise(orc, emb, 3, tau, m, [500, 499, 250, 3], chunk_tokens=32, what="tau/floor")


def test_denoise_onehot_exact(orc):
    """One-hot tokens: every cosine is exactly 0 or 1 in any precision, so
    the GPU's kept set must equal the oracle's own (fp64) decisions."""
    classes = np.random.default_rng(8).integers(0, 6, size=(2, 400))
    e = np.eye(8, dtype=np.float32)[classes]
    r = cmc.cmc_denoise(to_dev(e), g=3, tau=1.0, keep_min_every=16, chunk_tokens=16)
    torch.cuda.synchronize()
    ref = orc.denoise_select(orc.denoise_scores(e, 3), 1.0, 16, None, 16)
    assert (to_host(r["kept_idx"]) == ref["kept_idx"]).all()
    assert (to_host(r["chunk_offset"]) == ref["chunk_offset"]).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_denoise_zero_rows(orc, dtype):
    """Zero embeddings: the 1e-8 norm clamp gives cosine 0, never NaN."""
    e = np.random.default_rng(9).standard_normal((1, 50, 16)).astype(np.float32)
    e[0, 10:14] = 0.0
    emb = wl.f32_to_bf16_bits(e) if dtype == "bf16" else e
    _check_denoise(orc, emb, 3, 0.0, 0, what="zeros")


@pytest.mark.timeout(600)
def test_full_denoise_gpt2l_batch64(orc):
    """The benchmark's denoising workload at full size (64 contexts of up
    to 3072 tokens, H = 1280, bf16)."""
    w = wl.DENOISE_WORKLOADS["denoise_gpt2l_batch64"]
    say(f"{w.name}: generating inputs")
    emb = wl.denoise_emb(w)
    ref = _check_denoise(orc, emb, w.g, w.tau, w.keep_min_every, wl.denoise_tokens(w), w.chunk_tokens,
                         what=w.name)
    ret = ref["kept_count"] / wl.denoise_tokens(w)
    say(f"{w.name}: retention {ret.mean():.3f} (min {ret.min():.3f}, max {ret.max():.3f})")
