"""CME-guided Tier-2 localization on the GPU vs the oracle, through the C
ABI: row norms (from the selection pass, and the CME norms |h_j| from the
MemoryBridge call, which localization ranks) within their fp32 bounds of the
fp64 norms, and the chosen chunk offset and window start (bit-exact, decided
on the same fp32 norms on both sides, and on the bridge workload against the
oracle's whole fp64 chain)."""
import numpy as np
import pytest
import torch

from paper_2609_25537_amd import cmc
from paper_2609_25537_amd import workloads as wl
from tests.gpu_util import DEV, say, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("B,N,D", [(3, 100, 8), (2, 4096, 256), (4, 32768, 8)])
def test_norms_from_selection_pass(orc, B, N, D):
    say(f"norms B={B} N={N} D={D}")
    rng = np.random.default_rng(N + D)
    keys = rng.standard_normal((B, N, D)).astype(np.float32)
    keys[0, 3] = 0.0
    qv = rng.standard_normal((B, D)).astype(np.float32)
    n_rows = np.array([N, N // 3, 0, 7][:B], np.int32)
    norms = torch.empty((B, N), dtype=torch.float32, device=DEV)
    cmc.cmc_select_cmes_ragged(to_dev(keys), to_dev(qv), to_dev(n_rows), 4, norms_out=norms)
    torch.cuda.synchronize()
    got = to_host(norms).astype(np.float64)
    ref = orc.row_norms(keys)
    for b in range(B):
        nb = int(n_rows[b])
        np.testing.assert_allclose(got[b, :nb], ref[b, :nb], rtol=1e-6, atol=1e-30)
        assert (got[b, nb:] == 0).all()


def _check_locate(orc, norms, ctx, W, m, n_rows=None, offsets=None, chunk_tokens=0, what=""):
    say(f"locate {what}: B={norms.shape[0]} N={norms.shape[1]} W={W} m={m}")
    d_norms = to_dev(norms.astype(np.float32))
    alpha, start = cmc.cmc_locate_window(d_norms, to_dev(ctx), W, m,
                                         n_rows=None if n_rows is None else to_dev(n_rows),
                                         chunk_offset=None if offsets is None else to_dev(offsets),
                                         chunk_tokens=chunk_tokens)
    torch.cuda.synchronize()
    ref_a, ref_s = orc.locate(to_host(d_norms).astype(np.float64), ctx, W, m, n_rows, offsets, chunk_tokens)
    assert (to_host(alpha) == ref_a).all(), f"{what}: alpha differs"
    assert (to_host(start) == ref_s).all(), f"{what}: start differs"


@pytest.mark.parametrize("B,N,m,W", [(5, 64, 4, 100), (3, 4096, 16, 1024), (2, 32768, 64, 140), (64, 300, 1, 7)])
def test_locate_offset_table(orc, B, N, m, W):
    rng = np.random.default_rng(B * N)
    norms = rng.random((B, N)) * 10
    n_chunks = -(-N // m)
    tok = rng.integers(1, 300, size=(B, n_chunks))
    offsets = np.cumsum(tok, axis=1).astype(np.int32) - tok.astype(np.int32)
    ctx = (offsets[:, -1] + rng.integers(1, 400, size=B)).astype(np.int32)
    n_rows = rng.integers(0, N + 5, size=B).astype(np.int32)
    n_rows[0] = N
    _check_locate(orc, norms, ctx, W, m, n_rows, offsets, what="table")


def test_locate_ties_and_chunk_tokens(orc):
    """Integer-valued norms: many exact ties, resolved to the earliest row."""
    rng = np.random.default_rng(9)
    norms = rng.integers(0, 6, size=(16, 2000)).astype(np.float64)
    ctx = rng.integers(1, 20000, size=16).astype(np.int32)
    n_rows = rng.integers(0, 2001, size=16).astype(np.int32)
    _check_locate(orc, norms, ctx, 512, 8, n_rows, None, chunk_tokens=32, what="ties")
    _check_locate(orc, norms, ctx, 0, 1, None, None, chunk_tokens=1, what="W=0")


def test_select_then_locate(orc):
    """Selection pass -> norms -> localization, against the oracle's fp64
    norms: the largest norm is planted well apart from the rest, so both
    sides choose the same row."""
    rng = np.random.default_rng(10)
    B, N, D, m = 4, 2048, 64, 8
    keys = rng.standard_normal((B, N, D)).astype(np.float32)
    star = [5, 700, 2047, 1000]
    for b in range(B):
        keys[b, star[b]] *= 3.0
    qv = rng.standard_normal((B, D)).astype(np.float32)
    n_rows = np.array([N, N, N, 999], np.int32)
    norms = torch.empty((B, N), dtype=torch.float32, device=DEV)
    cmc.cmc_select_cmes_ragged(to_dev(keys), to_dev(qv), to_dev(n_rows), 32, norms_out=norms)
    ctx = np.full(B, N * 4, np.int32)
    alpha, start = cmc.cmc_locate_window(norms, to_dev(ctx), 512, m, n_rows=to_dev(n_rows), chunk_tokens=4 * m)
    torch.cuda.synchronize()
    ref_a, ref_s = orc.locate(orc.row_norms(keys), ctx, 512, m, n_rows, None, 4 * m)
    assert (to_host(alpha) == ref_a).all() and (to_host(start) == ref_s).all()
    assert to_host(alpha).tolist()[:3] == [(s // m) * 4 * m for s in star[:3]]


def _norm_rel_bound(H: int) -> float:
    """Relative error bound of the kernel's fp32 norm of an H-wide bf16 row:
    each lane sums its squares in one chain of ceil(H / 512) * 8 fused
    multiply-adds, then a 6-step butterfly adds the 64 lane sums, so the
    squared norm is within gamma_n (n = chain + 6, gamma_n = n u / (1 - n u))
    of the exact one (all terms are non-negative); the square root halves
    that and adds one rounding."""
    u = 2.0 ** -24
    n = -(-H // 512) * 8 + 6
    return 0.5 * n * u / (1 - n * u) + u


@pytest.mark.timeout(300)
def test_bridge_cme_norms_then_locate(orc):
    """The MemoryBridge workload end to end: the bridge call returns the CME
    norms |h_j| of its 49,152 input rows (64 contexts x 12 chunks x 64 CMEs),
    localization ranks them per context.  Norms within their fp32 bound of
    the oracle's fp64 norms; alpha and start bit-exact against the oracle's
    chain (fp64 norms -> argmax -> chunk offset -> window start) wherever the
    two largest norms of a context are further apart than that bound, and
    otherwise equal to the oracle's decision on the kernel's own norms."""
    w = wl.BRIDGE_WORKLOADS["bridge_gpt2l_llama3_batch64"]
    B, N, m, chunk_tokens, ctx_len, W = 64, 768, 64, 256, 3072, 256
    assert B * N == w.M
    say(f"bridge -> locate: M={w.M} Hc={w.Hc}")
    h = wl.bridge_h(w)
    p = wl.bridge_params(w)
    bf = lambda a: to_dev(np.ascontiguousarray(a))
    hn = torch.empty((w.M,), dtype=torch.float32, device=DEV)
    cmc.cmc_memory_bridge(bf(h), bf(p["w1"]), to_dev(p["b1"]), bf(p["w2"]), to_dev(p["b2"]), to_dev(p["gamma"]),
                          to_dev(p["beta"]), w.nu, w.eps, h_norms_out=hn)
    ctx = np.full(B, ctx_len, np.int32)
    alpha, start = cmc.cmc_locate_window(hn.view(B, N), to_dev(ctx), W, m, chunk_tokens=chunk_tokens)
    torch.cuda.synchronize()
    got_n = to_host(hn).astype(np.float64).reshape(B, N)
    ref_n = orc.row_norms(h).reshape(B, N)
    rel = _norm_rel_bound(w.Hc)
    assert (np.abs(got_n - ref_n) <= rel * ref_n).all(), f"worst rel err {np.max(np.abs(got_n / ref_n - 1)):.2e}"
    ref_a, ref_s = orc.locate(ref_n, ctx, W, m, chunk_tokens=chunk_tokens)
    own_a, own_s = orc.locate(got_n, ctx, W, m, chunk_tokens=chunk_tokens)
    ga, gs = to_host(alpha), to_host(start)
    top2 = -np.partition(-ref_n, 1, axis=1)[:, :2]
    resolved = (top2[:, 0] - top2[:, 1]) > 2 * rel * top2[:, 0]
    assert resolved.sum() >= B - 2, "workload norms too close to rank in fp32"
    assert (ga[resolved] == ref_a[resolved]).all() and (gs[resolved] == ref_s[resolved]).all()
    assert (ga == own_a).all() and (gs == own_s).all()
    # the chosen chunks vary across contexts (the norms rank, they do not tie)
    assert len(np.unique(ga)) > 4
