"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and its host-side validation returns the documented codes before
touching the GPU (no compute calls here)."""
import ctypes
import os
import re

import pytest

from paper_2609_25537_amd import cmc
from tests import pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for f in os.listdir(os.path.join(ROOT, "include")):
        if f.endswith(".h"):
            src = open(os.path.join(ROOT, "include", f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(cmc_[a-z0-9_]+)\s*\(", src))
    return names


def test_exports_every_declared_symbol():
    declared = _declared()
    assert {"cmc_select_cmes", "cmc_window_append", "cmc_two_tier_decode"} <= declared
    L = cmc.lib()
    for name in sorted(declared):
        assert hasattr(L, name), name
    assert set(cmc.EXPORTED) == declared


def test_status_strings():
    assert cmc.status_string(cmc.CMC_OK) == "CMC_OK"
    assert cmc.status_string(cmc.CMC_ERR_WORKSPACE_TOO_SMALL) == "CMC_ERR_WORKSPACE_TOO_SMALL"
    assert "gfx950" in cmc.version()


def test_window_start_matches_golden():
    for c in pins._golden()["window_start"]["cases"]:
        assert cmc.cmc_window_start(c["ctx_len"], c["W"], c["alpha"]) == c["start"]


FAKE = 1 << 20  # 16-byte aligned non-null address, never dereferenced: calls below fail validation first


def _sel(**kw):
    a = dict(keys=FAKE, kd=cmc.CMC_F32, qv=FAKE, B=2, N=64, D=8, k=2, idx=FAKE, sc=None, ws=FAKE, wsb=1 << 20,
             s=None)
    a.update(kw)
    return cmc.lib().cmc_select_cmes(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(B=1, N=4, k=5), cmc.CMC_ERR_INVALID_ARGUMENT),        # k > N
    (dict(D=6), cmc.CMC_ERR_UNSUPPORTED),                       # D % 4 (fp32 keys)
    (dict(D=12, kd=cmc.CMC_BF16), cmc.CMC_ERR_UNSUPPORTED),     # D % 8 (bf16 keys)
    (dict(kd=5), cmc.CMC_ERR_UNSUPPORTED),                      # unknown key dtype
    (dict(N=40000), cmc.CMC_ERR_UNSUPPORTED),                   # N too big
    (dict(wsb=16), cmc.CMC_ERR_WORKSPACE_TOO_SMALL),
    (dict(keys=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(keys=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),             # alignment
    (dict(k=-1), cmc.CMC_ERR_INVALID_ARGUMENT),
])
def test_select_validation(kw, code):
    assert _sel(**kw) == code
    assert cmc.last_error()


def test_select_signature_takes_key_dtype():
    """The boundary's selection takes the key type right after the keys:
    (sel_keys, key_dtype, q_vec, B, N, D, k, idx_out, scores_out, workspace,
    workspace_bytes, stream); bf16 keys with D % 8 == 0 pass validation."""
    assert _sel(B=0, kd=cmc.CMC_BF16, D=16) == cmc.CMC_OK
    assert _sel(D=16, kd=cmc.CMC_BF16, wsb=16) == cmc.CMC_ERR_WORKSPACE_TOO_SMALL  # got past the dtype checks
    assert len(cmc.lib().cmc_select_cmes.argtypes) == 12
    assert len(cmc.lib().cmc_select_cmes_ragged.argtypes) == 17


def test_select_empty_is_ok():
    assert _sel(keys=None, qv=None, B=0, N=10, k=3, idx=None, ws=None, wsb=0) == cmc.CMC_OK
    assert cmc.last_error() == ""


def _dec(**kw):
    a = dict(q=FAKE, ck=FAKE, cv=FAKE, idx=FAKE, k=4, wk=FAKE, wv=FAKE, wc=FAKE, W=8, dt=cmc.CMC_BF16,
             B=1, Hq=8, Hkv=2, Dh=128, N=16, scale=0.1, out=FAKE, ws=FAKE, wsb=1 << 30, s=None)
    a.update(kw)
    return cmc.lib().cmc_two_tier_decode(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(Hq=6, Hkv=4), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(Hq=12, Hkv=4), cmc.CMC_ERR_UNSUPPORTED),       # G = 3
    (dict(Dh=96), cmc.CMC_ERR_UNSUPPORTED),
    (dict(k=0, W=0), cmc.CMC_ERR_INVALID_ARGUMENT),       # empty cache
    (dict(idx=None, k=17), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(k=3, N=0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(dt=7), cmc.CMC_ERR_UNSUPPORTED),
    (dict(wsb=64), cmc.CMC_ERR_WORKSPACE_TOO_SMALL),
    (dict(ws=None), cmc.CMC_ERR_WORKSPACE_TOO_SMALL),
    (dict(out=FAKE + 8), cmc.CMC_ERR_UNSUPPORTED),
    (dict(wc=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(q=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(scale=float("nan")), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(B=-1), cmc.CMC_ERR_INVALID_ARGUMENT),
])
def test_decode_validation(kw, code):
    assert _dec(**kw) == code


def test_decode_empty_batch_ok():
    assert _dec(B=0) == cmc.CMC_OK


def test_decode_workspace_query():
    assert cmc.cmc_decode_workspace_bytes(1, 32, 8, 128, 256, 512) > 0
    assert cmc.cmc_decode_workspace_bytes(1, 32, 7, 128, 256, 512) == 0
    assert cmc.cmc_decode_workspace_bytes(1, 32, 8, 100, 256, 512) == 0
    assert cmc.cmc_decode_workspace_bytes(1, 32, 8, 128, 0, 0) == 0


def _app(**kw):
    a = dict(wk=FAKE, wv=FAKE, dt=cmc.CMC_BF16, wc=FAKE, nk=FAKE, nv=FAKE, B=2, Hkv=2, W=8, Dh=128, T=1, s=None)
    a.update(kw)
    return cmc.lib().cmc_window_append(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(T=0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(T=9), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(Dh=80), cmc.CMC_ERR_UNSUPPORTED),
    (dict(Hkv=0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(nk=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(wc=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),
    (dict(dt=3), cmc.CMC_ERR_UNSUPPORTED),
])
def test_append_validation(kw, code):
    assert _app(**kw) == code


def test_append_without_window_is_noop():
    assert _app(W=0, wk=None, wv=None, wc=None, T=5) == cmc.CMC_OK


def _sel_r(**kw):
    a = dict(keys=FAKE, kd=cmc.CMC_F32, qv=FAKE, n=FAKE, qr=None, B=2, N=64, D=8, k=4, stride=6, idx=FAKE,
             kout=FAKE, sc=None, nrm=None, ws=FAKE, wsb=1 << 20, s=None)
    a.update(kw)
    return cmc.lib().cmc_select_cmes_ragged(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(n=None), cmc.CMC_ERR_INVALID_ARGUMENT),             # n_rows is required
    (dict(stride=3), cmc.CMC_ERR_INVALID_ARGUMENT),           # idx_stride < k
    (dict(idx=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(D=6), cmc.CMC_ERR_UNSUPPORTED),
    (dict(D=12, kd=cmc.CMC_BF16), cmc.CMC_ERR_UNSUPPORTED),   # D % 8 (bf16 keys)
    (dict(kd=3), cmc.CMC_ERR_UNSUPPORTED),
    (dict(N=40000), cmc.CMC_ERR_UNSUPPORTED),
    (dict(wsb=16), cmc.CMC_ERR_WORKSPACE_TOO_SMALL),
    (dict(qr=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),             # alignment
    (dict(kout=FAKE + 8), cmc.CMC_ERR_UNSUPPORTED),
    (dict(nrm=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),
    (dict(k=-1), cmc.CMC_ERR_INVALID_ARGUMENT),
])
def test_select_ragged_validation(kw, code):
    assert _sel_r(**kw) == code
    assert cmc.last_error()


def test_select_ragged_empty_batch_ok():
    assert _sel_r(B=0, n=None) == cmc.CMC_OK


def _dec_r(step=False, **kw):
    a = dict(q=FAKE, ck=FAKE, cv=FAKE, idx=FAKE, kl=FAKE, k=4, wk=FAKE, wv=FAKE, wc=FAKE, W=8)
    if step:
        a.update(nk=FAKE, nv=FAKE, T=1)
    a.update(dt=cmc.CMC_BF16, B=1, Hq=8, Hkv=2, Dh=128, N=16, scale=0.1, out=FAKE, ws=FAKE, wsb=1 << 30, s=None)
    a.update(kw)
    fn = cmc.lib().cmc_decode_step_ragged if step else cmc.lib().cmc_two_tier_decode_ragged
    return fn(*a.values())


@pytest.mark.parametrize("step", [False, True])
@pytest.mark.parametrize("kw,code", [
    (dict(kl=None), cmc.CMC_ERR_INVALID_ARGUMENT),            # k_len is required
    (dict(kl=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),             # alignment
    (dict(Hq=12, Hkv=4), cmc.CMC_ERR_UNSUPPORTED),
    (dict(k=0, W=0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(wsb=64), cmc.CMC_ERR_WORKSPACE_TOO_SMALL),
])
def test_decode_ragged_validation(step, kw, code):
    assert _dec_r(step=step, **kw) == code


def test_decode_step_ragged_needs_new_rows():
    assert _dec_r(step=True, T=0) == cmc.CMC_ERR_INVALID_ARGUMENT


def test_decode_offset_limits():
    """A bf16 (sequence, kv head) pool or ring of 4 GiB or more, and key
    lists longer than INT_MAX rows, are refused before anything is enqueued
    (the kernel addresses them with 32-bit offsets and indices); fp32 pools
    of that size are addressed in 64 bits and pass this check."""
    big = (1 << 32) // (128 * 2)  # rows of Dh = 128 bf16 in 4 GiB
    assert _dec_r(N=big) == cmc.CMC_ERR_UNSUPPORTED and "4 GiB" in cmc.last_error()
    assert _dec_r(W=big) == cmc.CMC_ERR_UNSUPPORTED and "4 GiB" in cmc.last_error()
    assert _dec_r(step=True, W=big) == cmc.CMC_ERR_UNSUPPORTED
    assert _dec_r(N=big - 1, wsb=64) == cmc.CMC_ERR_WORKSPACE_TOO_SMALL  # just under: passes this check
    assert _dec_r(dt=cmc.CMC_F32, N=big, wsb=64) == cmc.CMC_ERR_WORKSPACE_TOO_SMALL
    assert _dec_r(dt=cmc.CMC_F32, k=2**31 - 8, W=8, N=2**31 - 1) == cmc.CMC_ERR_UNSUPPORTED
    assert "INT_MAX" in cmc.last_error() or "2147483647" in cmc.last_error()


def test_decode_step_append_row_limit():
    """At most 65535 rows appended per call (the launch packs T_new into 16
    bits); beyond that the call is refused before anything is enqueued."""
    assert _dec_r(step=True, W=70000, T=65536) == cmc.CMC_ERR_UNSUPPORTED
    assert "65535" in cmc.last_error()


def _loc(**kw):
    a = dict(nrm=FAKE, n=None, ctx=FAKE, B=2, N=64, m=4, off=FAKE, nch=16, ct=0, W=32, al=FAKE, st=FAKE, s=None)
    a.update(kw)
    return cmc.lib().cmc_locate_window(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(m=0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(nch=15), cmc.CMC_ERR_INVALID_ARGUMENT),             # chunks do not cover N rows
    (dict(W=-1), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(ctx=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(st=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(nrm=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(off=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),
    (dict(B=70000), cmc.CMC_ERR_UNSUPPORTED),
])
def test_locate_validation(kw, code):
    assert _loc(**kw) == code


def test_locate_empty_batch_ok():
    assert _loc(B=0, nrm=None, ctx=None, st=None) == cmc.CMC_OK


def _den(**kw):
    a = dict(emb=FAKE, dt=cmc.CMC_BF16, nt=None, B=2, n=64, H=128, g=3, tau=0.05, m=16, t=0, mc=None, keep=None,
             idx=FAKE, cnt=FAKE, off=None, nch=None, ws=FAKE, wsb=1 << 20, s=None)
    a.update(kw)
    return cmc.lib().cmc_denoise(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(g=0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(g=5), cmc.CMC_ERR_UNSUPPORTED),
    (dict(H=12), cmc.CMC_ERR_UNSUPPORTED),                    # bf16 rows need H % 8 == 0
    (dict(dt=cmc.CMC_F32, H=6), cmc.CMC_ERR_UNSUPPORTED),
    (dict(tau=float("nan")), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(m=-1), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(idx=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(cnt=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(wsb=64), cmc.CMC_ERR_WORKSPACE_TOO_SMALL),
    (dict(emb=FAKE + 2), cmc.CMC_ERR_UNSUPPORTED),
    (dict(dt=5), cmc.CMC_ERR_UNSUPPORTED),
])
def test_denoise_validation(kw, code):
    assert _den(**kw) == code


def test_denoise_workspace_query():
    assert cmc.cmc_denoise_workspace_bytes(3, 1000) >= 3000
    assert cmc.cmc_denoise_workspace_bytes(-1, 10) == 0
    assert _den(B=0) == cmc.CMC_OK


def _bridge(**kw):
    a = dict(h=FAKE, w1=FAKE, b1=FAKE, w2=FAKE, b2=FAKE, g=FAKE, be=FAKE, nu=1.0, eps=1e-5, M=10, Hc=64, F=128,
             Hd=128, out=FAKE, hn=None, ws=FAKE, wsb=1 << 20, s=None)
    a.update(kw)
    return cmc.lib().cmc_memory_bridge(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(Hc=96), cmc.CMC_ERR_UNSUPPORTED),                   # Hc % 64
    (dict(F=192), cmc.CMC_ERR_UNSUPPORTED),                   # F % 128
    (dict(Hd=64), cmc.CMC_ERR_UNSUPPORTED),                   # Hd % 128
    (dict(nu=0.0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(nu=float("inf")), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(eps=-1.0), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(M=-1), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(b2=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(w1=FAKE + 2), cmc.CMC_ERR_UNSUPPORTED),
    (dict(hn=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),             # h_norms_out alignment
    (dict(wsb=100), cmc.CMC_ERR_WORKSPACE_TOO_SMALL),
])
def test_bridge_validation(kw, code):
    assert _bridge(**kw) == code


def test_bridge_empty_and_workspace():
    assert _bridge(M=0, h=None) == cmc.CMC_OK
    assert cmc.cmc_bridge_workspace_bytes(10, 128) == 2560  # M * F bf16, rounded up to 256
    need = 49152 * 4096 * 2
    assert cmc.cmc_bridge_workspace_bytes(49152, 4096) == need
    assert _bridge(M=49152, F=4096, Hd=4096, wsb=need - 1) == cmc.CMC_ERR_WORKSPACE_TOO_SMALL
    assert f"{need} bytes needed" in cmc.last_error()


def _gather(**kw):
    a = dict(ck=FAKE, cv=FAKE, dt=cmc.CMC_BF16, idx=FAKE, kl=None, stride=8, B=2, Hkv=2, N=16, k=8, Dh=128,
             ok=FAKE, ov=FAKE, s=None)
    a.update(kw)
    return cmc.lib().cmc_gather_tier1(*a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(stride=4), cmc.CMC_ERR_INVALID_ARGUMENT),            # idx_stride < k
    (dict(idx=None, k=17), cmc.CMC_ERR_INVALID_ARGUMENT),      # k > N without idx
    (dict(Dh=96), cmc.CMC_ERR_UNSUPPORTED),
    (dict(dt=9), cmc.CMC_ERR_UNSUPPORTED),
    (dict(ok=None), cmc.CMC_ERR_INVALID_ARGUMENT),
    (dict(kl=FAKE + 4), cmc.CMC_ERR_UNSUPPORTED),
    (dict(Hkv=0), cmc.CMC_ERR_INVALID_ARGUMENT),
])
def test_gather_validation(kw, code):
    assert _gather(**kw) == code


def test_gather_empty_ok():
    assert _gather(B=0) == cmc.CMC_OK and _gather(k=0) == cmc.CMC_OK


def _noalloc(**kw):
    a = dict(q=FAKE, ck=FAKE, cv=FAKE, idx=FAKE, k=4, wk=FAKE, wv=FAKE, wc=FAKE, W=8, nk=FAKE, nv=FAKE, T=1,
             dt=cmc.CMC_BF16, B=1, Hq=8, Hkv=2, Dh=128, N=16, scale=0.1, out=FAKE, s=None)
    a.update(kw)
    return cmc.lib().cmc_decode_step_noalloc(*a.values())


@pytest.mark.parametrize("kw", [
    dict(B=4096, Hkv=8, Hq=32),                            # 36864 arrival counters > 16384
    dict(B=2, Hkv=16, Hq=128, Dh=256, k=0, W=200000),      # split partials beyond the fixed array
])
def test_noalloc_rejects_sizes_beyond_its_scratch(kw):
    """The no-allocation decode step refuses sizes its fixed scratch cannot
    hold, before touching the GPU."""
    assert _noalloc(**kw) == cmc.CMC_ERR_UNSUPPORTED
    assert "scratch" in cmc.last_error()


def test_noalloc_validates_like_decode_step():
    assert _noalloc(T=0) == cmc.CMC_ERR_INVALID_ARGUMENT
    assert _noalloc(Dh=96) == cmc.CMC_ERR_UNSUPPORTED
    assert _noalloc(B=0) == cmc.CMC_OK



def test_binding_refuses_host_tensors():
    """A host tensor never reaches the library as an address (the kernels
    would read it as device memory); the check runs before any call."""
    import torch
    q = torch.zeros((1, 4, 64), dtype=torch.float32)
    pool = torch.zeros((1, 4, 8, 64), dtype=torch.float32)
    with pytest.raises(ValueError, match="device tensors"):
        cmc._ptr(q)
    with pytest.raises((ValueError, RuntimeError)):
        cmc.cmc_two_tier_decode(q, pool, pool, None, 4, None, None, None, 0.125, W=0,
                                out=torch.zeros((1, 4, 64)), workspace=torch.zeros(1024, dtype=torch.uint8))


def test_last_error_is_per_thread():
    """cmc_last_error() is thread-local: two threads failing validation with
    different arguments, many times over and at the same time (ctypes calls
    release the GIL), each read back their own message."""
    import threading
    L = cmc.lib()
    L.cmc_last_error.restype = ctypes.c_char_p
    bad = []

    def worker(k, n_iter=2000):
        for _ in range(n_iter):
            rc = _sel(B=1, N=4, k=k)  # k > N: the message names this thread's k
            msg = L.cmc_last_error().decode()
            if rc != cmc.CMC_ERR_INVALID_ARGUMENT or f"k={k} " not in msg:
                bad.append((k, rc, msg))
                return

    threads = [threading.Thread(target=worker, args=(k,)) for k in (5, 7, 9, 11)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not bad, bad[:3]
