"""CPU oracle for the CMC two-tier decode path (test infrastructure only).

Wraps ``liboracle.so`` (built from ``cmc_oracle.c`` with plain gcc, fp64
arithmetic, no fast-math) for numpy callers.  Only the tests, the smoke
check and the benchmark's CPU-baseline leg use this package; it shares no
code with the HIP library and never imports it.

Functions follow Sec. 2.5 of the paper ("Inference with Two-Tier KV Cache
Policy"): ``select`` (Tier-1 cosine score and top-K in document order),
``window_start`` (Tier-2 window equation), ``window_append`` (the ring that
keeps the cache bounded by K + W + |q|) and ``two_tier_decode`` (softmax
attention over the assembled cache).

``Oracle(path)`` binds any build of the same source (the tests use it to
load deliberately mutated builds and show that the pins reject them); the
module-level functions use the default build.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "cmc_oracle.c")
LIBRARY = os.path.join(_HERE, "liboracle.so")


class OracleError(RuntimeError):
    pass


def compile_source(src: str, out: str) -> str:
    """Compile one oracle C source into a shared library with gcc
    (-O2, OpenMP, no fast-math)."""
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-Wall", "-Wextra", "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Build liboracle.so next to its source."""
    if force or not os.path.exists(LIBRARY):
        compile_source(SOURCE, LIBRARY)
    return LIBRARY


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what}: oracle returned {rc}")


class Oracle:
    """numpy-facing wrapper of one oracle build."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        P, I = ctypes.c_void_p, ctypes.c_int
        lib.oracle_select.argtypes = [P, P, I, I, I, I, P, P, P]
        lib.oracle_select.restype = I
        lib.oracle_window_append.argtypes = [P, P, I, P, P, P, I, I, I, I, I]
        lib.oracle_window_append.restype = I
        lib.oracle_two_tier_decode.argtypes = [P, P, P, I, P, I, P, P, P, I,
                                               I, I, I, I, I, ctypes.c_double, P]
        lib.oracle_two_tier_decode.restype = I
        lib.oracle_window_start.argtypes = [ctypes.c_longlong] * 3
        lib.oracle_window_start.restype = ctypes.c_longlong
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = I
        lib.oracle_set_num_threads.argtypes = [I]
        lib.oracle_set_num_threads.restype = None
        self.lib = lib
        self.path = path

    def num_threads(self) -> int:
        return self.lib.oracle_num_threads()

    def set_num_threads(self, n: int) -> None:
        self.lib.oracle_set_num_threads(int(n))

    def select(self, sel_keys: np.ndarray, q_vec: np.ndarray, k: int
               ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """Tier-1 selection.  sel_keys [B][N][D] fp32, q_vec [B][D] fp32.

        Returns (idx [B][k] int32 ascending, scores [B][N] fp64, gap [B]
        fp64), gap being the relative gap between the k-th and (k+1)-th
        largest scores (+inf when k is 0 or N).
        """
        keys = np.ascontiguousarray(sel_keys, np.float32)
        q = np.ascontiguousarray(q_vec, np.float32)
        B, N, D = keys.shape
        assert q.shape == (B, D)
        idx = np.zeros((B, k), np.int32)
        scores = np.zeros((B, N), np.float64)
        gap = np.zeros((B,), np.float64)
        rc = self.lib.oracle_select(_ptr(keys), _ptr(q), B, N, D, int(k),
                                    _ptr(idx), _ptr(scores), _ptr(gap))
        _check(rc, "select")
        return idx, scores, gap

    def window_start(self, ctx_len: int, W: int, alpha: int) -> int:
        """Tier-2 window start, max(0, min(|C| - W, alpha - floor(W/2)))."""
        return int(self.lib.oracle_window_start(int(ctx_len), int(W), int(alpha)))

    def window_append(self, win_k: np.ndarray, win_v: np.ndarray, win_count: np.ndarray,
                      new_k: np.ndarray, new_v: np.ndarray) -> None:
        """Ring append in place.  win_* [B][Hkv][W][Dh], new_* [B][Hkv][T][Dh]
        (fp32, or bf16 bits as uint16), win_count [B] int32."""
        for a in (win_k, win_v, win_count):
            assert a.flags.c_contiguous
        B, Hkv, W, Dh = win_k.shape
        nk = np.ascontiguousarray(new_k)
        nv = np.ascontiguousarray(new_v)
        T = nk.shape[2]
        assert win_count.dtype == np.int32 and nk.dtype == win_k.dtype
        rc = self.lib.oracle_window_append(_ptr(win_k), _ptr(win_v), win_k.dtype.itemsize,
                                           _ptr(win_count), _ptr(nk), _ptr(nv),
                                           B, Hkv, W, Dh, T)
        _check(rc, "window_append")

    def two_tier_decode(self, q: np.ndarray, cme_k: np.ndarray, cme_v: np.ndarray,
                        idx: Optional[np.ndarray], k: int,
                        win_k: Optional[np.ndarray], win_v: Optional[np.ndarray],
                        win_count: Optional[np.ndarray], W: int, scale: float) -> np.ndarray:
        """Two-tier decode attention; returns out [B][Hq][Dh] fp64.

        q [B][Hq][Dh] fp32; cme_* [B][Hkv][N][Dh]; win_* [B][Hkv][W][Dh];
        K/V fp32 or bf16 bit patterns (uint16).  idx None means rows 0..k-1.
        """
        qq = np.ascontiguousarray(q, np.float32)
        B, Hq, Dh = qq.shape
        ck = np.ascontiguousarray(cme_k)
        cv = np.ascontiguousarray(cme_v)
        Hkv, N = ck.shape[1], ck.shape[2]
        assert ck.shape == (B, Hkv, N, Dh) and cv.shape == ck.shape
        is_bf16 = 1 if ck.dtype == np.uint16 else 0
        if W > 0:
            wk = np.ascontiguousarray(win_k)
            wv = np.ascontiguousarray(win_v)
            wc = np.ascontiguousarray(win_count, np.int32)
            assert wk.dtype == ck.dtype and wk.shape == (B, Hkv, W, Dh)
        else:
            wk = wv = None
            wc = np.zeros((B,), np.int32)
        ii = None if idx is None else np.ascontiguousarray(idx, np.int32)
        if ii is not None:
            assert ii.shape == (B, k)
        out = np.zeros((B, Hq, Dh), np.float64)
        rc = self.lib.oracle_two_tier_decode(_ptr(qq), _ptr(ck), _ptr(cv), is_bf16, _ptr(ii),
                                             int(k), _ptr(wk), _ptr(wv), _ptr(wc), int(W),
                                             B, Hq, Hkv, Dh, N, float(scale), _ptr(out))
        _check(rc, "two_tier_decode")
        return out


_default: Optional[Oracle] = None


def default() -> Oracle:
    global _default
    if _default is None:
        if not os.path.exists(LIBRARY):
            build(force=False)
        _default = Oracle(LIBRARY)
    return _default


def num_threads() -> int:
    return default().num_threads()


def set_num_threads(n: int) -> None:
    default().set_num_threads(n)


def select(sel_keys, q_vec, k):
    return default().select(sel_keys, q_vec, k)


def window_start(ctx_len, W, alpha):
    return default().window_start(ctx_len, W, alpha)


def window_append(win_k, win_v, win_count, new_k, new_v):
    return default().window_append(win_k, win_v, win_count, new_k, new_v)


def two_tier_decode(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, W, scale):
    return default().two_tier_decode(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, W, scale)
