"""CPU oracle for the CMC two-tier decode path (test infrastructure only).

Wraps ``liboracle.so`` (built from ``cmc_oracle.c`` with plain gcc, fp64
arithmetic, no fast-math) for numpy callers.  Only the tests, the smoke
check and the benchmark's CPU-baseline leg use this package; it shares no
code with the HIP library and never imports it.

Functions follow Sec. 2.5 of the paper ("Inference with Two-Tier KV Cache
Policy"): ``select`` (Tier-1 cosine score and top-K in document order),
``window_start`` (Tier-2 window equation), ``window_append`` (the ring that
keeps the cache bounded by K + W + |q|) and ``two_tier_decode`` (softmax
attention over the assembled cache), plus ``select_ragged`` and
``two_tier_decode_ragged`` (the same definitions per sequence, for batches
whose sequences differ in size), and ``row_norms`` / ``locate`` (CME-guided
Tier-2 localization, from the appendix on window localization, ranking the
norms of the encoder's CME vectors h of Sec. 2.2), and
``denoise_scores`` / ``denoise_select`` (graph-based context denoising,
Sec. 2.1 Eq. 3 with the minimum keep interval), and ``bridge_hidden`` /
``bridge_out`` (the MemoryBridge projection and its norm-calibrated tanh
cap, Sec. 2.3).

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


def _keys(a: np.ndarray):
    """(contiguous array, 1 if it holds bf16 bit patterns else 0); uint16
    arrays are bf16, anything else is taken as fp32."""
    if a.dtype == np.uint16:
        return np.ascontiguousarray(a), 1
    return np.ascontiguousarray(a, np.float32), 0


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what}: oracle returned {rc}")


class Oracle:
    """numpy-facing wrapper of one oracle build."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        P, I = ctypes.c_void_p, ctypes.c_int
        lib.oracle_select.argtypes = [P, I, P, I, I, I, I, P, P, P]
        lib.oracle_select.restype = I
        lib.oracle_window_append.argtypes = [P, P, I, P, P, P, I, I, I, I, I]
        lib.oracle_window_append.restype = I
        lib.oracle_two_tier_decode.argtypes = [P, P, P, I, P, I, P, P, P, I,
                                               I, I, I, I, I, ctypes.c_double, P]
        lib.oracle_two_tier_decode.restype = I
        lib.oracle_row_norms.argtypes = [P, I, ctypes.c_longlong, I, P]
        lib.oracle_row_norms.restype = I
        lib.oracle_locate.argtypes = [P, P, I, I, I, P, I, I, P, I, P, P]
        lib.oracle_locate.restype = I
        lib.oracle_denoise_scores.argtypes = [P, I, P, I, I, I, I, P]
        lib.oracle_denoise_scores.restype = I
        lib.oracle_denoise_select.argtypes = [P, P, I, I, ctypes.c_double, I, I, P, P, P, P, P]
        lib.oracle_denoise_select.restype = I
        lib.oracle_bridge_hidden.argtypes = [P, P, P, I, I, I, P]
        lib.oracle_bridge_hidden.restype = I
        lib.oracle_bridge_out.argtypes = [P, P, P, P, P, ctypes.c_double, ctypes.c_double, I, I, I, P]
        lib.oracle_bridge_out.restype = I
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
        """Tier-1 selection.  sel_keys [B][N][D] fp32 (or uint16: bf16 bit
        patterns), q_vec [B][D] fp32.

        Returns (idx [B][k] int32 ascending, scores [B][N] fp64, gap [B]
        fp64), gap being the relative gap between the k-th and (k+1)-th
        largest scores (+inf when k is 0 or N).
        """
        keys, bf = _keys(sel_keys)
        q = np.ascontiguousarray(q_vec, np.float32)
        B, N, D = keys.shape
        assert q.shape == (B, D)
        idx = np.zeros((B, k), np.int32)
        scores = np.zeros((B, N), np.float64)
        gap = np.zeros((B,), np.float64)
        rc = self.lib.oracle_select(_ptr(keys), bf, _ptr(q), B, N, D, int(k),
                                    _ptr(idx), _ptr(scores), _ptr(gap))
        _check(rc, "select")
        return idx, scores, gap

    def denoise_scores(self, emb: np.ndarray, g: int, n_tokens: Optional[np.ndarray] = None) -> np.ndarray:
        """Eq. 3's statistic: the largest cosine similarity of each token to
        its next g tokens, fp64 [B][n] (-inf where there is none).  emb
        [B][n][H] fp32 or bf16 bits (uint16)."""
        e = np.ascontiguousarray(emb)
        B, n, H = e.shape
        nt = None if n_tokens is None else np.ascontiguousarray(n_tokens, np.int32)
        out = np.zeros((B, n), np.float64)
        rc = self.lib.oracle_denoise_scores(_ptr(e), 1 if e.dtype == np.uint16 else 0, _ptr(nt), B, n, H,
                                            int(g), _ptr(out))
        _check(rc, "denoise_scores")
        return out

    def denoise_select(self, max_cos: np.ndarray, tau: float, keep_min_every: int,
                       n_tokens: Optional[np.ndarray] = None, chunk_tokens: int = 0):
        """Threshold, minimum keep interval and compaction on the given
        max_cos [B][n].  Returns dict(keep [B][n] uint8, kept_idx [B][n],
        kept_count [B], chunk_offset [B][ceil(n/chunk_tokens)], n_chunks
        [B]) (the last two only with chunk_tokens > 0)."""
        mc = np.ascontiguousarray(max_cos, np.float64)
        B, n = mc.shape
        nt = None if n_tokens is None else np.ascontiguousarray(n_tokens, np.int32)
        keep = np.zeros((B, n), np.uint8)
        idx = np.zeros((B, n), np.int32)
        cnt = np.zeros((B,), np.int32)
        nch = -(-n // chunk_tokens) if chunk_tokens > 0 else 0
        off = np.zeros((B, max(nch, 1)), np.int32)
        ncs = np.zeros((B,), np.int32)
        rc = self.lib.oracle_denoise_select(_ptr(mc), _ptr(nt), B, n, float(tau), int(keep_min_every),
                                            int(chunk_tokens), _ptr(keep), _ptr(idx), _ptr(cnt), _ptr(off),
                                            _ptr(ncs))
        _check(rc, "denoise_select")
        r = {"keep": keep, "kept_idx": idx, "kept_count": cnt}
        if chunk_tokens > 0:
            r["chunk_offset"] = off[:, :nch]
            r["n_chunks"] = ncs
        return r

    def bridge_hidden(self, h: np.ndarray, w1: np.ndarray, b1: np.ndarray) -> np.ndarray:
        """MemoryBridge hidden layer GELU(h w1^T + b1), fp64 [M][F]; h [M][Hc]
        and w1 [F][Hc] bf16 bits (uint16), b1 [F] fp32."""
        hh = np.ascontiguousarray(h, np.uint16)
        ww = np.ascontiguousarray(w1, np.uint16)
        bb = np.ascontiguousarray(b1, np.float32)
        M, Hc = hh.shape
        F = ww.shape[0]
        assert ww.shape == (F, Hc) and bb.shape == (F,)
        out = np.zeros((M, F), np.float64)
        _check(self.lib.oracle_bridge_hidden(_ptr(hh), _ptr(ww), _ptr(bb), M, Hc, F, _ptr(out)), "bridge_hidden")
        return out

    def bridge_out(self, hidden: np.ndarray, w2: np.ndarray, b2: np.ndarray, gamma: np.ndarray,
                   beta: np.ndarray, nu: float, eps: float = 1e-5) -> np.ndarray:
        """MemoryBridge output layer, LayerNorm and norm-calibrated tanh cap
        from the given hidden activations [M][F] (any float values); w2 [Hd][F]
        bf16 bits; b2, gamma, beta [Hd] fp32.  Returns fp64 [M][Hd]."""
        hd = np.ascontiguousarray(hidden, np.float64)
        ww = np.ascontiguousarray(w2, np.uint16)
        M, F = hd.shape
        Hd = ww.shape[0]
        vec = [np.ascontiguousarray(v, np.float32) for v in (b2, gamma, beta)]
        assert ww.shape == (Hd, F) and all(v.shape == (Hd,) for v in vec)
        out = np.zeros((M, Hd), np.float64)
        rc = self.lib.oracle_bridge_out(_ptr(hd), _ptr(ww), *[_ptr(v) for v in vec], float(nu), float(eps), M, F,
                                        Hd, _ptr(out))
        _check(rc, "bridge_out")
        return out

    def memory_bridge(self, h, w1, b1, w2, b2, gamma, beta, nu, eps=1e-5):
        """The whole MemoryBridge in fp64 (hidden layer not rounded)."""
        return self.bridge_out(self.bridge_hidden(h, w1, b1), w2, b2, gamma, beta, nu, eps)

    def row_norms(self, rows: np.ndarray) -> np.ndarray:
        """||x|| over the last axis of rows [..., D] (fp32, or uint16: bf16
        bit patterns), fp64 with the leading shape (e.g. the CME vectors h
        [M][Hc] -> [M], memory rows [B][N][D] -> [B][N])."""
        x, bf = _keys(rows)
        D = x.shape[-1]
        R = int(np.prod(x.shape[:-1]))
        out = np.zeros(x.shape[:-1], np.float64)
        _check(self.lib.oracle_row_norms(_ptr(x), bf, R, D, _ptr(out)), "row_norms")
        return out

    def locate(self, norms: np.ndarray, ctx_len: np.ndarray, W: int, mems_per_chunk: int,
               n_rows: Optional[np.ndarray] = None, chunk_offset: Optional[np.ndarray] = None,
               chunk_tokens: int = 0) -> Tuple[np.ndarray, np.ndarray]:
        """CME-guided Tier-2 localization: (alpha [B], start [B]) int32.
        norms [B][N] (taken as given: the decision is made on these values),
        ctx_len [B] tokens, chunk_offset [B][n_chunks] or None (chunk i at
        i * chunk_tokens)."""
        nr = np.ascontiguousarray(norms, np.float64)
        B, N = nr.shape
        ctx = np.ascontiguousarray(ctx_len, np.int32)
        rows = None if n_rows is None else np.ascontiguousarray(n_rows, np.int32)
        off = None if chunk_offset is None else np.ascontiguousarray(chunk_offset, np.int32)
        n_chunks = 0 if off is None else off.shape[1]
        alpha = np.zeros((B,), np.int32)
        start = np.zeros((B,), np.int32)
        rc = self.lib.oracle_locate(_ptr(nr), _ptr(rows), B, N, int(mems_per_chunk), _ptr(off), n_chunks,
                                    int(chunk_tokens), _ptr(ctx), int(W), _ptr(alpha), _ptr(start))
        _check(rc, "locate")
        return alpha, start

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

    # ------------------------------------------------------- ragged batches
    #
    # A ragged batch is the uniform definition applied to each sequence on
    # its own sizes (Sec. 2.3: the number of memory rows follows from the
    # context length; Sec. 2.5: the assembled cache is [M* || C_local || q],
    # so the question's rows stay beside the selected ones).

    def select_ragged(self, sel_keys: np.ndarray, q_vec: np.ndarray, n_rows: np.ndarray, k: int,
                      q_rows: Optional[np.ndarray] = None, idx_stride: Optional[int] = None
                      ) -> Tuple[np.ndarray, np.ndarray]:
        """Sequence b: candidates are its rows [0, n_b) (n_b clamped into
        [0, N]); it keeps k_b = min(k, n_b) of them by the Tier-1 rule
        (select on those rows alone), then lists its q_b question rows n_b,
        ..., n_b + q_b - 1 (q_b clamped into [0, idx_stride - k_b]), then -1
        up to idx_stride.  Returns (idx [B][idx_stride] int32, k_out [B] =
        k_b + q_b)."""
        keys, _ = _keys(sel_keys)
        B, N, D = keys.shape
        stride = k if idx_stride is None else int(idx_stride)
        idx = np.full((B, stride), -1, np.int32)
        k_out = np.zeros((B,), np.int32)
        for b in range(B):
            nb = min(max(int(n_rows[b]), 0), N)
            kb = min(k, nb)
            if kb > 0:
                sel, _, _ = self.select(keys[b:b + 1, :nb], np.asarray(q_vec, np.float32)[b:b + 1], kb)
                idx[b, :kb] = sel[0]
            qb = 0 if q_rows is None else min(max(int(q_rows[b]), 0), stride - kb)
            idx[b, kb:kb + qb] = nb + np.arange(qb, dtype=np.int32)
            k_out[b] = kb + qb
        return idx, k_out

    def two_tier_decode_ragged(self, q: np.ndarray, cme_k: np.ndarray, cme_v: np.ndarray,
                               idx: Optional[np.ndarray], k_len: np.ndarray, k: int,
                               win_k: Optional[np.ndarray], win_v: Optional[np.ndarray],
                               win_count: Optional[np.ndarray], W: int, scale: float) -> np.ndarray:
        """Two-tier decode where sequence b's pool rows are its first k_b =
        k_len[b] (clamped into [0, k]) entries of idx (or rows 0..k_b-1 when
        idx is None); k is the row stride of idx."""
        B = q.shape[0]
        out = np.zeros(q.shape, np.float64)
        for b in range(B):
            kb = min(max(int(k_len[b]), 0), k)
            sl = slice(b, b + 1)
            ib = None if idx is None else np.ascontiguousarray(idx[sl, :kb])
            wk = wv = wc = None
            if W > 0:
                wk, wv, wc = win_k[sl], win_v[sl], win_count[sl]
            out[sl] = self.two_tier_decode(q[sl], cme_k[sl], cme_v[sl], ib, kb, wk, wv, wc, W, scale)
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


def select_ragged(sel_keys, q_vec, n_rows, k, q_rows=None, idx_stride=None):
    return default().select_ragged(sel_keys, q_vec, n_rows, k, q_rows, idx_stride)


def two_tier_decode_ragged(q, cme_k, cme_v, idx, k_len, k, win_k, win_v, win_count, W, scale):
    return default().two_tier_decode_ragged(q, cme_k, cme_v, idx, k_len, k, win_k, win_v, win_count, W, scale)


def row_norms(sel_keys):
    return default().row_norms(sel_keys)


def locate(norms, ctx_len, W, mems_per_chunk, n_rows=None, chunk_offset=None, chunk_tokens=0):
    return default().locate(norms, ctx_len, W, mems_per_chunk, n_rows, chunk_offset, chunk_tokens)


def denoise_scores(emb, g, n_tokens=None):
    return default().denoise_scores(emb, g, n_tokens)


def denoise_select(max_cos, tau, keep_min_every, n_tokens=None, chunk_tokens=0):
    return default().denoise_select(max_cos, tau, keep_min_every, n_tokens, chunk_tokens)


def bridge_hidden(h, w1, b1):
    return default().bridge_hidden(h, w1, b1)


def bridge_out(hidden, w2, b2, gamma, beta, nu, eps=1e-5):
    return default().bridge_out(hidden, w2, b2, gamma, beta, nu, eps)
