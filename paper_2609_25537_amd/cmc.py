"""Thin Python binding of libcmc.so (the C ABI in include/cmc.h).

Argument marshalling only: tensors become device pointers, the current
torch stream becomes the HIP stream, status codes become exceptions.  Every
step of the computation runs in the library's HIP kernels; there is no
fallback path, and a missing library raises.

Names match the C entry points: ``cmc_select_cmes``, ``cmc_window_append``,
``cmc_two_tier_decode``, ``cmc_decode_step``, their ``*_ragged`` variants,
the two workspace queries and ``cmc_window_start``.
bf16 K/V tensors (torch.bfloat16) are passed through as their raw bits.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_PKG = os.path.dirname(os.path.abspath(__file__))
# CMC_LIBRARY may name another build of the same library (e.g. one built with
# different tuning knobs); by default the in-tree build is used.
LIBRARY = os.environ.get("CMC_LIBRARY") or os.path.join(_PKG, "libcmc.so")

CMC_OK = 0
CMC_ERR_INVALID_ARGUMENT = 1
CMC_ERR_UNSUPPORTED = 2
CMC_ERR_WORKSPACE_TOO_SMALL = 3
CMC_ERR_HIP = 4
CMC_F32 = 0
CMC_BF16 = 1

EXPORTED = [
    "cmc_select_workspace_bytes", "cmc_select_cmes", "cmc_select_cmes_ragged", "cmc_gather_tier1",
    "cmc_window_append",
    "cmc_window_start", "cmc_decode_workspace_bytes", "cmc_two_tier_decode", "cmc_decode_step",
    "cmc_two_tier_decode_ragged", "cmc_decode_step_ragged", "cmc_locate_window", "cmc_denoise_workspace_bytes",
    "cmc_denoise", "cmc_bridge_workspace_bytes", "cmc_memory_bridge", "cmc_status_string", "cmc_last_error",
    "cmc_version", "cmc_decode_step_noalloc",
]


class CmcError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            raise RuntimeError(f"{LIBRARY} is missing: build it with __graft_entry__.build() "
                               "(python -m paper_2609_25537_amd.build)")
        L = ctypes.CDLL(LIBRARY)
        P, I, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        L.cmc_select_workspace_bytes.argtypes = [I, I]
        L.cmc_select_workspace_bytes.restype = SZ
        L.cmc_select_cmes.argtypes = [P, I, P, I, I, I, I, P, P, P, SZ, P]
        L.cmc_select_cmes.restype = I
        L.cmc_window_append.argtypes = [P, P, I, P, P, P, I, I, I, I, I, P]
        L.cmc_window_append.restype = I
        L.cmc_window_start.argtypes = [ctypes.c_longlong] * 3
        L.cmc_window_start.restype = ctypes.c_longlong
        L.cmc_decode_workspace_bytes.argtypes = [I, I, I, I, I, I]
        L.cmc_decode_workspace_bytes.restype = SZ
        L.cmc_two_tier_decode.argtypes = [P, P, P, P, I, P, P, P, I, I, I, I, I, I, I,
                                          ctypes.c_float, P, P, SZ, P]
        L.cmc_two_tier_decode.restype = I
        L.cmc_decode_step.argtypes = [P, P, P, P, I, P, P, P, I, P, P, I, I, I, I, I, I, I,
                                      ctypes.c_float, P, P, SZ, P]
        L.cmc_decode_step.restype = I
        L.cmc_select_cmes_ragged.argtypes = [P, I, P, P, P, I, I, I, I, I, P, P, P, P, P, SZ, P]
        L.cmc_select_cmes_ragged.restype = I
        L.cmc_locate_window.argtypes = [P, P, P, I, I, I, P, I, I, I, P, P, P]
        L.cmc_locate_window.restype = I
        L.cmc_gather_tier1.argtypes = [P, P, I, P, P, I, I, I, I, I, I, P, P, P]
        L.cmc_gather_tier1.restype = I
        L.cmc_denoise_workspace_bytes.argtypes = [I, I]
        L.cmc_denoise_workspace_bytes.restype = SZ
        L.cmc_denoise.argtypes = [P, I, P, I, I, I, I, ctypes.c_float, I, I, P, P, P, P, P, P, P, SZ, P]
        L.cmc_denoise.restype = I
        L.cmc_bridge_workspace_bytes.argtypes = [I, I]
        L.cmc_bridge_workspace_bytes.restype = SZ
        L.cmc_memory_bridge.argtypes = [P, P, P, P, P, P, P, ctypes.c_float, ctypes.c_float, I, I, I, I, P, P, P,
                                        SZ, P]
        L.cmc_memory_bridge.restype = I
        L.cmc_select_cmes_ragged.restype = I
        L.cmc_two_tier_decode_ragged.argtypes = [P, P, P, P, P, I, P, P, P, I, I, I, I, I, I, I,
                                                 ctypes.c_float, P, P, SZ, P]
        L.cmc_two_tier_decode_ragged.restype = I
        L.cmc_decode_step_ragged.argtypes = [P, P, P, P, P, I, P, P, P, I, P, P, I, I, I, I, I, I, I,
                                             ctypes.c_float, P, P, SZ, P]
        L.cmc_decode_step_ragged.restype = I
        L.cmc_decode_step_noalloc.argtypes = [P, P, P, P, I, P, P, P, I, P, P, I, I, I, I, I, I, I,
                                              ctypes.c_float, P, P]
        L.cmc_decode_step_noalloc.restype = I
        L.cmc_status_string.argtypes = [I]
        L.cmc_status_string.restype = ctypes.c_char_p
        L.cmc_last_error.argtypes = []
        L.cmc_last_error.restype = ctypes.c_char_p
        L.cmc_version.argtypes = []
        L.cmc_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().cmc_status_string(int(s)).decode()


def last_error() -> str:
    return lib().cmc_last_error().decode()


def version() -> str:
    return lib().cmc_version().decode()


def _check(rc: int) -> None:
    if rc != CMC_OK:
        raise CmcError(rc, last_error())


def _ptr(t) -> Optional[int]:
    """Device address of a tensor (None and raw integer addresses pass
    through).  Host tensors are refused: the kernels would take their
    addresses as device memory."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError(f"cmc: tensor of shape {tuple(t.shape)} is on {t.device}; the library takes device tensors")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _kv_dtype(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return CMC_BF16
    if t.dtype == torch.float32:
        return CMC_F32
    raise TypeError(f"expected a float32 or bfloat16 tensor, got {t.dtype}")


def _need(cond: bool, msg: str) -> None:
    if not cond:
        raise ValueError(msg)


# ------------------------------------------------------------- selection

def cmc_select_workspace_bytes(B: int, N: int) -> int:
    return int(lib().cmc_select_workspace_bytes(int(B), int(N)))


def cmc_select_cmes(sel_keys, q_vec, k: int, idx_out=None, scores_out=None, workspace=None,
                    stream=None):
    """Tier-1 selection.  sel_keys [B][N][D] fp32 or bf16, q_vec [B][D] fp32
    (device).  Returns idx_out [B][k] int32 (ascending)."""
    import torch
    _need(sel_keys.dim() == 3 and sel_keys.is_contiguous(), "sel_keys must be contiguous [B][N][D]")
    B, N, D = sel_keys.shape
    _need(q_vec.shape == (B, D) and q_vec.is_contiguous(), "q_vec must be contiguous [B][D]")
    _need(q_vec.dtype == torch.float32, "q_vec must be fp32")
    if idx_out is None:
        idx_out = torch.empty((B, k), dtype=torch.int32, device=sel_keys.device)
    _need(idx_out.shape == (B, k) and idx_out.dtype == torch.int32 and idx_out.is_contiguous(),
          "idx_out must be contiguous int32 [B][k]")
    if scores_out is not None:
        _need(scores_out.shape == (B, N) and scores_out.dtype == torch.float32, "scores_out [B][N] fp32")
    ws_bytes = 0
    if scores_out is None and workspace is None:
        workspace = torch.empty(max(1, cmc_select_workspace_bytes(B, N)), dtype=torch.uint8,
                                device=sel_keys.device)
    if workspace is not None:
        ws_bytes = workspace.numel() * workspace.element_size()
    rc = lib().cmc_select_cmes(_ptr(sel_keys), _kv_dtype(sel_keys), _ptr(q_vec), B, N, D, int(k), _ptr(idx_out),
                               _ptr(scores_out), _ptr(workspace), ws_bytes, _stream(stream))
    _check(rc)
    return idx_out


def cmc_select_cmes_ragged(sel_keys, q_vec, n_rows, k: int, q_rows=None, idx_stride: Optional[int] = None,
                           idx_out=None, k_out=None, scores_out=None, norms_out=None, workspace=None,
                           stream=None):
    """Ragged Tier-1 selection: sequence b's candidates are its first
    n_rows[b] rows; q_rows[b] pinned question rows (pool rows n_b ..) follow
    the selected ones.  sel_keys fp32 or bf16; n_rows/q_rows [B] int32
    (device).  Returns (idx_out [B][idx_stride] int32, k_out [B] int32)."""
    import torch
    _need(sel_keys.dim() == 3 and sel_keys.is_contiguous(), "sel_keys must be contiguous [B][N][D]")
    B, N, D = sel_keys.shape
    _need(q_vec.shape == (B, D) and q_vec.is_contiguous(), "q_vec must be contiguous [B][D]")
    _need(q_vec.dtype == torch.float32, "q_vec must be fp32")
    _need(n_rows.shape == (B,) and n_rows.dtype == torch.int32 and n_rows.is_contiguous(), "n_rows [B] int32")
    if q_rows is not None:
        _need(q_rows.shape == (B,) and q_rows.dtype == torch.int32 and q_rows.is_contiguous(), "q_rows [B] int32")
    stride = int(k if idx_stride is None else idx_stride)
    dev = sel_keys.device
    if idx_out is None:
        idx_out = torch.empty((B, stride), dtype=torch.int32, device=dev)
    _need(idx_out.shape == (B, stride) and idx_out.dtype == torch.int32 and idx_out.is_contiguous(),
          "idx_out must be contiguous int32 [B][idx_stride]")
    if k_out is None:
        k_out = torch.empty((B,), dtype=torch.int32, device=dev)
    _need(k_out.shape == (B,) and k_out.dtype == torch.int32, "k_out [B] int32")
    if scores_out is not None:
        _need(scores_out.shape == (B, N) and scores_out.dtype == torch.float32, "scores_out [B][N] fp32")
    if norms_out is not None:
        _need(norms_out.shape == (B, N) and norms_out.dtype == torch.float32 and norms_out.is_contiguous(),
              "norms_out [B][N] fp32")
    ws_bytes = 0
    if scores_out is None and workspace is None:
        workspace = torch.empty(max(1, cmc_select_workspace_bytes(B, N)), dtype=torch.uint8, device=dev)
    if workspace is not None:
        ws_bytes = workspace.numel() * workspace.element_size()
    rc = lib().cmc_select_cmes_ragged(_ptr(sel_keys), _kv_dtype(sel_keys), _ptr(q_vec), _ptr(n_rows), _ptr(q_rows),
                                      B, N, D,
                                      int(k), stride, _ptr(idx_out), _ptr(k_out), _ptr(scores_out),
                                      _ptr(norms_out), _ptr(workspace), ws_bytes, _stream(stream))
    _check(rc)
    return idx_out, k_out


def cmc_locate_window(norms, ctx_len, W: int, mems_per_chunk: int, n_rows=None, chunk_offset=None,
                      chunk_tokens: int = 0, alpha_out=None, start_out=None, stream=None):
    """CME-guided Tier-2 window placement.  norms [B][N] fp32, ctx_len [B]
    int32, chunk_offset [B][n_chunks] int32 or None (chunk i at i *
    chunk_tokens).  Returns (alpha [B], start [B]) int32."""
    import torch
    _need(norms.dim() == 2 and norms.dtype == torch.float32 and norms.is_contiguous(), "norms [B][N] fp32")
    B, N = norms.shape
    _need(ctx_len.shape == (B,) and ctx_len.dtype == torch.int32 and ctx_len.is_contiguous(), "ctx_len [B] int32")
    if n_rows is not None:
        _need(n_rows.shape == (B,) and n_rows.dtype == torch.int32 and n_rows.is_contiguous(), "n_rows [B] int32")
    n_chunks = 0
    if chunk_offset is not None:
        _need(chunk_offset.dim() == 2 and chunk_offset.shape[0] == B and chunk_offset.dtype == torch.int32
              and chunk_offset.is_contiguous(), "chunk_offset [B][n_chunks] int32")
        n_chunks = int(chunk_offset.shape[1])
    if alpha_out is None:
        alpha_out = torch.empty((B,), dtype=torch.int32, device=norms.device)
    if start_out is None:
        start_out = torch.empty((B,), dtype=torch.int32, device=norms.device)
    _need(alpha_out.shape == (B,) and start_out.shape == (B,) and alpha_out.dtype == start_out.dtype == torch.int32,
          "alpha_out/start_out [B] int32")
    rc = lib().cmc_locate_window(_ptr(norms), _ptr(n_rows), _ptr(ctx_len), B, N, int(mems_per_chunk),
                                 _ptr(chunk_offset), n_chunks, int(chunk_tokens), int(W), _ptr(alpha_out),
                                 _ptr(start_out), _stream(stream))
    _check(rc)
    return alpha_out, start_out


# ----------------------------------------------------------- MemoryBridge

def cmc_bridge_workspace_bytes(M: int, F: int) -> int:
    return int(lib().cmc_bridge_workspace_bytes(int(M), int(F)))


def cmc_memory_bridge(h, w1, b1, w2, b2, ln_gamma, ln_beta, nu: float, ln_eps: float = 1e-5, out=None,
                      h_norms_out=None, workspace=None, stream=None):
    """MemoryBridge projection.  h [M][Hc] bf16, w1 [F][Hc] bf16, b1 [F] fp32,
    w2 [Hd][F] bf16, b2/ln_gamma/ln_beta [Hd] fp32 (device).  Returns out
    [M][Hd] fp32; the workspace (if given) then holds the hidden activations
    [M][F] bf16, and h_norms_out (if given, [M] fp32) the norms |h_j|."""
    import torch
    bf, f32 = torch.bfloat16, torch.float32
    _need(h.dim() == 2 and h.dtype == bf and h.is_contiguous(), "h must be contiguous bf16 [M][Hc]")
    M, Hc = h.shape
    _need(w1.dim() == 2 and w1.shape[1] == Hc and w1.dtype == bf and w1.is_contiguous(), "w1 [F][Hc] bf16")
    F = w1.shape[0]
    _need(w2.dim() == 2 and w2.shape[1] == F and w2.dtype == bf and w2.is_contiguous(), "w2 [Hd][F] bf16")
    Hd = w2.shape[0]
    for name, v, n in (("b1", b1, F), ("b2", b2, Hd), ("ln_gamma", ln_gamma, Hd), ("ln_beta", ln_beta, Hd)):
        _need(v.shape == (n,) and v.dtype == f32 and v.is_contiguous(), f"{name} [{n}] fp32")
    if out is None:
        out = torch.empty((M, Hd), dtype=f32, device=h.device)
    _need(out.shape == (M, Hd) and out.dtype == f32 and out.is_contiguous(), "out [M][Hd] fp32")
    if h_norms_out is not None:
        _need(h_norms_out.numel() == M and h_norms_out.dtype == f32 and h_norms_out.is_contiguous(),
              "h_norms_out [M] fp32")
    if workspace is None:
        workspace = torch.empty(max(1, cmc_bridge_workspace_bytes(M, F)), dtype=torch.uint8, device=h.device)
    ws_bytes = workspace.numel() * workspace.element_size()
    rc = lib().cmc_memory_bridge(_ptr(h), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), _ptr(ln_gamma), _ptr(ln_beta),
                                 float(nu), float(ln_eps), M, Hc, F, Hd, _ptr(out), _ptr(h_norms_out),
                                 _ptr(workspace), ws_bytes,
                                 _stream(stream))
    _check(rc)
    return out


# ------------------------------------------------------------- denoising

def cmc_denoise_workspace_bytes(B: int, n: int) -> int:
    return int(lib().cmc_denoise_workspace_bytes(int(B), int(n)))


def cmc_denoise(emb, g: int = 3, tau: float = 0.05, keep_min_every: int = 16, n_tokens=None,
                chunk_tokens: int = 0, max_cos_out=None, keep_out=None, kept_idx=None, kept_count=None,
                chunk_offset=None, n_chunks_out=None, workspace=None, stream=None):
    """Graph-based context denoising.  emb [B][n][H] fp32 or bf16 (device).
    Returns dict(kept_idx [B][n] int32, kept_count [B] int32, and when asked
    for (a tensor passed, or chunk_tokens > 0) max_cos, keep, chunk_offset,
    n_chunks)."""
    import torch
    _need(emb.dim() == 3 and emb.is_contiguous(), "emb must be contiguous [B][n][H]")
    B, n, H = emb.shape
    dev = emb.device
    dtype = _kv_dtype(emb)
    if n_tokens is not None:
        _need(n_tokens.shape == (B,) and n_tokens.dtype == torch.int32 and n_tokens.is_contiguous(),
              "n_tokens [B] int32")
    if kept_idx is None:
        kept_idx = torch.empty((B, n), dtype=torch.int32, device=dev)
    if kept_count is None:
        kept_count = torch.empty((B,), dtype=torch.int32, device=dev)
    _need(kept_idx.shape == (B, n) and kept_idx.dtype == torch.int32, "kept_idx [B][n] int32")
    _need(kept_count.shape == (B,) and kept_count.dtype == torch.int32, "kept_count [B] int32")
    if max_cos_out is not None:
        _need(max_cos_out.shape == (B, n) and max_cos_out.dtype == torch.float32, "max_cos_out [B][n] fp32")
    if keep_out is not None:
        _need(keep_out.shape == (B, n) and keep_out.dtype == torch.uint8, "keep_out [B][n] uint8")
    nch = -(-n // chunk_tokens) if chunk_tokens > 0 else 0
    if chunk_tokens > 0:
        if chunk_offset is None:
            chunk_offset = torch.empty((B, max(nch, 1)), dtype=torch.int32, device=dev)
        if n_chunks_out is None:
            n_chunks_out = torch.empty((B,), dtype=torch.int32, device=dev)
        _need(chunk_offset.dtype == torch.int32 and chunk_offset.shape[0] == B and chunk_offset.shape[1] >= nch,
              "chunk_offset [B][ceil(n/chunk_tokens)] int32")
    if workspace is None:
        workspace = torch.empty(max(1, cmc_denoise_workspace_bytes(B, n)), dtype=torch.uint8, device=dev)
    ws_bytes = workspace.numel() * workspace.element_size()
    rc = lib().cmc_denoise(_ptr(emb), dtype, _ptr(n_tokens), B, n, H, int(g), float(tau), int(keep_min_every),
                           int(chunk_tokens), _ptr(max_cos_out), _ptr(keep_out), _ptr(kept_idx), _ptr(kept_count),
                           _ptr(chunk_offset), _ptr(n_chunks_out), _ptr(workspace), ws_bytes, _stream(stream))
    _check(rc)
    r = {"kept_idx": kept_idx, "kept_count": kept_count}
    if max_cos_out is not None:
        r["max_cos"] = max_cos_out
    if keep_out is not None:
        r["keep"] = keep_out
    if chunk_tokens > 0:
        r["chunk_offset"] = chunk_offset[:, :nch]
        r["n_chunks"] = n_chunks_out
    return r


def cmc_gather_tier1(cme_k, cme_v, idx, k: int, k_len=None, out_k=None, out_v=None, stream=None):
    """Copy the selected rows' K/V into contiguous [B][Hkv][k][Dh] blocks
    (row j = pool row idx[b][j]; idx [B][idx_stride] int32 or None for rows
    0..k-1; k_len [B] int32 or None).  Returns (out_k, out_v)."""
    import torch
    _need(cme_k.dim() == 4 and cme_k.is_contiguous() and cme_v.is_contiguous() and cme_v.shape == cme_k.shape,
          "cme_k/v [B][Hkv][N][Dh]")
    B, Hkv, N, Dh = cme_k.shape
    stride = 0
    if idx is not None:
        _need(idx.dim() == 2 and idx.shape[0] == B and idx.dtype == torch.int32 and idx.is_contiguous(),
              "idx [B][idx_stride] int32")
        stride = int(idx.shape[1])
    if k_len is not None:
        _need(k_len.shape == (B,) and k_len.dtype == torch.int32 and k_len.is_contiguous(), "k_len [B] int32")
    if out_k is None:
        out_k = torch.empty((B, Hkv, k, Dh), dtype=cme_k.dtype, device=cme_k.device)
    if out_v is None:
        out_v = torch.empty((B, Hkv, k, Dh), dtype=cme_k.dtype, device=cme_k.device)
    _need(out_k.shape == (B, Hkv, k, Dh) and out_v.shape == out_k.shape and out_k.dtype == out_v.dtype == cme_k.dtype,
          "out_k/v [B][Hkv][k][Dh]")
    rc = lib().cmc_gather_tier1(_ptr(cme_k), _ptr(cme_v), _kv_dtype(cme_k), _ptr(idx), _ptr(k_len), stride, B, Hkv,
                                N, int(k), Dh, _ptr(out_k), _ptr(out_v), _stream(stream))
    _check(rc)
    return out_k, out_v


# ---------------------------------------------------------------- window

def cmc_window_start(ctx_len: int, W: int, alpha: int) -> int:
    return int(lib().cmc_window_start(int(ctx_len), int(W), int(alpha)))


def cmc_window_append(win_k, win_v, win_count, new_k, new_v, stream=None) -> None:
    """Ring append in place.  win_* [B][Hkv][W][Dh], new_* [B][Hkv][T][Dh],
    win_count [B] int32 (all on the device)."""
    import torch
    _need(win_k.dim() == 4 and win_k.is_contiguous() and win_v.is_contiguous(), "win_k/v [B][Hkv][W][Dh]")
    B, Hkv, W, Dh = win_k.shape
    _need(win_v.shape == win_k.shape and win_v.dtype == win_k.dtype, "win_v must match win_k")
    _need(new_k.dim() == 4 and new_k.shape[:2] == (B, Hkv) and new_k.shape[3] == Dh, "new_k [B][Hkv][T][Dh]")
    _need(new_v.shape == new_k.shape and new_k.dtype == win_k.dtype == new_v.dtype, "new_k/v must match")
    _need(new_k.is_contiguous() and new_v.is_contiguous(), "new_k/v must be contiguous")
    _need(win_count.shape == (B,) and win_count.dtype == torch.int32, "win_count [B] int32")
    rc = lib().cmc_window_append(_ptr(win_k), _ptr(win_v), _kv_dtype(win_k), _ptr(win_count),
                                 _ptr(new_k), _ptr(new_v), B, Hkv, W, Dh, int(new_k.shape[2]),
                                 _stream(stream))
    _check(rc)


# ---------------------------------------------------------------- decode

def cmc_decode_workspace_bytes(B: int, Hq: int, Hkv: int, Dh: int, k: int, W: int) -> int:
    return int(lib().cmc_decode_workspace_bytes(int(B), int(Hq), int(Hkv), int(Dh), int(k), int(W)))


def decode_workspace(B: int, Hq: int, Hkv: int, Dh: int, k: int, W: int, device):
    """A zero-filled decode workspace (the library keeps it zeroed)."""
    import torch
    return torch.zeros(max(1, cmc_decode_workspace_bytes(B, Hq, Hkv, Dh, k, W)), dtype=torch.uint8,
                       device=device)


def _decode_args(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, new_k, new_v, out, workspace, W, k_len,
                 noalloc=False):
    """Checks shared by the decode wrappers; returns the C call's sizes and
    the (possibly allocated) out and workspace (none with noalloc)."""
    import torch
    _need(q.dim() == 3 and q.is_contiguous() and q.dtype == torch.float32, "q must be contiguous fp32 [B][Hq][Dh]")
    B, Hq, Dh = q.shape
    _need(cme_k.dim() == 4 and cme_k.is_contiguous() and cme_v.is_contiguous(), "cme_k/v [B][Hkv][N][Dh]")
    _need(cme_k.shape[0] == B and cme_k.shape[3] == Dh and cme_v.shape == cme_k.shape, "pool shape")
    _need(cme_v.dtype == cme_k.dtype, "cme_v dtype must match cme_k")
    Hkv, N = cme_k.shape[1], cme_k.shape[2]
    if W is None:
        W = 0 if win_k is None else win_k.shape[2]
    T = 0
    if W > 0:
        _need(win_k.shape == (B, Hkv, W, Dh) and win_v.shape == win_k.shape, "window shape")
        _need(win_k.dtype == cme_k.dtype == win_v.dtype, "window dtype must match pool")
        _need(win_k.is_contiguous() and win_v.is_contiguous(), "window must be contiguous")
        _need(win_count is not None and win_count.shape == (B,) and win_count.dtype == torch.int32,
              "win_count [B] int32")
        if new_k is not None:
            _need(new_k.dim() == 4 and new_k.shape[:2] == (B, Hkv) and new_k.shape[3] == Dh,
                  "new_k [B][Hkv][T][Dh]")
            _need(new_v.shape == new_k.shape and new_k.dtype == new_v.dtype == cme_k.dtype, "new_k/v must match")
            _need(new_k.is_contiguous() and new_v.is_contiguous(), "new_k/v must be contiguous")
            T = int(new_k.shape[2])
    if idx is not None:
        _need(idx.shape == (B, k) and idx.dtype == torch.int32 and idx.is_contiguous(), "idx [B][k] int32")
    if k_len is not None:
        _need(k_len.shape == (B,) and k_len.dtype == torch.int32 and k_len.is_contiguous(), "k_len [B] int32")
    if out is None:
        out = torch.empty((B, Hq, Dh), dtype=torch.float32, device=q.device)
    _need(out.shape == (B, Hq, Dh) and out.dtype == torch.float32 and out.is_contiguous(), "out [B][Hq][Dh] fp32")
    ws_bytes = 0
    if not noalloc:
        if workspace is None:
            workspace = decode_workspace(B, Hq, Hkv, Dh, k, W, q.device)
        ws_bytes = workspace.numel() * workspace.element_size()
    win = ((_ptr(win_k), _ptr(win_v), _ptr(win_count)) if W > 0 else (None, None, None))
    new = ((_ptr(new_k), _ptr(new_v)) if W > 0 and new_k is not None else (None, None))
    return dict(B=B, Hq=Hq, Hkv=Hkv, Dh=Dh, N=N, W=int(W), T=T, win=win, new=new, out=out, workspace=workspace,
                ws_bytes=ws_bytes, dtype=_kv_dtype(cme_k))


def cmc_two_tier_decode(q, cme_k, cme_v, idx, k: int, win_k, win_v, win_count, scale: float,
                        out=None, workspace=None, W: Optional[int] = None, stream=None):
    """One decode step over [pool rows idx || ring slots].  q [B][Hq][Dh] fp32,
    cme_* [B][Hkv][N][Dh], idx [B][k] int32 or None, win_* [B][Hkv][W][Dh] or
    None (W = 0), win_count [B] int32.  Returns out [B][Hq][Dh] fp32."""
    a = _decode_args(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, None, None, out, workspace, W, None)
    rc = lib().cmc_two_tier_decode(_ptr(q), _ptr(cme_k), _ptr(cme_v), _ptr(idx), int(k), *a["win"], a["W"],
                                   a["dtype"], a["B"], a["Hq"], a["Hkv"], a["Dh"], a["N"], float(scale),
                                   _ptr(a["out"]), _ptr(a["workspace"]), a["ws_bytes"], _stream(stream))
    _check(rc)
    return a["out"]


def cmc_decode_step(q, cme_k, cme_v, idx, k: int, win_k, win_v, win_count, new_k, new_v, scale: float,
                    out=None, workspace=None, W: Optional[int] = None, stream=None):
    """Ring append of new_k/new_v [B][Hkv][T][Dh] followed by the two-tier
    decode, in one launch.  Same arguments as cmc_two_tier_decode plus the
    new rows.  Returns out [B][Hq][Dh] fp32."""
    a = _decode_args(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, new_k, new_v, out, workspace, W, None)
    rc = lib().cmc_decode_step(_ptr(q), _ptr(cme_k), _ptr(cme_v), _ptr(idx), int(k), *a["win"], a["W"],
                               *a["new"], a["T"], a["dtype"], a["B"], a["Hq"], a["Hkv"], a["Dh"], a["N"],
                               float(scale), _ptr(a["out"]), _ptr(a["workspace"]), a["ws_bytes"], _stream(stream))
    _check(rc)
    return a["out"]


def cmc_two_tier_decode_ragged(q, cme_k, cme_v, idx, k_len, k: int, win_k, win_v, win_count, scale: float,
                               out=None, workspace=None, W: Optional[int] = None, stream=None):
    """cmc_two_tier_decode with per-sequence pool-row counts k_len [B] int32
    (device); k is the row stride of idx."""
    a = _decode_args(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, None, None, out, workspace, W, k_len)
    rc = lib().cmc_two_tier_decode_ragged(_ptr(q), _ptr(cme_k), _ptr(cme_v), _ptr(idx), _ptr(k_len), int(k),
                                          *a["win"], a["W"], a["dtype"], a["B"], a["Hq"], a["Hkv"], a["Dh"],
                                          a["N"], float(scale), _ptr(a["out"]), _ptr(a["workspace"]),
                                          a["ws_bytes"], _stream(stream))
    _check(rc)
    return a["out"]


def cmc_decode_step_ragged(q, cme_k, cme_v, idx, k_len, k: int, win_k, win_v, win_count, new_k, new_v,
                           scale: float, out=None, workspace=None, W: Optional[int] = None, stream=None):
    """cmc_decode_step with per-sequence pool-row counts k_len [B] int32."""
    a = _decode_args(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, new_k, new_v, out, workspace, W, k_len)
    rc = lib().cmc_decode_step_ragged(_ptr(q), _ptr(cme_k), _ptr(cme_v), _ptr(idx), _ptr(k_len), int(k),
                                      *a["win"], a["W"], *a["new"], a["T"], a["dtype"], a["B"], a["Hq"], a["Hkv"],
                                      a["Dh"], a["N"], float(scale), _ptr(a["out"]), _ptr(a["workspace"]),
                                      a["ws_bytes"], _stream(stream))
    _check(rc)
    return a["out"]


def cmc_decode_step_noalloc(q, cme_k, cme_v, idx, k: int, win_k, win_v, win_count, new_k, new_v, scale: float,
                            out=None, W: Optional[int] = None, stream=None):
    """cmc_decode_step without a workspace: the library's fixed scratch holds
    the counters and split partials (no device allocation in the call; `out`
    must then be passed by callers that cannot allocate)."""
    a = _decode_args(q, cme_k, cme_v, idx, k, win_k, win_v, win_count, new_k, new_v, out, None, W, None,
                     noalloc=True)
    rc = lib().cmc_decode_step_noalloc(_ptr(q), _ptr(cme_k), _ptr(cme_v), _ptr(idx), int(k), *a["win"], a["W"],
                                       *a["new"], a["T"], a["dtype"], a["B"], a["Hq"], a["Hkv"], a["Dh"], a["N"],
                                       float(scale), _ptr(a["out"]), _stream(stream))
    _check(rc)
    return a["out"]
