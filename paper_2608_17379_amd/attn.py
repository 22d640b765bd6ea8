"""ctypes binding of libattn.so (the C ABI declared in include/attn.h).

Argument marshalling only: every function checks the tensors it is given
(device, dtype, contiguity, shapes), passes raw device pointers, the sizes and
the current HIP stream to the C entry point of the same name, and turns a
non-zero status into ``AttnError``.  All arithmetic runs in the library's HIP
kernels; there is no fallback of any kind, and loading fails loudly when the
library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libattn.so")

ATTN_OK = 0
STATUS_NAMES = {
    0: "ATTN_OK", -1: "ATTN_ERR_NULL", -2: "ATTN_ERR_SHAPE", -3: "ATTN_ERR_GQA",
    -4: "ATTN_ERR_HEAD_DIM", -5: "ATTN_ERR_ALIGN", -6: "ATTN_ERR_WORKSPACE",
    -7: "ATTN_ERR_HIP", -8: "ATTN_ERR_VALUE", -9: "ATTN_ERR_SCRATCH",
}
EXPORTS = ("attn_fwd", "attn_bwd", "attn_bwd_workspace_size", "attn_fwd_varlen",
           "attn_bwd_varlen", "attn_bwd_varlen_workspace_size", "attn_bwd_phases",
           "attn_bwd_noalloc",
           "attn_bwd_varlen_phases", "attn_bwd_dkdv_form", "attn_fwd_paged_workspace_size",
           "attn_fwd_paged_form", "attn_fwd_paged",
           "attn_decode_paged_workspace_size",
           "attn_decode_paged", "attn_decode_paged_phases", "attn_gemm_bf16_nt",
           "attn_status_string")
ATTN_BWD_DQ = 1
ATTN_BWD_DKDV = 2
ATTN_BWD_DKDV_ONE_PER_CU = 4
ATTN_BWD_DKDV_TWO_PER_CU = 8
ATTN_FWD_PAGED_UNSPLIT = 0
ATTN_FWD_PAGED_KEY_HALVES = 1
ATTN_FWD_PAGED_SPLIT = 2
ATTN_DECODE_SPLIT = 1
ATTN_DECODE_MERGE = 2
ATTN_BWD_NOALLOC_SCRATCH_BYTES = 16 << 20


class AttnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} ({attn_status_string(status)})")


_lib = None
_P, _I, _F, _Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """Load libattn.so once; raise if it is missing (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_17379_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        l.attn_fwd.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _P]
        l.attn_fwd.restype = _I
        l.attn_bwd_workspace_size.argtypes = [_I, _I, _I, _I, _I]
        l.attn_bwd_workspace_size.restype = _Z
        l.attn_bwd.argtypes = [_P] * 9 + [_I] * 6 + [_F, _P, _Z, _P]
        l.attn_bwd.restype = _I
        l.attn_fwd_varlen.argtypes = [_P] * 6 + [_I] * 7 + [_F, _P]
        l.attn_fwd_varlen.restype = _I
        l.attn_bwd_varlen_workspace_size.argtypes = [_I, _I, _I, _I]
        l.attn_bwd_varlen_workspace_size.restype = _Z
        l.attn_bwd_varlen.argtypes = [_P] * 10 + [_I] * 7 + [_F, _P, _Z, _P]
        l.attn_bwd_varlen.restype = _I
        l.attn_bwd_noalloc.argtypes = [_P] * 9 + [_I] * 6 + [_F, _P]
        l.attn_bwd_noalloc.restype = _I
        l.attn_bwd_phases.argtypes = [_P] * 9 + [_I] * 6 + [_F, _P, _Z, _I, _P]
        l.attn_bwd_phases.restype = _I
        l.attn_bwd_varlen_phases.argtypes = [_P] * 10 + [_I] * 7 + [_F, _P, _Z, _I, _P]
        l.attn_bwd_varlen_phases.restype = _I
        l.attn_bwd_dkdv_form.argtypes = [_I] * 7
        l.attn_bwd_dkdv_form.restype = _I
        l.attn_fwd_paged_workspace_size.argtypes = [_I] * 7
        l.attn_fwd_paged_workspace_size.restype = _Z
        l.attn_fwd_paged_form.argtypes = [_I] * 5
        l.attn_fwd_paged_form.restype = _I
        l.attn_fwd_paged.argtypes = [_P] * 8 + [_I] * 10 + [_F, _P, _Z, _P]
        l.attn_fwd_paged.restype = _I
        l.attn_decode_paged_workspace_size.argtypes = [_I] * 5
        l.attn_decode_paged_workspace_size.restype = _Z
        l.attn_decode_paged.argtypes = [_P] * 7 + [_I] * 7 + [_F, _P, _Z, _P]
        l.attn_decode_paged.restype = _I
        l.attn_decode_paged_phases.argtypes = [_P] * 7 + [_I] * 7 + [_F, _P, _Z, _I, _P]
        l.attn_decode_paged_phases.restype = _I
        l.attn_gemm_bf16_nt.argtypes = [_P, _P, _P, _I, _I, _I, _P]
        l.attn_gemm_bf16_nt.restype = _I
        l.attn_status_string.argtypes = [_I]
        l.attn_status_string.restype = ctypes.c_char_p
        _lib = l
    return _lib


def attn_status_string(status: int) -> str:
    return lib().attn_status_string(int(status)).decode()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _ptr(t: Optional[torch.Tensor], name: str, dtype=torch.bfloat16) -> int:
    if t is None:
        return 0
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _shape(t: torch.Tensor, want, name: str):
    if tuple(t.shape) != tuple(want):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(want)}")


def _check(status: int, where: str):
    if status != ATTN_OK:
        raise AttnError(status, where)


# --------------------------------------------------------------------------
# Fixed length [B, H, S, D]
# --------------------------------------------------------------------------

def attn_bwd_workspace_size(B: int, Hq: int, Hkv: int, S: int, D: int) -> int:
    return int(lib().attn_bwd_workspace_size(B, Hq, Hkv, S, D))


def attn_fwd(q, k, v, o, lse, causal: bool, scale: float, stream=None) -> None:
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    _shape(k, (B, Hkv, S, D), "k")
    _shape(v, (B, Hkv, S, D), "v")
    _shape(o, (B, Hq, S, D), "o")
    _shape(lse, (B, Hq, S), "lse")
    st = lib().attn_fwd(_ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"), _ptr(o, "o"),
                        _ptr(lse, "lse", torch.float32), B, Hq, Hkv, S, D, int(bool(causal)),
                        float(scale), _stream(stream))
    _check(st, "attn_fwd")


def attn_bwd_phases(q, k, v, o, lse, dO, dq, dk, dv, causal: bool, scale: float,
                    workspace: torch.Tensor, phases: int, stream=None) -> None:
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    for t, n, hh in ((k, "k", Hkv), (v, "v", Hkv), (o, "o", Hq), (dO, "dO", Hq),
                     (dq, "dq", Hq), (dk, "dk", Hkv), (dv, "dv", Hkv)):
        _shape(t, (B, hh, S, D), n)
    _shape(lse, (B, Hq, S), "lse")
    st = lib().attn_bwd_phases(_ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"), _ptr(o, "o"),
                               _ptr(lse, "lse", torch.float32), _ptr(dO, "dO"), _ptr(dq, "dq"),
                               _ptr(dk, "dk"), _ptr(dv, "dv"), B, Hq, Hkv, S, D,
                               int(bool(causal)), float(scale),
                               _ptr(workspace, "workspace", torch.uint8), workspace.numel(),
                               int(phases), _stream(stream))
    _check(st, "attn_bwd_phases")


def attn_bwd(q, k, v, o, lse, dO, dq, dk, dv, causal: bool, scale: float,
             workspace: torch.Tensor, stream=None) -> None:
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    for t, n, hh in ((k, "k", Hkv), (v, "v", Hkv), (o, "o", Hq), (dO, "dO", Hq),
                     (dq, "dq", Hq), (dk, "dk", Hkv), (dv, "dv", Hkv)):
        _shape(t, (B, hh, S, D), n)
    _shape(lse, (B, Hq, S), "lse")
    st = lib().attn_bwd(_ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"), _ptr(o, "o"),
                        _ptr(lse, "lse", torch.float32), _ptr(dO, "dO"), _ptr(dq, "dq"),
                        _ptr(dk, "dk"), _ptr(dv, "dv"), B, Hq, Hkv, S, D, int(bool(causal)),
                        float(scale), _ptr(workspace, "workspace", torch.uint8),
                        workspace.numel(), _stream(stream))
    _check(st, "attn_bwd")


def attn_bwd_noalloc(q, k, v, o, lse, dO, dq, dk, dv, causal: bool, scale: float,
                     stream=None) -> None:
    """attn_bwd with the library's own device scratch instead of a
    workspace (for callers that cannot allocate); calls that can overlap on
    one GPU race."""
    B, Hq, S, D = q.shape
    Hkv = k.shape[1]
    for t, n, hh in ((k, "k", Hkv), (v, "v", Hkv), (o, "o", Hq), (dO, "dO", Hq),
                     (dq, "dq", Hq), (dk, "dk", Hkv), (dv, "dv", Hkv)):
        _shape(t, (B, hh, S, D), n)
    _shape(lse, (B, Hq, S), "lse")
    st = lib().attn_bwd_noalloc(_ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"), _ptr(o, "o"),
                                _ptr(lse, "lse", torch.float32), _ptr(dO, "dO"), _ptr(dq, "dq"),
                                _ptr(dk, "dk"), _ptr(dv, "dv"), B, Hq, Hkv, S, D,
                                int(bool(causal)), float(scale), _stream(stream))
    _check(st, "attn_bwd_noalloc")


def attn_bwd_dkdv_form(nseg: int, Hkv: int, S: int, total: int, D: int, causal: bool,
                       packed: bool) -> int:
    """The dK/dV form the library picks (ATTN_BWD_DKDV_ONE_PER_CU or
    ATTN_BWD_DKDV_TWO_PER_CU; always the latter at D = 64)."""
    st = lib().attn_bwd_dkdv_form(nseg, Hkv, S, total, D, int(bool(causal)), int(bool(packed)))
    if st < 0:
        _check(st, "attn_bwd_dkdv_form")
    return st


# --------------------------------------------------------------------------
# Packed variable length [T, H, D]
# --------------------------------------------------------------------------

def attn_bwd_varlen_workspace_size(total: int, Hq: int, Hkv: int, D: int) -> int:
    return int(lib().attn_bwd_varlen_workspace_size(total, Hq, Hkv, D))


def check_cu_seqlens(cu_host: Sequence[int], total: int, max_seqlen: int) -> None:
    """Host-side check of the offsets the library cannot read itself."""
    cu = [int(c) for c in cu_host]
    if not cu or cu[0] != 0 or cu[-1] != total:
        raise ValueError("cu_seqlens must start at 0 and end at total")
    if any(b < a for a, b in zip(cu, cu[1:])):
        raise ValueError("cu_seqlens must be non-decreasing")
    if any(b - a > max_seqlen for a, b in zip(cu, cu[1:])):
        raise ValueError("a sequence is longer than max_seqlen")


def _varlen_common(q, k, cu_seqlens, max_seqlen, cu_seqlens_host):
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    nseq = cu_seqlens.numel() - 1
    host = cu_seqlens_host if cu_seqlens_host is not None else cu_seqlens.cpu().tolist()
    check_cu_seqlens(host, T, max_seqlen)
    return T, Hq, Hkv, D, nseq


def attn_fwd_varlen(q, k, v, o, lse, cu_seqlens, max_seqlen: int, causal: bool, scale: float,
                    stream=None, cu_seqlens_host: Optional[Sequence[int]] = None) -> None:
    T, Hq, Hkv, D, nseq = _varlen_common(q, k, cu_seqlens, max_seqlen, cu_seqlens_host)
    _shape(k, (T, Hkv, D), "k")
    _shape(v, (T, Hkv, D), "v")
    _shape(o, (T, Hq, D), "o")
    _shape(lse, (Hq, T), "lse")
    st = lib().attn_fwd_varlen(_ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"), _ptr(o, "o"),
                               _ptr(lse, "lse", torch.float32),
                               _ptr(cu_seqlens, "cu_seqlens", torch.int32), nseq, int(max_seqlen),
                               T, Hq, Hkv, D, int(bool(causal)), float(scale), _stream(stream))
    _check(st, "attn_fwd_varlen")


def attn_bwd_varlen_phases(q, k, v, o, lse, dO, dq, dk, dv, cu_seqlens, max_seqlen: int,
                           causal: bool, scale: float, workspace: torch.Tensor, phases: int,
                           stream=None, cu_seqlens_host: Optional[Sequence[int]] = None) -> None:
    T, Hq, Hkv, D, nseq = _varlen_common(q, k, cu_seqlens, max_seqlen, cu_seqlens_host)
    for t, n, hh in ((k, "k", Hkv), (v, "v", Hkv), (o, "o", Hq), (dO, "dO", Hq),
                     (dq, "dq", Hq), (dk, "dk", Hkv), (dv, "dv", Hkv)):
        _shape(t, (T, hh, D), n)
    _shape(lse, (Hq, T), "lse")
    st = lib().attn_bwd_varlen_phases(
        _ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"), _ptr(o, "o"), _ptr(lse, "lse", torch.float32),
        _ptr(dO, "dO"), _ptr(dq, "dq"), _ptr(dk, "dk"), _ptr(dv, "dv"),
        _ptr(cu_seqlens, "cu_seqlens", torch.int32), nseq, int(max_seqlen), T, Hq, Hkv, D,
        int(bool(causal)), float(scale), _ptr(workspace, "workspace", torch.uint8),
        workspace.numel(), int(phases), _stream(stream))
    _check(st, "attn_bwd_varlen_phases")


def attn_bwd_varlen(q, k, v, o, lse, dO, dq, dk, dv, cu_seqlens, max_seqlen: int, causal: bool,
                    scale: float, workspace: torch.Tensor, stream=None,
                    cu_seqlens_host: Optional[Sequence[int]] = None) -> None:
    T, Hq, Hkv, D, nseq = _varlen_common(q, k, cu_seqlens, max_seqlen, cu_seqlens_host)
    for t, n, hh in ((k, "k", Hkv), (v, "v", Hkv), (o, "o", Hq), (dO, "dO", Hq),
                     (dq, "dq", Hq), (dk, "dk", Hkv), (dv, "dv", Hkv)):
        _shape(t, (T, hh, D), n)
    _shape(lse, (Hq, T), "lse")
    st = lib().attn_bwd_varlen(_ptr(q, "q"), _ptr(k, "k"), _ptr(v, "v"), _ptr(o, "o"),
                               _ptr(lse, "lse", torch.float32), _ptr(dO, "dO"), _ptr(dq, "dq"),
                               _ptr(dk, "dk"), _ptr(dv, "dv"),
                               _ptr(cu_seqlens, "cu_seqlens", torch.int32), nseq, int(max_seqlen),
                               T, Hq, Hkv, D, int(bool(causal)), float(scale),
                               _ptr(workspace, "workspace", torch.uint8), workspace.numel(),
                               _stream(stream))
    _check(st, "attn_bwd_varlen")


# --------------------------------------------------------------------------
# Paged key/value cache, page size 1 (forward only)
# --------------------------------------------------------------------------

def _host_list(t, host):
    return [int(x) for x in (host if host is not None else t.cpu().tolist())]


def check_paged_host(kv_host: Sequence[int], idx_host: Sequence[int], num_pages: int,
                     max_kvlen: Optional[int] = None) -> None:
    """Host-side check of the page arrays the library cannot read itself."""
    if not kv_host or kv_host[0] != 0 or kv_host[-1] != len(idx_host):
        raise ValueError("kv_indptr must start at 0 and end at len(kv_indices)")
    if any(b < a for a, b in zip(kv_host, kv_host[1:])):
        raise ValueError("kv_indptr must be non-decreasing")
    if any(p < 0 or p >= num_pages for p in idx_host):
        raise ValueError("a page index is outside the cache")
    if max_kvlen is not None and any(b - a > max_kvlen for a, b in zip(kv_host, kv_host[1:])):
        raise ValueError("a request has more than max_kvlen keys")


def attn_fwd_paged_workspace_size(batch: int, max_qlen: int, total_q: int, max_kvlen: int,
                                  Hq: int, Hkv: int, D: int) -> int:
    return int(lib().attn_fwd_paged_workspace_size(batch, max_qlen, total_q, max_kvlen, Hq,
                                                   Hkv, D))


def attn_fwd_paged(q, k_cache, v_cache, o, lse, qo_indptr, kv_indptr, kv_indices,
                   max_qlen: int, max_kvlen: int, causal: bool, scale: float, workspace=None,
                   stream=None, qo_indptr_host=None, kv_indptr_host=None, kv_indices_host=None,
                   checked: bool = False) -> None:
    """Paged prefill.  The index arrays are checked on the host (from the
    *_host copies when given, else from a device-to-host copy) unless
    `checked` says the caller has already done so with check_cu_seqlens and
    check_paged_host for these arrays.  `workspace` None runs the prefill
    unsplit (see attn_fwd_paged_workspace_size)."""
    Tq, Hq, D = q.shape
    P, Hkv = k_cache.shape[0], k_cache.shape[1]
    _shape(k_cache, (P, Hkv, D), "k_cache")
    _shape(v_cache, (P, Hkv, D), "v_cache")
    _shape(o, (Tq, Hq, D), "o")
    _shape(lse, (Hq, Tq), "lse")
    batch = qo_indptr.numel() - 1
    if kv_indptr.numel() != batch + 1:
        raise ValueError("qo_indptr and kv_indptr must have the same length")
    if not checked:
        check_cu_seqlens(_host_list(qo_indptr, qo_indptr_host), Tq, max_qlen)
        check_paged_host(_host_list(kv_indptr, kv_indptr_host),
                         _host_list(kv_indices, kv_indices_host), P, max_kvlen)
    nnz = kv_indices.numel()
    st = lib().attn_fwd_paged(_ptr(q, "q"), _ptr(k_cache, "k_cache"), _ptr(v_cache, "v_cache"),
                              _ptr(o, "o"), _ptr(lse, "lse", torch.float32),
                              _ptr(qo_indptr, "qo_indptr", torch.int32),
                              _ptr(kv_indptr, "kv_indptr", torch.int32),
                              _ptr(kv_indices, "kv_indices", torch.int32) if nnz else 0,
                              batch, int(max_qlen), Tq, int(max_kvlen), nnz, P, Hq, Hkv, D,
                              int(bool(causal)), float(scale),
                              _ptr(workspace, "workspace", torch.uint8) if workspace is not None
                              else 0,
                              workspace.numel() if workspace is not None else 0, _stream(stream))
    _check(st, "attn_fwd_paged")


def attn_decode_paged_workspace_size(batch: int, max_kvlen: int, Hq: int, Hkv: int, D: int) -> int:
    return int(lib().attn_decode_paged_workspace_size(batch, max_kvlen, Hq, Hkv, D))


def attn_decode_paged(q, k_cache, v_cache, o, lse, kv_indptr, kv_indices, max_kvlen: int,
                      scale: float, workspace: torch.Tensor, stream=None,
                      kv_indptr_host=None, kv_indices_host=None, checked: bool = False) -> None:
    """Paged decode (see attn_fwd_paged for `checked` and the host copies)."""
    attn_decode_paged_phases(q, k_cache, v_cache, o, lse, kv_indptr, kv_indices, max_kvlen,
                             scale, workspace, ATTN_DECODE_SPLIT | ATTN_DECODE_MERGE, stream,
                             kv_indptr_host, kv_indices_host, checked)


def attn_decode_paged_phases(q, k_cache, v_cache, o, lse, kv_indptr, kv_indices, max_kvlen: int,
                             scale: float, workspace: torch.Tensor, phases: int, stream=None,
                             kv_indptr_host=None, kv_indices_host=None,
                             checked: bool = False) -> None:
    batch, Hq, D = q.shape
    P, Hkv = k_cache.shape[0], k_cache.shape[1]
    _shape(k_cache, (P, Hkv, D), "k_cache")
    _shape(v_cache, (P, Hkv, D), "v_cache")
    _shape(o, (batch, Hq, D), "o")
    _shape(lse, (Hq, batch), "lse")
    _shape(kv_indptr, (batch + 1,), "kv_indptr")
    if not checked:
        check_paged_host(_host_list(kv_indptr, kv_indptr_host),
                         _host_list(kv_indices, kv_indices_host), P, max_kvlen)
    nnz = kv_indices.numel()
    st = lib().attn_decode_paged_phases(
        _ptr(q, "q"), _ptr(k_cache, "k_cache"), _ptr(v_cache, "v_cache"), _ptr(o, "o"),
        _ptr(lse, "lse", torch.float32), _ptr(kv_indptr, "kv_indptr", torch.int32),
        _ptr(kv_indices, "kv_indices", torch.int32) if nnz else 0, batch, int(max_kvlen), nnz, P,
        Hq, Hkv, D, float(scale), _ptr(workspace, "workspace", torch.uint8), workspace.numel(),
        int(phases), _stream(stream))
    _check(st, "attn_decode_paged_phases")


# --------------------------------------------------------------------------
# BF16 GEMM C = A B^T
# --------------------------------------------------------------------------

def attn_gemm_bf16_nt(a, b, c, stream=None) -> None:
    M, K = a.shape
    N = b.shape[0]
    _shape(b, (N, K), "b")
    _shape(c, (M, N), "c")
    st = lib().attn_gemm_bf16_nt(_ptr(a, "a"), _ptr(b, "b"), _ptr(c, "c"), M, N, K,
                                 _stream(stream))
    _check(st, "attn_gemm_bf16_nt")


def gemm_nt(a, b):
    """Return C = A B^T (bf16) for A [M, K], B [N, K]."""
    c = torch.empty((a.shape[0], b.shape[0]), dtype=torch.bfloat16, device=a.device)
    attn_gemm_bf16_nt(a, b, c)
    return c


# --------------------------------------------------------------------------
# Allocating conveniences (torch allocates the outputs; the library fills them)
# --------------------------------------------------------------------------

def attn_fwd_paged_form(batch: int, max_qlen: int, max_kvlen: int, Hq: int,
                        with_workspace: bool) -> int:
    """The form attn_fwd_paged runs (ATTN_FWD_PAGED_UNSPLIT, _KEY_HALVES or
    _SPLIT) for these shapes, with or without a workspace."""
    st = lib().attn_fwd_paged_form(batch, max_qlen, max_kvlen, Hq, int(bool(with_workspace)))
    if st < 0:
        _check(st, "attn_fwd_paged_form")
    return st


def prefill_workspace_for(q, k_cache, batch: int, max_qlen: int, max_kvlen: int):
    """The workspace attn_fwd_paged needs for these shapes, or None when it
    runs unsplit."""
    Tq, Hq, D = q.shape
    n = attn_fwd_paged_workspace_size(batch, max_qlen, Tq, max_kvlen, Hq, k_cache.shape[1], D)
    return torch.empty(n, dtype=torch.uint8, device=q.device) if n else None


def forward_paged(q, k_cache, v_cache, qo_indptr, kv_indptr, kv_indices, max_qlen: int,
                  causal: bool, scale: float, max_kvlen: Optional[int] = None,
                  split: bool = True, **host):
    """Return (o, lse) of a paged prefill (packed queries).  max_kvlen
    defaults to the longest request of kv_indptr; split False runs the
    prefill unsplit."""
    if max_kvlen is None:
        kv = _host_list(kv_indptr, host.get("kv_indptr_host"))
        max_kvlen = max((b - a for a, b in zip(kv, kv[1:])), default=0)
    o = torch.empty_like(q)
    lse = torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32, device=q.device)
    ws = (prefill_workspace_for(q, k_cache, qo_indptr.numel() - 1, max_qlen, max_kvlen)
          if split else None)
    attn_fwd_paged(q, k_cache, v_cache, o, lse, qo_indptr, kv_indptr, kv_indices, max_qlen,
                   max_kvlen, causal, scale, ws, **host)
    return o, lse


def decode_workspace_for(q, k_cache, max_kvlen: int) -> torch.Tensor:
    batch, Hq, D = q.shape
    n = attn_decode_paged_workspace_size(batch, max_kvlen, Hq, k_cache.shape[1], D)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=q.device)


def decode_paged(q, k_cache, v_cache, kv_indptr, kv_indices, max_kvlen: int, scale: float,
                 workspace=None, **host):
    """Return (o, lse) of a paged decode step (one query per request)."""
    o = torch.empty_like(q)
    lse = torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32, device=q.device)
    ws = workspace if workspace is not None else decode_workspace_for(q, k_cache, max_kvlen)
    attn_decode_paged(q, k_cache, v_cache, o, lse, kv_indptr, kv_indices, max_kvlen, scale, ws,
                      **host)
    return o, lse

def forward(q, k, v, causal: bool, scale: float, cu_seqlens=None, max_seqlen: int = 0,
            cu_seqlens_host=None):
    """Return (o, lse) for fixed-length or packed inputs."""
    o = torch.empty_like(q)
    if cu_seqlens is None:
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
        attn_fwd(q, k, v, o, lse, causal, scale)
    else:
        lse = torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32, device=q.device)
        attn_fwd_varlen(q, k, v, o, lse, cu_seqlens, max_seqlen, causal, scale,
                        cu_seqlens_host=cu_seqlens_host)
    return o, lse


def workspace_for(q, k, cu_seqlens=None) -> torch.Tensor:
    if cu_seqlens is None:
        B, Hq, S, D = q.shape
        n = attn_bwd_workspace_size(B, Hq, k.shape[1], S, D)
    else:
        T, Hq, D = q.shape
        n = attn_bwd_varlen_workspace_size(T, Hq, k.shape[1], D)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=q.device)


def backward(q, k, v, o, lse, dO, causal: bool, scale: float, cu_seqlens=None,
             max_seqlen: int = 0, workspace=None, cu_seqlens_host=None, dkdv_form: int = 0):
    """Return (dq, dk, dv) for fixed-length or packed inputs.  dkdv_form 0
    lets the library choose the dK/dV kernel's form; ATTN_BWD_DKDV_ONE_PER_CU
    or ATTN_BWD_DKDV_TWO_PER_CU forces one."""
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = workspace if workspace is not None else workspace_for(q, k, cu_seqlens)
    phases = ATTN_BWD_DQ | ATTN_BWD_DKDV | int(dkdv_form)
    if cu_seqlens is None:
        if dkdv_form:
            attn_bwd_phases(q, k, v, o, lse, dO, dq, dk, dv, causal, scale, ws, phases)
        else:
            attn_bwd(q, k, v, o, lse, dO, dq, dk, dv, causal, scale, ws)
    elif dkdv_form:
        attn_bwd_varlen_phases(q, k, v, o, lse, dO, dq, dk, dv, cu_seqlens, max_seqlen, causal,
                               scale, ws, phases, cu_seqlens_host=cu_seqlens_host)
    else:
        attn_bwd_varlen(q, k, v, o, lse, dO, dq, dk, dv, cu_seqlens, max_seqlen, causal, scale,
                        ws, cu_seqlens_host=cu_seqlens_host)
    return dq, dk, dv
