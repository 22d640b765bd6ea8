"""Attention over a paged key/value cache (page size 1), forward, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring): never used by the
library itself.

What is computed (PTXBench, Appendix A, paragraph "Generalization attention
workloads": paged causal prefill and paged decode, page size 1, grouped-query
heads, each returning the attention output and the fp32 log-sum-exp): the
cache holds one token per page, k_cache and v_cache are [num_pages, Hkv, D];
request b owns the query rows qo_indptr[b] .. qo_indptr[b+1]-1 of the packed
query tensor q [Tq, Hq, D] and the keys/values of pages
kv_indices[kv_indptr[b]], ..., kv_indices[kv_indptr[b+1]-1], in that order.
The result per request is plain attention of its queries over those keys:

    O   = softmax(scale Q K^T + mask) V,   LSE = log sum_j exp(scale q.k_j)

with O [Tq, Hq, D] and LSE [Hq, Tq].

Reading of the causal mask when a request has fewer queries than keys (the
paper's prefill has as many of each, and a decode request has one query): the
q_len queries are the last q_len of the request's kv_len positions, so query
i (0-based within the request) sees keys j <= i + kv_len - q_len.  With
q_len = kv_len this is the lower-triangular mask; a decode query sees every
key.  Rows that see no key get O = 0 and LSE = -inf.
"""
from __future__ import annotations

import math
from typing import Sequence

import torch

from .attention import _F64, _as64, _head_forward


def attention_forward_paged(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                            qo_indptr: Sequence[int], kv_indptr: Sequence[int],
                            kv_indices: Sequence[int], causal: bool, scale: float,
                            block_rows: int = 512):
    """Return (O [Tq, Hq, D], LSE [Hq, Tq]) in fp64."""
    if q.dim() != 3 or k_cache.dim() != 3 or v_cache.shape != k_cache.shape:
        raise ValueError("q is [Tq, Hq, D]; k_cache and v_cache are [num_pages, Hkv, D]")
    qo = [int(x) for x in qo_indptr]
    kv = [int(x) for x in kv_indptr]
    idx = [int(x) for x in kv_indices]
    if len(qo) != len(kv) or qo[0] != 0 or qo[-1] != q.shape[0] or kv[0] != 0 \
            or kv[-1] != len(idx):
        raise ValueError("indptr arrays must have batch+1 entries from 0 to their totals")
    if any(b < a for a, b in zip(qo, qo[1:])) or any(b < a for a, b in zip(kv, kv[1:])):
        raise ValueError("indptr arrays must be non-decreasing")
    if any(p < 0 or p >= k_cache.shape[0] for p in idx):
        raise ValueError("page index out of range")
    hq, hkv = q.shape[1], k_cache.shape[1]
    if hq % hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    group = hq // hkv
    q64, k64, v64 = _as64(q), _as64(k_cache), _as64(v_cache)
    o = torch.zeros(q64.shape, dtype=_F64)
    lse = torch.full((hq, q64.shape[0]), -math.inf, dtype=_F64)
    for b in range(len(qo) - 1):
        qa, qb = qo[b], qo[b + 1]
        pages = torch.tensor(idx[kv[b]:kv[b + 1]], dtype=torch.long)
        kb, vb = k64[pages], v64[pages]          # [kv_len, Hkv, D], gathered in order
        q_len, kv_len = qb - qa, kb.shape[0]
        if q_len == 0:
            continue
        for h in range(hq):
            g = h // group
            oh, lh = _head_forward(q64[qa:qb, h], kb[:, g], vb[:, g], causal, scale,
                                   block_rows, pos0=kv_len - q_len)
            o[qa:qb, h] = oh
            lse[h, qa:qb] = lh
    return o, lse
