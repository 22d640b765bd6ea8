"""Plain fp64 definition of scaled-dot-product attention and its gradients.

TEST INFRASTRUCTURE ONLY (see the package docstring): never used by the
library itself.

What is computed (PTXBench, Appendix A, paragraph "Workloads"): the forward
returns the attention output O, of the same shape as Q, and the fp32
log-sum-exp L of every query row; the backward consumes Q, K, V, O, dO and L
and returns dQ, dK, dV.  Causal variants apply a lower-triangular mask (key j
visible to query i iff j <= i).  The log-sum-exp is L_i = m_i + log(l_i) with
m_i the row maximum and l_i the sum of exp(s_ij - m_i) (epilogue of the
corrected FlashAttention-3 Algorithm 2, Appendix A), i.e. the natural log of
sum_j exp(scale * q_i . k_j) over the visible keys.

Readings of points the paper leaves open (each is listed in the design notes):
  * the softmax scale is an explicit argument (1/sqrt(D) in every workload);
  * grouped-query attention maps query head h to key/value head h // (Hq/Hkv)
    and dK, dV are summed over each query-head group;
  * packed variable-length input is [T, H, D] with sequence s occupying rows
    cu_seqlens[s] .. cu_seqlens[s+1]-1; no attention crosses sequences and the
    causal mask uses positions local to each sequence;
  * a row with no visible key (only possible for empty inputs) has O = 0 and
    L = -inf.

The arithmetic is the textbook one, in fp64:
    X  = scale * Q K^T          (masked entries -inf)
    m  = rowmax X,  E = exp(X - m),  l = rowsum E,  P = E / l,  L = m + ln l
    O  = P V
    dP = dO V^T,  Delta = rowsum(P * dP),  dS = P * (dP - Delta)
    dQ = scale * dS K,  dK = scale * dS^T Q,  dV = P^T dO
Query rows are independent in this definition, so rows are processed in
blocks of at most ``block_rows`` purely to bound the fp64 temporaries; each
block still sees whole key rows (two-pass softmax, no online rescaling).
Under the causal mask a block's scores stop at the last key any of its rows
can see: the keys after it are masked for every row of the block, so they
would only contribute exact zeros to P, O and the gradients.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import torch

_F64 = torch.float64


def _as64(x: torch.Tensor) -> torch.Tensor:
    return x.detach().to(device="cpu", dtype=_F64)


def _scores(qb: torch.Tensor, kh: torch.Tensor, row0: int, causal: bool,
            scale: float) -> torch.Tensor:
    """X = scale * Q_I K^T for the query rows I = row0 .. row0+len(qb)-1."""
    x = (qb @ kh.transpose(0, 1)).mul_(scale)
    if causal:
        rows = torch.arange(row0, row0 + qb.shape[0]).unsqueeze(1)
        cols = torch.arange(kh.shape[0]).unsqueeze(0)
        x.masked_fill_(cols > rows, -math.inf)
    return x


def _softmax_rows(x: torch.Tensor):
    """Two-pass softmax of whole rows: returns P and L = m + ln(l)."""
    m = x.max(dim=1, keepdim=True).values
    # A row with every entry masked has m = -inf; it gets P = 0 and L = -inf.
    empty = torch.isinf(m) & (m < 0)
    m_safe = torch.where(empty, torch.zeros_like(m), m)
    e = (x - m_safe).exp_()   # 0 wherever x is -inf, so on every entry of an empty row
    l = e.sum(dim=1, keepdim=True)
    p = e.div_(torch.where(empty, torch.ones_like(l), l))
    lse = torch.where(empty, torch.full_like(m, -math.inf), m_safe + torch.log(l))
    return p, lse.squeeze(1)


def _visible_keys(nkeys: int, last_pos: int, causal: bool) -> int:
    """Number of leading keys a block of query rows can see: under the causal
    mask no row at a position <= last_pos sees key last_pos + 1 or later, and
    such keys would only add exact zeros to P, so they are left out."""
    return max(0, min(nkeys, last_pos + 1)) if causal else nkeys


def _head_forward(qh, kh, vh, causal, scale, block_rows, pos0=0):
    """One query head.  Query row i sits at key position pos0 + i (0 unless
    the queries are the last rows of a longer key sequence)."""
    n = qh.shape[0]
    o = torch.zeros(n, vh.shape[1], dtype=_F64)
    lse = torch.full((n,), -math.inf, dtype=_F64)
    for r0 in range(0, n, block_rows):
        r1 = min(n, r0 + block_rows)
        kend = _visible_keys(kh.shape[0], pos0 + r1 - 1, causal)
        if kend == 0:   # no row of the block sees a key: O = 0, L = -inf
            continue
        p, l = _softmax_rows(_scores(qh[r0:r1], kh[:kend], pos0 + r0, causal, scale))
        o[r0:r1] = p @ vh[:kend]
        lse[r0:r1] = l
    return o, lse


def _head_backward(qh, kh, vh, doh, causal, scale, block_rows):
    """Gradients of one query head; dk, dv are this head's share."""
    n = qh.shape[0]
    dq = torch.zeros_like(qh)
    dk = torch.zeros_like(kh)
    dv = torch.zeros_like(vh)
    for r0 in range(0, n, block_rows):
        r1 = min(n, r0 + block_rows)
        kend = _visible_keys(kh.shape[0], r1 - 1, causal)
        if kend == 0:
            continue
        kb, vb = kh[:kend], vh[:kend]
        p, _ = _softmax_rows(_scores(qh[r0:r1], kb, r0, causal, scale))
        dp = doh[r0:r1] @ vb.transpose(0, 1)
        delta = (p * dp).sum(dim=1, keepdim=True)
        ds = dp.sub_(delta).mul_(p)   # dS = P * (dP - Delta)
        dq[r0:r1] = scale * (ds @ kb)
        dk[:kend] += scale * (ds.transpose(0, 1) @ qh[r0:r1])
        dv[:kend] += p.transpose(0, 1) @ doh[r0:r1]
    return dq, dk, dv


def _segments(q, cu_seqlens):
    """Yield (segment id, row range) per batch entry or packed sequence.

    Fixed layout [B, H, S, D]: one segment per batch entry, range None.
    Packed layout [T, H, D]: one segment per sequence, range (start, end).
    """
    if cu_seqlens is None:
        for b in range(q.shape[0]):
            yield b, None
    else:
        cu = [int(c) for c in cu_seqlens]
        for s in range(len(cu) - 1):
            yield s, (cu[s], cu[s + 1])


def _check(q, k, v, cu_seqlens):
    if cu_seqlens is None:
        if q.dim() != 4 or k.dim() != 4 or v.dim() != 4:
            raise ValueError("fixed-length inputs are [B, H, S, D]")
        hq, hkv = q.shape[1], k.shape[1]
    else:
        if q.dim() != 3 or k.dim() != 3 or v.dim() != 3:
            raise ValueError("packed inputs are [T, H, D]")
        hq, hkv = q.shape[1], k.shape[1]
        cu = [int(c) for c in cu_seqlens]
        if cu[0] != 0 or any(b < a for a, b in zip(cu, cu[1:])) or cu[-1] != q.shape[0]:
            raise ValueError("cu_seqlens must start at 0, be non-decreasing and end at T")
    if hq % hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    return hq, hkv


def _head_slices(q, k, v, extra, seg, h, g, fixed):
    """fp64 2-D [L, D] slices of query head h and kv head g for one segment."""
    if fixed:
        b = seg
        sl = lambda t, hh: t[b, hh]
    else:
        a, e = seg
        sl = lambda t, hh: t[a:e, hh]
    out = [sl(q, h), sl(k, g), sl(v, g)]
    out += [sl(t, h) for t in extra]
    return out


def attention_forward(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                      causal: bool, scale: float,
                      cu_seqlens: Optional[Sequence[int]] = None,
                      block_rows: int = 512):
    """Return (O, LSE) in fp64.

    Fixed-length: q [B, Hq, S, D], k, v [B, Hkv, S, D] -> O [B, Hq, S, D],
    LSE [B, Hq, S].  Packed: q [T, Hq, D], k, v [T, Hkv, D], cu_seqlens of
    length nseq+1 -> O [T, Hq, D], LSE [Hq, T].
    """
    hq, hkv = _check(q, k, v, cu_seqlens)
    q64, k64, v64 = _as64(q), _as64(k), _as64(v)
    group = hq // hkv
    fixed = cu_seqlens is None
    o = torch.zeros(q64.shape, dtype=_F64)
    if fixed:
        lse = torch.full(q64.shape[:3], -math.inf, dtype=_F64)
    else:
        lse = torch.full((hq, q64.shape[0]), -math.inf, dtype=_F64)
    for seg_id, seg in _segments(q64, cu_seqlens):
        key = seg_id if fixed else seg
        for h in range(hq):
            g = h // group
            qh, kh, vh = _head_slices(q64, k64, v64, [], key, h, g, fixed)
            if qh.shape[0] == 0:
                continue
            oh, lh = _head_forward(qh, kh, vh, causal, scale, block_rows)
            if fixed:
                o[seg_id, h] = oh
                lse[seg_id, h] = lh
            else:
                o[seg[0]:seg[1], h] = oh
                lse[h, seg[0]:seg[1]] = lh
    return o, lse


def attention_backward(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                       do: torch.Tensor, causal: bool, scale: float,
                       cu_seqlens: Optional[Sequence[int]] = None,
                       block_rows: int = 512):
    """Return (dQ, dK, dV) in fp64 for the loss sum(dO * O).

    The probabilities are recomputed from the definition (the oracle uses its
    own exact softmax, not a caller-supplied O or LSE).  dK and dV have the
    key/value head count and are summed over each query-head group.
    """
    hq, hkv = _check(q, k, v, cu_seqlens)
    q64, k64, v64, do64 = _as64(q), _as64(k), _as64(v), _as64(do)
    group = hq // hkv
    fixed = cu_seqlens is None
    dq = torch.zeros(q64.shape, dtype=_F64)
    dk = torch.zeros(k64.shape, dtype=_F64)
    dv = torch.zeros(v64.shape, dtype=_F64)
    for seg_id, seg in _segments(q64, cu_seqlens):
        key = seg_id if fixed else seg
        for h in range(hq):
            g = h // group
            qh, kh, vh, doh = _head_slices(q64, k64, v64, [do64], key, h, g, fixed)
            if qh.shape[0] == 0:
                continue
            a, b_, c = _head_backward(qh, kh, vh, doh, causal, scale, block_rows)
            if fixed:
                dq[seg_id, h] = a
                dk[seg_id, g] += b_
                dv[seg_id, g] += c
            else:
                dq[seg[0]:seg[1], h] = a
                dk[seg[0]:seg[1], g] += b_
                dv[seg[0]:seg[1], g] += c
    return dq, dk, dv


def attention_probs(q: torch.Tensor, k: torch.Tensor, causal: bool,
                    scale: float) -> torch.Tensor:
    """Softmax probabilities P [B, Hq, S, S] for small fixed-length inputs."""
    hq, hkv = _check(q, k, k, None)
    q64, k64 = _as64(q), _as64(k)
    group = hq // hkv
    bsz, _, s, _ = q64.shape
    p = torch.zeros(bsz, hq, s, s, dtype=_F64)
    for b in range(bsz):
        for h in range(hq):
            p[b, h], _ = _softmax_rows(_scores(q64[b, h], k64[b, h // group], 0, causal, scale))
    return p
