"""Seeded synthetic attention workloads.

This module only draws inputs; it holds none of the attention arithmetic, so
both the HIP library's tests and the fp64 oracle can be fed from it without
sharing any computation.

Every input is i.i.d. N(0, 1) drawn in fp32 on the CPU and rounded to bf16
with round-to-nearest-even (torch's cast), so the GPU and the oracle see the
same bits.  One ``torch.Generator`` seeded with ``seed`` draws, in order: the
packed sequence lengths (variable-length workload only), then Q, K, V and dO.
The long-sequence workload multiplies Q and K by 2 after the cast (exact in
bf16), which makes the softmax rows peaky (logit std about 4).

Shapes follow the attention workloads of PTXBench (Appendix A, "Workloads"
and "Generalization attention workloads"): bf16 Q, K, V of shape
[B, H, S, D], an fp32 log-sum-exp of shape [B, H, S], causal variants with a
lower-triangular mask, grouped-query variants with fewer key/value heads, and
ragged causal prefill over packed sequences.  The sizes below are the ones this
library is measured on; the paper's own trace files are not available, so
these synthetic tensors stand in for them.  The paper gives the ragged
prefill workload only as a sequence count and a token total, so its lengths
are drawn as a uniformly random composition of the total.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    B: int            # batch (fixed-length) or number of sequences (packed)
    Hq: int
    Hkv: int
    S: int            # sequence length (fixed-length) or max length (packed)
    D: int
    causal: bool
    qk_mult: float = 1.0
    varlen: bool = False
    len_lo: int = 0   # packed: lengths drawn uniformly in [len_lo, len_hi]
    len_hi: int = 0
    total: int = 0    # packed: if > 0, lengths are a random composition of
                      # `total` into B positive parts instead

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)


WORKLOADS = {
    "mha_b1_h1_s128_d64": Workload("mha_b1_h1_s128_d64", 1, 1, 1, 128, 64, False),
    "mha_causal_b4_h16_s2048_d128": Workload(
        "mha_causal_b4_h16_s2048_d128", 4, 16, 16, 2048, 128, True),
    "gqa_causal_b2_hq32_hkv8_s4096_d128": Workload(
        "gqa_causal_b2_hq32_hkv8_s4096_d128", 2, 32, 8, 4096, 128, True),
    "long_causal_b1_h16_s16384_d128_qk2": Workload(
        "long_causal_b1_h16_s16384_d128_qk2", 1, 16, 16, 16384, 128, True, qk_mult=2.0),
    "varlen_causal_n8_l512_8192_h32_d64": Workload(
        "varlen_causal_n8_l512_8192_h32_d64", 8, 32, 32, 8192, 64, True,
        varlen=True, len_lo=512, len_hi=8192),
    # The paper's own attention shape (B4 H48 S4096), at its three head
    # dimensions, non-causal and causal.
    **{f"mha{c}_b4_h48_s4096_d{d}": Workload(f"mha{c}_b4_h48_s4096_d{d}", 4, 48, 48, 4096, d,
                                             c == "_causal")
       for d in (64, 96, 128) for c in ("", "_causal")},
    # The paper's ragged causal prefill: 33 sequences, 16,294 tokens in all,
    # 32 query heads over 4 key/value heads, D = 128.
    "ragged_gqa_causal_n33_t16294_hq32_hkv4_d128": Workload(
        "ragged_gqa_causal_n33_t16294_hq32_hkv4_d128", 33, 32, 4, 16294, 128, True,
        varlen=True, total=16294),
}

# The configuration the headline throughput is quoted on.
HEADLINE = "mha_causal_b4_h16_s2048_d128"


@dataclass
class Inputs:
    workload: Workload
    q: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    do: torch.Tensor
    cu_seqlens: Optional[List[int]] = None

    @property
    def total(self) -> int:
        return self.q.shape[0] if self.cu_seqlens is not None else 0

    @property
    def max_seqlen(self) -> int:
        if self.cu_seqlens is None:
            return self.q.shape[2]
        cu = self.cu_seqlens
        return max(b - a for a, b in zip(cu, cu[1:]))


def random_composition(gen: torch.Generator, total: int, parts: int) -> List[int]:
    """`parts` positive lengths summing to `total`, uniform over all such
    compositions: the gaps between `parts - 1` distinct cut points drawn
    without replacement from 1 .. total - 1."""
    if parts < 1 or total < parts:
        raise ValueError("need total >= parts >= 1")
    cuts = (torch.randperm(total - 1, generator=gen)[:parts - 1] + 1).sort().values.tolist()
    bounds = [0] + cuts + [total]
    return [b - a for a, b in zip(bounds, bounds[1:])]


def _randn_bf16(gen: torch.Generator, shape) -> torch.Tensor:
    return torch.randn(*shape, generator=gen, dtype=torch.float32).to(torch.bfloat16)


def make_inputs(w: Workload, seed: int = 0, lengths: Optional[List[int]] = None) -> Inputs:
    """Draw the bf16 inputs of workload ``w`` on the CPU.

    ``lengths`` overrides the drawn packed sequence lengths (tests use it for
    ragged and empty sequences); it is ignored for fixed-length workloads.
    """
    gen = torch.Generator().manual_seed(seed)
    if w.varlen:
        if lengths is None and w.total:
            lengths = random_composition(gen, w.total, w.B)
        elif lengths is None:
            lengths = torch.randint(w.len_lo, w.len_hi + 1, (w.B,), generator=gen).tolist()
        cu = [0]
        for n in lengths:
            cu.append(cu[-1] + int(n))
        t = cu[-1]
        q = _randn_bf16(gen, (t, w.Hq, w.D))
        k = _randn_bf16(gen, (t, w.Hkv, w.D))
        v = _randn_bf16(gen, (t, w.Hkv, w.D))
        do = _randn_bf16(gen, (t, w.Hq, w.D))
    else:
        cu = None
        q = _randn_bf16(gen, (w.B, w.Hq, w.S, w.D))
        k = _randn_bf16(gen, (w.B, w.Hkv, w.S, w.D))
        v = _randn_bf16(gen, (w.B, w.Hkv, w.S, w.D))
        do = _randn_bf16(gen, (w.B, w.Hq, w.S, w.D))
    if w.qk_mult != 1.0:
        q = q * w.qk_mult
        k = k * w.qk_mult
    return Inputs(w, q, k, v, do, cu)


# ---------------------------------------------------------------------------
# Paged key/value cache (page size 1): the paper's paged causal prefill and
# paged decode workloads give head counts, the request count, the number of
# page indices and the cache size; the lengths and the pages are drawn here.
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class PagedWorkload:
    name: str
    batch: int        # requests
    Hq: int
    Hkv: int
    D: int
    nnz: int          # page indices over all requests (total keys)
    num_pages: int    # pages in the cache
    decode: bool      # one query per request (else as many queries as keys)
    causal: bool = True

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)


PAGED_WORKLOADS = {
    "paged_prefill_causal_q892_p43676_hq24_hkv8_d128": PagedWorkload(
        "paged_prefill_causal_q892_p43676_hq24_hkv8_d128", 1, 24, 8, 128, 892, 43676, False),
    "paged_decode_b15_nnz9625_p42784_hq24_hkv8_d128": PagedWorkload(
        "paged_decode_b15_nnz9625_p42784_hq24_hkv8_d128", 15, 24, 8, 128, 9625, 42784, True),
}


@dataclass
class PagedInputs:
    workload: PagedWorkload
    q: torch.Tensor            # [Tq, Hq, D] (decode: [batch, Hq, D])
    k_cache: torch.Tensor      # [num_pages, Hkv, D]
    v_cache: torch.Tensor
    qo_indptr: List[int]
    kv_indptr: List[int]
    kv_indices: List[int]

    @property
    def max_qlen(self) -> int:
        return max(b - a for a, b in zip(self.qo_indptr, self.qo_indptr[1:]))

    @property
    def max_kvlen(self) -> int:
        return max(b - a for a, b in zip(self.kv_indptr, self.kv_indptr[1:]))


def make_paged_inputs(w: PagedWorkload, seed: int = 0,
                      kv_lens: Optional[List[int]] = None) -> PagedInputs:
    """Draw, in order: the key count of each request (a random composition of
    nnz), the page of every key (distinct pages, a uniformly random subset of
    the cache in random order), then Q, the K cache and the V cache, i.i.d.
    N(0, 1) rounded to bf16.  ``kv_lens`` overrides the drawn counts (their
    sum must then be nnz)."""
    gen = torch.Generator().manual_seed(seed)
    if kv_lens is None:
        kv_lens = random_composition(gen, w.nnz, w.batch) if w.nnz >= w.batch else None
    if kv_lens is None or sum(kv_lens) != w.nnz or len(kv_lens) != w.batch:
        raise ValueError("kv_lens must be batch counts summing to nnz")
    if w.nnz > w.num_pages:
        raise ValueError("more keys than pages")
    pages = torch.randperm(w.num_pages, generator=gen)[:w.nnz].tolist()
    q_lens = [1] * w.batch if w.decode else list(kv_lens)
    qo, kv = [0], [0]
    for a, b in zip(q_lens, kv_lens):
        qo.append(qo[-1] + a)
        kv.append(kv[-1] + b)
    q = _randn_bf16(gen, (qo[-1], w.Hq, w.D))
    kc = _randn_bf16(gen, (w.num_pages, w.Hkv, w.D))
    vc = _randn_bf16(gen, (w.num_pages, w.Hkv, w.D))
    return PagedInputs(w, q, kc, vc, qo, kv, pages)


# ---------------------------------------------------------------------------
# BF16 GEMM C = A B^T (the paper's fifth primary workload)
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class GemmWorkload:
    name: str
    M: int
    N: int
    K: int


GEMM_WORKLOADS = {
    "gemm_bf16_nt_m8192_n7168_k5120": GemmWorkload("gemm_bf16_nt_m8192_n7168_k5120",
                                                   8192, 7168, 5120),
}


def make_gemm_inputs(w: GemmWorkload, seed: int = 0):
    """A [M, K] then B [N, K], i.i.d. N(0, 1) rounded to bf16."""
    gen = torch.Generator().manual_seed(seed)
    return _randn_bf16(gen, (w.M, w.K)), _randn_bf16(gen, (w.N, w.K))


def small(name: str, B: int, Hq: int, Hkv: int, S: int, D: int, causal: bool,
          varlen: bool = False, qk_mult: float = 1.0) -> Workload:
    """An ad-hoc workload for shape sweeps (same drawing recipe)."""
    return Workload(name, B, Hq, Hkv, S, D, causal, qk_mult=qk_mult, varlen=varlen,
                    len_lo=1, len_hi=max(1, S))
