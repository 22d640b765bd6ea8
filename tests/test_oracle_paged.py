"""Pins of the paged-cache oracle (page size 1) against facts fixed by the
definition: a pure-Python brute force of the bottom-right causal mask,
torch's own fp64 SDPA for decode, identity pages against the packed oracle
(pinned separately), invariance under a relabelling of the cache pages, and
empty requests.  ``test_planted_paged_mistakes_are_caught`` shows that a
plausible mistake in the gather or the mask alignment fails one of them.
"""
import math

import pytest
import torch

import oracle
from oracle import paged as opaged

F64 = torch.float64


def _rnd(gen, *shape, mult=1.0):
    return torch.randn(*shape, generator=gen, dtype=F64) * mult


def _case(gen, q_lens, kv_lens, hq, hkv, d, num_pages):
    """Random queries, a random cache and distinct random pages per request."""
    qo = [0]
    for n in q_lens:
        qo.append(qo[-1] + n)
    kv = [0]
    for n in kv_lens:
        kv.append(kv[-1] + n)
    q = _rnd(gen, qo[-1], hq, d)
    kc = _rnd(gen, num_pages, hkv, d)
    vc = _rnd(gen, num_pages, hkv, d)
    idx = torch.randperm(num_pages, generator=gen)[:kv[-1]].tolist()
    return q, kc, vc, qo, kv, idx


def _brute(q, kc, vc, qo, kv, idx, causal, scale):
    """Pure-Python loops over the definition: query i of a request with q_len
    queries and kv_len keys sees key j iff j <= i + kv_len - q_len (causal)."""
    tq, hq, d = q.shape
    hkv = kc.shape[1]
    g = hq // hkv
    o = [[[0.0] * d for _ in range(hq)] for _ in range(tq)]
    lse = [[-math.inf] * tq for _ in range(hq)]
    for b in range(len(qo) - 1):
        q_len, kv_len = qo[b + 1] - qo[b], kv[b + 1] - kv[b]
        pages = idx[kv[b]:kv[b + 1]]
        for i in range(q_len):
            row = qo[b] + i
            for h in range(hq):
                vis = [j for j in range(kv_len) if not causal or j <= i + kv_len - q_len]
                if not vis:
                    continue
                s = [scale * sum(float(q[row, h, t]) * float(kc[pages[j], h // g, t])
                                 for t in range(d)) for j in vis]
                m = max(s)
                e = [math.exp(x - m) for x in s]
                den = sum(e)
                lse[h][row] = m + math.log(den)
                for t in range(d):
                    o[row][h][t] = sum(e[n] * float(vc[pages[j], h // g, t])
                                       for n, j in enumerate(vis)) / den
    return torch.tensor(o, dtype=F64), torch.tensor(lse, dtype=F64)


@pytest.mark.parametrize("causal", [False, True])
def test_paged_matches_brute_force(causal):
    """Requests with fewer, equal and (for causal) more queries than keys."""
    gen = torch.Generator().manual_seed(11)
    q, kc, vc, qo, kv, idx = _case(gen, [3, 5, 1, 4], [7, 5, 6, 2], 4, 2, 3, 40)
    o, lse = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, causal, 0.7)
    bo, bl = _brute(q, kc, vc, qo, kv, idx, causal, 0.7)
    fin = torch.isfinite(bl)
    assert torch.equal(torch.isfinite(lse), fin)
    assert torch.allclose(lse[fin], bl[fin], atol=1e-12)
    assert torch.allclose(o, bo, atol=1e-12)
    if causal:
        # 4 queries over 2 keys: the first two see nothing.
        assert torch.isinf(lse[:, 9:11]).all() and (o[9:11] == 0).all()


def test_identity_pages_equal_packed_oracle():
    """Cache = the packed K/V, pages = their row numbers: the packed result."""
    gen = torch.Generator().manual_seed(12)
    lens = [9, 1, 14, 6]
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    q = _rnd(gen, cu[-1], 6, 8)
    k = _rnd(gen, cu[-1], 2, 8)
    v = _rnd(gen, cu[-1], 2, 8)
    for causal in (False, True):
        po, pl = oracle.attention_forward_paged(q, k, v, cu, cu, list(range(cu[-1])), causal, 0.3)
        ro, rl = oracle.attention_forward(q, k, v, causal, 0.3, cu_seqlens=cu)
        assert torch.allclose(po, ro, atol=1e-14) and torch.allclose(pl, rl, atol=1e-14)


def test_page_relabelling_invariance():
    """Moving every page to another slot of a larger cache (and remapping the
    indices) leaves O and LSE unchanged."""
    gen = torch.Generator().manual_seed(13)
    q, kc, vc, qo, kv, idx = _case(gen, [4, 6], [9, 6], 4, 1, 5, 30)
    perm = torch.randperm(50, generator=gen)[:30]   # old page p -> new slot perm[p]
    kc2 = _rnd(gen, 50, 1, 5)
    vc2 = _rnd(gen, 50, 1, 5)
    kc2[perm] = kc
    vc2[perm] = vc
    idx2 = [int(perm[p]) for p in idx]
    for causal in (False, True):
        a = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, causal, 0.5)
        b = oracle.attention_forward_paged(q, kc2, vc2, qo, kv, idx2, causal, 0.5)
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_decode_is_softmax_over_every_key():
    """One query per request (decode): the causal mask hides nothing, and the
    result is torch's fp64 SDPA over the gathered keys (GQA by repetition)."""
    gen = torch.Generator().manual_seed(14)
    q, kc, vc, qo, kv, idx = _case(gen, [1, 1, 1], [5, 1, 12], 6, 2, 8, 64)
    o, lse = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, True, 0.35)
    o2, lse2 = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, False, 0.35)
    assert torch.equal(o, o2) and torch.equal(lse, lse2)
    for b in range(3):
        pages = torch.tensor(idx[kv[b]:kv[b + 1]])
        kb = kc[pages].repeat_interleave(3, dim=1).transpose(0, 1)   # [Hq, kv_len, D]
        vb = vc[pages].repeat_interleave(3, dim=1).transpose(0, 1)
        qb = q[b:b + 1].transpose(0, 1)                               # [Hq, 1, D]
        ref = torch.nn.functional.scaled_dot_product_attention(qb, kb, vb, scale=0.35)
        assert torch.allclose(o[b], ref[:, 0], atol=1e-13)
        ref_l = torch.logsumexp(0.35 * (qb @ kb.transpose(1, 2)), dim=-1)[:, 0]
        assert torch.allclose(lse[:, b], ref_l, atol=1e-13)


def test_empty_requests():
    gen = torch.Generator().manual_seed(15)
    q, kc, vc, qo, kv, idx = _case(gen, [2, 0, 3], [0, 4, 3], 2, 1, 4, 10)
    o, lse = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, True, 0.5)
    assert (o[0:2] == 0).all() and torch.isinf(lse[:, 0:2]).all()
    assert torch.isfinite(lse[:, 2:5]).all()


def test_paged_input_validation():
    gen = torch.Generator().manual_seed(16)
    q, kc, vc, qo, kv, idx = _case(gen, [2], [3], 2, 1, 4, 10)
    with pytest.raises(ValueError):
        oracle.attention_forward_paged(q, kc, vc, qo, kv, [0, 1, 10], True, 0.5)
    with pytest.raises(ValueError):
        oracle.attention_forward_paged(q, kc, vc, [0, 1], kv, idx, True, 0.5)


def _paged_pins_hold():
    try:
        for causal in (False, True):
            test_paged_matches_brute_force(causal)
        test_identity_pages_equal_packed_oracle()
        test_page_relabelling_invariance()
        test_decode_is_softmax_over_every_key()
    except AssertionError:
        return False
    return True


def test_planted_paged_mistakes_are_caught(monkeypatch):
    """Top-left mask alignment, ignoring the page indices, and reversed page
    order are each rejected by the pins above."""
    orig = opaged._head_forward

    def top_left(qh, kh, vh, causal, scale, block_rows, pos0=0):
        return orig(qh, kh, vh, causal, scale, block_rows, pos0=0)

    monkeypatch.setattr(opaged, "_head_forward", top_left)
    assert not _paged_pins_hold()
    monkeypatch.undo()

    orig_fn = opaged.attention_forward_paged

    def ignore_pages(q, kc, vc, qo, kv, idx, causal, scale, block_rows=512):
        return orig_fn(q, kc, vc, qo, kv, list(range(len(idx))), causal, scale, block_rows)

    def reversed_pages(q, kc, vc, qo, kv, idx, causal, scale, block_rows=512):
        rev = []
        for b in range(len(kv) - 1):
            rev += list(reversed(idx[kv[b]:kv[b + 1]]))
        return orig_fn(q, kc, vc, qo, kv, rev, causal, scale, block_rows)

    for bad in (ignore_pages, reversed_pages):
        monkeypatch.setattr(oracle, "attention_forward_paged", bad)
        assert not _paged_pins_hold(), bad.__name__
        monkeypatch.undo()
    assert _paged_pins_hold()
