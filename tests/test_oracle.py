"""Pins of the fp64 oracle against facts fixed by the mathematics.

None of these compares the oracle with itself: each check is a closed form,
an invariant, finite differences, a pure-Python brute force, or torch's own
independent fp64 SDPA.  Between them, a dropped term, a wrong sign, a wrong
index or a transposed operand anywhere in the oracle fails at least one
(``test_planted_mistakes_are_caught`` demonstrates it for a set of such
mistakes).
"""
import math

import pytest
import torch

import oracle
from oracle import attention as oatt
from paper_2608_17379_amd import workloads as wl

F64 = torch.float64


def rnd(gen, *shape, mult=1.0):
    return torch.randn(*shape, generator=gen, dtype=F64) * mult


# --------------------------------------------------------------------------
# closed forms
# --------------------------------------------------------------------------

def test_hand_worked_example():
    """Two keys, D=1, scale 1: scores [0, ln 3] give softmax [1/4, 3/4]."""
    q = torch.tensor([[[[1.0], [1.0]]]], dtype=F64)
    k = torch.tensor([[[[0.0], [math.log(3.0)]]]], dtype=F64)
    v = torch.tensor([[[[1.0], [5.0]]]], dtype=F64)
    do = torch.ones(1, 1, 2, 1, dtype=F64)
    o, lse = oracle.attention_forward(q, k, v, causal=False, scale=1.0)
    assert torch.allclose(o.flatten(), torch.tensor([4.0, 4.0], dtype=F64), atol=1e-14)
    assert torch.allclose(lse.flatten(), torch.full((2,), math.log(4.0), dtype=F64), atol=1e-14)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, causal=False, scale=1.0)
    # dP_ij = v_j, Delta = 4, dS = [-3/4, 3/4], dQ = dS k, dK = dS^T q, dV = P^T dO
    assert torch.allclose(dq.flatten(), torch.full((2,), 0.75 * math.log(3.0), dtype=F64), atol=1e-14)
    assert torch.allclose(dk.flatten(), torch.tensor([-1.5, 1.5], dtype=F64), atol=1e-14)
    assert torch.allclose(dv.flatten(), torch.tensor([0.5, 1.5], dtype=F64), atol=1e-14)
    # causal: row 0 sees key 0 only
    o, lse = oracle.attention_forward(q, k, v, causal=True, scale=1.0)
    assert torch.allclose(o.flatten(), torch.tensor([1.0, 4.0], dtype=F64), atol=1e-14)
    assert torch.allclose(lse.flatten(), torch.tensor([0.0, math.log(4.0)], dtype=F64), atol=1e-14)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, causal=True, scale=1.0)
    assert torch.allclose(dq.flatten(), torch.tensor([0.0, 0.75 * math.log(3.0)], dtype=F64), atol=1e-14)
    assert torch.allclose(dk.flatten(), torch.tensor([-0.75, 0.75], dtype=F64), atol=1e-14)
    assert torch.allclose(dv.flatten(), torch.tensor([1.25, 0.75], dtype=F64), atol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_equal_keys_give_mean_of_values(causal):
    gen = torch.Generator().manual_seed(1)
    B, H, S, D = 2, 3, 9, 5
    scale = 0.37
    q = rnd(gen, B, H, S, D)
    c = rnd(gen, D)
    k = c.expand(B, H, S, D).clone()
    v = rnd(gen, B, H, S, D)
    o, lse = oracle.attention_forward(q, k, v, causal, scale)
    n = torch.arange(1, S + 1, dtype=F64) if causal else torch.full((S,), float(S), dtype=F64)
    if causal:
        mean_v = v.cumsum(dim=2) / n.view(1, 1, S, 1)
    else:
        mean_v = v.mean(dim=2, keepdim=True).expand_as(v)
    assert torch.allclose(o, mean_v, atol=1e-13)
    want_lse = scale * (q @ c) + torch.log(n)
    assert torch.allclose(lse, want_lse, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_zero_queries_give_uniform_attention(causal):
    gen = torch.Generator().manual_seed(2)
    B, H, S, D = 1, 2, 7, 4
    q = torch.zeros(B, H, S, D, dtype=F64)
    k = rnd(gen, B, H, S, D)
    v = rnd(gen, B, H, S, D)
    o, lse = oracle.attention_forward(q, k, v, causal, 0.5)
    n = torch.arange(1, S + 1, dtype=F64) if causal else torch.full((S,), float(S), dtype=F64)
    want = v.cumsum(2) / n.view(1, 1, S, 1) if causal else v.mean(2, keepdim=True).expand_as(v)
    assert torch.allclose(o, want, atol=1e-13)
    assert torch.allclose(lse, torch.log(n).expand_as(lse), atol=1e-13)


def test_single_key():
    gen = torch.Generator().manual_seed(3)
    q, k, v, do = (rnd(gen, 2, 2, 1, 6) for _ in range(4))
    for causal in (False, True):
        o, lse = oracle.attention_forward(q, k, v, causal, 0.3)
        assert torch.allclose(o, v, atol=1e-15)
        assert torch.allclose(lse, 0.3 * (q * k).sum(-1), atol=1e-14)
        dq, dk, dv = oracle.attention_backward(q, k, v, do, causal, 0.3)
        assert dq.abs().max() < 1e-14 and dk.abs().max() < 1e-14
        assert torch.allclose(dv, do, atol=1e-15)


# --------------------------------------------------------------------------
# invariants
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
def test_probabilities_rows_sum_to_one(causal):
    gen = torch.Generator().manual_seed(4)
    q = rnd(gen, 2, 4, 11, 8, mult=3.0)
    k = rnd(gen, 2, 2, 11, 8, mult=3.0)
    p = oracle.attention_probs(q, k, causal, 0.35)
    assert (p >= 0).all()
    assert torch.allclose(p.sum(-1), torch.ones(2, 4, 11, dtype=F64), atol=1e-12)
    if causal:
        assert (p.triu(diagonal=1) == 0).all()


def test_causal_future_keys_do_not_matter():
    gen = torch.Generator().manual_seed(5)
    B, H, S, D = 1, 2, 10, 4
    q, k, v, do = (rnd(gen, B, H, S, D) for _ in range(4))
    i0 = 4
    k2, v2 = k.clone(), v.clone()
    k2[:, :, i0 + 1:] += rnd(gen, B, H, S - i0 - 1, D)
    v2[:, :, i0 + 1:] += rnd(gen, B, H, S - i0 - 1, D)
    o1, l1 = oracle.attention_forward(q, k, v, True, 0.5, block_rows=1)
    o2, l2 = oracle.attention_forward(q, k2, v2, True, 0.5, block_rows=1)
    assert torch.equal(o1[:, :, :i0 + 1], o2[:, :, :i0 + 1])
    assert torch.equal(l1[:, :, :i0 + 1], l2[:, :, :i0 + 1])
    assert not torch.allclose(o1[:, :, i0 + 1:], o2[:, :, i0 + 1:])
    # dO of earlier queries cannot reach later keys
    j0 = 6
    do2 = do.clone()
    do2[:, :, :j0] += rnd(gen, B, H, j0, D)
    _, dk1, dv1 = oracle.attention_backward(q, k, v, do, True, 0.5)
    _, dk2, dv2 = oracle.attention_backward(q, k, v, do2, True, 0.5)
    assert torch.allclose(dk1[:, :, j0:], dk2[:, :, j0:], atol=1e-14, rtol=0)
    assert torch.allclose(dv1[:, :, j0:], dv2[:, :, j0:], atol=1e-14, rtol=0)
    assert not torch.allclose(dv1[:, :, :j0], dv2[:, :, :j0])


@pytest.mark.parametrize("causal", [False, True])
def test_gqa_equals_repeated_kv_heads(causal):
    gen = torch.Generator().manual_seed(6)
    B, Hq, Hkv, S, D = 2, 6, 2, 8, 4
    G = Hq // Hkv
    q, do = rnd(gen, B, Hq, S, D), rnd(gen, B, Hq, S, D)
    k, v = rnd(gen, B, Hkv, S, D), rnd(gen, B, Hkv, S, D)
    kr, vr = k.repeat_interleave(G, dim=1), v.repeat_interleave(G, dim=1)
    o1, l1 = oracle.attention_forward(q, k, v, causal, 0.4)
    o2, l2 = oracle.attention_forward(q, kr, vr, causal, 0.4)
    assert torch.allclose(o1, o2, atol=1e-14) and torch.allclose(l1, l2, atol=1e-14)
    dq1, dk1, dv1 = oracle.attention_backward(q, k, v, do, causal, 0.4)
    dq2, dk2, dv2 = oracle.attention_backward(q, kr, vr, do, causal, 0.4)
    assert torch.allclose(dq1, dq2, atol=1e-13)
    assert torch.allclose(dk1, dk2.view(B, Hkv, G, S, D).sum(2), atol=1e-13)
    assert torch.allclose(dv1, dv2.view(B, Hkv, G, S, D).sum(2), atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_key_shift_invariance(causal):
    gen = torch.Generator().manual_seed(7)
    q, k, v = (rnd(gen, 1, 2, 9, 5) for _ in range(3))
    u = rnd(gen, 5)
    o1, l1 = oracle.attention_forward(q, k, v, causal, 0.6)
    o2, l2 = oracle.attention_forward(q, k + u, v, causal, 0.6)
    assert torch.allclose(o1, o2, atol=1e-13)
    assert torch.allclose(l2 - l1, 0.6 * (q @ u), atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_gradient_identities(causal):
    gen = torch.Generator().manual_seed(8)
    B, Hq, Hkv, S, D = 2, 4, 2, 12, 6
    q, do = rnd(gen, B, Hq, S, D), rnd(gen, B, Hq, S, D)
    k, v = rnd(gen, B, Hkv, S, D), rnd(gen, B, Hkv, S, D)
    o, _ = oracle.attention_forward(q, k, v, causal, 0.4)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, causal, 0.4)
    # each row of dS sums to zero, so sum_j dK_j = 0
    assert dk.sum(2).abs().max() < 1e-12
    # each row of P sums to one, so sum_j dV_j = sum_i dO_i over the group
    G = Hq // Hkv
    assert torch.allclose(dv.sum(2), do.sum(2).view(B, Hkv, G, D).sum(2), atol=1e-12)
    # sum_ij P_ij dP_ij = sum_i dO_i . O_i
    p = oracle.attention_probs(q, k, causal, 0.4)
    dp = do @ v.repeat_interleave(G, 1).transpose(-1, -2)
    assert torch.allclose((p * dp).sum(-1), (do * o).sum(-1), atol=1e-12)


def test_row_blocking_is_exact():
    gen = torch.Generator().manual_seed(9)
    q, k, v, do = (rnd(gen, 1, 2, 37, 8) for _ in range(4))
    for causal in (False, True):
        a = oracle.attention_forward(q, k, v, causal, 0.3, block_rows=5)
        b = oracle.attention_forward(q, k, v, causal, 0.3, block_rows=512)
        assert all(torch.allclose(x, y, atol=1e-14) for x, y in zip(a, b))
        a = oracle.attention_backward(q, k, v, do, causal, 0.3, block_rows=3)
        b = oracle.attention_backward(q, k, v, do, causal, 0.3, block_rows=512)
        assert all(torch.allclose(x, y, atol=1e-13) for x, y in zip(a, b))


# --------------------------------------------------------------------------
# finite differences and brute force
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
def test_gradients_match_central_finite_differences(causal):
    gen = torch.Generator().manual_seed(10)
    B, Hq, Hkv, S, D = 1, 2, 1, 6, 4
    scale = 0.45
    q, do = rnd(gen, B, Hq, S, D), rnd(gen, B, Hq, S, D)
    k, v = rnd(gen, B, Hkv, S, D), rnd(gen, B, Hkv, S, D)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, causal, scale)

    def loss(q_, k_, v_):
        o, _ = oracle.attention_forward(q_, k_, v_, causal, scale)
        return float((o * do).sum())

    h = 1e-6
    for name, t, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = torch.zeros_like(t)
        flat, nflat = t.view(-1), num.view(-1)
        for i in range(flat.numel()):
            old = float(flat[i])
            flat[i] = old + h
            lp = loss(q, k, v)
            flat[i] = old - h
            lm = loss(q, k, v)
            flat[i] = old
            nflat[i] = (lp - lm) / (2 * h)
        err = (num - g).norm() / g.norm()
        assert err < 1e-6, (name, float(err))


def _brute_forward(q, k, v, causal, scale):
    """Scalar loops with math.exp: an implementation independent of torch ops."""
    B, H, S, D = q.shape
    Hkv = k.shape[1]
    G = H // Hkv
    o = [[[[0.0] * D for _ in range(S)] for _ in range(H)] for _ in range(B)]
    lse = [[[0.0] * S for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            g = h // G
            for i in range(S):
                logits = []
                for j in range(S):
                    if causal and j > i:
                        continue
                    s = 0.0
                    for d in range(D):
                        s += float(q[b, h, i, d]) * float(k[b, g, j, d])
                    logits.append((j, scale * s))
                mx = max(x for _, x in logits)
                den = sum(math.exp(x - mx) for _, x in logits)
                lse[b][h][i] = mx + math.log(den)
                for d in range(D):
                    o[b][h][i][d] = sum(math.exp(x - mx) / den * float(v[b, g, j, d]) for j, x in logits)
    return torch.tensor(o, dtype=F64), torch.tensor(lse, dtype=F64)


@pytest.mark.parametrize("causal", [False, True])
def test_forward_matches_brute_force(causal):
    gen = torch.Generator().manual_seed(11)
    q = rnd(gen, 1, 4, 7, 3, mult=2.0)
    k = rnd(gen, 1, 2, 7, 3, mult=2.0)
    v = rnd(gen, 1, 2, 7, 3)
    o, lse = oracle.attention_forward(q, k, v, causal, 0.7)
    ob, lb = _brute_forward(q, k, v, causal, 0.7)
    assert torch.allclose(o, ob, atol=1e-13)
    assert torch.allclose(lse, lb, atol=1e-13)


# --------------------------------------------------------------------------
# torch's independent fp64 SDPA (library special case)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("hq,hkv,s,d", [(2, 2, 33, 16), (8, 2, 50, 8), (3, 1, 1, 4), (4, 4, 129, 64)])
def test_matches_torch_sdpa_fp64(causal, hq, hkv, s, d):
    gen = torch.Generator().manual_seed(12)
    B = 2
    scale = 1.0 / math.sqrt(d)
    q = rnd(gen, B, hq, s, d, mult=1.5)
    k = rnd(gen, B, hkv, s, d, mult=1.5)
    v = rnd(gen, B, hkv, s, d)
    do = rnd(gen, B, hq, s, d)
    qa, ka, va = (t.clone().requires_grad_(True) for t in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(
        qa, ka, va, is_causal=causal, scale=scale, enable_gqa=(hq != hkv))
    ref.backward(do)
    G = hq // hkv
    logits = scale * (q @ k.repeat_interleave(G, 1).transpose(-1, -2))
    if causal:
        logits = logits.masked_fill(torch.ones(s, s, dtype=torch.bool).triu(1), -math.inf)
    ref_lse = torch.logsumexp(logits, dim=-1)
    o, lse = oracle.attention_forward(q, k, v, causal, scale)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, causal, scale)
    assert torch.allclose(o, ref.detach(), atol=1e-12)
    assert torch.allclose(lse, ref_lse, atol=1e-12)
    assert torch.allclose(dq, qa.grad, atol=1e-11)
    assert torch.allclose(dk, ka.grad, atol=1e-11)
    assert torch.allclose(dv, va.grad, atol=1e-11)


# --------------------------------------------------------------------------
# packed variable-length layout
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
def test_packed_equals_per_sequence(causal):
    gen = torch.Generator().manual_seed(13)
    lens = [5, 1, 0, 9, 3]
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    T, Hq, Hkv, D = cu[-1], 4, 2, 6
    q, do = rnd(gen, T, Hq, D), rnd(gen, T, Hq, D)
    k, v = rnd(gen, T, Hkv, D), rnd(gen, T, Hkv, D)
    o, lse = oracle.attention_forward(q, k, v, causal, 0.5, cu_seqlens=cu)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, causal, 0.5, cu_seqlens=cu)
    assert o.shape == (T, Hq, D) and lse.shape == (Hq, T)
    for s in range(len(lens)):
        a, b = cu[s], cu[s + 1]
        if a == b:
            continue
        per = lambda t: t[a:b].permute(1, 0, 2).unsqueeze(0)
        o1, l1 = oracle.attention_forward(per(q), per(k), per(v), causal, 0.5)
        g1 = oracle.attention_backward(per(q), per(k), per(v), per(do), causal, 0.5)
        assert torch.allclose(o[a:b], o1[0].permute(1, 0, 2), atol=1e-14)
        assert torch.allclose(lse[:, a:b], l1[0], atol=1e-14)
        for got, want in zip((dq, dk, dv), g1):
            assert torch.allclose(got[a:b], want[0].permute(1, 0, 2), atol=1e-13)


def test_invalid_inputs_raise():
    q = torch.zeros(1, 3, 4, 2)
    k = torch.zeros(1, 2, 4, 2)
    with pytest.raises(ValueError):
        oracle.attention_forward(q, k, k, False, 1.0)
    with pytest.raises(ValueError):
        oracle.attention_forward(torch.zeros(4, 2, 2), torch.zeros(4, 2, 2), torch.zeros(4, 2, 2),
                                 False, 1.0, cu_seqlens=[0, 3, 2, 4])


# --------------------------------------------------------------------------
# the pins catch planted mistakes
# --------------------------------------------------------------------------

def _run_pins():
    """A compact subset of the pins above; returns True if all hold."""
    gen = torch.Generator().manual_seed(14)
    B, Hq, Hkv, S, D = 1, 2, 1, 6, 4
    q, do = rnd(gen, B, Hq, S, D), rnd(gen, B, Hq, S, D)
    k, v = rnd(gen, B, Hkv, S, D), rnd(gen, B, Hkv, S, D)
    ok = True
    for causal in (False, True):
        qa, ka, va = (t.clone().requires_grad_(True) for t in (q, k, v))
        ref = torch.nn.functional.scaled_dot_product_attention(
            qa, ka, va, is_causal=causal, scale=0.45, enable_gqa=True)
        ref.backward(do)
        o, lse = oracle.attention_forward(q, k, v, causal, 0.45)
        dq, dk, dv = oracle.attention_backward(q, k, v, do, causal, 0.45)
        ok &= torch.allclose(o, ref.detach(), atol=1e-10)
        ok &= bool(torch.allclose(dq, qa.grad, atol=1e-10) and torch.allclose(dk, ka.grad, atol=1e-10)
                   and torch.allclose(dv, va.grad, atol=1e-10))
        c = rnd(gen, D)
        ke = c.expand(B, Hkv, S, D).clone()
        _, l2 = oracle.attention_forward(q, ke, v, causal, 0.45)
        n = torch.arange(1, S + 1, dtype=F64) if causal else torch.full((S,), float(S), dtype=F64)
        ok &= torch.allclose(l2, 0.45 * (q @ c) + torch.log(n), atol=1e-12)
    return bool(ok)


def test_planted_mistakes_are_caught(monkeypatch):
    assert _run_pins()
    orig_scores, orig_soft, orig_bwd = oatt._scores, oatt._softmax_rows, oatt._head_backward

    def mask_diag(qb, kh, row0, causal, scale):       # strict mask hides the diagonal
        x = orig_scores(qb, kh, row0, False, scale)
        if causal:
            rows = torch.arange(row0, row0 + qb.shape[0]).unsqueeze(1)
            x = x.masked_fill(torch.arange(kh.shape[0]).unsqueeze(0) >= rows, -math.inf)
            x[:, 0] = torch.where(torch.isinf(x[:, 0]), torch.zeros_like(x[:, 0]), x[:, 0])
        return x

    def no_scale(qb, kh, row0, causal, scale):         # forgets the softmax scale
        return orig_scores(qb, kh, row0, causal, 1.0)

    def lse_no_max(x):                                 # drops m from L = m + ln l
        p, l = orig_soft(x)
        m = x.max(dim=1).values
        return p, l - m

    def bwd_no_delta(qh, kh, vh, doh, causal, scale, block_rows):  # dS = P dP
        n = qh.shape[0]
        p, _ = orig_soft(orig_scores(qh, kh, 0, causal, scale))
        ds = p * (doh @ vh.T)
        return scale * ds @ kh, scale * ds.T @ qh, p.T @ doh

    def bwd_transposed(qh, kh, vh, doh, causal, scale, block_rows):  # dV = P dO
        dq, dk, dv = orig_bwd(qh, kh, vh, doh, causal, scale, block_rows)
        p, _ = orig_soft(orig_scores(qh, kh, 0, causal, scale))
        return dq, dk, p @ doh

    for name, fn in (("_scores", mask_diag), ("_scores", no_scale), ("_softmax_rows", lse_no_max),
                     ("_head_backward", bwd_no_delta), ("_head_backward", bwd_transposed)):
        monkeypatch.setattr(oatt, name, fn)
        assert not _run_pins(), fn.__name__
        monkeypatch.undo()
    assert _run_pins()


# --------------------------------------------------------------------------
# input generator (host logic shared by both sides; no attention arithmetic)
# --------------------------------------------------------------------------

def test_workload_inputs_are_seeded_and_shaped():
    w = wl.WORKLOADS["mha_b1_h1_s128_d64"]
    a, b = wl.make_inputs(w, 0), wl.make_inputs(w, 0)
    assert a.q.dtype == torch.bfloat16 and a.q.shape == (1, 1, 128, 64)
    assert torch.equal(a.q, b.q) and torch.equal(a.do, b.do)
    assert not torch.equal(a.q, wl.make_inputs(w, 1).q)
    wv = wl.small("vl", 3, 4, 2, 64, 64, True, varlen=True)
    x = wl.make_inputs(wv, 0, lengths=[5, 0, 17])
    assert x.cu_seqlens == [0, 5, 5, 22] and x.q.shape == (22, 4, 64) and x.k.shape == (22, 2, 64)
    assert x.max_seqlen == 17


def test_ragged_prefill_lengths_are_a_composition():
    """33 positive lengths summing to 16,294 tokens, the same for a seed."""
    w = wl.WORKLOADS["ragged_gqa_causal_n33_t16294_hq32_hkv4_d128"]
    gen = torch.Generator().manual_seed(0)
    lens = wl.random_composition(gen, w.total, w.B)
    assert len(lens) == 33 and sum(lens) == 16294 and min(lens) >= 1
    assert lens == wl.random_composition(torch.Generator().manual_seed(0), w.total, w.B)
    assert wl.random_composition(torch.Generator().manual_seed(1), 5, 5) == [1] * 5
    assert wl.random_composition(torch.Generator().manual_seed(1), 7, 1) == [7]


def test_oracle_regression_fixture():
    """Oracle output on the smallest workload equals the committed fixture."""
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "oracle_mha_b1_h1_s128_d64_seed0.json")
    fx = json.load(open(path))
    w = wl.WORKLOADS[fx["workload"]]
    x = wl.make_inputs(w, fx["seed"])
    o, lse = oracle.attention_forward(x.q, x.k, x.v, w.causal, w.scale)
    dq, dk, dv = oracle.attention_backward(x.q, x.k, x.v, x.do, w.causal, w.scale)
    for i, r in enumerate(fx["rows"]):
        assert abs(float(lse[0, 0, r]) - fx["lse_rows"][i]) < 1e-12
        assert torch.allclose(o[0, 0, r, :8], torch.tensor(fx["o_rows_first8"][i], dtype=F64), atol=1e-12)
    for n, t in (("o", o), ("dq", dq), ("dk", dk), ("dv", dv)):
        assert abs(float(t.norm()) - fx["norms"][n]) < 1e-9
