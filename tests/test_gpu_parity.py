"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Small shapes are compared element by element over whole tensors and span
several tiles plus ragged tails (tiles are 128 query rows x 64 keys forward,
128 keys x 64 queries for dK/dV), at head dimensions 64, 96 and 128.  The
measured workloads run at full size in the benchmark's launch configuration
and are compared over whole output tensors: the oracle computes them slice
by slice (one segment and one key/value head with its whole query-head
group is an independent problem), and the metrics are accumulated over all
slices.  The paper's B4 H48 S4096 shapes are compared on sampled slices.
"""
import math

import pytest
import torch

import oracle
from paper_2608_17379_amd import attn
from paper_2608_17379_amd import workloads as wl

from parity import (GRAD_RELL2, LSE_MAXABS, O_MAXABS, WholeTensorParity, announce, check_all,
                    gpu_fwd_bwd, max_abs, oracle_all, rel_l2, to_gpu)

pytestmark = pytest.mark.gpu


def _fixed_case(S, D, causal, Hq=2, Hkv=2, B=1, seed=0, qk_mult=1.0, dkdv_form=0):
    w = wl.small(f"b{B}_hq{Hq}_hkv{Hkv}_s{S}_d{D}_c{int(causal)}", B, Hq, Hkv, S, D, causal,
                 qk_mult=qk_mult)
    x = wl.make_inputs(w, seed)
    announce(f"fixed {w.name} seed={seed} dkdv_form={dkdv_form}")
    got = gpu_fwd_bwd(x, causal, w.scale, dkdv_form)
    ref = oracle_all(x, causal, w.scale)
    return check_all(got, ref, w.name)


def test_smallest_workload_exact_shape():
    w = wl.WORKLOADS["mha_b1_h1_s128_d64"]
    x = wl.make_inputs(w, 0)
    announce(f"workload {w.name}")
    check_all(gpu_fwd_bwd(x, w.causal, w.scale), oracle_all(x, w.causal, w.scale), w.name)


@pytest.mark.parametrize("D", [64, 96, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("S", [1, 2, 17, 63, 64, 65, 127, 128, 129, 200, 383])
def test_shapes_mha(S, D, causal):
    _fixed_case(S, D, causal)


@pytest.mark.parametrize("D", [64, 96, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Hq,Hkv", [(4, 2), (8, 2), (8, 1)])
def test_shapes_gqa(Hq, Hkv, D, causal):
    _fixed_case(190, D, causal, Hq=Hq, Hkv=Hkv, B=2)


def test_workgroup_order_short_last_window():
    """17 key/value head groups (not a multiple of the 8 XCDs) of 16 query
    heads and 8 causal blocks of 128 queries: the forward's and dQ's
    workgroup order then takes windows of two groups per XCD, the last one
    short, and leaves unused slots on some XCDs."""
    _fixed_case(1024, 64, True, Hq=16, Hkv=1, B=17)


@pytest.mark.parametrize("D", [64, 96, 128])
def test_long_ragged_sequence(D):
    _fixed_case(1000, D, True, Hq=2, Hkv=1)


def test_peaky_rows():
    _fixed_case(300, 128, True, qk_mult=4.0)


FORMS = [attn.ATTN_BWD_DKDV_ONE_PER_CU, attn.ATTN_BWD_DKDV_TWO_PER_CU]
# D = 64 has the four-wavefront (two-per-CU) form only: the one-per-CU bit
# is ignored there, so it is not crossed with D = 64.
D_FORMS = [(96, f) for f in FORMS] + [(128, f) for f in FORMS] + \
    [(64, attn.ATTN_BWD_DKDV_TWO_PER_CU)]


@pytest.mark.parametrize("D,form", D_FORMS)
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("S", [17, 65, 129, 383])
def test_dkdv_forms(S, causal, D, form):
    """Both forms of the dK/dV kernel, whichever the library would pick:
    tails inside the first and later key blocks and the causal diagonal."""
    _fixed_case(S, D, causal, dkdv_form=form)


def test_dkdv_phase_repeated_after_one_dq_phase():
    """A second dK/dV phase on the workspace of one dQ phase gives the same
    bits (the dK/dV kernels only read the workspace)."""
    w = wl.small("dkdv_repeat", 2, 4, 2, 700, 128, True)
    x = wl.make_inputs(w, 7)
    q, k, v, do, _ = to_gpu(x)
    o, lse = attn.forward(q, k, v, True, w.scale)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = attn.workspace_for(q, k)
    two = attn.ATTN_BWD_DKDV | attn.ATTN_BWD_DKDV_TWO_PER_CU
    attn.attn_bwd_phases(q, k, v, o, lse, do, dq, dk, dv, True, w.scale, ws, attn.ATTN_BWD_DQ)
    attn.attn_bwd_phases(q, k, v, o, lse, do, dq, dk, dv, True, w.scale, ws, two)
    torch.cuda.synchronize()
    first = (dk.clone(), dv.clone())
    dk.zero_()
    dv.zero_()
    attn.attn_bwd_phases(q, k, v, o, lse, do, dq, dk, dv, True, w.scale, ws, two)
    torch.cuda.synchronize()
    assert torch.equal(first[0], dk) and torch.equal(first[1], dv)
    ref = oracle_all(x, True, w.scale)
    check_all((o.cpu(), lse.cpu(), dq.cpu(), dk.cpu(), dv.cpu()), ref, "dkdv repeated")


@pytest.mark.parametrize("D,form", D_FORMS)
def test_dkdv_forms_gqa_and_packed(D, form):
    _fixed_case(190, D, True, Hq=8, Hkv=2, B=2, dkdv_form=form)
    w = wl.small(f"varlen_forms_d{D}", 6, 4, 1, 300, D, True, varlen=True)
    x = wl.make_inputs(w, 3, lengths=[1, 17, 64, 0, 130, 300])
    announce(f"packed {w.name} dkdv_form={form}")
    check_all(gpu_fwd_bwd(x, True, w.scale, form), oracle_all(x, True, w.scale), w.name)


@pytest.mark.parametrize("D", [64, 96, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 1)])
def test_packed_ragged(D, causal, Hq, Hkv):
    w = wl.small(f"varlen_hq{Hq}_hkv{Hkv}_d{D}_c{int(causal)}", 6, Hq, Hkv, 300, D, causal,
                 varlen=True)
    x = wl.make_inputs(w, 3, lengths=[1, 17, 64, 0, 130, 300])
    announce(f"packed {w.name} lengths={x.cu_seqlens}")
    check_all(gpu_fwd_bwd(x, causal, w.scale), oracle_all(x, causal, w.scale), w.name)


def test_backward_isolated_from_forward():
    """The GPU backward fed the oracle's O (as bf16) and LSE (as fp32)."""
    w = wl.small("bwd_iso", 2, 4, 2, 257, 128, True)
    x = wl.make_inputs(w, 5)
    announce("bwd isolation")
    ro, rlse = oracle.attention_forward(x.q, x.k, x.v, True, w.scale)
    rdq, rdk, rdv = oracle.attention_backward(x.q, x.k, x.v, x.do, True, w.scale)
    q, k, v, do, _ = to_gpu(x)
    o = ro.to(torch.bfloat16).cuda()
    lse = rlse.to(torch.float32).cuda()
    dq, dk, dv = attn.backward(q, k, v, o, lse, do, True, w.scale)
    torch.cuda.synchronize()
    assert rel_l2(dq, rdq) <= GRAD_RELL2
    assert rel_l2(dk, rdk) <= GRAD_RELL2
    assert rel_l2(dv, rdv) <= GRAD_RELL2


def test_deterministic_and_guard_bands():
    """Two runs are bitwise equal; nothing is written outside the outputs."""
    w = wl.small("guard", 2, 4, 2, 333, 128, True)
    x = wl.make_inputs(w, 6)
    announce("determinism + guard bands")
    q, k, v, do, _ = to_gpu(x)
    pad = 4096

    sentinel = -1536.0   # exactly representable in bf16 and fp32

    def guarded(like):
        buf = torch.full((like.numel() + 2 * pad,), sentinel, dtype=like.dtype, device=like.device)
        return buf, buf[pad:pad + like.numel()].view(like.shape)

    ob, o = guarded(q)
    lb, lse = guarded(torch.empty(x.q.shape[:3], dtype=torch.float32, device=q.device))
    attn.attn_fwd(q, k, v, o, lse, True, w.scale)
    dqb, dq = guarded(q)
    dkb, dk = guarded(k)
    dvb, dv = guarded(v)
    wsz = attn.attn_bwd_workspace_size(2, 4, 2, 333, 128)
    wsb = torch.full((wsz + 2 * pad,), 7, dtype=torch.uint8, device=q.device)
    ws = wsb[pad:pad + wsz]
    attn.attn_bwd(q, k, v, o, lse, do, dq, dk, dv, True, w.scale, ws)
    first = [t.clone() for t in (o, lse, dq, dk, dv)]
    attn.attn_fwd(q, k, v, o, lse, True, w.scale)
    attn.attn_bwd(q, k, v, o, lse, do, dq, dk, dv, True, w.scale, ws)
    torch.cuda.synchronize()
    for a, b in zip(first, (o, lse, dq, dk, dv)):
        assert torch.equal(a, b)
    for buf in (ob, lb, dqb, dkb, dvb):
        assert (buf[:pad].float() == sentinel).all() and (buf[-pad:].float() == sentinel).all()
    assert (wsb[:pad] == 7).all() and (wsb[-pad:] == 7).all()


def test_gradient_identities_on_gpu_outputs():
    """sum_j dK_j ~ 0 and sum_j dV_j ~ sum_i dO_i (per key/value head)."""
    w = wl.small("ident", 1, 4, 2, 512, 64, True)
    x = wl.make_inputs(w, 7)
    announce("gradient identities")
    o, lse, dq, dk, dv = gpu_fwd_bwd(x, True, w.scale)
    dks = dk.double().sum(2)
    assert float(dks.abs().max()) < 0.05 * float(dk.double().abs().sum(2).max())
    want = x.do.double().sum(2).view(1, 2, 2, 64).sum(2)
    assert rel_l2(dv.double().sum(2), want) < 1e-2


def test_empty_inputs_are_noops():
    dev = torch.device("cuda", 0)
    e = torch.empty(0, 2, 0, 64, dtype=torch.bfloat16, device=dev)
    lse = torch.empty(0, 2, 0, dtype=torch.float32, device=dev)
    attn.attn_fwd(e, e, e, e.clone(), lse, True, 0.125)
    q = torch.zeros(0, 2, 64, dtype=torch.bfloat16, device=dev)
    cu = torch.zeros(1, dtype=torch.int32, device=dev)
    attn.attn_fwd_varlen(q, q, q, q.clone(), torch.empty(2, 0, device=dev), cu, 1, True, 0.125,
                         cu_seqlens_host=[0])
    torch.cuda.synchronize()


# ---------------------------------------------------------------------------
# The measured workloads at full size, every head compared
# ---------------------------------------------------------------------------

def _slices(w, x):
    """Every (segment, key/value head) of a workload: with its whole
    query-head group, a slice is an independent attention problem, and the
    slices together cover every element of every output."""
    nseg = len(x.cu_seqlens) - 1 if x.cu_seqlens is not None else w.B
    return [(seg, g) for seg in range(nseg) for g in range(w.Hkv)]


def _full_size(name, heads=None, seed=0):
    """Run the workload at full size in the benchmark's launch configuration
    and compare with the oracle slice by slice: every slice when `heads` is
    None (whole-tensor metrics), else only the listed ones."""
    w = wl.WORKLOADS[name]
    x = wl.make_inputs(w, seed)
    announce(f"full-size {name}")
    q, k, v, do, cu = to_gpu(x)
    ms = x.max_seqlen if cu is not None else 0
    o, lse = attn.forward(q, k, v, w.causal, w.scale, cu_seqlens=cu, max_seqlen=ms,
                          cu_seqlens_host=x.cu_seqlens)
    dq, dk, dv = attn.backward(q, k, v, o, lse, do, w.causal, w.scale, cu_seqlens=cu,
                               max_seqlen=ms, cu_seqlens_host=x.cu_seqlens)
    torch.cuda.synchronize()
    o, lse, dq, dk, dv = (t.cpu() for t in (o, lse, dq, dk, dv))
    for t in (o, lse, dq, dk, dv):
        assert torch.isfinite(t.float()).all()
    G = w.Hq // w.Hkv
    acc = WholeTensorParity(name)
    for seg, g in (_slices(w, x) if heads is None else heads):
        hs = list(range(g * G, (g + 1) * G))
        if cu is None:
            sl = lambda t, hh: t[seg:seg + 1, hh]
            qs, dos = sl(x.q, hs), sl(x.do, hs)
            ks, vs = sl(x.k, [g]), sl(x.v, [g])
            ro, rl = oracle.attention_forward(qs, ks, vs, w.causal, w.scale)
            rdq, rdk, rdv = oracle.attention_backward(qs, ks, vs, dos, w.causal, w.scale)
            got = (sl(o, hs), sl(lse, hs), sl(dq, hs), sl(dk, [g]), sl(dv, [g]))
        else:
            a, b = x.cu_seqlens[seg], x.cu_seqlens[seg + 1]
            sl = lambda t, hh: t[a:b, hh]
            qs, dos = sl(x.q, hs), sl(x.do, hs)
            ks, vs = sl(x.k, [g]), sl(x.v, [g])
            cu1 = [0, b - a]
            ro, rl = oracle.attention_forward(qs, ks, vs, w.causal, w.scale, cu_seqlens=cu1)
            rdq, rdk, rdv = oracle.attention_backward(qs, ks, vs, dos, w.causal, w.scale,
                                                      cu_seqlens=cu1)
            got = (sl(o, hs), lse[hs, a:b], sl(dq, hs), sl(dk, [g]), sl(dv, [g]))
        acc.add(got, (ro, rl, rdq, rdk, rdv), f"seg={seg} kvhead={g}")
    if heads is None:
        assert acc.slices == len(_slices(w, x))
    return acc.finish()


@pytest.mark.parametrize("name", ["mha_causal_b4_h16_s2048_d128",
                                  "gqa_causal_b2_hq32_hkv8_s4096_d128",
                                  "long_causal_b1_h16_s16384_d128_qk2",
                                  "varlen_causal_n8_l512_8192_h32_d64",
                                  "ragged_gqa_causal_n33_t16294_hq32_hkv4_d128"])
def test_full_workload_every_head(name):
    """The four measured configurations beyond the smallest and the paper's
    ragged GQA prefill: whole output tensors against the oracle."""
    _full_size(name)


@pytest.mark.parametrize("name", [f"mha{c}_b4_h48_s4096_d{d}" for d in (64, 96, 128)
                                  for c in ("", "_causal")])
def test_full_paper_shape(name):
    """The paper's own B4 H48 S4096 shape at its three head dimensions,
    compared on sampled heads (first, middle and last batch entry)."""
    _full_size(name, [(0, 0), (1, 23), (3, 47)])
