"""GPU parity of the paged-cache entry points (page size 1) against the fp64
oracle: paged prefill through attn_fwd_paged and decode through
attn_decode_paged, called through the C ABI by the binding.

Small cases span several key tiles (64 keys forward), several decode chunks
(64 keys) and ragged tails, with head dimensions 64, 96 and 128, grouped
query heads, requests with fewer queries than keys, and empty requests.
Paged prefill runs in each of its three forms: split into 256-key chunks
with a merge (what the library does, given a workspace, when the unsplit
grid would leave more than half the CUs idle: the two-head cases here),
the 8-wavefront key-halves form (an unsplit grid with fewer workgroups
than CUs: the two-head cases without a workspace, the grouped four-head
cases, 192 workgroups, either way, and the paper's prefill) and the plain
unsplit form (the six-head cases, 288 workgroups).  The
split cases include blocks of one to four chunks and ragged last chunks;
the key-halves cases include requests whose keys all fall in one tile (one
half sees none) and rows that see no key.  The paper's two paged workloads
run at full size, compared on every head.
"""
import pytest
import torch

import oracle
from paper_2608_17379_amd import attn
from paper_2608_17379_amd import workloads as wl

from parity import LSE_MAXABS, O_MAXABS, announce, max_abs

pytestmark = pytest.mark.gpu


def _indptr(lens):
    out = [0]
    for n in lens:
        out.append(out[-1] + n)
    return out


def _draw(seed, q_lens, kv_lens, hq, hkv, d, num_pages):
    gen = torch.Generator().manual_seed(seed)
    nnz = sum(kv_lens)
    pages = torch.randperm(num_pages, generator=gen)[:nnz].tolist()
    q = torch.randn(sum(q_lens), hq, d, generator=gen).to(torch.bfloat16)
    kc = torch.randn(num_pages, hkv, d, generator=gen).to(torch.bfloat16)
    vc = torch.randn(num_pages, hkv, d, generator=gen).to(torch.bfloat16)
    return q, kc, vc, _indptr(q_lens), _indptr(kv_lens), pages


def _dev(*ts):
    return [t.cuda() for t in ts]


def _i32(xs):
    return torch.tensor(xs, dtype=torch.int32, device="cuda")


def _check(o, lse, ro, rl, label):
    eo, el = max_abs(o.cpu(), ro), max_abs(lse.cpu(), rl)
    announce(f"{label}: o_maxabs={eo:.3g} lse_maxabs={el:.3g}")
    assert eo <= O_MAXABS, (label, eo)
    assert el <= LSE_MAXABS, (label, el)


def _prefill(q, kc, vc, qo, kv, idx, causal, scale, label, split=True, form=None):
    """Paged prefill against the oracle; `form`, when given, is the form
    (attn.ATTN_FWD_PAGED_*) the library must report for these shapes."""
    if form is not None:
        got = attn.attn_fwd_paged_form(len(qo) - 1, max(b - a for a, b in zip(qo, qo[1:])),
                                       max(b - a for a, b in zip(kv, kv[1:])), q.shape[1],
                                       split)
        assert got == form, (label, got, form)
    dq, dkc, dvc = _dev(q, kc, vc)
    o, lse = attn.forward_paged(dq, dkc, dvc, _i32(qo), _i32(kv), _i32(idx),
                                max(b - a for a, b in zip(qo, qo[1:])), causal, scale,
                                split=split, qo_indptr_host=qo, kv_indptr_host=kv,
                                kv_indices_host=idx)
    torch.cuda.synchronize()
    ro, rl = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, causal, scale)
    _check(o, lse, ro, rl, label)


@pytest.mark.parametrize("split", [True, False])
@pytest.mark.parametrize("D", [64, 96, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 2), (6, 2)])
def test_paged_prefill(D, causal, Hq, Hkv, split):
    # q_len == kv_len, q_len < kv_len (a continued prefill), one key, a
    # request with more queries than keys, an empty request, a request of
    # blocks with one to four 256-key chunks (the last ragged), and one with
    # more queries than keys over several chunks
    q_lens = [200, 37, 1, 70, 0, 129, 700, 600]
    kv_lens = [200, 300, 1, 5, 0, 129, 900, 520]
    args = _draw(1, q_lens, kv_lens, Hq, Hkv, D, 4000)
    # 8 requests x Hq heads x 6 blocks of 128 queries: 96, 192 or 288 workgroups
    form = {2: attn.ATTN_FWD_PAGED_SPLIT if split else attn.ATTN_FWD_PAGED_KEY_HALVES,
            4: attn.ATTN_FWD_PAGED_KEY_HALVES, 6: attn.ATTN_FWD_PAGED_UNSPLIT}[Hq]
    announce(f"paged prefill D={D} causal={causal} Hq={Hq} Hkv={Hkv} split={split} form={form}")
    _prefill(*args, causal, D ** -0.5, f"prefill d{D} c{int(causal)} g{Hq // Hkv} s{int(split)}",
             split, form)


def _decode(q, kc, vc, kv, idx, max_kvlen, scale, label):
    dq, dkc, dvc = _dev(q, kc, vc)
    o, lse = attn.decode_paged(dq, dkc, dvc, _i32(kv), _i32(idx), max_kvlen, scale,
                               kv_indptr_host=kv, kv_indices_host=idx)
    torch.cuda.synchronize()
    qo = list(range(q.shape[0] + 1))
    ro, rl = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, True, scale)
    _check(o, lse, ro, rl, label)


@pytest.mark.parametrize("D", [64, 96, 128])
@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (24, 8), (32, 4), (32, 1)])
def test_paged_decode(D, Hq, Hkv):
    # one key, one chunk (64 keys) and its neighbours, two chunks and their
    # neighbours, many chunks (up to 19), no keys
    kv_lens = [1, 63, 64, 65, 127, 128, 129, 700, 0, 256, 1200]
    q, kc, vc, _, kv, idx = _draw(2, [1] * len(kv_lens), kv_lens, Hq, Hkv, D, 4000)
    announce(f"paged decode D={D} Hq={Hq} Hkv={Hkv}")
    _decode(q, kc, vc, kv, idx, max(kv_lens), D ** -0.5, f"decode d{D} g{Hq // Hkv}")


def test_decode_peaky_rows_across_chunks():
    """Scores with a large spread, so the chunks' maxima differ widely and the
    merge's rescaling matters."""
    kv_lens = [1000, 333]
    q, kc, vc, _, kv, idx = _draw(3, [1, 1], kv_lens, 8, 2, 128, 2000)
    q, kc = q * 4, kc * 4   # exact in bf16
    _decode(q, kc, vc, kv, idx, 1000, 128 ** -0.5, "decode peaky")


def test_decode_workspace_larger_max_kvlen_and_guard_bands():
    """max_kvlen above every request (extra chunks do nothing); nothing is
    written outside o and lse."""
    kv_lens = [300, 5]
    q, kc, vc, _, kv, idx = _draw(4, [1, 1], kv_lens, 8, 2, 64, 1000)
    dq, dkc, dvc = _dev(q, kc, vc)
    pad, sent = 4096, -1536.0
    ob = torch.full((q.numel() + 2 * pad,), sent, dtype=torch.bfloat16, device="cuda")
    lb = torch.full((16 + 2 * pad,), sent, dtype=torch.float32, device="cuda")
    o = ob[pad:pad + q.numel()].view(q.shape)
    lse = lb[pad:pad + 16].view(8, 2)
    ws = attn.decode_workspace_for(dq, dkc, 2000)
    attn.attn_decode_paged(dq, dkc, dvc, o, lse, _i32(kv), _i32(idx), 2000, 0.125, ws,
                           kv_indptr_host=kv, kv_indices_host=idx)
    torch.cuda.synchronize()
    ro, rl = oracle.attention_forward_paged(q, kc, vc, [0, 1, 2], kv, idx, True, 0.125)
    _check(o, lse, ro, rl, "decode max_kvlen 2000")
    for b in (ob, lb):
        assert (b[:pad].float() == sent).all() and (b[-pad:].float() == sent).all()


@pytest.mark.parametrize("split", [True, False])
def test_paged_prefill_guard_bands_and_determinism(split):
    """Nothing is written outside o and lse; two calls give the same bits
    (split: the second call reuses the first call's workspace)."""
    q_lens, kv_lens = [150, 64], [600, 90]
    q, kc, vc, qo, kv, idx = _draw(5, q_lens, kv_lens, 4, 2, 128, 1000)
    dq, dkc, dvc = _dev(q, kc, vc)
    Tq = sum(q_lens)
    pad, sent = 4096, -1536.0
    ob = torch.full((q.numel() + 2 * pad,), sent, dtype=torch.bfloat16, device="cuda")
    lb = torch.full((4 * Tq + 2 * pad,), sent, dtype=torch.float32, device="cuda")
    o = ob[pad:pad + q.numel()].view(q.shape)
    lse = lb[pad:pad + 4 * Tq].view(4, Tq)
    ws = attn.prefill_workspace_for(dq, dkc, 2, 150, 600) if split else None
    assert (ws is not None) == split   # these shapes are split when a workspace is given
    outs = []
    for _ in range(2):
        attn.attn_fwd_paged(dq, dkc, dvc, o, lse, _i32(qo), _i32(kv), _i32(idx), 150, 600, True,
                            128 ** -0.5, ws)
        torch.cuda.synchronize()
        outs.append((o.clone(), lse.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    ro, rl = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, True, 128 ** -0.5)
    _check(o, lse, ro, rl, f"prefill guard split={split}")
    for b in (ob, lb):
        assert (b[:pad].float() == sent).all() and (b[-pad:].float() == sent).all()


def test_paged_prefill_max_kvlen_above_every_request():
    """A larger max_kvlen only adds empty chunks."""
    q, kc, vc, qo, kv, idx = _draw(6, [300, 40], [300, 500], 4, 2, 128, 1000)
    dq, dkc, dvc = _dev(q, kc, vc)
    o, lse = attn.forward_paged(dq, dkc, dvc, _i32(qo), _i32(kv), _i32(idx), 300, True,
                                128 ** -0.5, max_kvlen=2000, qo_indptr_host=qo,
                                kv_indptr_host=kv, kv_indices_host=idx)
    torch.cuda.synchronize()
    ro, rl = oracle.attention_forward_paged(q, kc, vc, qo, kv, idx, True, 128 ** -0.5)
    _check(o, lse, ro, rl, "prefill max_kvlen 2000")


@pytest.mark.parametrize("name", list(wl.PAGED_WORKLOADS))
def test_full_paged_workload(name):
    w = wl.PAGED_WORKLOADS[name]
    x = wl.make_paged_inputs(w, 0)
    announce(f"full-size {name}")
    if w.decode:
        _decode(x.q, x.k_cache, x.v_cache, x.kv_indptr, x.kv_indices, x.max_kvlen, w.scale, name)
    else:
        for split in (True, False):
            _prefill(x.q, x.k_cache, x.v_cache, x.qo_indptr, x.kv_indptr, x.kv_indices, w.causal,
                     w.scale, f"{name} split={split}", split, attn.ATTN_FWD_PAGED_KEY_HALVES)
