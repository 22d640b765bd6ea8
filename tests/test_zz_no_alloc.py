"""attn_bwd_noalloc (the backward for callers that cannot allocate: its
scratch is the library's own device array) against attn_bwd with a caller
workspace, through the C ABI.

Both run the same kernels on the same inputs, and the backward is
deterministic, so the outputs must be bitwise equal.  Two calls in a row
share the one scratch array: the second, on a smaller problem, must not see
anything left by the first.
"""
import pytest
import torch

from paper_2608_17379_amd import attn
from paper_2608_17379_amd import workloads as wl

from parity import announce, check_all, oracle_all, to_gpu

pytestmark = pytest.mark.gpu


def _run(w, seed):
    x = wl.make_inputs(w, seed)
    announce(f"noalloc {w.name} seed={seed}")
    q, k, v, do, _ = to_gpu(x)
    o, lse = attn.forward(q, k, v, w.causal, w.scale)
    ref = [torch.empty_like(t) for t in (q, k, v)]
    attn.attn_bwd(q, k, v, o, lse, do, *ref, w.causal, w.scale, attn.workspace_for(q, k))
    got = [torch.full_like(t, -1536.0) for t in (q, k, v)]
    attn.attn_bwd_noalloc(q, k, v, o, lse, do, *got, w.causal, w.scale)
    torch.cuda.synchronize()
    for r, g in zip(ref, got):
        assert torch.equal(r, g), w.name
    return x, (o.cpu(), lse.cpu(), *(g.cpu() for g in got))


def test_noalloc_equals_workspace_backward_twice():
    big = wl.small("noalloc_big", 2, 8, 2, 1000, 128, True)
    small = wl.small("noalloc_small", 1, 4, 4, 300, 64, False)
    x, got = _run(big, 11)
    check_all(got, oracle_all(x, big.causal, big.scale), big.name)
    x, got = _run(small, 12)
    check_all(got, oracle_all(x, small.causal, small.scale), small.name)


def test_noalloc_rejects_problems_beyond_its_scratch():
    q = torch.zeros(1, 32, 65600, 128, dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros(1, 32, 65600, dtype=torch.float32, device="cuda")
    with pytest.raises(attn.AttnError) as e:
        attn.attn_bwd_noalloc(q, q, q, q, lse, q, q, q, q, True, 0.125)
    assert e.value.status == -9
