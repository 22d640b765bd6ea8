"""GPU parity of the BF16 GEMM C = A B^T (attn_gemm_bf16_nt) against the fp64
oracle.

Tolerance, derived from the arithmetic (no source states one for the GEMM):
bf16 x bf16 products are exact in fp32, so the only errors are the fp32
summation of K products and the final rounding to bf16.  Any summation order
with at most 2 fp32 units of rounding per addition errs by at most
gamma * S with gamma = K 2^-23 / (1 - K 2^-23) and S = sum_k |a_k b_k|; the
bf16 rounding (round to nearest even, 8 significant bits) adds at most
2^-8 of the result.  Every element must satisfy

    |c - r| <= 2^-8 |r| + (1 + 2^-8) gamma S,

and, as a typical-error check, the relative L2 error must be at most 5e-3
(bf16 rounding alone gives about 2e-3).  The paper's own checker,
allclose(atol=rtol=1e-2), is reported as well.

Small shapes cover every tail (M, N not multiples of the 256 x 256 tile; K
not a multiple of the 64-wide K step); the paper's 8192 x 7168 x 5120
workload is compared over its whole output.
"""
import math

import pytest
import torch

import oracle
from paper_2608_17379_amd import attn
from paper_2608_17379_amd import workloads as wl

from parity import announce

pytestmark = pytest.mark.gpu


def _check(c, a, b, label):
    r = oracle.gemm_nt(a, b)
    s = oracle.abs_products(a, b)
    K = a.shape[1]
    gamma = K * 2.0 ** -23 / (1 - K * 2.0 ** -23)
    bound = 2.0 ** -8 * r.abs() + (1 + 2.0 ** -8) * gamma * s
    c64 = c.double().cpu()
    err = (c64 - r).abs()
    rel = float((c64 - r).norm() / r.norm()) if r.norm() > 0 else float(err.max())
    ok_close = bool(torch.allclose(c64, r, atol=1e-2, rtol=1e-2))
    announce(f"{label}: max err/bound={float((err / bound.clamp_min(1e-300)).max()):.3g} "
             f"rel_l2={rel:.3g} allclose(1e-2)={ok_close}")
    assert (err <= bound).all(), label
    assert rel <= 5e-3, (label, rel)


def _draw(seed, M, N, K):
    gen = torch.Generator().manual_seed(seed)
    a = torch.randn(M, K, generator=gen).to(torch.bfloat16)
    b = torch.randn(N, K, generator=gen).to(torch.bfloat16)
    return a, b


@pytest.mark.parametrize("M,N,K", [(1, 8, 8), (256, 256, 64), (255, 264, 72), (300, 520, 200),
                                   (513, 1000, 1024), (64, 2048, 136), (1024, 256, 5120),
                                   (2048, 2048, 512),
                                   # more tiles than CUs with a small last round: one
                                   # launch runs the full tiles in rounds, then that
                                   # round as 128-row half tiles (ragged M, K tail;
                                   # ragged N; 3 half-tiled tiles, whose 6 halves do
                                   # not divide among the 8 XCDs)
                                   (4252, 4096, 136), (4352, 4072, 520), (1792, 9472, 64)])
def test_gemm_shapes(M, N, K):
    a, b = _draw(M + N + K, M, N, K)
    announce(f"gemm M={M} N={N} K={K}")
    c = attn.gemm_nt(a.cuda(), b.cuda())
    torch.cuda.synchronize()
    _check(c, a, b, f"gemm {M}x{N}x{K}")


def test_gemm_k_zero_and_guard_bands():
    a, b = _draw(1, 300, 264, 64)
    da, db = a.cuda(), b.cuda()
    pad, sent = 4096, -1536.0
    cb = torch.full((300 * 264 + 2 * pad,), sent, dtype=torch.bfloat16, device="cuda")
    c = cb[pad:pad + 300 * 264].view(300, 264)
    attn.attn_gemm_bf16_nt(da, db, c)
    torch.cuda.synchronize()
    _check(c, a, b, "gemm guard")
    assert (cb[:pad].float() == sent).all() and (cb[-pad:].float() == sent).all()
    z = attn.gemm_nt(torch.empty(5, 0, dtype=torch.bfloat16, device="cuda"),
                     torch.empty(8, 0, dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    assert (z.float() == 0).all()


def test_gemm_deterministic():
    a, b = _draw(2, 512, 512, 640)
    da, db = a.cuda(), b.cuda()
    c1, c2 = attn.gemm_nt(da, db), attn.gemm_nt(da, db)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)


@pytest.mark.parametrize("name", list(wl.GEMM_WORKLOADS))
def test_full_gemm_workload(name):
    """The paper's GEMM at full size: every element of C against the oracle
    and its per-element bound (the rows are compared in blocks only to bound
    the fp64 temporaries; the relative L2 error is taken over the whole
    output)."""
    w = wl.GEMM_WORKLOADS[name]
    a, b = wl.make_gemm_inputs(w, 0)
    announce(f"full-size {name}")
    c = attn.gemm_nt(a.cuda(), b.cuda())
    torch.cuda.synchronize()
    c = c.cpu()
    assert torch.isfinite(c.float()).all()
    K = w.K
    gamma = K * 2.0 ** -23 / (1 - K * 2.0 ** -23)
    sq_err = sq_ref = 0.0
    worst, close_fail = 0.0, 0
    for r0 in range(0, w.M, 1024):
        r1 = min(w.M, r0 + 1024)
        r = oracle.gemm_nt(a[r0:r1], b)
        bound = 2.0 ** -8 * r.abs() + (1 + 2.0 ** -8) * gamma * oracle.abs_products(a[r0:r1], b)
        err = (c[r0:r1].double() - r).abs()
        assert (err <= bound).all(), (name, r0)
        worst = max(worst, float((err / bound.clamp_min(1e-300)).max()))
        sq_err += float((err ** 2).sum())
        sq_ref += float((r ** 2).sum())
        close_fail += int((err > 1e-2 + 1e-2 * r.abs()).sum())
    rel = math.sqrt(sq_err / sq_ref)
    announce(f"{name} whole output: max err/bound={worst:.3g} rel_l2={rel:.3g} "
             f"allclose(1e-2) failing {close_fail / (w.M * w.N):.2e}")
    assert rel <= 5e-3, (name, rel)
