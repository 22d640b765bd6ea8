"""Shared helpers of the GPU parity tests (not a test module).

Tolerances (bf16 inputs, fp32 accumulation, bf16 outputs):
  O        max-abs error <= 2e-2 against the fp64 oracle
  dQ,dK,dV relative L2 error <= 3e-2 over the compared tensor
  LSE      max-abs error <= 1e-3 (fp32 output; expected error ~1e-5: the
           score products are exact in fp32 and only the fp32 summation and
           the ~1-ulp hardware exp2/log2 contribute)
"""
import sys

import torch

import oracle
from paper_2608_17379_amd import attn
from paper_2608_17379_amd import workloads as wl

O_MAXABS = 2e-2
GRAD_RELL2 = 3e-2
LSE_MAXABS = 1e-3


def announce(msg: str) -> None:
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


def rel_l2(x: torch.Tensor, ref: torch.Tensor) -> float:
    x64, r64 = x.detach().double().cpu(), ref.detach().double().cpu()
    den = float(r64.norm())
    return float((x64 - r64).norm()) / (den if den > 0 else 1.0)


def max_abs(x: torch.Tensor, ref: torch.Tensor) -> float:
    x64, r64 = x.detach().double().cpu(), ref.detach().double().cpu()
    if x64.numel() == 0:
        return 0.0
    fin = torch.isfinite(r64)
    if not torch.equal(torch.isfinite(x64), fin):
        return float("inf")
    d = (x64 - r64)[fin].abs()
    return float(d.max()) if d.numel() else 0.0


def to_gpu(x: wl.Inputs):
    dev = torch.device("cuda", 0)
    q, k, v, do = (t.to(dev) for t in (x.q, x.k, x.v, x.do))
    cu = None
    if x.cu_seqlens is not None:
        cu = torch.tensor(x.cu_seqlens, dtype=torch.int32, device=dev)
    return q, k, v, do, cu


def gpu_fwd_bwd(x: wl.Inputs, causal: bool, scale: float, dkdv_form: int = 0):
    q, k, v, do, cu = to_gpu(x)
    ms = x.max_seqlen if cu is not None else 0
    o, lse = attn.forward(q, k, v, causal, scale, cu_seqlens=cu, max_seqlen=ms,
                          cu_seqlens_host=x.cu_seqlens)
    dq, dk, dv = attn.backward(q, k, v, o, lse, do, causal, scale, cu_seqlens=cu, max_seqlen=ms,
                               cu_seqlens_host=x.cu_seqlens, dkdv_form=dkdv_form)
    torch.cuda.synchronize()
    return o.cpu(), lse.cpu(), dq.cpu(), dk.cpu(), dv.cpu()


def check_all(got, ref, label: str):
    """got = (o, lse, dq, dk, dv) from the GPU; ref = fp64 oracle values."""
    o, lse, dq, dk, dv = got
    ro, rlse, rdq, rdk, rdv = ref
    errs = {
        "o_maxabs": max_abs(o, ro),
        "lse_maxabs": max_abs(lse, rlse),
        "dq_rel": rel_l2(dq, rdq),
        "dk_rel": rel_l2(dk, rdk),
        "dv_rel": rel_l2(dv, rdv),
    }
    announce(f"{label}: " + " ".join(f"{k}={v:.3g}" for k, v in errs.items()))
    assert errs["o_maxabs"] <= O_MAXABS, (label, errs)
    assert errs["lse_maxabs"] <= LSE_MAXABS, (label, errs)
    for n in ("dq_rel", "dk_rel", "dv_rel"):
        assert errs[n] <= GRAD_RELL2, (label, n, errs)
    return errs


def oracle_all(x: wl.Inputs, causal: bool, scale: float):
    o, lse = oracle.attention_forward(x.q, x.k, x.v, causal, scale, cu_seqlens=x.cu_seqlens)
    dq, dk, dv = oracle.attention_backward(x.q, x.k, x.v, x.do, causal, scale,
                                           cu_seqlens=x.cu_seqlens)
    return o, lse, dq, dk, dv
