"""Host-only tests of the C ABI: the library loads, exports every symbol of
include/attn.h, and rejects every invalid argument with its status code
before any GPU call (pointers here are fake integers; they are never
dereferenced because validation fails first)."""
import ctypes
import os
import re

import pytest

from paper_2608_17379_amd import attn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
A = 0x10000   # a fake, 16-byte aligned "device address"


def header_symbols():
    text = open(os.path.join(ROOT, "include", "attn.h")).read()
    return set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(attn_\w+)\s*\(", text, re.M))


def test_phase_mask_validation():
    l = attn.lib()
    args = [A] * 9 + [1, 2, 2, 64, 64, 1, 0.125, A, 1 << 20]
    # 4 and 8 pick the dK/dV form: only with the dK/dV phase, never both
    bad_masks = (0, 4, 8, 12, -1, 16, 5, 9, 13, 14, 15)
    for bad in bad_masks:
        assert l.attn_bwd_phases(*args, bad, None) == -8
    argsv = [A] * 10 + [2, 64, 100, 2, 1, 128, 1, 0.1, A, 1 << 20]
    for bad in bad_masks:
        assert l.attn_bwd_varlen_phases(*argsv, bad, None) == -8
    assert l.attn_bwd_phases(*(args[:-2] + [A, 1]), 2, None) == -6


def test_library_exports_every_declared_symbol():
    syms = header_symbols()
    assert syms == set(attn.EXPORTS)
    l = attn.lib()
    for s in syms:
        assert hasattr(l, s), s


def fwd(**kw):
    args = dict(q=A, k=A, v=A, o=A, lse=A, B=1, Hq=2, Hkv=2, S=64, D=64, causal=0, scale=0.125)
    args.update(kw)
    return attn.lib().attn_fwd(args["q"], args["k"], args["v"], args["o"], args["lse"], args["B"],
                               args["Hq"], args["Hkv"], args["S"], args["D"], args["causal"],
                               args["scale"], None)


def bwd(**kw):
    args = dict(q=A, k=A, v=A, o=A, lse=A, dO=A, dq=A, dk=A, dv=A, B=1, Hq=2, Hkv=2, S=64, D=64,
                causal=1, scale=0.125, ws=A, wsb=1 << 20)
    args.update(kw)
    return attn.lib().attn_bwd(*(args[n] for n in ("q", "k", "v", "o", "lse", "dO", "dq", "dk",
                                                    "dv", "B", "Hq", "Hkv", "S", "D", "causal",
                                                    "scale", "ws", "wsb")), None)


def fwdv(**kw):
    args = dict(q=A, k=A, v=A, o=A, lse=A, cu=A, nseq=2, ms=64, T=100, Hq=2, Hkv=1, D=128,
                causal=1, scale=0.1)
    args.update(kw)
    return attn.lib().attn_fwd_varlen(*(args[n] for n in ("q", "k", "v", "o", "lse", "cu", "nseq",
                                                           "ms", "T", "Hq", "Hkv", "D", "causal",
                                                           "scale")), None)


def bwdv(**kw):
    args = dict(q=A, k=A, v=A, o=A, lse=A, dO=A, dq=A, dk=A, dv=A, cu=A, nseq=2, ms=64, T=100,
                Hq=2, Hkv=1, D=128, causal=1, scale=0.1, ws=A, wsb=1 << 20)
    args.update(kw)
    return attn.lib().attn_bwd_varlen(*(args[n] for n in (
        "q", "k", "v", "o", "lse", "dO", "dq", "dk", "dv", "cu", "nseq", "ms", "T", "Hq", "Hkv",
        "D", "causal", "scale", "ws", "wsb")), None)


@pytest.mark.parametrize("call", [fwd, bwd, fwdv, bwdv])
def test_scalar_validation(call):
    assert call(Hq=0) == -2
    assert call(Hkv=0) == -2
    assert call(Hq=3, Hkv=2) == -3
    assert call(D=80) == -4
    assert call(D=32) == -4
    assert call(D=256) == -4
    assert call(causal=2) == -8
    assert call(scale=float("nan")) == -8
    assert call(scale=float("inf")) == -8
    assert call(scale=0.0) == -8
    assert call(scale=-0.125) == -8
    assert call(Hq=65536, Hkv=1, D=128) == -2
    assert call(q=0) == -1
    assert call(k=A + 8) == -5
    assert call(lse=A + 4) == -5


@pytest.mark.parametrize("call", [fwd, bwd])
def test_fixed_shape_validation(call):
    assert call(B=-1) == -2
    assert call(S=-5) == -2
    assert call(S=65535 * 128 + 1) == -2
    # empty problems are no-ops and may carry null pointers
    assert call(B=0, q=0, k=0, v=0, o=0, lse=0) == 0
    assert call(S=0, q=0, k=0, v=0, o=0, lse=0) == 0


@pytest.mark.parametrize("call", [fwdv, bwdv])
def test_packed_shape_validation(call):
    assert call(nseq=-1) == -2
    assert call(T=-1) == -2
    assert call(ms=0) == -8
    assert call(cu=0) == -1
    assert call(cu=A + 2) == -5
    assert call(nseq=0, q=0, cu=0) == 0
    assert call(T=0, q=0, cu=0) == 0


def test_workspace_validation():
    need = attn.attn_bwd_workspace_size(1, 2, 2, 64, 64)
    assert need >= 1 * 2 * 64 * 4 and need % 256 == 0
    assert bwd(wsb=need - 1) == -6
    assert bwd(ws=0) == -6
    assert bwd(ws=A + 8) == -5
    needv = attn.attn_bwd_varlen_workspace_size(100, 2, 1, 128)
    assert needv >= 100 * 2 * 4
    assert bwdv(wsb=needv - 1) == -6
    assert attn.attn_bwd_workspace_size(0, 2, 2, 64, 64) == 0


def test_status_strings():
    for code in range(-9, 1):
        s = attn.attn_status_string(code)
        assert s and s != "unknown status"
    assert attn.attn_status_string(-99) == "unknown status"


def test_binding_rejects_host_tensors():
    import torch
    q = torch.zeros(1, 1, 4, 64, dtype=torch.bfloat16)
    lse = torch.zeros(1, 1, 4)
    with pytest.raises(ValueError):
        attn.attn_fwd(q, q, q, q.clone(), lse, False, 0.125)


def test_cu_seqlens_host_check():
    attn.check_cu_seqlens([0, 3, 3, 10], 10, 7)
    for bad, total, ms in (([1, 3], 3, 5), ([0, 4, 3], 3, 5), ([0, 3], 4, 5), ([0, 9], 9, 5)):
        with pytest.raises(ValueError):
            attn.check_cu_seqlens(bad, total, ms)


def fwdp(**kw):
    # A split-size prefill (8 unsplit workgroups, 600 keys) with a workspace
    # one byte short, so that no valid combination reaches a launch.
    args = dict(q=A, k=A, v=A, o=A, lse=A, qo=A, kv=A, idx=A, batch=2, mq=64, Tq=100, mk=600,
                nnz=120, P=1000, Hq=4, Hkv=2, D=128, causal=1, scale=0.1, ws=A,
                wsb=attn.attn_fwd_paged_workspace_size(2, 64, 100, 600, 4, 2, 128) - 1)
    args.update(kw)
    return attn.lib().attn_fwd_paged(*(args[n] for n in (
        "q", "k", "v", "o", "lse", "qo", "kv", "idx", "batch", "mq", "Tq", "mk", "nnz", "P", "Hq",
        "Hkv", "D", "causal", "scale", "ws", "wsb")), None)


def dec(**kw):
    args = dict(q=A, k=A, v=A, o=A, lse=A, kv=A, idx=A, batch=3, mk=500, nnz=900, P=1000, Hq=24,
                Hkv=8, D=128, scale=0.1, ws=A, wsb=1 << 24)
    args.update(kw)
    return attn.lib().attn_decode_paged(*(args[n] for n in (
        "q", "k", "v", "o", "lse", "kv", "idx", "batch", "mk", "nnz", "P", "Hq", "Hkv", "D",
        "scale", "ws", "wsb")), None)


@pytest.mark.parametrize("call", [fwdp, dec])
def test_paged_validation(call):
    assert call(Hq=3, Hkv=2) == -3
    assert call(D=80) == -4
    assert call(scale=0.0) == -8
    assert call(batch=-1) == -2
    assert call(nnz=-1) == -2
    assert call(nnz=(1 << 29) + 1) == -2
    assert call(P=-1) == -2
    assert call(P=(1 << 31) // (2 * 128 * 2) + 1) == -2   # cache bytes beyond 2^31
    assert call(kv=0) == -1
    assert call(idx=0) == -1
    assert call(kv=A + 2) == -5
    assert call(idx=A + 1) == -5
    assert call(q=A + 8) == -5
    assert call(batch=0, q=0, kv=0, idx=0) == 0


def test_paged_prefill_specific_validation():
    assert fwdp(causal=2) == -8
    assert fwdp(mq=0) == -8
    assert fwdp(qo=0) == -1
    assert fwdp(Tq=-1) == -2
    assert fwdp(mk=-1) == -2
    assert fwdp(Tq=0, q=0, qo=0) == 0
    assert fwdp() == -6                                  # workspace one byte short
    assert fwdp(wsb=1 << 30, ws=A + 8) == -5             # misaligned workspace


def test_paged_prefill_form():
    form = attn.attn_fwd_paged_form
    # the paper's paged prefill: 7 blocks x 24 heads = 168 workgroups
    assert form(1, 892, 892, 24, True) == attn.ATTN_FWD_PAGED_KEY_HALVES
    assert form(1, 892, 892, 24, False) == attn.ATTN_FWD_PAGED_KEY_HALVES
    # 5 x 24 = 120 workgroups: split when a workspace is given
    assert form(1, 640, 892, 24, True) == attn.ATTN_FWD_PAGED_SPLIT
    assert form(1, 640, 892, 24, False) == attn.ATTN_FWD_PAGED_KEY_HALVES
    assert form(1, 640, 256, 24, True) == attn.ATTN_FWD_PAGED_KEY_HALVES   # one chunk
    assert form(64, 4096, 4096, 32, True) == attn.ATTN_FWD_PAGED_UNSPLIT
    assert form(2, 128, 600, 128, False) == attn.ATTN_FWD_PAGED_UNSPLIT      # exactly 256
    assert form(1, 128, 600, 255, False) == attn.ATTN_FWD_PAGED_KEY_HALVES   # 255
    # the workspace size agrees: non-zero exactly when the form is the split
    for args in [(1, 892, 892, 24), (1, 640, 892, 24), (2, 150, 600, 4), (64, 4096, 4096, 32)]:
        b, mq, mk, hq = args
        split = form(b, mq, mk, hq, True) == attn.ATTN_FWD_PAGED_SPLIT
        assert (attn.attn_fwd_paged_workspace_size(b, mq, b * mq, mk, hq, 1, 128) > 0) == split
    for bad in [(0, 892, 892, 24, True), (1, 0, 892, 24, True), (1, 892, -1, 24, True),
                (1, 892, 892, 0, True)]:
        assert attn.lib().attn_fwd_paged_form(*[int(v) for v in bad]) == -2
    assert attn.lib().attn_fwd_paged_form(1, 892, 892, 24, 2) == -8


def test_paged_prefill_workspace_size():
    size = attn.attn_fwd_paged_workspace_size
    # split: 2 x 4 x 1 unsplit workgroups, 600 keys -> 3 chunks of 256
    slots = 100 * 4 * 3
    assert size(2, 64, 100, 600, 4, 2, 128) == (slots * 128 * 4 + 255) // 256 * 256 + \
        (slots * 4 + 255) // 256 * 256
    assert size(2, 64, 100, 256, 4, 2, 128) == 0         # one chunk: no split
    assert size(64, 4096, 64 * 4096, 4096, 32, 8, 128) == 0   # the grid fills the chip
    # the paper's paged prefill: 7 blocks x 24 heads = 168 workgroups, fewer
    # than the 256 CUs but more than half: the key-halves form, no split
    assert size(1, 892, 892, 892, 24, 8, 128) == 0
    assert size(1, 640, 640, 892, 24, 8, 128) > 0        # 5 x 24 = 120 < 128: split
    assert size(0, 64, 100, 600, 4, 2, 128) == 0
    assert size(2, 64, 100, 0, 4, 2, 128) == 0


def test_decode_specific_validation():
    assert dec(Hq=66, Hkv=2) == -3     # more than 32 query heads per kv head
    assert dec(mk=0) == -8
    need = attn.attn_decode_paged_workspace_size(3, 500, 24, 8, 128)
    assert need >= 3 * 24 * 4 * 129 * 4 and need % 256 == 0
    assert dec(wsb=need - 1) == -6
    assert dec(ws=0) == -6
    assert dec(ws=A + 8) == -5
    assert attn.attn_decode_paged_workspace_size(0, 500, 24, 8, 128) == 0


def test_paged_host_check():
    attn.check_paged_host([0, 2, 2, 5], [4, 1, 0, 2, 3], 5, 3)
    for kv, idx, p, mk in (([1, 2], [0, 1], 5, None), ([0, 2, 1], [0, 1], 5, None),
                           ([0, 2], [0, 5], 5, None), ([0, 2], [0, -1], 5, None),
                           ([0, 3], [0, 1, 2], 5, 2), ([0, 2], [0, 1, 2], 5, None)):
        with pytest.raises(ValueError):
            attn.check_paged_host(kv, idx, p, mk)


def test_decode_phase_mask_validation():
    l = attn.lib()
    args = [A] * 7 + [3, 500, 900, 1000, 24, 8, 128, 0.1, A, 1 << 24]
    for bad in (0, 4, -1):
        assert l.attn_decode_paged_phases(*args, bad, None) == -8


def test_gemm_validation():
    l = attn.lib()
    g = lambda a=A, b=A, c=A, M=64, N=64, K=64: l.attn_gemm_bf16_nt(a, b, c, M, N, K, None)
    assert g(M=-1) == -2
    assert g(K=12) == -2          # K % 8
    assert g(N=20) == -2          # N % 8
    assert g(K=1 << 23) == -2     # 256 rows beyond 31-bit offsets
    assert g(a=0) == -1
    assert g(c=A + 8) == -5
    assert g(M=0, a=0, b=0, c=0) == 0
    assert g(N=0, a=0, b=0, c=0) == 0


def test_gemm_empty_k_allows_null_operands():
    l = attn.lib()
    assert l.attn_gemm_bf16_nt(A, A, 0, 64, 64, 0, None) == -1   # c is still needed


def test_dkdv_form_rule():
    form = attn.attn_bwd_dkdv_form
    one, two = attn.ATTN_BWD_DKDV_ONE_PER_CU, attn.ATTN_BWD_DKDV_TWO_PER_CU
    assert form(4, 16, 2048, 0, 128, True, False) == two      # 1024 causal key blocks
    assert form(2, 8, 4096, 0, 128, True, False) == one       # 512: one round at two per CU
    assert form(2, 8, 4096, 0, 128, False, False) == two      # non-causal blocks are equal
    assert form(1, 16, 16384, 0, 96, True, False) == two
    assert form(33, 4, 1500, 16294, 128, True, True) == one   # ~640 packed blocks
    assert form(4, 48, 4096, 0, 64, True, False) == two       # D = 64: one form
    assert form(2, 8, 4096, 0, 64, True, False) == two
    l = attn.lib()
    assert l.attn_bwd_dkdv_form(1, 1, 128, 0, 80, 1, 0) == -4
    assert l.attn_bwd_dkdv_form(-1, 1, 128, 0, 128, 1, 0) == -2
    assert l.attn_bwd_dkdv_form(1, 1, 128, 0, 128, 2, 0) == -8
    with pytest.raises(attn.AttnError):
        form(1, 1, 128, 0, 80, True, False)


def test_noalloc_validation_before_any_gpu_call():
    """attn_bwd_noalloc checks its sizes, its scratch limit and its pointers
    on the host and returns before any GPU call."""
    l = attn.lib()

    def call(**kw):
        a = dict(p=A, B=1, Hq=2, Hkv=2, S=64, D=64, causal=1, scale=0.125)
        a.update(kw)
        ptrs = [a.get(n, a["p"]) for n in ("q", "k", "v", "o", "lse", "dO", "dq", "dk", "dv")]
        return l.attn_bwd_noalloc(*ptrs, a["B"], a["Hq"], a["Hkv"], a["S"], a["D"], a["causal"],
                                  a["scale"], None)

    limit = attn.ATTN_BWD_NOALLOC_SCRATCH_BYTES
    assert limit == 16 << 20
    # B * Hq * S = 2^21 rows x heads fit exactly (two 4-byte arrays); one more
    # 64-row block does not.
    assert attn.attn_bwd_workspace_size(1, 32, 32, 65536, 128) == limit
    assert call(B=1, Hq=32, Hkv=32, S=65536 + 64, D=128, p=0) == -9
    assert call(B=2, Hq=32, Hkv=32, S=65536, D=128) == -9
    assert call(B=1, Hq=32, Hkv=32, S=65536, D=128, p=0) == -1   # fits: pointers checked next
    assert call(q=0) == -1
    assert call(dv=A + 8) == -5
    assert call(D=80) == -4
    assert call(Hq=3, Hkv=2) == -3
    assert call(scale=0.0) == -8
    assert call(B=-1) == -2
    assert call(B=0, p=0) == 0   # no rows: a no-op
    assert "noalloc" in attn.attn_status_string(-9)


def test_forward_and_dq_grid_must_fit_one_launch():
    """The forward and dQ kernels run one 1-D grid over (query block, query
    head) in the XCD-aware order; shapes whose grid exceeds 2^31 - 1
    workgroups are refused before any GPU call."""
    big_s = 128 * 65535   # the largest S check_rows allows
    assert fwd(B=1 << 14, Hq=1 << 14, Hkv=1 << 14, S=big_s) == -2
    assert bwd(B=1 << 14, Hq=1 << 14, Hkv=1 << 14, S=big_s) == -2


def test_calibration_library_exports():
    """The benchmark's MFMA-rate calibration library (measurement support,
    not part of the attention ABI) is built beside libattn.so and exports
    its two entry points."""
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "paper_2608_17379_amd", "libcalib.so")
    lib = ctypes.CDLL(path)
    for name in ("calib_mfma_rate", "calib_mfma_chains"):
        assert hasattr(lib, name), name
    assert lib.calib_mfma_chains() == 8

