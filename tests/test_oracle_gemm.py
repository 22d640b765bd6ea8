"""Pins of the GEMM oracle C = A B^T: a hand-worked product, a pure-Python
triple loop, one-hot rows of A that pick out columns of B (which tells
A B^T from A B and from A^T B), and the bound quantity sum_k |a_k b_k|.
``test_planted_gemm_mistakes_are_caught`` shows that a missing transpose or a
dropped reduction term fails them."""
import pytest
import torch

import oracle
from oracle import gemm as ogemm

F64 = torch.float64


def test_hand_worked_product():
    a = torch.tensor([[1.0, 2.0, 3.0], [0.0, -1.0, 4.0]], dtype=F64)
    b = torch.tensor([[1.0, 0.0, 1.0], [2.0, 1.0, 0.0], [-1.0, 1.0, 1.0], [0.5, 0.5, 0.5]],
                     dtype=F64)
    # C[m, n] = a_m . b_n
    want = torch.tensor([[4.0, 4.0, 4.0, 3.0], [4.0, -1.0, 3.0, 1.5]], dtype=F64)
    assert torch.equal(oracle.gemm_nt(a, b), want)
    assert torch.equal(oracle.abs_products(a, b),
                       torch.tensor([[4.0, 4.0, 6.0, 3.0], [4.0, 1.0, 5.0, 2.5]], dtype=F64))


def test_brute_force_triple_loop():
    gen = torch.Generator().manual_seed(21)
    a = torch.randn(5, 7, generator=gen, dtype=F64)
    b = torch.randn(3, 7, generator=gen, dtype=F64)
    c = oracle.gemm_nt(a, b)
    for m in range(5):
        for n in range(3):
            s = 0.0
            for k in range(7):
                s += float(a[m, k]) * float(b[n, k])
            assert abs(float(c[m, n]) - s) < 1e-12


def test_one_hot_rows_select_columns_of_b():
    """Row m of A = e_{i(m)} gives C[m, :] = B[:, i(m)] (column i of B)."""
    gen = torch.Generator().manual_seed(22)
    K = 6
    b = torch.randn(K, K, generator=gen, dtype=F64)   # square: a transposition mistake still runs
    sel = [4, 0, 5, 2]
    a = torch.zeros(len(sel), K, dtype=F64)
    for m, i in enumerate(sel):
        a[m, i] = 1.0
    c = oracle.gemm_nt(a, b)
    for m, i in enumerate(sel):
        assert torch.equal(c[m], b[:, i])


def test_bf16_inputs_are_read_exactly():
    gen = torch.Generator().manual_seed(23)
    a = torch.randn(4, 16, generator=gen).to(torch.bfloat16)
    b = torch.randn(3, 16, generator=gen).to(torch.bfloat16)
    c = oracle.gemm_nt(a, b)
    assert c.dtype == F64
    assert torch.equal(c, a.double() @ b.double().T)


def test_shape_validation():
    with pytest.raises(ValueError):
        oracle.gemm_nt(torch.zeros(2, 3), torch.zeros(2, 4))


def _pins_hold():
    try:
        test_hand_worked_product()
        test_brute_force_triple_loop()
        test_one_hot_rows_select_columns_of_b()
    except AssertionError:
        return False
    return True


def test_planted_gemm_mistakes_are_caught(monkeypatch):
    def no_transpose(a, b):
        return ogemm._as64(a) @ ogemm._as64(b) if a.shape[1] == b.shape[0] else \
            ogemm._as64(a) @ ogemm._as64(b).T

    def dropped_term(a, b):
        return ogemm._as64(a)[:, :-1] @ ogemm._as64(b)[:, :-1].T

    for bad in (no_transpose, dropped_term):
        monkeypatch.setattr(oracle, "gemm_nt", bad)
        assert not _pins_hold(), bad.__name__
        monkeypatch.undo()
    assert _pins_hold()
