"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before any launch (runs without a GPU)."""
import ctypes
import os
import re

import pytest

from oracle import locks_oracle as O

from paper_2607_24555_amd import locks as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "locks.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(locks_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return B.lib()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) == 23
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B._SIGS), "binding and header disagree"


def cfg(**kw):
    c = B.Config(num_seqs=2, num_q_heads=8, num_kv_heads=2, rank=8, budget_tokens=256,
                 max_pages_per_seq=64, num_blocks=128)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_payload_and_stride_per_page_size_match_the_oracle(lib):
    for Bp in (16, 32, 64):
        for r in (1, 2, 4, 8, 15):
            assert B.summary_payload_bytes_ex(r, 0, Bp) == O.payload_bytes(r, B=Bp)
            assert B.summary_stride(r, 0, Bp) == O.record_stride(r, "int4", Bp)
    assert B.summary_stride(8, 0, 48) == 0 and B.summary_payload_bytes_ex(8, 0, 8) == 0


def test_payload_and_stride(lib):
    assert [B.summary_payload_bytes(r) for r in (8, 4, 2)] == [818, 490, 326]
    assert [B.summary_stride(r) for r in (8, 4, 2)] == [832, 496, 336]
    assert B.summary_payload_bytes(0) == 0 and B.summary_stride(16) == 0


@pytest.mark.parametrize("basis,name", [(B.LOCKS_BASIS_INT4, "int4"), (B.LOCKS_BASIS_INT8, "int8"),
                                        (B.LOCKS_BASIS_BF16, "bf16")])
def test_payload_and_stride_per_basis_match_the_oracle_layout(lib, basis, name):
    for r in (1, 2, 4, 8, 15):
        assert B.summary_payload_bytes_ex(r, basis) == O.payload_bytes(r, basis=name)
        assert B.summary_stride(r, basis) == O.record_stride(r, name)
    assert B.summary_stride(8, 3) == 0 and B.summary_stride(0, basis) == 0


@pytest.mark.parametrize("bad,code", [(dict(basis=3), -1), (dict(basis=-1), -1),
                                      (dict(basis=1, rank=3), -2), (dict(basis=2, rank=15), -2)])
def test_bad_basis_is_rejected(lib, bad, code):
    c = cfg(**bad).c()
    assert lib.locks_workspace_bytes(ctypes.byref(c)) == 0
    fake = ctypes.c_void_p(0x1000)
    assert lib.locks_build_summaries(ctypes.byref(c), fake, fake, fake, None, 0, fake, None) == code


@pytest.mark.parametrize("bad,code", [
    (dict(head_dim=64), -2), (dict(page_size=8), -2), (dict(page_size=48), -2),
    (dict(page_size=128), -2), (dict(page_size=32, basis=1), -2),
    (dict(page_size=64, budget_tokens=64), -1), (dict(kv_dtype=7), -2),
    (dict(rank=0), -1), (dict(rank=16), -1), (dict(num_q_heads=7), -1),
    (dict(budget_tokens=16), -1), (dict(budget_tokens=0), -1), (dict(max_pages_per_seq=0), -1),
    (dict(num_blocks=0), -1), (dict(num_kv_heads=0), -1), (dict(num_seqs=-1), -1),
    (dict(num_q_heads=34, num_kv_heads=2), -2),
])
def test_bad_config_is_rejected_before_launch(lib, bad, code):
    c = cfg(**bad).c()
    assert lib.locks_workspace_bytes(ctypes.byref(c)) == 0
    fake = ctypes.c_void_p(0x1000)
    rc = lib.locks_select(ctypes.byref(c), fake, fake, fake, fake, fake, fake, None, fake, 1 << 30, None)
    assert rc == code
    rc = lib.locks_build_summaries(ctypes.byref(c), fake, fake, fake, None, 0, fake, None)
    assert rc == code


def test_null_pointers_and_workspace(lib):
    c = cfg().c()
    need = lib.locks_workspace_bytes(ctypes.byref(c))
    assert need > 0
    fake = ctypes.c_void_p(0x1000)
    # null query
    assert lib.locks_select(ctypes.byref(c), None, fake, fake, fake, fake, fake, None, fake, need, None) == -1
    # workspace too small / missing / misaligned
    assert lib.locks_select(ctypes.byref(c), fake, fake, fake, fake, fake, fake, None, fake, need - 1, None) == -3
    assert lib.locks_select(ctypes.byref(c), fake, fake, fake, fake, fake, fake, None, None, need, None) == -3
    assert lib.locks_select(ctypes.byref(c), fake, fake, fake, fake, fake, fake, None,
                            ctypes.c_void_p(0x1010), need, None) == -3
    assert lib.locks_sparse_attend(ctypes.byref(c), fake, fake, fake, fake, fake, None, fake, None,
                                   fake, need, None) == -1
    assert lib.locks_dense_attend(ctypes.byref(c), fake, None, fake, fake, fake, fake, None, fake,
                                  need, None) == -1
    assert lib.locks_decode_step(ctypes.byref(c), fake, fake, fake, fake, fake, fake, None, 3, fake,
                                 fake, fake, None, fake, need, None) == -1
    assert lib.locks_build_summaries(ctypes.byref(c), fake, fake, fake, None, -1, fake, None) == -1
    assert lib.locks_build_factors(ctypes.byref(c), fake, fake, fake, None, 4, fake, fake, fake,
                                   fake, None) == -1
    assert lib.locks_strerror(-3).decode().startswith("workspace")
    assert lib.locks_last_hip_error() == 0


def test_empty_batch_is_a_no_op(lib):
    c = cfg(num_seqs=0).c()
    need = lib.locks_workspace_bytes(ctypes.byref(c))
    fake = ctypes.c_void_p(0x1000)
    ws = ctypes.c_void_p(0x10000)
    assert lib.locks_select(ctypes.byref(c), fake, fake, fake, fake, fake, fake, None, ws, need, None) == 0
    assert lib.locks_decode_step(ctypes.byref(c), fake, fake, fake, fake, fake, fake, None, 0, fake,
                                 fake, fake, None, ws, need, None) == 0


def test_workspace_grows_with_shape(lib):
    small = cfg().c()
    big = cfg(max_pages_per_seq=4096).c()
    assert lib.locks_workspace_bytes(ctypes.byref(big)) > lib.locks_workspace_bytes(ctypes.byref(small))


@pytest.mark.parametrize("kv,code", [
    (dict(bits=0), -1), (dict(bits=9), -1), (dict(v_group=24), -1), (dict(v_group=256), -1),
    (dict(v_group=4), -1), (dict(stage=2), -1), (dict(stage=-1), -1),
])
def test_kivi_bad_arguments_are_rejected_before_launch(lib, kv, code):
    c = cfg().c()
    k = B.Kivi(4, 32, B.LOCKS_KIVI_POST)
    for name, val in kv.items():
        setattr(k, name, val)
    fake = ctypes.c_void_p(0x1000)
    assert lib.locks_kivi_quantize(ctypes.byref(c), ctypes.byref(k), fake, fake, fake, fake, None, 0,
                                   None) == code
    need = lib.locks_workspace_bytes(ctypes.byref(c))
    o = B.StepOpts(ctypes.pointer(k), None, None)
    assert lib.locks_decode_step_ex(ctypes.byref(c), ctypes.byref(o), fake, fake, fake, fake, fake,
                                    fake, fake, 1, fake, fake, fake, None, fake, need, None) == code


def test_kivi_null_pointers_dtype_and_empty_batch(lib):
    c = cfg().c()
    k = B.Kivi(2, 32, B.LOCKS_KIVI_PRE)
    fake = ctypes.c_void_p(0x1000)
    q = lib.locks_kivi_quantize
    assert q(ctypes.byref(c), None, fake, fake, fake, fake, None, 0, None) == -1
    assert q(ctypes.byref(c), ctypes.byref(k), None, fake, fake, fake, None, 0, None) == -1
    assert q(ctypes.byref(c), ctypes.byref(k), fake, fake, fake, None, None, 0, None) == -1
    assert q(ctypes.byref(c), ctypes.byref(k), fake, fake, fake, fake, None, 3, None) == -1
    assert q(ctypes.byref(c), ctypes.byref(k), fake, fake, fake, fake, fake, -1, None) == -1
    # fake quantisation rounds to bfloat16: an fp32 cache is not supported
    c32 = cfg(kv_dtype=B.LOCKS_FP32, q_dtype=B.LOCKS_FP32).c()
    assert q(ctypes.byref(c32), ctypes.byref(k), fake, fake, fake, fake, None, 0, None) == -2
    need32 = lib.locks_workspace_bytes(ctypes.byref(c32))
    o = B.StepOpts(ctypes.pointer(k), None, None)
    assert lib.locks_decode_step_ex(ctypes.byref(c32), ctypes.byref(o), fake, fake, fake, fake,
                                    fake, fake, fake, 1, fake, fake, fake, None, fake, need32,
                                    None) == -2
    # no sequences: nothing launched
    c0 = cfg(num_seqs=0).c()
    assert q(ctypes.byref(c0), ctypes.byref(k), fake, fake, fake, fake, None, 0, None) == 0
    need0 = lib.locks_workspace_bytes(ctypes.byref(c0))
    ws = ctypes.c_void_p(0x10000)
    assert lib.locks_decode_step_ex(ctypes.byref(c0), ctypes.byref(o), fake, fake, fake, fake,
                                    fake, fake, None, 0, fake, fake, fake, None, ws, need0,
                                    None) == 0
    # null options are the plain step (its own argument checks apply)
    need = lib.locks_workspace_bytes(ctypes.byref(c))
    assert lib.locks_decode_step_ex(ctypes.byref(c), None, None, fake, fake, fake, fake, fake,
                                    None, 0, fake, fake, fake, None, fake, need, None) == -1


def test_append_and_step_options_are_checked(lib):
    c = cfg().c()
    fake = ctypes.c_void_p(0x1000)
    ap = lib.locks_append_kv
    assert ap(ctypes.byref(c), None, fake, fake, fake, fake, fake, None) == -1
    assert ap(ctypes.byref(c), fake, None, fake, fake, fake, fake, None) == -1
    assert ap(ctypes.byref(c), fake, fake, fake, fake, fake, None, None) == -1
    assert ap(ctypes.byref(cfg(head_dim=64).c()), fake, fake, fake, fake, fake, fake, None) == -2
    assert ap(ctypes.byref(cfg(num_seqs=0).c()), fake, fake, fake, fake, fake, fake, None) == 0
    need = lib.locks_workspace_bytes(ctypes.byref(c))
    for kn, vn in ((fake, None), (None, fake)):   # both new rows or neither
        o = B.StepOpts(None, kn, vn)
        assert lib.locks_decode_step_ex(ctypes.byref(c), ctypes.byref(o), fake, fake, fake, fake,
                                        fake, fake, None, 0, fake, fake, fake, None, fake, need,
                                        None) == -1


def test_table_checks_switch_and_error_offset(lib):
    """The switch returns the previous setting; the error word sits inside the
    workspace, after every other region, with one word per sequence behind it."""
    try:
        assert B.set_table_checks(True) is False
        assert B.set_table_checks(True) is True
    finally:
        B.set_table_checks(False)
    c = cfg()
    off = int(lib.locks_table_error_offset(ctypes.byref(c.c())))
    ws = B.workspace_bytes(c)
    assert off % 256 == 0 and off + 4 * (1 + c.num_seqs) <= ws
    bad = cfg(rank=0)
    assert lib.locks_table_error_offset(ctypes.byref(bad.c())) == ctypes.c_size_t(-1).value
