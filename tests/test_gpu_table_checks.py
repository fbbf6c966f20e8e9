"""Table checks, the device-side guard of page-table and sequence-length reads
(locks_set_table_checks): valid tables give the same outputs bit for bit and a
zero error word; an out-of-range block id or sequence length is clamped on the
device, reported in the workspace's error word (and the per-sequence words
behind it), and leaves the other sequences' outputs untouched."""
import pytest
import torch

from paper_2607_24555_amd import locks as B
from tests._gpu_common import Dev
from workloads import WorkloadSpec, build_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _checks_off_afterwards():
    yield
    B.set_table_checks(False)


@pytest.fixture(scope="module")
def dev():
    print("[table checks] S=3 Hq=8 Hkv=2 lens=[700, 1500, 333] r=8 b=256", flush=True)
    spec = WorkloadSpec("table-checks", 3, 8, 2, [700, 1500, 333], 8, 256, "bf16", "bf16")
    d = Dev(build_workload(spec, 5, device="cpu"))
    store = B.alloc_summaries(d.cfg, d.device)
    B.build_summaries(d.cfg, d.k, d.pt, d.sl, store)
    torch.cuda.synchronize()
    return d, store


def _step(d, store, pt, sl):
    ids, sel, out, lse = B.decode_step(d.cfg, d.q, d.k, d.v, pt, sl, store, d.ws)
    torch.cuda.synchronize()
    return ids.clone(), sel.clone(), out.clone(), lse.clone()


def _same(a, b):
    return all(torch.equal(torch.nan_to_num(x, nan=123.0), torch.nan_to_num(y, nan=123.0))
               for x, y in zip(a, b))


def test_valid_tables_pass_unchanged(dev):
    d, store = dev
    plain = _step(d, store, d.pt, d.sl)
    dense_plain = B.dense_attend(d.cfg, d.q, d.k, d.v, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    dense_plain = tuple(t.clone() for t in dense_plain)
    B.set_table_checks(True)
    checked = _step(d, store, d.pt, d.sl)
    assert B.table_errors(d.cfg, d.ws) == (0, [0, 0, 0])
    assert _same(plain, checked)
    dense_checked = B.dense_attend(d.cfg, d.q, d.k, d.v, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    assert B.table_errors(d.cfg, d.ws)[0] == 0
    assert _same(dense_plain, dense_checked)
    # the static entry point reads the checked copies as well
    static = B.decode_step_static(d.cfg, d.q, d.k, d.v, d.pt, d.sl, store)
    torch.cuda.synchronize()
    assert _same(plain, static)


def test_bad_block_ids_are_clamped_and_reported(dev):
    d, store = dev
    plain = _step(d, store, d.pt, d.sl)
    pt = d.pt.clone()
    pt[1, 3] = d.cfg.num_blocks + 5   # page 3 of sequence 1 (94 pages)
    pt[2, 0] = -7                     # the sink page of sequence 2
    B.set_table_checks(True)
    got = _step(d, store, pt, d.sl)
    word, rows = B.table_errors(d.cfg, d.ws)
    assert word == B.LOCKS_TABLE_E_BLOCK
    assert rows == [0, B.LOCKS_TABLE_E_BLOCK, B.LOCKS_TABLE_E_BLOCK]
    # sequence 0 is computed from its own rows only
    for p, g in zip(plain, got):
        assert torch.equal(torch.nan_to_num(p[0], nan=123.0), torch.nan_to_num(g[0], nan=123.0))
    # the word follows the last checked call
    _step(d, store, d.pt, d.sl)
    assert B.table_errors(d.cfg, d.ws) == (0, [0, 0, 0])


def test_bad_lengths_are_clamped_and_reported(dev):
    d, store = dev
    plain = _step(d, store, d.pt, d.sl)
    sl = d.sl.clone()
    sl[1] = d.cfg.page_size * d.cfg.max_pages_per_seq + 100
    sl[2] = -3
    B.set_table_checks(True)
    got = _step(d, store, d.pt, sl)
    word, rows = B.table_errors(d.cfg, d.ws)
    assert word & B.LOCKS_TABLE_E_LENGTH
    assert rows[0] == 0 and rows[1] & B.LOCKS_TABLE_E_LENGTH and rows[2] == B.LOCKS_TABLE_E_LENGTH
    for p, g in zip(plain, got):
        assert torch.equal(torch.nan_to_num(p[0], nan=123.0), torch.nan_to_num(g[0], nan=123.0))
    # the empty (clamped) sequence selects nothing
    assert bool((got[0][2] == -1).all())
