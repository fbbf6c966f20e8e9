"""GPU checks of the new token's KV write (App. E schedule: the KV write beside the
selection) through the C ABI: locks_append_kv writes exactly the slot of token
seq_lens[s] - 1 of every sequence and KV head, and the fused step given the new rows
(locks_decode_step_ex) returns bit for bit what writing the rows first and running
the plain step returns, with and without KIVI, with and without pages to build."""
import numpy as np
import pytest
import torch

from paper_2607_24555_amd import locks as B
from tests._gpu_common import Dev
from workloads import WorkloadSpec, build_workload

pytestmark = pytest.mark.gpu
PAGE = 16


def _expected(d, k_new, v_new):
    kc, vc = d.k.clone(), d.v.clone()
    for s, L in enumerate(d.w.spec.seq_lens):
        if L < 1:
            continue
        t = L - 1
        blk = int(d.w.page_table[s, t // PAGE])
        kc[blk, :, t % PAGE] = k_new[s]
        vc[blk, :, t % PAGE] = v_new[s]
    return kc, vc


def _rows(d, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    shape = (d.cfg.num_seqs, d.cfg.num_kv_heads, 128)
    dt = d.k.dtype
    return (torch.randn(shape, generator=g).to(dt).to(d.device),
            torch.randn(shape, generator=g).to(dt).to(d.device))


@pytest.mark.parametrize("kv", ["bf16", "fp32"])
def test_append_writes_only_the_newest_token(kv):
    lens = [0, 1, 16, 17, 31, 32, 16 * 9 + 5]
    spec = WorkloadSpec("append", len(lens), 8, 2, lens, 8, 64, kv, kv, spare_pages_per_seq=1)
    d = Dev(build_workload(spec, 21))
    print(f"[append] {kv} lens {lens}", flush=True)
    k_new, v_new = _rows(d, 1)
    kc, vc = _expected(d, k_new, v_new)
    B.append_kv(d.cfg, k_new, v_new, d.k, d.v, d.pt, d.sl)
    torch.cuda.synchronize()
    assert torch.equal(d.k, kc) and torch.equal(d.v, vc)


@pytest.mark.parametrize("kivi_stage", [None, B.LOCKS_KIVI_POST, B.LOCKS_KIVI_PRE])
@pytest.mark.parametrize("filled", [True, False])
def test_step_with_new_rows_equals_write_then_step(kivi_stage, filled):
    """`filled`: the new token completes a page in some sequences, which the step
    builds (beside the scan); otherwise no page is built this step."""
    lens = [16 * 300, 16 * 200 + 9, 16 * 150, 16 * 90 + 1] if filled else \
        [16 * 300 + 1, 16 * 200 + 9, 16 * 150 + 4, 16 * 90 + 1]
    spec = WorkloadSpec("append-step", len(lens), 16, 4, lens, 2, 256, "bf16", "bf16")
    w = build_workload(spec, 23)
    a, b = Dev(w), Dev(w)
    cfg = a.cfg
    print(f"[append step] kivi {kivi_stage} filled {filled}", flush=True)
    k_new, v_new = _rows(a, 2)
    listed = [(s, L // PAGE - 1) for s, L in enumerate(lens) if L % PAGE == 0]
    bl = torch.tensor(listed, dtype=torch.int32, device=a.device).reshape(-1, 2) if listed else None
    kv = None if kivi_stage is None else B.Kivi(4, 32, kivi_stage)
    store_a, store_b = B.alloc_summaries(cfg), B.alloc_summaries(cfg)
    B.build_summaries(cfg, a.k, a.pt, a.sl, store_a)
    B.build_summaries(cfg, b.k, b.pt, b.sl, store_b)
    # a: the caller writes the rows, then the plain (or KIVI) step
    ka, va = _expected(a, k_new, v_new)
    a.k.copy_(ka)
    a.v.copy_(va)
    ra = B.decode_step(cfg, a.q, a.k, a.v, a.pt, a.sl, store_a, a.ws, build_list=bl, kivi=kv)
    # b: the step writes the rows itself
    rb = B.decode_step(cfg, b.q, b.k, b.v, b.pt, b.sl, store_b, b.ws, build_list=bl, kivi=kv,
                       k_new=k_new, v_new=v_new)
    torch.cuda.synchronize()
    assert torch.equal(a.k, b.k) and torch.equal(a.v, b.v)
    assert torch.equal(store_a, store_b)
    for x, y in zip(ra, rb):
        assert torch.equal(x.cpu(), y.cpu()) or np.array_equal(
            x.cpu().numpy(), y.cpu().numpy(), equal_nan=True)
