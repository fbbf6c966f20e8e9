"""locks_decode_step_static -- the fused step on the library's static device scratch,
for callers that cannot allocate -- against locks_decode_step with a caller
workspace on the same inputs: two calls in a row, the second on a smaller input,
32- and 64-token pages, a step with a build list, a HIP-graph capture of the static
step, and the size limit."""
import numpy as np
import pytest
import torch

from paper_2607_24555_amd import locks as B
from tests._gpu_common import LSE_TOL, OUT_TOL, OVERLAP_TOL, Dev, ids_of, rel_l2
from workloads import WorkloadSpec, build_workload

pytestmark = pytest.mark.gpu


def _dev(S, Hq, Hkv, lens, rank, budget, seed):
    print(f"[static] S={S} Hq={Hq} Hkv={Hkv} lens={lens} r={rank} b={budget}", flush=True)
    spec = WorkloadSpec("static", S, Hq, Hkv, list(lens), rank, budget, "bf16", "bf16")
    d = Dev(build_workload(spec, seed, device="cuda"))
    store = B.alloc_summaries(d.cfg, d.device)
    B.build_summaries(d.cfg, d.k, d.pt, d.sl, store)
    return d, store


def _same(a, b):
    ids, sel, out, lse = a
    ids2, sel2, out2, lse2 = b
    assert torch.equal(ids, ids2)
    assert torch.equal(out, out2) and torch.equal(lse, lse2)
    assert torch.equal(torch.nan_to_num(sel, nan=-7.0), torch.nan_to_num(sel2, nan=-7.0))


def _close(a, b, k):
    """Tables by the overlap rule, outputs and LSEs within the parity tolerances."""
    ids, sel, out, lse = a
    ids2, sel2, out2, lse2 = b
    inter = tot = 0
    for r1, r2 in zip(ids.view(-1, k).tolist(), ids2.view(-1, k).tolist()):
        inter += len(set(ids_of(r1)) & set(ids_of(r2)))
        tot += len(ids_of(r1))
    assert inter >= OVERLAP_TOL * tot, (inter, tot)
    o1, o2 = out.double().cpu().numpy(), out2.double().cpu().numpy()
    worst = max(rel_l2(x, y) for x, y in zip(o1.reshape(-1, 128), o2.reshape(-1, 128)))
    assert worst <= OUT_TOL, worst
    assert float((lse - lse2).abs().max()) <= LSE_TOL
    fin = torch.isfinite(sel) & torch.isfinite(sel2)
    assert float((sel[fin] - sel2[fin]).abs().max()) <= LSE_TOL


def _both(d, store, bl=None):
    cfg = d.cfg
    ref = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws, build_list=bl)
    got = B.decode_step_static(cfg, d.q, d.k, d.v, d.pt, d.sl, store, build_list=bl)
    torch.cuda.synchronize()
    return ref, got


def test_static_step_matches_workspace_step_twice_then_smaller():
    # the larger input first, then a smaller one over the scratch the first left behind
    d, store = _dev(2, 32, 8, [16 * 2500 + 7, 16 * 1800 + 3], 8, 2048, 31)
    assert B.workspace_bytes(d.cfg) <= B.STATIC_SCRATCH_BYTES
    ref, got = _both(d, store)
    _same(ref, got)
    d2, store2 = _dev(1, 8, 2, [16 * 300 + 5], 4, 512, 32)
    assert B.workspace_bytes(d2.cfg) < B.workspace_bytes(d.cfg)
    ref2, got2 = _both(d2, store2)
    _same(ref2, got2)
    print("[static] two calls in a row (second smaller) equal the workspace step bit for bit")


@pytest.mark.parametrize("Bp,G", [(32, 16), (64, 4)])
def test_static_step_large_pages(Bp, G):
    """Pages of 32 and 64 tokens (their scans run as 16-token sub-pages): the static
    step equals the workspace step bit for bit."""
    print(f"[static] page {Bp}: S=2 G={G} Hkv=2 r=8 b=2048", flush=True)
    spec = WorkloadSpec("static-large", 2, 2 * G, 2, [Bp * 900 + 5, Bp * 260], 8, 2048, "bf16",
                        "bf16", page_size=Bp)
    d = Dev(build_workload(spec, 35, device="cuda"))
    store = B.alloc_summaries(d.cfg, d.device)
    B.build_summaries(d.cfg, d.k, d.pt, d.sl, store)
    ref, got = _both(d, store)
    _same(ref, got)
    print(f"[static] page {Bp}: equal to the workspace step")


def test_static_step_with_build_list():
    """The pages that just filled, listed: built beside the scan when the device's
    side stream exists, else before it on the caller's stream -- the same step."""
    d, store = _dev(3, 32, 8, [16 * 700, 16 * 420, 16 * 333], 8, 2048, 33)
    lens = [int(x) for x in d.w.spec.seq_lens]
    bl = torch.tensor([[s, L // 16 - 1] for s, L in enumerate(lens)], dtype=torch.int32,
                      device=d.device)
    ref_store = store.clone()
    ref, got = _both(d, store, bl)
    assert torch.equal(store, ref_store)      # rebuilt bytes equal the store's
    _close(ref, got, d.cfg.k)
    B.init()                                  # the side stream exists from here on
    ref, got = _both(d, store, bl)
    _same(ref, got)
    print("[static] build-list step agrees with the workspace step")


def test_static_step_replays_from_a_graph():
    d, store = _dev(1, 32, 2, [16 * 4000 + 9], 8, 2048, 34)
    cfg = d.cfg
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    gids, gsel = B.alloc_select_outputs(cfg, d.device)
    gout, glse = B.alloc_attend_outputs(cfg, d.device)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        B.decode_step_static(cfg, d.q, d.k, d.v, d.pt, d.sl, store, out_ids=gids,
                             out_sel_lse=gsel, out=gout, out_lse=glse)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (gids, gsel, gout, glse):
            t.zero_()
        # eager work of the program between replays, on the same static scratch
        B.decode_step_static(cfg, d.q, d.k, d.v, d.pt, d.sl, store)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _same((ids, sel, out, lse), (gids, gsel, gout, glse))
    print("[static] graph replays equal the eager workspace step")


def test_static_step_rejects_a_configuration_beyond_its_scratch():
    cfg = B.Config(num_seqs=64, num_q_heads=32, num_kv_heads=8, rank=2, budget_tokens=256,
                   max_pages_per_seq=8192, num_blocks=1)
    assert B.workspace_bytes(cfg) > B.STATIC_SCRATCH_BYTES
    dev = torch.device("cuda")
    q = torch.zeros(64, 32, 128, dtype=torch.bfloat16, device=dev)
    kc = torch.zeros(1, 8, 16, 128, dtype=torch.bfloat16, device=dev)
    pt = torch.zeros(64, 8192, dtype=torch.int32, device=dev)
    sl = torch.zeros(64, dtype=torch.int32, device=dev)
    summ = B.alloc_summaries(cfg, dev)
    with pytest.raises(B.LocksError, match="status -3"):
        B.decode_step_static(cfg, q, kc, kc, pt, sl, summ)
