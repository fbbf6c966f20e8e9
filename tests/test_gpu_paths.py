"""Every kernel instance and step branch the library dispatches to, reached through
the C ABI and held to the oracle: the generic scan at every rank and both query
types, the specialised scans for each (rank, group size, query type, wave steps),
the attention kernels for every pairing of query and KV types and every split
shape, both selection paths (fast, and the block-level path with survivors
re-read from memory), and the fused step's build-list branches (wider bases,
fp32 KV, KIVI before and after the build, the KV write).  Tolerances as in the
other parity tests: page LSE 1e-3 absolute, output 2e-3 rel-L2, tables by the
gap rule."""
import numpy as np
import pytest
import torch

from oracle import locks_oracle as O
from paper_2607_24555_amd import locks as B
from tests._gpu_common import (LSE_TOL, OUT_TOL, Dev, check_attention_on_table, check_sel_lse,
                               check_table, ids_of, near_tie_overlap, rel_l2)
from workloads import WorkloadSpec, build_workload, gather_unit

pytestmark = pytest.mark.gpu

DT = {"bf16": B.LOCKS_BF16, "fp32": B.LOCKS_FP32}


def _dev(name, S, G, Hkv, lens, rank, budget, kv, q, basis=B.LOCKS_BASIS_INT4, seed=21,
         spare=0, on_gpu=False):
    print(f"[paths {name}] S={S} G={G} Hkv={Hkv} lens={lens[:4]} r={rank} b={budget} kv={kv} "
          f"q={q} basis={basis}", flush=True)
    spec = WorkloadSpec(name, S, G * Hkv, Hkv, list(lens), rank, budget, kv, q,
                        spare_pages_per_seq=spare)
    d = Dev(build_workload(spec, seed, device="cuda" if on_gpu else "cpu"))
    if basis != B.LOCKS_BASIS_INT4:
        d.cfg.basis = basis
        d.ws = B.alloc_workspace(d.cfg, d.device)
    return d


def _scores_against_oracle(d, store, recs):
    cfg, G = d.cfg, d.cfg.group
    all_lse = torch.full((cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq), float("nan"),
                         device=d.device)
    B.score_pages(cfg, d.q, store, d.pt, d.sl, d.ws, all_lse)
    torch.cuda.synchronize()
    worst = 0.0
    refs = {}
    basis = B.BASIS_NAMES[cfg.basis]
    for (s, h), rec in recs.items():
        k, v, qg = d.unit(s, h)
        ref = O.decode_step(qg, k, v, rec, cfg.rank, cfg.budget_tokens, basis)
        refs[(s, h)] = (k, v, qg, ref)
        n_c = k.shape[0] // 16
        if n_c:
            got = all_lse[s, h * G:(h + 1) * G, :n_c].double().cpu().numpy()
            worst = max(worst, float(np.max(np.abs(got - ref["s_hat"]))))
    assert worst <= LSE_TOL, worst
    return refs, worst


def _step_against_oracle(d, refs, ids, sel, out, lse):
    cfg, G = d.cfg, d.cfg.group
    results, worst = [], 0.0
    for (s, h), (k, v, qg, ref) in refs.items():
        n_c, n = k.shape[0] // 16, -(-k.shape[0] // 16)
        got = ids_of(ids[s, h].tolist())
        results.append(check_table(got, ref, n, cfg.k))
        hs = slice(h * G, (h + 1) * G)
        worst = max(worst, check_attention_on_table(qg, k, v, got, out[s, hs].double().cpu().numpy(),
                                                    lse[s, hs].double().cpu().numpy()))
        check_sel_lse(sel[s, hs].double().cpu().numpy(), got, ref["s_hat"], n_c)
    return near_tie_overlap(results), worst


def _attend_on_oracle_tables(d, refs):
    cfg, G = d.cfg, d.cfg.group
    ids = torch.full((cfg.num_seqs, cfg.num_kv_heads, cfg.k), -1, dtype=torch.int32)
    for (s, h), (_, _, _, ref) in refs.items():
        ids[s, h, :len(ref["ids"])] = torch.tensor(ref["ids"], dtype=torch.int32)
    out, lse = B.sparse_attend(cfg, d.q, d.k, d.v, d.pt, d.sl, ids.to(d.device), d.ws)
    dout, dlse = B.dense_attend(cfg, d.q, d.k, d.v, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    worst = 0.0
    for (s, h), (k, v, qg, ref) in refs.items():
        hs = slice(h * G, (h + 1) * G)
        o = out[s, hs].double().cpu().numpy()
        worst = max(worst, max(rel_l2(o[g], ref["out"][g]) for g in range(G)))
        np.testing.assert_allclose(lse[s, hs].double().cpu().numpy(), ref["lse"], atol=LSE_TOL)
        o_d, l_d = O.dense_step(qg, k, v)
        od = dout[s, hs].double().cpu().numpy()
        worst = max(worst, max(rel_l2(od[g], o_d[g]) for g in range(G)))
        np.testing.assert_allclose(dlse[s, hs].double().cpu().numpy(), l_d, atol=LSE_TOL)
    assert worst <= OUT_TOL, worst
    return worst


@pytest.mark.parametrize("q", ["bf16", "fp32"])
@pytest.mark.parametrize("rank", list(range(1, 16)))
def test_generic_scan_every_rank(rank, q):
    """Two-head groups take the generic matrix-core scan at every rank."""
    d = _dev("generic", 1, 2, 2, [16 * 130 + 5], rank, 256, q, q)
    store, recs = d.oracle_summaries()
    _, worst = _scores_against_oracle(d, store, recs)
    print(f"[paths generic] r={rank} q={q}: max |hat s err| {worst:.2e}")


STEP_CASES = {
    # name: (G, rank, kv dtype, q dtype)
    "G16-r2": (16, 2, "bf16", "bf16"),
    "G16-r4": (16, 4, "bf16", "bf16"),
    "G16-r2-fp32": (16, 2, "fp32", "fp32"),
    "G16-r4-fp32q": (16, 4, "bf16", "fp32"),
    "G16-r8-fp32q": (16, 8, "bf16", "fp32"),
    "G4-r2-fp32q": (4, 2, "bf16", "fp32"),
    "G4-r4-fp32kv": (4, 4, "fp32", "bf16"),
    "G4-r4-fp32": (4, 4, "fp32", "fp32"),
    "G4-r8-fp32q": (4, 8, "bf16", "fp32"),
}


@pytest.mark.parametrize("name", sorted(STEP_CASES))
def test_step_kernel_variants(name):
    """Scan, fused step, attention on the oracle's tables and the dense baseline for
    the specialised scans and every pairing of query and KV types."""
    G, rank, kv, q = STEP_CASES[name]
    d = _dev(name, 1, G, 2, [16 * 1100 + 3], rank, 2048, kv, q)
    store, recs = d.oracle_summaries()
    refs, err = _scores_against_oracle(d, store, recs)
    ids, sel, out, lse = B.decode_step(d.cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    ov, worst = _step_against_oracle(d, refs, ids, sel, out, lse)
    worst_a = _attend_on_oracle_tables(d, refs)
    print(f"[paths {name}] hat s err {err:.2e}; step near-tie overlap {ov:.4f}, rel-L2 "
          f"{worst:.2e}; attend/dense on oracle tables rel-L2 {worst_a:.2e}")


BIG_CASES = {
    # four 16-page steps per scan wave, fp32 queries
    "G16-r8-fp32q-4steps": (2, 16, 2, [16 * 16384 + 7, 16 * 16000 + 2], 8),
    "G4-r8-fp32q-4steps": (1, 4, 8, [16 * 8192 + 5], 8),
}


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", sorted(BIG_CASES))
def test_step_four_step_scans_fp32_queries(name):
    S, G, Hkv, lens, rank = BIG_CASES[name]
    d = _dev(name, S, G, Hkv, lens, rank, 2048, "bf16", "fp32", on_gpu=True)
    store, recs = d.oracle_summaries()
    refs, err = _scores_against_oracle(d, store, recs)
    ids, sel, out, lse = B.decode_step(d.cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    ov, worst = _step_against_oracle(d, refs, ids, sel, out, lse)
    print(f"[paths {name}] hat s err {err:.2e}; near-tie overlap {ov:.4f}; rel-L2 {worst:.2e}")


SPLIT_CASES = {
    # 32 (seq, KV head) units of 128 table entries: two entries per attention wave
    "two-per-wave": (4, [16 * 256 + 9, 16 * 300, 16 * 129 + 1, 16 * 400 + 15]),
    # 128 units: eight entries per wave
    "eight-per-wave": (16, [16 * 260 + 3 * i for i in range(16)]),
}


@pytest.mark.parametrize("name", sorted(SPLIT_CASES))
def test_attention_split_shapes(name):
    S, lens = SPLIT_CASES[name]
    d = _dev(name, S, 4, 8, lens, 8, 2048, "bf16", "bf16", on_gpu=True)
    store, recs = d.oracle_summaries()
    refs, _ = _scores_against_oracle(d, store, recs)
    ids, sel, out, lse = B.decode_step(d.cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    ov, worst = _step_against_oracle(d, refs, ids, sel, out, lse)
    worst_a = _attend_on_oracle_tables(d, refs)
    print(f"[paths {name}] step rel-L2 {worst:.2e}, near-tie overlap {ov:.4f}; attend on "
          f"oracle tables {worst_a:.2e}")


@pytest.mark.timeout(600)
def test_block_level_selection_rereads_survivors():
    """A 4096-token budget over 33,001 pages: the block-level selection path, whose
    final cut holds more survivors than its registers and re-reads them."""
    d = _dev("many-survivors", 1, 2, 1, [16 * 33000 + 5], 8, 4096, "bf16", "bf16", on_gpu=True)
    store, recs = d.oracle_summaries()
    refs, _ = _scores_against_oracle(d, store, recs)
    ids, sel, out, lse = B.decode_step(d.cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    ids2, sel2 = B.select(d.cfg, d.q, store, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    assert torch.equal(ids, ids2)
    ov, worst = _step_against_oracle(d, refs, ids, sel, out, lse)
    print(f"[paths many-survivors] near-tie overlap {ov:.4f}, rel-L2 {worst:.2e}")


BUILD_CASES = {
    # name: (kv, q, basis, kivi stage or None, budget, kv write inside the step)
    "int8-basis": ("bf16", "bf16", B.LOCKS_BASIS_INT8, None, 256, False),
    "bf16-basis-kivi-post": ("bf16", "bf16", B.LOCKS_BASIS_BF16, B.LOCKS_KIVI_POST, 256, False),
    "fp32-kv": ("fp32", "fp32", B.LOCKS_BASIS_INT4, None, 256, True),
    "fp32-q-kivi-pre": ("bf16", "fp32", B.LOCKS_BASIS_INT4, B.LOCKS_KIVI_PRE, 256, True),
    "block-select-kv-write": ("bf16", "bf16", B.LOCKS_BASIS_INT4, None, 4096, True),
    "int8-basis-kv-write-kivi-pre": ("bf16", "bf16", B.LOCKS_BASIS_INT8, B.LOCKS_KIVI_PRE, 256,
                                     True),
}


@pytest.mark.parametrize("name", sorted(BUILD_CASES))
def test_step_build_list_branches(name):
    """A fused step with a build list (and optionally KIVI and the new token's KV
    write) on the step branches other than the overlapped int4 build: it must equal,
    bit for bit, the same work done by the separate entry points in order (KV
    write, KIVI PRE, build, KIVI POST, then a step without a list), and its output
    must match the oracle's attention over its own table on the final caches."""
    kv, q, basis, stage, budget, write = BUILD_CASES[name]
    rank = 4
    lens = [16 * 300 - 1, 16 * 200 + 9, 16 * 150 + 15]   # the new token fills page 299 of seq 0
    d = _dev(name, 3, 4, 2, lens, rank, budget, kv, q, basis=basis, spare=1)
    cfg = d.cfg
    dev = d.device
    store = B.alloc_summaries(cfg, dev)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    kivi = None if stage is None else B.Kivi(4, 32, stage)
    gen = torch.Generator().manual_seed(5)
    kt = torch.bfloat16 if kv == "bf16" else torch.float32
    k_new = torch.randn(3, 2, 128, generator=gen).to(kt).to(dev) if write else None
    v_new = torch.randn(3, 2, 128, generator=gen).to(kt).to(dev) if write else None
    new_lens = [L + 1 if write else L for L in lens]
    sl = torch.tensor(new_lens, dtype=torch.int32, device=dev)
    listed = [(s, L // 16 - 1) for s, L in enumerate(new_lens)] + [(1, 3), (2, 77)]
    bl = torch.tensor(listed, dtype=torch.int32, device=dev)
    blocks = torch.tensor([int(d.w.page_table[s, j]) for s, j in listed], device=dev).long()
    store[blocks] = 0                                   # the build must rewrite them
    # reference: the separate entry points in the step's order
    rk, rv, rstore = d.k.clone(), d.v.clone(), store.clone()
    if write:
        B.append_kv(cfg, k_new, v_new, rk, rv, d.pt, sl)
    if kivi is not None and stage == B.LOCKS_KIVI_PRE:
        B.kivi_quantize(cfg, kivi, rk, rv, d.pt, sl, bl)
    B.build_summaries(cfg, rk, d.pt, sl, rstore, build_list=bl)
    if kivi is not None and stage == B.LOCKS_KIVI_POST:
        B.kivi_quantize(cfg, kivi, rk, rv, d.pt, sl, bl)
    r_ids, r_sel, r_out, r_lse = B.decode_step(cfg, d.q, rk, rv, d.pt, sl, rstore, d.ws)
    torch.cuda.synchronize()
    ws2 = B.alloc_workspace(cfg, dev)
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, sl, store, ws2, build_list=bl,
                                       kivi=kivi, k_new=k_new, v_new=v_new)
    torch.cuda.synchronize()
    assert torch.equal(d.k, rk) and torch.equal(d.v, rv)
    assert torch.equal(store, rstore)
    assert torch.equal(ids, r_ids)
    assert torch.equal(out, r_out) and torch.equal(lse, r_lse)
    assert torch.equal(torch.nan_to_num(sel, nan=-7.0), torch.nan_to_num(r_sel, nan=-7.0))
    # the output against the oracle's attention over the step's table, final caches
    d.w.k_cache, d.w.v_cache = d.k, d.v
    d.w.spec.seq_lens = new_lens
    G = cfg.group
    worst = 0.0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg = gather_unit(d.w, s, h)
            got = ids_of(ids[s, h].tolist())
            assert len(got) == min(cfg.k, -(-new_lens[s] // 16))
            hs = slice(h * G, (h + 1) * G)
            worst = max(worst, check_attention_on_table(qg, k, v, got, out[s, hs].double().cpu().numpy(),
                                                        lse[s, hs].double().cpu().numpy()))
    print(f"[paths {name}] equals the separate calls bit for bit; rel-L2 on its tables "
          f"{worst:.2e}")
