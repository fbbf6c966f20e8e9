"""GPU parity: liblocks (through its C ABI) against the CPU fp64 oracle on the same
seeded inputs.  Tolerances: page LSE 1e-3 absolute; attention output 2e-3 relative
L2; selected sets identical where the oracle's ranking gap exceeds 1e-3, else an
aggregate overlap of at least 99%."""
import math

import numpy as np
import pytest
import torch

from oracle import locks_oracle as O
from paper_2607_24555_amd import locks as B
from tests._gpu_common import (LSE_TOL, OUT_TOL, OVERLAP_TOL, Dev, check_attention_on_table,
                               check_sel_lse, check_table, ids_of, near_tie_overlap, parse_codes,
                               rel_l2)
from workloads import WorkloadSpec, build_workload, config_spec, make_workload

pytestmark = pytest.mark.gpu

CASES = {
    "cfg0": (0, {}),
    "cfg0-ragged": (0, dict(seq_len=4096 - 5)),
    "cfg1-ragged": (1, dict(seq_len=32768 - 3)),
    "cfg1-r2-b256": (1, dict(seq_len=8192 + 16, rank=2, budget_tokens=256)),
    "r4-G4": (1, dict(seq_len=4096 + 7, rank=4, num_kv_heads=2, num_q_heads=8)),
    "G16": (3, dict(seq_len=16384 + 9)),
    "mixed-lens": (4, dict(num_seqs=5)),
}


def _mk(name):
    cfg_id, ov = CASES[name]
    print(f"[case {name}] cfg {cfg_id} {ov}", flush=True)
    return Dev(make_workload(cfg_id, seed=1, **ov))


def _edge_workload(G, lens, rank=8, budget=64, kv="bf16", seed=3):
    spec = WorkloadSpec("edge", len(lens), 2 * G, 2, list(lens), rank, budget, kv, kv)
    return Dev(build_workload(spec, seed))


@pytest.fixture(scope="module", params=sorted(CASES))
def case(request):
    d = _mk(request.param)
    store, recs = d.oracle_summaries()
    return request.param, d, store, recs


def _oracle_unit(d, recs, s, h):
    k, v, qg = d.unit(s, h)
    return k, v, qg, O.decode_step(qg, k, v, recs[(s, h)], d.cfg.rank, d.cfg.budget_tokens)


def test_scan_and_select_on_oracle_bytes(case):
    name, d, store, recs = case
    cfg = d.cfg
    all_lse = torch.full((cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq), float("nan"),
                         device=d.device)
    ids, sel = B.select(cfg, d.q, store, d.pt, d.sl, d.ws, out_all_lse=all_lse)
    torch.cuda.synchronize()
    G = cfg.group
    results = []
    worst = 0.0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg, ref = _oracle_unit(d, recs, s, h)
            n_c, n = k.shape[0] // 16, -(-k.shape[0] // 16)
            got = all_lse[s, h * G:(h + 1) * G, :n_c].double().cpu().numpy()
            if n_c:
                worst = max(worst, float(np.max(np.abs(got - ref["s_hat"]))))
            g_ids = ids_of(ids[s, h].tolist())
            results.append(check_table(g_ids, ref, n, cfg.k))
            assert ids[s, h].tolist()[len(g_ids):] == [-1] * (cfg.k - len(g_ids))
            gsel = sel[s, h * G:(h + 1) * G].double().cpu().numpy()
            # the returned LSEs are exactly the scan's scores of the table's pages
            for t, j in enumerate(g_ids):
                if j < n_c:
                    np.testing.assert_allclose(gsel[:, t], got[:, j], atol=0, rtol=0)
            check_sel_lse(gsel, g_ids, ref["s_hat"], n_c)
    overlap = near_tie_overlap(results)
    print(f"[{name}] max |hat s gpu - oracle| = {worst:.3e}; near-tie overlap {overlap:.4f}")
    assert worst <= LSE_TOL


def test_attend_on_oracle_table(case):
    name, d, store, recs = case
    cfg = d.cfg
    ids = torch.full((cfg.num_seqs, cfg.num_kv_heads, cfg.k), -1, dtype=torch.int32)
    refs = {}
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg, ref = _oracle_unit(d, recs, s, h)
            ids[s, h, :len(ref["ids"])] = torch.tensor(ref["ids"], dtype=torch.int32)
            refs[(s, h)] = ref
    out, lse = B.sparse_attend(cfg, d.q, d.k, d.v, d.pt, d.sl, ids.to(d.device), d.ws)
    torch.cuda.synchronize()
    G = cfg.group
    worst = 0.0
    for (s, h), ref in refs.items():
        o = out[s, h * G:(h + 1) * G].double().cpu().numpy()
        for g in range(G):
            worst = max(worst, rel_l2(o[g], ref["out"][g]))
        np.testing.assert_allclose(lse[s, h * G:(h + 1) * G].double().cpu().numpy(), ref["lse"],
                                   atol=LSE_TOL)
    print(f"[{name}] sparse attend worst rel-L2 = {worst:.3e}")
    assert worst <= OUT_TOL


def test_dense_attend(case):
    name, d, store, recs = case
    cfg = d.cfg
    out, lse = B.dense_attend(cfg, d.q, d.k, d.v, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    G = cfg.group
    worst = 0.0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg = d.unit(s, h)
            o_ref, l_ref = O.dense_step(qg, k, v)
            o = out[s, h * G:(h + 1) * G].double().cpu().numpy()
            for g in range(G):
                worst = max(worst, rel_l2(o[g], o_ref[g]))
            np.testing.assert_allclose(lse[s, h * G:(h + 1) * G].double().cpu().numpy(), l_ref,
                                       atol=LSE_TOL)
    print(f"[{name}] dense worst rel-L2 = {worst:.3e}")
    assert worst <= OUT_TOL


def _check_step_against_oracle(name, d, recs, ids, out, lse, sel=None):
    """Every unit of a fused step on oracle bytes: the table by the gap rule (and
    the tolerance band at near ties), the output and LSE against the oracle's
    attention over the GPU's own table, and the returned page LSEs."""
    cfg = d.cfg
    G = cfg.group
    results, same, worst = [], 0, 0.0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg, ref = _oracle_unit(d, recs, s, h)
            n_c, n = k.shape[0] // 16, -(-k.shape[0] // 16)
            got = ids_of(ids[s, h].tolist())
            results.append(check_table(got, ref, n, cfg.k))
            same += got == ref["ids"]
            o = out[s, h * G:(h + 1) * G].double().cpu().numpy()
            l = lse[s, h * G:(h + 1) * G].double().cpu().numpy()
            worst = max(worst, check_attention_on_table(qg, k, v, got, o, l))
            if sel is not None:
                check_sel_lse(sel[s, h * G:(h + 1) * G].double().cpu().numpy(), got,
                              ref["s_hat"], n_c)
    overlap = near_tie_overlap(results)
    print(f"[{name}] tables identical on {same}/{len(results)} units, near-tie overlap "
          f"{overlap:.4f}, worst rel-L2 {worst:.3e}")


def test_decode_step_on_oracle_bytes(case):
    name, d, store, recs = case
    ids, sel, out, lse = B.decode_step(d.cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    _check_step_against_oracle(name, d, recs, ids, out, lse, sel)


def test_decode_step_with_gpu_built_summaries(case):
    """The fused step over summaries the GPU built itself.  int4 codes may flip
    between an fp32 and an fp64 build, so tables are held to the overlap rule;
    every unit's output is checked against the oracle's attention over the GPU's
    own table."""
    name, d, store_ref, recs = case
    cfg = d.cfg
    store = B.alloc_summaries(cfg, d.device)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    G = cfg.group
    inter = tot = 0
    worst = 0.0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg, ref = _oracle_unit(d, recs, s, h)
            got = ids_of(ids[s, h].tolist())
            inter += len(set(got) & set(ref["ids"]))
            tot += len(ref["ids"])
            o = out[s, h * G:(h + 1) * G].double().cpu().numpy()
            l = lse[s, h * G:(h + 1) * G].double().cpu().numpy()
            worst = max(worst, check_attention_on_table(qg, k, v, got, o, l))
    print(f"[{name}] gpu-built summaries: table overlap {inter / max(tot, 1):.4f}, "
          f"worst rel-L2 on the GPU's tables {worst:.2e}")
    assert inter / max(tot, 1) >= OVERLAP_TOL


def test_build_codes_match_oracle(case):
    """GPU-built records against oracle-built records: every code within +-1 and at
    least 99.9% identical on pages with a clear spectral gap at r."""
    name, d, store_ref, recs = case
    cfg = d.cfg
    store = B.alloc_summaries(cfg, d.device)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    torch.cuda.synchronize()
    r = cfg.rank
    same = total = 0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            rec = recs[(s, h)]
            n_c = rec.shape[0]
            if n_c == 0:
                continue
            k, _, _ = d.unit(s, h)
            f = O.build_factors(k[:n_c * 16].reshape(n_c, 16, 128), r)
            lam = f["sigma2"]
            gapped = (lam[:, r - 1] - lam[:, r]) > 1e-3 * lam[:, r - 1]
            blocks = d.w.page_table[s, :n_c].long().to(d.device)
            got = parse_codes(store[blocks, h].cpu().numpy(), r)
            want = parse_codes(rec, r)
            for key in ("vcodes", "ccodes", "mcodes"):
                a, b = got[key][gapped], want[key][gapped]
                assert np.max(np.abs(a - b)) <= 1, (key, s, h)
                same += int(np.sum(a == b))
                total += a.size
    frac = same / max(total, 1)
    print(f"[{name}] identical codes on gapped pages: {frac:.5f}")
    assert frac >= 0.999


def test_build_factors_reconstruct_like_oracle(case):
    """Unquantised GPU factors: eigenvalues, and logits q^T(mu + V c_i)/sqrt d for the
    group queries and fresh N(0,1) queries, on pages with a spectral gap at r."""
    name, d, store_ref, recs = case
    cfg = d.cfg
    r = cfg.rank
    rng = np.random.default_rng(5)
    for s in range(min(cfg.num_seqs, 2)):
        L = int(d.w.spec.seq_lens[s])
        n_c = L // 16
        if n_c == 0:
            continue
        pages = np.arange(0, n_c, max(1, n_c // 64))
        lst = torch.tensor([[s, int(j)] for j in pages], dtype=torch.int32, device=d.device)
        mu, basis, coef, sig2 = B.build_factors(cfg, d.k, d.pt, d.sl, lst)
        torch.cuda.synchronize()
        for h in range(cfg.num_kv_heads):
            k, _, qg = d.unit(s, h)
            f = O.build_factors(k[:n_c * 16].reshape(n_c, 16, 128)[pages], r)
            lam = f["sigma2"]
            gapped = (lam[:, r - 1] - lam[:, r]) > 1e-3 * lam[:, r - 1]
            g2 = sig2[:, h].double().cpu().numpy()
            assert np.all(np.abs(g2 - lam) <= 1e-4 * lam[:, :1] + 1e-4 * np.abs(lam))
            qs = np.concatenate([qg, rng.standard_normal((4, 128))])
            rec_g = mu[:, h].double().cpu().numpy()[:, None, :] + np.einsum(
                "pil,pcl->pic", coef[:, h].double().cpu().numpy(), basis[:, h].double().cpu().numpy())
            rec_o = f["mu"][:, None, :] + np.einsum("pil,pcl->pic", f["C"], f["V"])
            zg = np.einsum("gc,pic->gpi", qs, rec_g) / math.sqrt(128)
            zo = np.einsum("gc,pic->gpi", qs, rec_o) / math.sqrt(128)
            err = np.max(np.abs(zg - zo)[:, gapped]) if gapped.any() else 0.0
            print(f"[{name}] factors s{s} h{h}: max logit diff {err:.2e} on {gapped.sum()} pages")
            assert err <= LSE_TOL


@pytest.mark.parametrize("G,lens,rank,budget,kv", [
    (1, [0, 5, 16, 17, 48, 200, 1000], 8, 64, "bf16"),
    (8, [0, 15, 16, 33, 160, 161, 2000], 1, 48, "bf16"),
    (4, [2048, 1, 999, 32], 15, 512, "fp32"),
    (4, [16 * 300 + 5, 777, 16 * 64], 8, 256, "fp32"),
    (2, [4096 * 4 + 3, 64], 8, 2048, "bf16"),
    # budget above 2080 tokens: the block-level (generic) selection path
    (4, [16 * 700 + 7, 16 * 300, 5000, 16 * 257], 8, 4096, "bf16"),
    # more than 4096 pages per sequence: several wave-level selection chunks
    (2, [4096 * 16 * 2 + 37, 4096 * 16 + 80], 2, 256, "bf16"),
    # 20,001 pages: each 1024-page chunk keeps fewer survivors than the table needs
    (4, [16 * 20000 + 5], 8, 2048, "bf16"),
])
def test_edge_batches(G, lens, rank, budget, kv):
    """Empty, sub-page, exact-page, tiny-budget and n <= k sequences in one batch."""
    print(f"[edge] G={G} lens={lens} r={rank} b={budget} {kv}", flush=True)
    d = _edge_workload(G, lens, rank, budget, kv)
    cfg = d.cfg
    store, recs = d.oracle_summaries()
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    _check_step_against_oracle("edge", d, recs, ids, out, lse, sel)
    # a second call on the same workspace gives bit-identical results (no state)
    ids2, sel2, out2, lse2 = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    assert torch.equal(ids, ids2) and torch.equal(out, out2)


def test_clustered_top_pages_exact_recut():
    """The best pages crowd into two selection chunks (far more of them than a
    chunk keeps as survivors), so the table must come from the exact recut over
    every page's key; it must still equal the oracle's."""
    n = 20001
    spec = WorkloadSpec("clustered", 1, 8, 2, [16 * (n - 1) + 3], 8, 2048, "bf16", "bf16")
    w = build_workload(spec, 7)
    G = 4
    for h in range(2):
        qhat = w.q[0, h * G:(h + 1) * G].float().mean(0)
        qhat = qhat / qhat.norm()
        blocks = w.page_table[0, 3000:3200].long()
        w.k_cache[blocks, h] = (w.k_cache[blocks, h].float() + 3.0 * qhat).to(w.k_cache.dtype)
    print("[clustered] pages 3000..3199 raised", flush=True)
    d = Dev(w)
    cfg = d.cfg
    store, recs = d.oracle_summaries()
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    for h in range(2):
        _, _, _, ref = _oracle_unit(d, recs, 0, h)
        inside = sum(3000 <= j < 3200 for j in ref["ids"])
        assert inside > 64, inside  # more than any chunk's survivor row holds
    _check_step_against_oracle("clustered", d, recs, ids, out, lse, sel)
    ids2, sel2 = B.select(cfg, d.q, store, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    assert torch.equal(ids2, ids)


def test_reasoning_steps_build_filled_pages_inline():
    """The reasoning workload's step loop (32 q / 8 kv heads, r = 2, b = 256): every
    step writes one new token per sequence into the paged cache, bumps seq_lens
    and lists the pages that just filled as the step's build list.  After the loop
    the incrementally built summary store equals a fresh build of every complete
    page bit for bit, and the last step agrees with the oracle run from scratch
    on the final keys (GPU-built summaries: tables by the overlap rule)."""
    spec = config_spec(4, num_seqs=4, seed=2)
    # one sequence fills a page on the first append, one on the fifth, one sits
    # exactly on a page boundary, one is arbitrary
    spec.seq_lens = [16 * 600 - 1, 16 * 800 - 5, 16 * 512, spec.seq_lens[3]]
    w = build_workload(spec, 2)
    d = Dev(w)
    cfg = d.cfg
    print(f"[reasoning] lens {spec.seq_lens} r={cfg.rank} b={cfg.budget_tokens}", flush=True)
    store = B.alloc_summaries(cfg, d.device)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    gen = torch.Generator().manual_seed(11)
    lens = list(spec.seq_lens)
    built = 0
    ids = out = lse = None
    for step in range(20):
        pairs = []
        for s in range(cfg.num_seqs):
            j, r = divmod(lens[s], 16)
            blk = int(w.page_table[s, j])
            assert blk >= 0
            # the new token: an earlier key of the sequence plus noise; value N(0, 1)
            kn = (w.k_cache[int(w.page_table[s, j - 1]), :, r].float()
                  + 0.3 * torch.randn(cfg.num_kv_heads, 128, generator=gen)).to(w.k_cache.dtype)
            vn = torch.randn(cfg.num_kv_heads, 128, generator=gen).to(w.v_cache.dtype)
            w.k_cache[blk, :, r] = kn
            w.v_cache[blk, :, r] = vn
            d.k[blk, :, r] = kn.to(d.device)
            d.v[blk, :, r] = vn.to(d.device)
            lens[s] += 1
            if lens[s] % 16 == 0:
                pairs.append((s, j))
        d.sl.copy_(torch.tensor(lens, dtype=torch.int32))
        bl = torch.tensor(pairs, dtype=torch.int32, device=d.device) if pairs else None
        built += len(pairs)
        ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws,
                                           build_list=bl)
    torch.cuda.synchronize()
    assert built >= 4, built
    spec.seq_lens = lens
    w.seq_lens = torch.tensor(lens, dtype=torch.int32)
    fresh = B.alloc_summaries(cfg, d.device)
    B.build_summaries(cfg, d.k, d.pt, d.sl, fresh)
    torch.cuda.synchronize()
    for s in range(cfg.num_seqs):
        blocks = w.page_table[s, :lens[s] // 16].long().to(d.device)
        assert torch.equal(store[blocks], fresh[blocks]), s
    inter, tot = 0, 0
    G = cfg.group
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg = d.unit(s, h)
            ref = O.decode_step(qg, k, v, O.unit_summaries(k, cfg.rank), cfg.rank,
                                cfg.budget_tokens)
            got = ids_of(ids[s, h].tolist())
            inter += len(set(got) & set(ref["ids"]))
            tot += len(ref["ids"])
            check_attention_on_table(qg, k, v, got, out[s, h * G:(h + 1) * G].double().cpu().numpy(),
                                     lse[s, h * G:(h + 1) * G].double().cpu().numpy())
    print(f"[reasoning] {built} pages built inline; final table overlap {inter / tot:.4f}")
    assert inter / tot >= OVERLAP_TOL


@pytest.mark.parametrize("n,budget,rank", [(5001, 1024, 4), (16389, 2048, 2)])
def test_identical_pages_tie_break(n, budget, rank):
    """Every page holds the same keys, so all page scores tie exactly: the table
    is the sink, the k - 2 lowest candidate pages and the recent page (ties go
    to the lower page), across several selection chunks (the larger case keeps
    more tied survivors than the compacted final cut holds)."""
    print(f"[ties] n={n} b={budget} r={rank}", flush=True)
    spec = WorkloadSpec("ties", 1, 8, 2, [16 * (n - 1) + 3], rank, budget, "bf16", "bf16")
    w = build_workload(spec, 5)
    w.k_cache[:] = w.k_cache[:1].clone()
    d = Dev(w)
    cfg = d.cfg
    store, recs = d.oracle_summaries()
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    want = [0] + list(range(1, cfg.k - 1)) + [n - 1]
    for h in range(cfg.num_kv_heads):
        assert ids_of(ids[0, h].tolist()) == want
    ids2, sel2 = B.select(cfg, d.q, store, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    assert torch.equal(ids2, ids)
    _check_step_against_oracle("ties", d, recs, ids, out, lse, sel)


def test_decode_step_builds_last_pages_beside_the_scan():
    """A step whose build list holds the last complete page of every sequence: those
    pages are built and scored beside the scan of the others (side stream).  The
    rebuilt bytes equal the store's, the outputs match the same step without a
    build list (the scored pages differ only by rounding), and a HIP graph of the
    step replays the eager result exactly (the first such call, which creates the
    side stream, is eager)."""
    d = _mk("mixed-lens")
    cfg, dev = d.cfg, d.device
    store = B.alloc_summaries(cfg, dev)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    torch.cuda.synchronize()
    ref = store.clone()
    lens = [int(x) for x in d.w.spec.seq_lens]
    bl = torch.tensor([[s, L // 16 - 1] for s, L in enumerate(lens) if L >= 16], dtype=torch.int32,
                      device=dev)
    print(f"[builds] {bl.shape[0]} last pages listed, lens {lens}", flush=True)
    ids0, sel0, out0, lse0 = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    ids, sel = B.alloc_select_outputs(cfg, dev)
    out, lse = B.alloc_attend_outputs(cfg, dev)
    B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws, build_list=bl, out_ids=ids,
                  out_sel_lse=sel, out=out, out_lse=lse)
    torch.cuda.synchronize()
    assert torch.equal(store, ref)
    assert float((out - out0).abs().max()) <= 1e-4
    assert float((lse - lse0).abs().max()) <= 1e-4
    same = sum(len(set(a) & set(b)) for a, b in zip(ids.view(-1, ids.shape[-1]).tolist(),
                                                     ids0.view(-1, ids0.shape[-1]).tolist()))
    assert same >= 0.99 * ids.numel(), (same, ids.numel())
    fin = torch.isfinite(sel0)
    assert torch.equal(fin, torch.isfinite(sel))
    assert float((sel[fin] - sel0[fin]).abs().max()) <= 1e-3
    gids, gsel = B.alloc_select_outputs(cfg, dev)
    gout, glse = B.alloc_attend_outputs(cfg, dev)
    ws2 = B.alloc_workspace(cfg, dev)

    def call():
        B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, ws2, build_list=bl, out_ids=gids,
                      out_sel_lse=gsel, out=gout, out_lse=glse)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (gids, gsel, gout, glse):
            t.zero_()
        B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws, build_list=bl)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(gids, ids), rep
        assert torch.equal(gout, out) and torch.equal(glse, lse), rep
        assert torch.equal(torch.nan_to_num(gsel, nan=-7.0), torch.nan_to_num(sel, nan=-7.0)), rep
        assert torch.equal(store, ref), rep
    print("[builds] overlapped builds: eager and 3 graph replays agree")


@pytest.mark.parametrize("name", ["G16", "r4-G4"])
def test_decode_step_graph_replay(name):
    """The fused step captured in a HIP graph gives the eager result on every
    replay, with eager library work and host synchronisation between replays."""
    d = _mk(name)
    cfg, dev = d.cfg, d.device
    store = B.alloc_summaries(cfg, dev)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    ids, sel = B.alloc_select_outputs(cfg, dev)
    out, lse = B.alloc_attend_outputs(cfg, dev)
    B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws, out_ids=ids, out_sel_lse=sel,
                  out=out, out_lse=lse)
    torch.cuda.synchronize()
    ws2 = B.alloc_workspace(cfg, dev)
    gids, gsel = B.alloc_select_outputs(cfg, dev)
    gout, glse = B.alloc_attend_outputs(cfg, dev)

    def call():
        B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, ws2, out_ids=gids, out_sel_lse=gsel,
                      out=gout, out_lse=glse)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (gids, gsel, gout, glse):
            t.zero_()
        # eager work of the program between replays (another step, another workspace)
        B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(gids, ids), rep
        assert torch.equal(gout, out) and torch.equal(glse, lse), rep
        assert torch.equal(torch.nan_to_num(gsel, nan=-7.0), torch.nan_to_num(sel, nan=-7.0)), rep
    print(f"[{name}] graph replay matches the eager step on 3 replays")
