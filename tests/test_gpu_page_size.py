"""GPU parity at page sizes B = 32 and 64 (App. D.3 "Page size"): the build of the
B x B Gram's eigenpairs (unquantised factors through reconstructed logits, stored
codes), the scan of B-token records, the selection with k = ceil(b / B) and the
attention over B-token pages, each through the C ABI against the oracle at the
same tolerances as 16-token pages (page LSE 1e-3, output 2e-3 rel-L2, tables by
the gap rule)."""
import math

import numpy as np
import pytest
import torch

from oracle import locks_oracle as O
from paper_2607_24555_amd import locks as B
from tests._gpu_common import (LSE_TOL, OVERLAP_TOL, Dev, check_attention_on_table, check_sel_lse,
                               check_table, ids_of, near_tie_overlap, rel_l2)
from workloads import WorkloadSpec, build_workload, gather_unit

pytestmark = pytest.mark.gpu


def _dev(name, Bp, S, G, Hkv, lens, rank, budget, kv="bf16", q="bf16", seed=41, spare=0,
         on_gpu=False):
    print(f"[page {Bp}] {name}: S={S} G={G} Hkv={Hkv} lens={lens[:4]} r={rank} b={budget} "
          f"kv={kv} q={q}", flush=True)
    spec = WorkloadSpec(name, S, G * Hkv, Hkv, list(lens), rank, budget, kv, q,
                        spare_pages_per_seq=spare, page_size=Bp)
    return Dev(build_workload(spec, seed, device="cuda" if on_gpu else "cpu"))


def _well_posed(f, r, rel=1e-3):
    lam = f["sigma2"]
    ok = np.ones(lam.shape[0], bool)
    for l in range(r):
        ok &= (lam[:, l] - lam[:, l + 1]) > rel * lam[:, l]
    a = np.sort(np.abs(f["V"]), axis=1)
    ok &= np.all(a[:, -1, :] - a[:, -2, :] > rel * a[:, -1, :], axis=1)
    return ok


def _codes(rec, r, Bp):
    """Integer codes of int4-basis records of B-token pages (parsed here, by hand)."""
    rec = rec.astype(np.int64)
    v = np.empty((rec.shape[0], 128, r), np.int64)
    for l in range(r):
        b = rec[:, 64 * l:64 * l + 64]
        v[:, 0::2, l] = (b & 15) - 8
        v[:, 1::2, l] = (b >> 4) - 8
    c = rec[:, 64 * r:64 * r + Bp * r] - 128
    m = rec[:, 64 * r + Bp * r:64 * r + Bp * r + 128] - 128
    return {"vcodes": v, "ccodes": c, "mcodes": m}


@pytest.mark.parametrize("Bp,rank,kv", [(32, 8, "bf16"), (64, 8, "bf16"), (32, 2, "fp32"),
                                        (64, 15, "bf16"), (32, 1, "bf16")])
def test_build_factors_and_codes(Bp, rank, kv):
    """Unquantised factors: every eigenvalue of the B x B Gram (within 1e-4 of the
    largest), reconstructed logits q^T(mu + V c_i)/sqrt d for the group queries and
    fresh ones on pages with a gap at r (1e-3); stored codes within +-1 and 99.9%
    identical on well-posed pages."""
    d = _dev("build", Bp, 1, 4, 2, [Bp * 300 + 7], rank, 2048, kv, kv)
    cfg = d.cfg
    r = rank
    L = int(d.w.spec.seq_lens[0])
    n_c = L // Bp
    pages = np.arange(0, n_c, 3)
    lst = torch.tensor([[0, int(j)] for j in pages], dtype=torch.int32, device=d.device)
    mu, basis, coef, sig2 = B.build_factors(cfg, d.k, d.pt, d.sl, lst)
    store = B.alloc_summaries(cfg, d.device)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    for h in range(cfg.num_kv_heads):
        k, _, qg = d.unit(0, h)
        f = O.build_factors(k[:n_c * Bp].reshape(n_c, Bp, 128), r)
        lam = f["sigma2"][pages]
        g2 = sig2[:, h].double().cpu().numpy()
        assert g2.shape == lam.shape
        assert np.all(np.abs(g2 - lam) <= 1e-4 * lam[:, :1] + 1e-4 * np.abs(lam))
        gapped = (lam[:, r - 1] - lam[:, r]) > 1e-3 * lam[:, r - 1]
        qs = np.concatenate([qg, rng.standard_normal((4, 128))])
        rec_g = mu[:, h].double().cpu().numpy()[:, None, :] + np.einsum(
            "pil,pcl->pic", coef[:, h].double().cpu().numpy(), basis[:, h].double().cpu().numpy())
        rec_o = f["mu"][pages][:, None, :] + np.einsum("pil,pcl->pic", f["C"][pages], f["V"][pages])
        zg = np.einsum("gc,pic->gpi", qs, rec_g) / math.sqrt(128)
        zo = np.einsum("gc,pic->gpi", qs, rec_o) / math.sqrt(128)
        err = np.max(np.abs(zg - zo)[:, gapped]) if gapped.any() else 0.0
        # orthonormal basis columns for the kept modes
        Vg = basis[:, h].double().cpu().numpy()
        kept = np.sum(lam[:, :r] > 1e-6 * lam[:, :1], axis=1)
        for p in range(Vg.shape[0]):
            kk = int(kept[p])
            np.testing.assert_allclose(Vg[p, :, :kk].T @ Vg[p, :, :kk], np.eye(kk), atol=1e-4)
        # stored codes
        rec = O.encode(f["mu"], f["V"], f["C"])
        posed = _well_posed(f, r)
        blocks = d.w.page_table[0, :n_c].long().to(d.device)
        got, want = _codes(store[blocks, h].cpu().numpy(), r, Bp), _codes(rec, r, Bp)
        same = total = 0
        for key in want:
            a, b = got[key][posed], want[key][posed]
            assert np.max(np.abs(a - b), initial=0) <= 1, key
            same += int(np.sum(a == b))
            total += a.size
        print(f"[page {Bp}] r={r} {kv} h{h}: max logit diff {err:.2e} on {int(gapped.sum())} "
              f"pages; identical codes {same / max(total, 1):.5f} on {int(posed.sum())}/{n_c}",
              flush=True)
        assert err <= LSE_TOL
        assert same >= 0.999 * total


STEP = {
    # name: (B, S, G, Hkv, lens, rank, budget, kv, q)
    "B32-G4-r8": (32, 3, 4, 2, [32 * 700 + 5, 32 * 130 + 31, 32 * 40], 8, 2048, "bf16", "bf16"),
    "B64-G4-r8": (64, 3, 4, 2, [64 * 500 + 63, 64 * 90, 64 * 20 + 1], 8, 2048, "bf16", "bf16"),
    "B32-G16-r8": (32, 1, 16, 2, [32 * 1500 + 9], 8, 2048, "bf16", "bf16"),
    "B64-G16-r2": (64, 1, 16, 2, [64 * 900 + 9], 2, 2048, "bf16", "bf16"),
    "B32-G8-r4-fp32": (32, 2, 8, 2, [32 * 400 + 3, 32 * 9], 4, 512, "fp32", "fp32"),
    "B64-G2-r15-fp32q": (64, 2, 2, 2, [64 * 300 + 33, 17], 15, 1024, "bf16", "fp32"),
    "B32-G4-r8-fp32kv": (32, 2, 4, 2, [32 * 350 + 1, 0], 8, 256, "fp32", "bf16"),
    "B64-b256": (64, 2, 4, 2, [64 * 200 + 11, 64 * 3 + 5], 8, 256, "bf16", "bf16"),
    # four pages per stage-2 pass (four-head groups) at the other ranks and fp32 q
    "B32-G4-r2-fp32q": (32, 2, 4, 2, [32 * 300 + 7, 32 * 40], 2, 1024, "bf16", "fp32"),
    "B64-G4-r4": (64, 2, 4, 2, [64 * 150 + 3, 64 * 30], 4, 1024, "bf16", "bf16"),
    # r = 8 with sixteen-head groups: 16-token sub-pages whose LSEs are merged per
    # page; ragged lengths, a sequence without a complete page, fp32 queries
    "B64-G16-r8": (64, 3, 16, 2, [64 * 700 + 40, 63, 64 * 77], 8, 2048, "bf16", "bf16"),
    "B32-G16-r8-fp32q": (32, 3, 16, 1, [32 * 900 + 31, 32 * 5, 32 * 260 + 1], 8, 1024, "bf16",
                         "fp32"),
    "B64-G4-r8-fp32q": (64, 3, 4, 2, [64 * 400 + 5, 64 * 61, 40], 8, 1024, "bf16", "fp32"),
    "B64-G16-r8-fp32q": (64, 2, 16, 2, [64 * 500 + 17, 64 * 90], 8, 2048, "bf16", "fp32"),
    "B32-G4-r8-fp32q": (32, 3, 4, 2, [32 * 640 + 9, 32 * 33, 31], 8, 1024, "bf16", "fp32"),
}


@pytest.mark.parametrize("name", sorted(STEP))
def test_scan_select_attend_on_oracle_bytes(name):
    Bp, S, G, Hkv, lens, rank, budget, kv, q = STEP[name]
    d = _dev(name, Bp, S, G, Hkv, lens, rank, budget, kv, q)
    cfg = d.cfg
    assert cfg.k == -(-budget // Bp)
    store, recs = d.oracle_summaries()
    all_lse = torch.full((cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq), float("nan"),
                         device=d.device)
    B.score_pages(cfg, d.q, store, d.pt, d.sl, d.ws, all_lse)
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    ids2, sel2 = B.select(cfg, d.q, store, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    assert torch.equal(ids, ids2)
    Gq = cfg.group
    worst, results, worst_o = 0.0, [], 0.0
    oracle_ids = torch.full((cfg.num_seqs, cfg.num_kv_heads, cfg.k), -1, dtype=torch.int32)
    refs = {}
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg = d.unit(s, h)
            ref = O.decode_step(qg, k, v, recs[(s, h)], rank, budget, "int4", Bp)
            refs[(s, h)] = (k, v, qg, ref)
            L = k.shape[0]
            n_c, n = L // Bp, -(-L // Bp)
            hs = slice(h * Gq, (h + 1) * Gq)
            if n_c:
                got = all_lse[s, hs, :n_c].double().cpu().numpy()
                worst = max(worst, float(np.max(np.abs(got - ref["s_hat"]))))
            g_ids = ids_of(ids[s, h].tolist())
            results.append(check_table(g_ids, ref, n, cfg.k))
            worst_o = max(worst_o, check_attention_on_table(
                qg, k, v, g_ids, out[s, hs].double().cpu().numpy(),
                lse[s, hs].double().cpu().numpy(), Bp))
            check_sel_lse(sel[s, hs].double().cpu().numpy(), g_ids, ref["s_hat"], n_c)
            oracle_ids[s, h, :len(ref["ids"])] = torch.tensor(ref["ids"], dtype=torch.int32)
    ov = near_tie_overlap(results)
    # attention on the oracle's own tables, and the dense baseline
    o2, l2 = B.sparse_attend(cfg, d.q, d.k, d.v, d.pt, d.sl, oracle_ids.to(d.device), d.ws)
    od, ld = B.dense_attend(cfg, d.q, d.k, d.v, d.pt, d.sl, d.ws)
    torch.cuda.synchronize()
    worst_a = 0.0
    for (s, h), (k, v, qg, ref) in refs.items():
        hs = slice(h * Gq, (h + 1) * Gq)
        oo = o2[s, hs].double().cpu().numpy()
        worst_a = max(worst_a, max(rel_l2(oo[g], ref["out"][g]) for g in range(Gq)))
        np.testing.assert_allclose(l2[s, hs].double().cpu().numpy(), ref["lse"], atol=LSE_TOL)
        o_d, l_d = O.dense_step(qg, k, v)
        odd = od[s, hs].double().cpu().numpy()
        worst_a = max(worst_a, max(rel_l2(odd[g], o_d[g]) for g in range(Gq)))
        np.testing.assert_allclose(ld[s, hs].double().cpu().numpy(), l_d, atol=LSE_TOL)
    print(f"[page {Bp}] {name}: max |hat s err| {worst:.2e}; near-tie overlap {ov:.4f}; step "
          f"rel-L2 {worst_o:.2e}; attend / dense on oracle tables {worst_a:.2e}")
    assert worst <= LSE_TOL
    assert worst_a <= 2e-3


@pytest.mark.parametrize("Bp", [32, 64])
def test_gpu_built_summaries_and_build_list_step(Bp):
    """The fused step on summaries the GPU built (tables by the overlap rule, every
    output against the oracle's attention over the GPU's table), and a step whose
    build list names the pages that just filled and which writes the new token
    itself: bit for bit the KV write, the build and a plain step called apart."""
    lens = [Bp * 400 - 1, Bp * 150 + 5, Bp * 77 - 1]
    d = _dev("built", Bp, 3, 4, 2, lens, 8, 2048, spare=1)
    cfg, dev = d.cfg, d.device
    store = B.alloc_summaries(cfg, dev)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    inter = tot = 0
    Gq = cfg.group
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg = d.unit(s, h)
            ref = O.decode_step(qg, k, v, O.unit_summaries(k, 8, "int4", Bp), 8, cfg.budget_tokens,
                                "int4", Bp)
            got = ids_of(ids[s, h].tolist())
            inter += len(set(got) & set(ref["ids"]))
            tot += len(ref["ids"])
            hs = slice(h * Gq, (h + 1) * Gq)
            check_attention_on_table(qg, k, v, got, out[s, hs].double().cpu().numpy(),
                                     lse[s, hs].double().cpu().numpy(), Bp)
    print(f"[page {Bp}] gpu-built summaries: table overlap {inter / tot:.4f}", flush=True)
    assert inter >= OVERLAP_TOL * tot
    # the step that appends a token, completing the last page of sequences 0 and 2
    gen = torch.Generator().manual_seed(9)
    kt = d.k.dtype
    k_new = torch.randn(3, 2, 128, generator=gen).to(kt).to(dev)
    v_new = torch.randn(3, 2, 128, generator=gen).to(kt).to(dev)
    new_lens = [L + 1 for L in lens]
    sl = torch.tensor(new_lens, dtype=torch.int32, device=dev)
    listed = [(s, L // Bp - 1) for s, L in enumerate(new_lens)]
    bl = torch.tensor(listed, dtype=torch.int32, device=dev)
    rk, rv, rstore = d.k.clone(), d.v.clone(), store.clone()
    B.append_kv(cfg, k_new, v_new, rk, rv, d.pt, sl)
    B.build_summaries(cfg, rk, d.pt, sl, rstore, build_list=bl)
    r_out = B.decode_step(cfg, d.q, rk, rv, d.pt, sl, rstore, d.ws)
    torch.cuda.synchronize()
    ws2 = B.alloc_workspace(cfg, dev)
    got = B.decode_step(cfg, d.q, d.k, d.v, d.pt, sl, store, ws2, build_list=bl, k_new=k_new,
                        v_new=v_new)
    torch.cuda.synchronize()
    assert torch.equal(d.k, rk) and torch.equal(d.v, rv) and torch.equal(store, rstore)
    assert torch.equal(got[0], r_out[0]) and torch.equal(got[2], r_out[2])
    assert torch.equal(got[3], r_out[3])
    assert torch.equal(torch.nan_to_num(got[1], nan=-7.0), torch.nan_to_num(r_out[1], nan=-7.0))
    # a fresh build of every complete page equals the store the step left
    fresh = B.alloc_summaries(cfg, dev)
    B.build_summaries(cfg, d.k, d.pt, sl, fresh)
    torch.cuda.synchronize()
    for s, L in enumerate(new_lens):
        blocks = d.w.page_table[s, :L // Bp].long().to(dev)
        assert torch.equal(store[blocks], fresh[blocks]), s
    print(f"[page {Bp}] build-list step with the KV write equals the separate calls")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("Bp", [32, 64])
def test_full_size_128k_large_pages(Bp):
    """The 8 x 128K Llama-shaped workload at B = 32 and 64 (r = 8, b = 2048): the GPU builds
    every summary; on two sampled units with the oracle's bytes installed, every
    page score, the table, the page LSEs and the output."""
    d = _dev(f"128k-B{Bp}", Bp, 8, 4, 8, [131072] * 8, 8, 2048, on_gpu=True)
    cfg = d.cfg
    store = B.alloc_summaries(cfg, d.device)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    torch.cuda.synchronize()
    units = [(0, 0), (5, 6)]
    store_o, recs = d.oracle_summaries(units=set(units))
    for (s, h), rec in recs.items():
        blocks = d.w.page_table[s, :rec.shape[0]].long()
        store[blocks, h] = store_o[blocks, h]
    all_lse = torch.full((cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq), float("nan"),
                         device=d.device)
    B.score_pages(cfg, d.q, store, d.pt, d.sl, d.ws, all_lse)
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    Gq = cfg.group
    for (s, h) in units:
        k, v, qg = gather_unit(d.w, s, h)
        ref = O.decode_step(qg, k, v, recs[(s, h)], 8, 2048, "int4", Bp)
        n = -(-k.shape[0] // Bp)
        hs = slice(h * Gq, (h + 1) * Gq)
        err = float(np.max(np.abs(all_lse[s, hs, :n].double().cpu().numpy() - ref["s_hat"])))
        got = ids_of(ids[s, h].tolist())
        check_table(got, ref, n, cfg.k)
        w = check_attention_on_table(qg, k, v, got, out[s, hs].double().cpu().numpy(),
                                     lse[s, hs].double().cpu().numpy(), Bp)
        check_sel_lse(sel[s, hs].double().cpu().numpy(), got, ref["s_hat"], n)
        print(f"[page {Bp}] 128K unit ({s}, {h}): hat s err {err:.2e}, same table "
              f"{got == ref['ids']}, rel-L2 {w:.2e}", flush=True)
        assert err <= LSE_TOL
