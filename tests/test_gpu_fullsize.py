"""Parity at the benchmark's full sizes, in the launch configuration bench.py times:
the eager fused locks_decode_step over every page of every sequence of the
GLM-4-9B 1M-token (16-, 32- and 64-token pages), Llama-3.1-8B 8 x 128K (r = 8
and r = 2) and Qwen3-4B reasoning workloads.  The GPU builds every summary; for a few sampled (sequence, KV head)
units the oracle builds that unit's summaries itself and computes the whole step
of that unit (every page scored, the shared table, attention).  On those units:
GPU-built codes against the oracle's (within +-1, >= 99.9% identical on gapped
pages); then, with the oracle's bytes installed for the unit, page scores
(<= 1e-3 absolute), the table (identical where the ranking gap exceeds 1e-3, else
overlap), the selected page LSEs, the output (rel-L2 <= 2e-3) and its LSE."""
import numpy as np
import pytest
import torch

from oracle import locks_oracle as O
from paper_2607_24555_amd import locks as B
from tests._gpu_common import (LSE_TOL, check_attention_on_table, check_sel_lse, check_table,
                               ids_of, parse_codes, rel_l2)
from workloads import gather_unit, make_workload

pytestmark = pytest.mark.gpu

FULL = {
    # name: (workload id, overrides, sampled (seq, KV head) units)
    "glm4-9b-1m": (3, {}, [(0, 1)]),
    "glm4-9b-1m-B32": (3, {"page_size": 32}, [(0, 0)]),
    "glm4-9b-1m-B64": (3, {"page_size": 64}, [(0, 1)]),
    "llama-8x128k-r8": (2, {}, [(0, 0), (3, 5), (7, 7)]),
    "llama-8x128k-r2": (2, {"rank": 2}, [(1, 2), (6, 4)]),
    "qwen3-reasoning": (4, {}, [(0, 0), (17, 3), (42, 6), (63, 7)]),
}


def _well_posed(f, r, rel=1e-3):
    """Pages whose stored codes are fixed by the definition up to rounding: every
    one of the r kept modes is separated from its neighbours by a relative
    eigen-gap above `rel` (else the basis may rotate inside a near-degenerate pair:
    Cor. "The per-page basis is residual-optimal" fixes the subspace, not a basis), and each basis column's
    largest-magnitude entry leads the runner-up by more than `rel` (else the sign
    convention may pick the other sign)."""
    lam = f["sigma2"]
    ok = np.ones(lam.shape[0], bool)
    for l in range(r):
        ok &= (lam[:, l] - lam[:, l + 1]) > rel * lam[:, l]
    a = np.sort(np.abs(f["V"]), axis=1)                  # [P][d][r] ascending along d
    ok &= np.all(a[:, -1, :] - a[:, -2, :] > rel * a[:, -1, :], axis=1)
    return ok


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", sorted(FULL))
def test_full_size_step_on_sampled_units(name):
    wid, ov, units = FULL[name]
    print(f"[full {name}] generating", flush=True)
    w = make_workload(wid, seed=0, device="cuda", **ov)
    cfg = B.config_for(w.spec, w.num_blocks, w.max_pages)
    r, G, P = cfg.rank, cfg.group, cfg.page_size
    store = B.alloc_summaries(cfg)
    B.build_summaries(cfg, w.k_cache, w.page_table, w.seq_lens, store)
    torch.cuda.synchronize()
    ref = {}
    for s, h in units:
        k, v, qg = gather_unit(w, s, h)
        n_c = k.shape[0] // P
        print(f"[full {name}] oracle build of unit ({s}, {h}): {n_c} pages", flush=True)
        f = O.build_factors(k[:n_c * P].reshape(n_c, P, 128), r)
        rec = O.encode(f["mu"], f["V"], f["C"])
        posed = _well_posed(f, r)
        blocks = w.page_table[s, :n_c].long()
        got, want = parse_codes(store[blocks, h].cpu().numpy(), r, P), parse_codes(rec, r, P)
        far = np.zeros(n_c, bool)
        for key in want:
            far |= (np.abs(got[key] - want[key]) > 1).reshape(n_c, -1).any(axis=1)
        for j in np.flatnonzero(far)[:5]:
            lam = f["sigma2"][j]
            print(f"[full {name}] page {j}: codes differ by > 1; eigen-gaps "
                  f"{np.round((lam[:r] - lam[1:r + 1]) / lam[:r], 5).tolist()}, "
                  f"well posed {bool(posed[j])}", flush=True)
        assert not np.any(far & posed), np.flatnonzero(far & posed)[:10]
        same = total = 0
        for key in want:
            a, b = got[key][posed], want[key][posed]
            same += int(np.sum(a == b))
            total += a.size
        print(f"[full {name}] unit ({s}, {h}): identical codes {same / total:.5f} on "
              f"{int(posed.sum())}/{n_c} well-posed pages; {int(far.sum())} pages with a "
              f"code off by more than 1", flush=True)
        assert same / total >= 0.999
        store[blocks, h] = torch.from_numpy(rec).to(store.device)
        ref[(s, h)] = (qg, O.decode_step(qg, k, v, rec, r, cfg.budget_tokens, "int4", P), n_c)

    ws = B.alloc_workspace(cfg)
    ids, sel, out, lse = B.decode_step(cfg, w.q, w.k_cache, w.v_cache, w.page_table, w.seq_lens,
                                       store, ws)
    all_lse = torch.full((cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq), float("nan"),
                         device=store.device)
    B.score_pages(cfg, w.q, store, w.page_table, w.seq_lens, ws, all_lse)
    torch.cuda.synchronize()
    for (s, h), (qg, rf, n_c) in ref.items():
        hs = slice(h * G, (h + 1) * G)
        s_hat = all_lse[s, hs, :n_c].double().cpu().numpy()
        err = float(np.max(np.abs(s_hat - rf["s_hat"])))
        got = ids_of(ids[s, h].tolist())
        o = out[s, hs].double().cpu().numpy()
        l = lse[s, hs].double().cpu().numpy()
        worst = max(rel_l2(o[g], rf["out"][g]) for g in range(G))
        print(f"[full {name}] unit ({s}, {h}): max |hat s err| {err:.2e}, gap {rf['gap']:.2e}, "
              f"same table {got == rf['ids']}, overlap "
              f"{len(set(got) & set(rf['ids'])) / len(rf['ids']):.4f}, rel-L2 {worst:.2e}",
              flush=True)
        assert err <= LSE_TOL
        check_table(got, rf, -(-int(w.spec.seq_lens[s]) // P), cfg.k)
        k, v, _ = gather_unit(w, s, h)
        check_attention_on_table(qg, k, v, got, o, l, P)
        check_sel_lse(sel[s, hs].double().cpu().numpy(), got, rf["s_hat"], n_c)
