"""GPU parity of the basis-precision variants: an int8 or bfloat16 basis in place
of the int4 one, coefficients and centroid still int8 (Sec. 5 "Ablations"; the
r8fp control of the retention remark).  Same tolerances as the int4 summaries:
page LSE 1e-3 absolute, attention output 2e-3 relative L2, tables by the gap
rule."""
import numpy as np
import pytest
import torch

from oracle import locks_oracle as O
from paper_2607_24555_amd import locks as B
from tests._gpu_common import (LSE_TOL, Dev, check_attention_on_table, check_sel_lse, check_table,
                               ids_of, near_tie_overlap)
from workloads import make_workload

pytestmark = pytest.mark.gpu

CASES = {
    "G4-r8": (1, dict(seq_len=8192 + 21)),
    "G4-r4-h2": (1, dict(seq_len=4096 + 7, rank=4, num_kv_heads=2, num_q_heads=8)),
    "G16-r8": (3, dict(seq_len=16384 + 9)),
    "G4-r2-mixed": (4, dict(num_seqs=3)),
}
BASES = {"int8": B.LOCKS_BASIS_INT8, "bf16": B.LOCKS_BASIS_BF16}


def _dev(case, basis):
    cid, ov = CASES[case]
    print(f"[basis {basis}] case {case}: cfg {cid} {ov}", flush=True)
    d = Dev(make_workload(cid, seed=7, **ov))
    d.cfg.basis = BASES[basis]
    d.ws = B.alloc_workspace(d.cfg, d.device)
    return d


def _oracle(d, recs, s, h, basis):
    k, v, qg = d.unit(s, h)
    return k, v, qg, O.decode_step(qg, k, v, recs[(s, h)], d.cfg.rank, d.cfg.budget_tokens, basis)


@pytest.mark.parametrize("basis", sorted(BASES))
@pytest.mark.parametrize("case", sorted(CASES))
def test_scan_and_step_on_oracle_bytes(case, basis):
    """Oracle-encoded records: every page score, then the fused step."""
    d = _dev(case, basis)
    cfg, G = d.cfg, d.cfg.group
    store, recs = d.oracle_summaries()
    all_lse = torch.full((cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq), float("nan"),
                         device=d.device)
    B.score_pages(cfg, d.q, store, d.pt, d.sl, d.ws, all_lse)
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws)
    torch.cuda.synchronize()
    worst, results, same, worst_o = 0.0, [], 0, 0.0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k, v, qg, ref = _oracle(d, recs, s, h, basis)
            n_c, n = k.shape[0] // 16, -(-k.shape[0] // 16)
            if n_c:
                got = all_lse[s, h * G:(h + 1) * G, :n_c].double().cpu().numpy()
                worst = max(worst, float(np.max(np.abs(got - ref["s_hat"]))))
            g_ids = ids_of(ids[s, h].tolist())
            results.append(check_table(g_ids, ref, n, cfg.k))
            same += g_ids == ref["ids"]
            o = out[s, h * G:(h + 1) * G].double().cpu().numpy()
            l = lse[s, h * G:(h + 1) * G].double().cpu().numpy()
            worst_o = max(worst_o, check_attention_on_table(qg, k, v, g_ids, o, l))
            check_sel_lse(sel[s, h * G:(h + 1) * G].double().cpu().numpy(), g_ids, ref["s_hat"], n_c)
    overlap = near_tie_overlap(results)
    print(f"[basis {basis}] {case}: max |hat s - oracle| {worst:.2e}, tables {same}/{len(results)}, "
          f"near-tie overlap {overlap:.4f}, worst out rel-L2 {worst_o:.2e}")
    assert worst <= LSE_TOL


@pytest.mark.parametrize("basis", sorted(BASES))
@pytest.mark.parametrize("case", ["G4-r8", "G4-r4-h2", "G4-r2-mixed"])
def test_build_matches_oracle_records(case, basis):
    """GPU-built records against oracle-built ones on pages whose top r directions
    are isolated: coefficient and centroid codes within +-1; basis codes (int8) or
    values (bf16) within one step plus the fp32 eigensolver's perturbation bound;
    99.9% of the codes identical and 99% of the bf16 values within the step alone."""
    d = _dev(case, basis)
    cfg = d.cfg
    r = cfg.rank
    store = B.alloc_summaries(cfg, d.device)
    B.build_summaries(cfg, d.k, d.pt, d.sl, store)
    torch.cuda.synchronize()
    _, recs = d.oracle_summaries()
    same = total = in_step = n_v = 0
    worst_v = 0.0
    for (s, h), rec in recs.items():
        n_c = rec.shape[0]
        if n_c == 0:
            continue
        k, _, _ = d.unit(s, h)
        lam = O.build_factors(k[:n_c * 16].reshape(n_c, 16, 128), r)["sigma2"]
        # every one of the top r directions isolated: an 8-bit code resolves a
        # rotation inside the subspace that a 4-bit one does not
        gapped = np.all((lam[:, :r] - lam[:, 1:r + 1]) > 1e-3 * lam[:, :r], axis=1)
        blocks = d.w.page_table[s, :n_c].long().to(d.device)
        got = O.decode(store[blocks, h].cpu().numpy(), r, basis)
        want = O.decode(rec, r, basis)
        for key in ("ccodes", "mcodes"):
            a, b = got[key][gapped], want[key][gapped]
            assert np.max(np.abs(a - b)) <= 1, (key, s, h)
            same += int(np.sum(a == b))
            total += a.size
        if not gapped.any():
            continue
        # the eigensolver's own error: it stops once the off-diagonal Frobenius
        # mass is 1e-10 of the diagonal's, a residual E with |E| <= 1e-5 |lambda|,
        # which moves v_l = D^T u_l / sigma_l by at most |E| max_j sigma_j /
        # (sigma_l |lambda_l - lambda_j|) to first order (Davis-Kahan); 4x margin
        # for the fp32 Gram's rounding
        lg = np.maximum(lam[gapped], 0.0)
        sg = np.sqrt(lg)
        diff = np.abs(lg[:, :r, None] - lg[:, None, :])
        diff[:, np.arange(r), np.arange(r)] = np.inf
        amp = np.max(sg[:, None, :] / (sg[:, :r, None] * diff), axis=2)
        eig = 4 * 1e-5 * np.linalg.norm(lg, axis=1)[:, None] * amp          # [P][r]
        if basis == "int8":
            # one code step of rounding plus that error in steps of the column scale
            a, b = got["vcodes"][gapped], want["vcodes"][gapped]
            lim = 1 + eig / want["vscale"][gapped]
            assert np.all(np.abs(a - b) <= lim[:, None, :]), (s, h)
            same += int(np.sum(a == b))
            total += a.size
        else:
            # one bfloat16 step of the stored value plus that error
            w = want["V"][gapped]
            dv = np.abs(got["V"][gapped] - w)
            step = 2.0 ** -7 * np.abs(w) + 1e-6
            worst_v = max(worst_v, float(np.max(dv / (step + eig[:, None, :]))))
            in_step += int(np.sum(dv <= step))
            n_v += dv.size
    frac = same / max(total, 1)
    frac_v = in_step / max(n_v, 1)
    print(f"[basis {basis}] {case}: identical codes {frac:.5f}; bf16 basis values within one "
          f"step {frac_v:.5f}, worst {worst_v:.3f} of the bound")
    assert frac >= 0.999
    assert worst_v <= 1.0
    assert basis != "bf16" or frac_v >= 0.99
