"""Shared plumbing for the GPU parity tests (inputs on the device, oracle on the host)."""
import math

import numpy as np
import torch

from oracle import locks_oracle as O
from paper_2607_24555_amd import locks as B
from workloads import gather_unit

PAGE = 16
LSE_TOL = 1e-3        # page-LSE absolute error bound
OUT_TOL = 2e-3        # attention output relative L2 bound (bf16 KV)
GAP_TOL = 1e-3        # selection: identical sets when the ranking gap exceeds this
OVERLAP_TOL = 0.99    # ... otherwise aggregate overlap at least this


class Dev:
    """A workload's tensors on the GPU plus its liblocks configuration."""

    def __init__(self, w, device="cuda"):
        self.w = w
        self.cfg = B.config_for(w.spec, w.num_blocks, w.max_pages)
        self.q = w.q.to(device)
        self.k = w.k_cache.to(device)
        self.v = w.v_cache.to(device)
        self.pt = w.page_table.to(device)
        self.sl = w.seq_lens.to(device)
        self.ws = B.alloc_workspace(self.cfg, device)
        self.device = device

    def oracle_summaries(self, units=None):
        """Summary store filled with oracle-encoded records (and the per-unit records)."""
        store = B.alloc_summaries(self.cfg, self.device)
        recs = {}
        S, H = self.cfg.num_seqs, self.cfg.num_kv_heads
        for s in range(S):
            for h in range(H):
                if units is not None and (s, h) not in units:
                    continue
                k, _, _ = gather_unit(self.w, s, h)
                rec = O.unit_summaries(k, self.cfg.rank, B.BASIS_NAMES[self.cfg.basis],
                                       self.cfg.page_size)
                recs[(s, h)] = rec
                n_c = rec.shape[0]
                if n_c:
                    blocks = self.w.page_table[s, :n_c].long()
                    store[blocks.to(self.device), h] = torch.from_numpy(rec).to(self.device)
        return store, recs

    def unit(self, s, h):
        return gather_unit(self.w, s, h)


def check_table(got, ref, n, k):
    """One (sequence, KV head) table against the oracle's selection (Sec. 4 "Score";
    Cor. "Group-shared selection").

    The table must be well formed: ascending, no repeats, min(k, n) entries, the
    sink (page 0) and the most recent page (n - 1) included.  Where the oracle's
    ranking gap exceeds GAP_TOL it must equal the oracle's table.  Otherwise it may
    differ only by candidate pages whose share-average key lies within
    4 * LSE_TOL (natural log) of the oracle's cut: each page score and each log Z_g
    may move by LSE_TOL, so log mbar of a page by 2 LSE_TOL and the difference of
    two pages' keys by 4 LSE_TOL; a swapped pair straddles the cut, so each of its
    pages lies within that difference of it.
    Returns (near_tie, common, size): whether the unit is a near tie, and the
    number of the oracle's pages the table holds out of the oracle's count."""
    assert got == sorted(set(got)), got
    assert len(got) == min(k, n), (len(got), k, n)
    if n == 0:
        return False, 0, 0
    assert got[0] == 0 and got[-1] == n - 1, got
    want = ref["ids"]
    if ref["gap"] > GAP_TOL:
        assert got == want, (got, want, ref["gap"])
        return False, len(want), len(want)
    lm = ref["log_mbar"]
    cand = sorted(range(1, n - 1), key=lambda j: (-lm[j], j))
    cut = lm[cand[k - 3]]
    for j in set(got) ^ set(want):
        assert 0 < j < n - 1 and abs(lm[j] - cut) <= 4 * LSE_TOL, (j, lm[j], cut, ref["gap"])
    return True, len(set(got) & set(want)), len(want)


def near_tie_overlap(results):
    """results: check_table returns.  Over the near-tie units only, the fraction of
    the oracle's pages the GPU tables hold must be at least OVERLAP_TOL, or at most
    one page may be missed in all (below 100 pages one legitimate swap already
    costs more than 1%).  Returns that fraction (1.0 with no near-tie unit)."""
    common = sum(c for nt, c, t in results if nt)
    total = sum(t for nt, c, t in results if nt)
    assert common >= OVERLAP_TOL * total or total - common <= 1, (common, total)
    return common / total if total else 1.0


def check_attention_on_table(qg, k, v, got, o, l, page_size=PAGE):
    """GPU output o [G][d] and LSE l [G] of one (sequence, KV head) against the
    oracle's attention over the GPU's own table of pages of page_size tokens
    (Sec. 2): rel-L2 <= OUT_TOL per head, LSE within LSE_TOL; an empty table gives
    0 and -inf.  Returns the worst rel-L2."""
    if not got:
        assert np.all(o == 0) and np.all(np.isneginf(l)), (o, l)
        return 0.0
    o_ref, l_ref = O.attend(qg, k, v, got, page_size)
    worst = max(rel_l2(o[g], o_ref[g]) for g in range(qg.shape[0]))
    assert worst <= OUT_TOL, worst
    np.testing.assert_allclose(l, l_ref, atol=LSE_TOL)
    return worst


def check_sel_lse(gsel, got, s_hat_ref, n_c):
    """Estimated page LSEs returned with a table: gsel [G][k] holds the oracle's
    page score (within LSE_TOL) of every table entry with a summary, NaN for the
    partial recent page and for padding."""
    for t in range(gsel.shape[1]):
        j = got[t] if t < len(got) else -1
        if 0 <= j < n_c:
            np.testing.assert_allclose(gsel[:, t], s_hat_ref[:, j], atol=LSE_TOL, rtol=0)
        else:
            assert np.isnan(gsel[:, t]).all(), (t, j, gsel[:, t])


def rel_l2(a, b):
    n = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (n if n > 0 else 1.0)


def ids_of(row):
    return [int(x) for x in row if int(x) >= 0]


def parse_codes(rec, r, P=16):
    """Integer codes of int4-basis records of P-token pages laid out as
    include/locks.h documents (test-local parser, independent of the oracle's
    decoder)."""
    rec = rec.astype(np.int64)
    v = np.empty((rec.shape[0], 128, r), np.int64)
    for l in range(r):
        b = rec[:, 64 * l:64 * l + 64]
        v[:, 0::2, l] = (b & 15) - 8
        v[:, 1::2, l] = (b >> 4) - 8
    c = rec[:, 64 * r:(64 + P) * r] - 128
    m = rec[:, (64 + P) * r:(64 + P) * r + 128] - 128
    return {"vcodes": v, "ccodes": c, "mcodes": m}
