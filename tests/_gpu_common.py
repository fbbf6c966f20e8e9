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
                rec = O.unit_summaries(k, self.cfg.rank, B.BASIS_NAMES[self.cfg.basis])
                recs[(s, h)] = rec
                n_c = rec.shape[0]
                if n_c:
                    blocks = self.w.page_table[s, :n_c].long()
                    store[blocks.to(self.device), h] = torch.from_numpy(rec).to(self.device)
        return store, recs

    def unit(self, s, h):
        return gather_unit(self.w, s, h)


def selection_agreement(pairs):
    """pairs: list of (gpu_ids, oracle_ids, gap).  Sets must be identical where the
    oracle's gap exceeds GAP_TOL; elsewhere the aggregate overlap is returned."""
    inter = tot = 0
    for got, ref, gap in pairs:
        if gap > GAP_TOL:
            assert sorted(got) == sorted(ref), (got, ref, gap)
        inter += len(set(got) & set(ref))
        tot += len(ref)
    return inter / max(tot, 1)


def rel_l2(a, b):
    n = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (n if n > 0 else 1.0)


def ids_of(row):
    return [int(x) for x in row if int(x) >= 0]


def parse_codes(rec, r):
    """Integer codes of int4-basis records laid out as include/locks.h documents
    (test-local parser, independent of the oracle's decoder)."""
    rec = rec.astype(np.int64)
    v = np.empty((rec.shape[0], 128, r), np.int64)
    for l in range(r):
        b = rec[:, 64 * l:64 * l + 64]
        v[:, 0::2, l] = (b & 15) - 8
        v[:, 1::2, l] = (b >> 4) - 8
    c = rec[:, 64 * r:80 * r] - 128
    m = rec[:, 80 * r:80 * r + 128] - 128
    return {"vcodes": v, "ccodes": c, "mcodes": m}
