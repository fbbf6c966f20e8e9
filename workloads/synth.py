"""Seeded synthetic decode-step inputs shaped like the paper's workloads.

This module only draws random tensors and lays them out in a paged KV cache.
It contains none of the method's arithmetic (no centering, eigenbasis,
quantisation, scoring or attention), so both the HIP path and the CPU oracle
can consume its output without sharing any of the method's code.

Key recipe (one recipe for every workload; a reading of the paper's setting of
per-page low-rank key structure, Sec. 3 / App. B, not a copy of its traces):

* every (sequence, KV head) draws a global key mean: N(0, 1) per channel, except
  four outlier channels (chosen once per seed) set to +/-8 with a seeded sign;
* every 16-token page draws its own orthonormal 8-dimensional subspace of R^128
  (Gaussian matrix, modified Gram-Schmidt) and per-token coefficients
  c_l ~ N(0, (4 * 0.7^l)^2), l = 0..7;
* key = mean + U_page c + N(0, 0.05^2) noise per element;
* queries are N(0, 1) with the four outlier channels set to the mean's value,
  one query per query head of the GQA group;
* carrier tokens: min(round(0.01 L), 40) tokens spread over 5 random pages that
  are neither the first nor the last page; each gets 6 * q_hat added to its key,
  q_hat being the normalised mean of the group's queries;
* values are N(0, 1);
* bf16 workloads round keys, values and queries to bf16 (round-to-nearest-even).

Physical layout: k_cache / v_cache are [num_blocks][H_kv][B][128] for pages of
B = page_size tokens (16 unless stated); logical page j of sequence s lives in
block page_table[s][j]; blocks are a seeded random permutation, so consecutive
logical pages are scattered in memory.  The tokens do not depend on the page size
(the per-page subspace above is drawn per 16 tokens), so workloads of different
page sizes hold the same keys and values.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import torch

PAGE = 16
HEAD_DIM = 128
SUB_RANK = 8
COEF_SCALE0 = 4.0
COEF_DECAY = 0.7
NOISE_STD = 0.05
OUTLIER_MAG = 8.0
N_OUTLIERS = 4
CARRIER_GAIN = 6.0
CARRIER_PAGES = 5
CARRIER_CAP = 40
CHUNK_PAGES = 4096  # generation chunk (part of the recipe: fixes the RNG stream)


@dataclass
class WorkloadSpec:
    name: str
    num_seqs: int
    num_q_heads: int
    num_kv_heads: int
    seq_lens: List[int]
    rank: int
    budget_tokens: int
    kv_dtype: str  # "bf16" | "fp32"
    q_dtype: str
    spare_pages_per_seq: int = 0  # free blocks reserved for appended tokens
    page_size: int = PAGE         # tokens per KV page (16, 32 or 64); the key recipe
                                  # below is the same for every page size


def config_spec(cfg_id: int, *, rank: Optional[int] = None, seed: int = 0,
                num_seqs: Optional[int] = None, seq_len: Optional[int] = None,
                num_kv_heads: Optional[int] = None, num_q_heads: Optional[int] = None,
                budget_tokens: Optional[int] = None,
                spare_pages: Optional[int] = None,
                page_size: Optional[int] = None) -> WorkloadSpec:
    """The five decode-step workloads; keyword overrides shrink them for tests."""
    if cfg_id == 0:
        s = WorkloadSpec("tiny-1h-4k", 1, 1, 1, [4096], 8, 256, "fp32", "fp32")
    elif cfg_id == 1:
        s = WorkloadSpec("llama8b-32k", 1, 32, 8, [32768], 8, 2048, "bf16", "bf16")
    elif cfg_id == 2:
        s = WorkloadSpec("llama8b-8x128k", 8, 32, 8, [131072] * 8, 8, 2048, "bf16", "bf16")
    elif cfg_id == 3:
        s = WorkloadSpec("glm4-9b-1m", 1, 32, 2, [1048576], 8, 2048, "bf16", "bf16")
    elif cfg_id == 4:
        g = torch.Generator().manual_seed(1_000_003 * (seed + 1) + 4)
        n = 64 if num_seqs is None else num_seqs
        lo, hi = 8192, 65536
        lens = torch.randint(lo, hi + 1, (n,), generator=g).tolist()
        s = WorkloadSpec("qwen3-4b-reasoning", n, 32, 8, lens, 2, 256, "bf16", "bf16",
                         spare_pages_per_seq=8)
    else:
        raise ValueError(f"unknown workload {cfg_id}")
    if num_seqs is not None and cfg_id != 4:
        s.num_seqs = num_seqs
        s.seq_lens = (s.seq_lens * num_seqs)[:num_seqs]
    if seq_len is not None:
        s.seq_lens = [seq_len] * s.num_seqs
    if num_kv_heads is not None:
        s.num_kv_heads = num_kv_heads
    if num_q_heads is not None:
        s.num_q_heads = num_q_heads
    if rank is not None:
        s.rank = rank
    if budget_tokens is not None:
        s.budget_tokens = budget_tokens
    if spare_pages is not None:
        s.spare_pages_per_seq = spare_pages
    if page_size is not None:
        s.page_size = page_size
    return s


@dataclass
class Workload:
    spec: WorkloadSpec
    q: torch.Tensor            # [S][H_q][128]
    k_cache: torch.Tensor      # [num_blocks][H_kv][page_size][128]
    v_cache: torch.Tensor
    page_table: torch.Tensor   # int32 [S][max_pages]
    seq_lens: torch.Tensor     # int32 [S]
    carrier_pages: Dict[tuple, List[int]] = field(default_factory=dict)

    @property
    def num_blocks(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.page_table.shape[1])


def _torch_dtype(name: str) -> torch.dtype:
    return {"bf16": torch.bfloat16, "fp32": torch.float32}[name]


def _gen(seed: int, *tags: int, device) -> torch.Generator:
    x = seed & 0xFFFFFFFF
    for t in tags:
        x = (x * 6364136223846793005 + 1442695040888963407 + (t & 0xFFFFFFFF)) & ((1 << 63) - 1)
    g = torch.Generator(device=torch.device(device))
    g.manual_seed(x)
    return g


def _orthonormal(a: torch.Tensor) -> torch.Tensor:
    """Modified Gram-Schmidt over the last axis of [..., d, r] (fp64 for accuracy)."""
    a = a.double()
    cols = []
    for l in range(a.shape[-1]):
        v = a[..., l]
        for u in cols:
            v = v - (u * v).sum(-1, keepdim=True) * u
        v = v / v.norm(dim=-1, keepdim=True)
        cols.append(v)
    return torch.stack(cols, dim=-1)


def _round(x: torch.Tensor, dtype: torch.dtype) -> torch.Tensor:
    return x.to(dtype)


def unit_mean(seed: int, seq: int, kvh: int, outliers: torch.Tensor, device) -> torch.Tensor:
    """Global key mean of one (sequence, KV head): N(0,1) plus four +/-8 outlier channels."""
    g = _gen(seed, 11, seq, kvh, device=device)
    mean = torch.randn(HEAD_DIM, generator=g, device=device)
    signs = torch.where(torch.rand(N_OUTLIERS, generator=g, device=device) < 0.5, -1.0, 1.0)
    mean[outliers] = OUTLIER_MAG * signs
    return mean


def unit_tokens(spec: WorkloadSpec, seed: int, seq: int, kvh: int, mean: torch.Tensor,
                q_group: torch.Tensor, device) -> tuple:
    """Keys [L][128] (fp32, before dtype rounding), values [L][128], carrier pages."""
    L = spec.seq_lens[seq]
    n_pages = (L + PAGE - 1) // PAGE
    g = _gen(seed, 17, seq, kvh, device=device)
    scales = COEF_SCALE0 * (COEF_DECAY ** torch.arange(SUB_RANK, device=device, dtype=torch.float64))
    keys = torch.empty(n_pages * PAGE, HEAD_DIM, device=device, dtype=torch.float32)
    for p0 in range(0, n_pages, CHUNK_PAGES):
        p1 = min(n_pages, p0 + CHUNK_PAGES)
        m = p1 - p0
        a = torch.randn(m, HEAD_DIM, SUB_RANK, generator=g, device=device)
        U = _orthonormal(a)
        c = torch.randn(m, PAGE, SUB_RANK, generator=g, device=device).double() * scales
        noise = torch.randn(m, PAGE, HEAD_DIM, generator=g, device=device).double() * NOISE_STD
        k = mean.double() + torch.einsum("pdr,pir->pid", U, c) + noise
        keys[p0 * PAGE:p1 * PAGE] = k.reshape(m * PAGE, HEAD_DIM).float()
    # carrier tokens (a handful of distinctive keys aligned with the group query)
    carriers: List[int] = []
    n_car = min(int(round(0.01 * L)), CARRIER_CAP)
    if n_pages >= CARRIER_PAGES + 2 and n_car > 0:
        qm = q_group.double().mean(0)
        qhat = (qm / qm.norm()).float()
        cand = torch.randperm(n_pages - 2, generator=g, device=device)[:CARRIER_PAGES] + 1
        carriers = sorted(int(x) for x in cand.tolist())
        per = [n_car // CARRIER_PAGES + (1 if i < n_car % CARRIER_PAGES else 0)
               for i in range(CARRIER_PAGES)]
        for pg, cnt in zip(carriers, per):
            slots = torch.randperm(PAGE, generator=g, device=device)[:cnt]
            idx = pg * PAGE + slots
            keys[idx] += CARRIER_GAIN * qhat
    vals = torch.randn(n_pages * PAGE, HEAD_DIM, generator=g, device=device)
    return keys[:L], vals[:L], carriers


def make_workload(cfg_id: int, seed: int = 0, device="cpu", **overrides) -> Workload:
    spec = config_spec(cfg_id, seed=seed, **overrides)
    return build_workload(spec, seed, device)


def build_workload(spec: WorkloadSpec, seed: int = 0, device="cpu") -> Workload:
    dev = torch.device(device)
    S, Hq, Hkv = spec.num_seqs, spec.num_q_heads, spec.num_kv_heads
    if Hq % Hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    G = Hq // Hkv
    P = spec.page_size
    kvt, qt = _torch_dtype(spec.kv_dtype), _torch_dtype(spec.q_dtype)
    g0 = _gen(seed, 3, device="cpu")
    outliers = torch.randperm(HEAD_DIM, generator=g0)[:N_OUTLIERS].to(dev)
    n_pages = [(L + P - 1) // P for L in spec.seq_lens]
    max_pages = max(1, max(n + spec.spare_pages_per_seq for n in n_pages))
    total = sum(n + spec.spare_pages_per_seq for n in n_pages)
    total = max(total, 1)
    perm = torch.randperm(total, generator=g0).to(torch.int32)
    page_table = torch.full((S, max_pages), -1, dtype=torch.int32)
    off = 0
    for s in range(S):
        m = n_pages[s] + spec.spare_pages_per_seq
        page_table[s, :m] = perm[off:off + m]
        off += m
    k_cache = torch.zeros(total, Hkv, P, HEAD_DIM, dtype=kvt, device=dev)
    v_cache = torch.zeros(total, Hkv, P, HEAD_DIM, dtype=kvt, device=dev)
    q = torch.empty(S, Hq, HEAD_DIM, dtype=torch.float32, device=dev)
    carriers: Dict[tuple, List[int]] = {}
    pt_dev = page_table.to(dev).long()
    for s in range(S):
        L = spec.seq_lens[s]
        for h in range(Hkv):
            gq = _gen(seed, 29, s, h, device=device)
            qg = torch.randn(G, HEAD_DIM, generator=gq, device=dev)
            mean = unit_mean(seed, s, h, outliers, dev)
            qg[:, outliers] = mean[outliers]   # queries share the head's outlier channels
            car: List[int] = []
            if L > 0:
                keys, vals, car = unit_tokens(spec, seed, s, h, mean, qg, dev)
                n = (L + P - 1) // P
                kp = torch.zeros(n * P, HEAD_DIM, device=dev)
                vp = torch.zeros(n * P, HEAD_DIM, device=dev)
                kp[:L] = keys
                vp[:L] = vals
                blocks = pt_dev[s, :n]
                k_cache[blocks, h] = _round(kp.view(n, P, HEAD_DIM), kvt)
                v_cache[blocks, h] = _round(vp.view(n, P, HEAD_DIM), kvt)
            q[s, h * G:(h + 1) * G] = qg
            carriers[(s, h)] = car
    return Workload(spec, _round(q, qt), k_cache, v_cache, page_table.to(dev),
                    torch.tensor(spec.seq_lens, dtype=torch.int32, device=dev), carriers)


def gather_unit(w: Workload, seq: int, kvh: int):
    """Host fp64 copies of one (sequence, KV head): keys [L][d], values [L][d], q [G][d]."""
    L = int(w.spec.seq_lens[seq])
    P = w.spec.page_size
    n = (L + P - 1) // P
    G = w.spec.num_q_heads // w.spec.num_kv_heads
    blocks = w.page_table[seq, :n].long().cpu()
    k = w.k_cache.index_select(0, blocks.to(w.k_cache.device))[:, kvh].double().cpu()
    v = w.v_cache.index_select(0, blocks.to(w.v_cache.device))[:, kvh].double().cpu()
    q = w.q[seq, kvh * G:(kvh + 1) * G].double().cpu()
    return (k.reshape(n * P, HEAD_DIM)[:L].numpy(), v.reshape(n * P, HEAD_DIM)[:L].numpy(),
            q.numpy())
