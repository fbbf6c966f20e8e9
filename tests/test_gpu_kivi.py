"""GPU parity of the KIVI fake quantisation of finalised pages (Sec. 5 "KV-cache
quantization under extreme sparsity"; App. C, protocol of the KIVI grid) through
the C ABI.  The quantised caches are compared with the oracle bit for bit (the codes
are decided in float32 on both sides); the fused step on a quantised cache, in the
POST and PRE orders, is held to the step tolerances against the oracle's step on the
oracle's quantised cache."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import locks_oracle as O
from paper_2607_24555_amd import locks as B
from tests._gpu_common import OVERLAP_TOL, Dev, check_attention_on_table, ids_of
from workloads import WorkloadSpec, build_workload, gather_unit, make_workload

pytestmark = pytest.mark.gpu
PAGE = 16


def _bits(x) -> np.ndarray:
    """bfloat16 bit patterns of a bf16 torch tensor or of exact bf16 values (numpy)."""
    if isinstance(x, torch.Tensor):
        return x.detach().cpu().contiguous().view(torch.int16).numpy().astype(np.uint16)
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _oracle_page(kc, vc, blk, h, bits, g):
    k = kc[blk, h].double().numpy()
    v = vc[blk, h].double().numpy()
    return O.kivi_page(k, v, bits, g)


def _expected_caches(w, pages, bits, g):
    """The workload's caches with the listed (seq, page) pairs' K and V replaced by the
    oracle's fake quantisation (complete pages only, every KV head)."""
    kc, vc = w.k_cache.clone(), w.v_cache.clone()
    H = w.spec.num_kv_heads
    for s, j in pages:
        if not (0 <= s < w.spec.num_seqs) or not (0 <= j < int(w.seq_lens[s]) // PAGE):
            continue
        blk = int(w.page_table[s, j])
        for h in range(H):
            kq, vq = _oracle_page(w.k_cache, w.v_cache, blk, h, bits, g)
            kc[blk, h] = torch.from_numpy(kq).to(torch.bfloat16)
            vc[blk, h] = torch.from_numpy(vq).to(torch.bfloat16)
    return kc, vc


def _complete_pages(w):
    return [(s, j) for s in range(w.spec.num_seqs) for j in range(int(w.seq_lens[s]) // PAGE)]


def _ragged(G=4, lens=(16 * 40 + 5, 16 * 64, 7, 0, 16 * 3), seed=5, spare=2):
    spec = WorkloadSpec("kivi", len(lens), 2 * G, 2, list(lens), 8, 128, "bf16", "bf16",
                        spare_pages_per_seq=spare)
    return build_workload(spec, seed)


def _with_flat_slices(w):
    """Page 1 of sequence 0 gets identical keys (every key channel constant) and one
    token whose values are constant over the first 64 channels: scale 0 keeps them."""
    w = dataclasses.replace(w, k_cache=w.k_cache.clone(), v_cache=w.v_cache.clone())
    blk = int(w.page_table[0, 1])
    w.k_cache[blk, 0] = w.k_cache[blk, 0, 3].clone()
    w.v_cache[blk, 1, 5, :64] = 0.75
    return w


@pytest.mark.parametrize("bits,g", [(4, 32), (2, 32), (2, 128), (4, 8), (3, 16), (1, 64), (8, 32)])
def test_quantize_every_complete_page_bit_exact(bits, g):
    w = _with_flat_slices(_ragged())
    print(f"[kivi all] bits {bits} g {g} lens {w.spec.seq_lens}", flush=True)
    d = Dev(w)
    kv = B.Kivi(bits, g, B.LOCKS_KIVI_POST)
    B.kivi_quantize(d.cfg, kv, d.k, d.v, d.pt, d.sl)
    torch.cuda.synchronize()
    kc, vc = _expected_caches(w, _complete_pages(w), bits, g)
    np.testing.assert_array_equal(_bits(d.k), _bits(kc))
    np.testing.assert_array_equal(_bits(d.v), _bits(vc))
    # the flat slices kept their values; partial pages and spare blocks are untouched
    blk = int(w.page_table[0, 1])
    assert torch.equal(d.k[blk, 0].cpu(), w.k_cache[blk, 0])
    if g <= 64:
        assert torch.equal(d.v[blk, 1, 5, :64].cpu(), w.v_cache[blk, 1, 5, :64])
    tail = int(w.page_table[0, 40])
    assert torch.equal(d.k[tail].cpu(), w.k_cache[tail]) and torch.equal(d.v[tail].cpu(), w.v_cache[tail])
    # quantisation did act on the other pages
    assert not torch.equal(d.k.cpu(), w.k_cache)


def test_quantize_listed_pages_skips_invalid_entries():
    w = _ragged(seed=6)
    d = Dev(w)
    pages = [(0, 0), (0, 39), (1, 63), (4, 2), (1, 5)]
    invalid = [(0, 40), (2, 0), (3, 0), (5, 0), (-1, 3), (1, 64), (1, -2)]
    lst = torch.tensor(pages + invalid, dtype=torch.int32, device=d.device)
    kv = B.Kivi(2, 32, B.LOCKS_KIVI_PRE)
    print(f"[kivi list] {len(pages)} pages + {len(invalid)} invalid entries", flush=True)
    B.kivi_quantize(d.cfg, kv, d.k, d.v, d.pt, d.sl, page_list=lst)
    torch.cuda.synchronize()
    kc, vc = _expected_caches(w, pages, 2, 32)
    np.testing.assert_array_equal(_bits(d.k), _bits(kc))
    np.testing.assert_array_equal(_bits(d.v), _bits(vc))
    # an empty list launches nothing
    B.kivi_quantize(d.cfg, kv, d.k, d.v, d.pt, d.sl, page_list=lst[:0])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bits(d.k), _bits(kc))


@pytest.mark.parametrize("bits", [4, 2])
def test_quantize_full_size_sampled_pages(bits):
    """Every complete page of the Llama-3.1-8B-shaped 32K workload (2,048 pages x 8 KV
    heads) in one launch; 256 sampled page-heads checked one by one, and no block
    outside the sequence's pages changed."""
    w = make_workload(1, seed=2)
    d = Dev(w)
    print(f"[kivi 32k] bits {bits}", flush=True)
    B.kivi_quantize(d.cfg, B.Kivi(bits, 32, B.LOCKS_KIVI_POST), d.k, d.v, d.pt, d.sl)
    torch.cuda.synchronize()
    got_k, got_v = d.k.cpu(), d.v.cpu()
    rng = np.random.default_rng(bits)
    n_c = int(w.seq_lens[0]) // PAGE
    for _ in range(256):
        j, h = int(rng.integers(n_c)), int(rng.integers(w.spec.num_kv_heads))
        blk = int(w.page_table[0, j])
        kq, vq = _oracle_page(w.k_cache, w.v_cache, blk, h, bits, 32)
        np.testing.assert_array_equal(_bits(got_k[blk, h]), _bits(kq))
        np.testing.assert_array_equal(_bits(got_v[blk, h]), _bits(vq))
    used = set(int(x) for x in w.page_table[0, :n_c])
    other = [b for b in range(w.num_blocks) if b not in used]
    if other:
        idx = torch.tensor(other)
        assert torch.equal(got_k[idx], w.k_cache[idx]) and torch.equal(got_v[idx], w.v_cache[idx])


def _finalised_state(d, w, listed, kv, stage):
    """Caches and summaries as a serving loop leaves them: every complete page other
    than the listed ones finalised earlier (quantised, and summarised before (POST)
    or after (PRE) its quantisation)."""
    others = [p for p in _complete_pages(w) if p not in listed]
    lst = torch.tensor(others, dtype=torch.int32, device=d.device).reshape(-1, 2)
    store = B.alloc_summaries(d.cfg, d.device)
    if stage == B.LOCKS_KIVI_POST:
        B.build_summaries(d.cfg, d.k, d.pt, d.sl, store)
        B.kivi_quantize(d.cfg, kv, d.k, d.v, d.pt, d.sl, page_list=lst)
    else:
        B.kivi_quantize(d.cfg, kv, d.k, d.v, d.pt, d.sl, page_list=lst)
        B.build_summaries(d.cfg, d.k, d.pt, d.sl, store)
    return store


@pytest.mark.parametrize("stage", [B.LOCKS_KIVI_POST, B.LOCKS_KIVI_PRE])
@pytest.mark.parametrize("bits,inner", [(4, False), (2, False), (4, True)])
def test_decode_step_on_quantised_cache(stage, bits, inner):
    """The fused step with the pages that filled this step in its build list: the
    listed pages are quantised before (PRE) or after (POST) their build, the caches
    afterwards equal the oracle's quantised caches bit for bit, and tables and
    outputs follow the oracle's step on those caches, its summaries built from the
    quantised keys (PRE) or from the keys as written (POST)."""
    lens = [16 * 300, 16 * 200 + 9, 16 * 150, 16 * 90 + 1]
    spec = WorkloadSpec("kivi-step", len(lens), 16, 4, lens, 4, 256, "bf16", "bf16")
    w = build_workload(spec, 11)
    d = Dev(w)
    cfg = d.cfg
    listed = [(s, int(w.seq_lens[s]) // PAGE - 1) for s in range(spec.num_seqs)]
    if inner:   # pages other than the last complete one (built on the forked stream)
        listed += [(0, 7), (2, int(w.seq_lens[2]) // PAGE - 2), (3, 40)]
    kv = B.Kivi(bits, 32, stage)
    name = "POST" if stage == B.LOCKS_KIVI_POST else "PRE"
    print(f"[kivi step] {name} bits {bits} listed {listed}", flush=True)
    store = _finalised_state(d, w, listed, kv, stage)
    bl = torch.tensor(listed, dtype=torch.int32, device=d.device)
    ids, sel, out, lse = B.decode_step(cfg, d.q, d.k, d.v, d.pt, d.sl, store, d.ws,
                                       build_list=bl, kivi=kv)
    torch.cuda.synchronize()
    kc, vc = _expected_caches(w, _complete_pages(w), bits, 32)
    np.testing.assert_array_equal(_bits(d.k), _bits(kc))
    np.testing.assert_array_equal(_bits(d.v), _bits(vc))
    wq = dataclasses.replace(w, k_cache=kc, v_cache=vc)
    G = cfg.group
    inter = tot = same = 0
    worst = 0.0
    for s in range(cfg.num_seqs):
        for h in range(cfg.num_kv_heads):
            k0, _, _ = d.unit(s, h)
            kq, vq, qg = gather_unit(wq, s, h)
            keys_for_summary = kq if stage == B.LOCKS_KIVI_PRE else k0
            ref = O.decode_step(qg, kq, vq, O.unit_summaries(keys_for_summary, cfg.rank),
                                cfg.rank, cfg.budget_tokens)
            got = ids_of(ids[s, h].tolist())
            inter += len(set(got) & set(ref["ids"]))
            tot += len(ref["ids"])
            same += got == ref["ids"]
            # attention over the quantised caches, on the GPU's own table
            o = out[s, h * G:(h + 1) * G].double().cpu().numpy()
            l = lse[s, h * G:(h + 1) * G].double().cpu().numpy()
            worst = max(worst, check_attention_on_table(qg, kq, vq, got, o, l))
    print(f"[kivi step] {name} bits {bits}: overlap {inter / tot:.4f}, identical tables "
          f"{same}/{cfg.num_seqs * cfg.num_kv_heads}, worst rel-L2 {worst:.2e}")
    assert inter / tot >= OVERLAP_TOL
