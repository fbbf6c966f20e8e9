#!/usr/bin/env python
"""Decode-step benchmark of the Locks sparse decode attention on one MI355X.

One step = the fused locks_decode_step (summary scan -> share-average combine and
top-k table -> sparse attention over the table) on synthetic inputs resident in
HBM.  The headline workload is the 1,048,576-token GLM-4-9B-shaped decode
(1 sequence, 32 query heads over 2 KV heads, d = 128, page 16, r = 8, budget 2048
tokens, bf16 KV); the same line carries the metric's 128K point (8 sequences of
131,072 tokens, 32 q / 8 kv heads, r = 8) as a second block.  Each block rotates
over --copies independent copies of the KV cache and summary store so that the
256 MB last-level cache cannot serve repeats.

Timing protocol (after App. C.7 "Decode efficiency"): --warmup untimed steps,
then three windows of --steps steps, each bracketed by a device synchronisation
and timed by the wall clock and HIP events (a window more than 10% off the median
is timed again, at most three times), then one dispersion window with a HIP event
around every step for the per-step mean and sd (timed again if sd / mean exceeds
10%).  `value` is the mean over the three windows of the wall-clock time per
step, in microseconds.  After timing, the step's outputs for
one full (sequence, KV head) unit -- whose summaries are the oracle's own records
-- are checked against the CPU fp64 oracle (page LSEs, table, output, output LSE);
a failed check exits non-zero without a value.  That oracle step, timed, is the
CPU baseline.

Prints ONE JSON line.
"""
import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-step latency (µs) + achieved HBM GB/s vs peak at 128K/1M ctx, r=8"
HBM_PEAK_GBPS = 8000.0
FP32_VALU_PEAK_TFLOPS = 157.3
WINDOWS = 3
CV_LIMIT = 0.10
LSE_TOL, OUT_TOL, GAP_TOL = 1e-3, 2e-3, 1e-3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64, help="steps per timed window (3 windows)")
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--copies", type=int, default=3)
    ap.add_argument("--workload", choices=list(WORKLOADS), default="1m")
    ap.add_argument("--second", choices=list(WORKLOADS) + ["none"], default=None,
                    help="second block of the line (default: 128k when the workload is 1m)")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (CPU baseline and the parity gate)")
    ap.add_argument("--no-build", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step from captured HIP graphs instead of launching it")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--kivi", type=int, default=0, metavar="BITS",
                    help="KIVI fake quantisation of finalised pages at BITS bits (values in "
                         "groups of 32 channels): every complete page before timing, and in the "
                         "reasoning loop the pages that fill, inside the step")
    ap.add_argument("--kivi-stage", choices=("post", "pre"), default="post")
    ap.add_argument("--torch-kv-write", action="store_true",
                    help="reasoning loop: write the new token's K and V with torch copies "
                         "before the step instead of inside it")
    ap.add_argument("--no-kivi-pass", action="store_true",
                    help="skip the separately timed KIVI pass over every complete page")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="first run a plain fp32 copy of this many MiB four times (the "
                         "known-size reference that scales hardware byte counters)")
    return ap.parse_args()


WORKLOADS = {
    # name: (workload id, overrides, description)
    "1m": (3, {}, "glm4-9b-1m: 1 seq x 1,048,576 tokens, 32 q / 2 kv heads, d 128, "
                  "page 16, r 8, b 2048, bf16 KV"),
    "128k": (2, {}, "llama3.1-8b-128k: 8 seq x 131,072 tokens, 32 q / 8 kv heads, d 128, "
                    "page 16, r 8, b 2048, bf16 KV"),
    "128k-r2": (2, {"rank": 2}, "llama3.1-8b-128k: 8 seq x 131,072 tokens, 32 q / 8 kv heads, "
                                "d 128, page 16, r 2, b 2048, bf16 KV"),
    "128k-int8basis": (2, {"basis": 1}, "llama3.1-8b-128k: 8 seq x 131,072 tokens, 32 q / 8 kv "
                                        "heads, d 128, page 16, r 8, int8 basis, b 2048, bf16 KV"),
    "128k-bf16basis": (2, {"basis": 2}, "llama3.1-8b-128k: 8 seq x 131,072 tokens, 32 q / 8 kv "
                                        "heads, d 128, page 16, r 8, bf16 basis, b 2048, bf16 KV"),
    "32k": (1, {}, "llama3.1-8b-32k: 1 seq x 32,768 tokens, 32 q / 8 kv heads, d 128, page 16, "
                   "r 8, b 2048, bf16 KV"),
    # page sizes of App. D.3: the same keys and values in pages of 32 and 64 tokens
    "1m-B32": (3, {"page_size": 32}, "glm4-9b-1m: 1 seq x 1,048,576 tokens, 32 q / 2 kv heads, "
                                     "d 128, page 32, r 8, b 2048, bf16 KV"),
    "1m-B64": (3, {"page_size": 64}, "glm4-9b-1m: 1 seq x 1,048,576 tokens, 32 q / 2 kv heads, "
                                     "d 128, page 64, r 8, b 2048, bf16 KV"),
    "128k-B32": (2, {"page_size": 32}, "llama3.1-8b-128k: 8 seq x 131,072 tokens, 32 q / 8 kv "
                                       "heads, d 128, page 32, r 8, b 2048, bf16 KV"),
    "128k-B64": (2, {"page_size": 64}, "llama3.1-8b-128k: 8 seq x 131,072 tokens, 32 q / 8 kv "
                                       "heads, d 128, page 64, r 8, b 2048, bf16 KV"),
    "reasoning": (4, {}, "qwen3-4b-reasoning: 64 seq x U[8K,64K] tokens, 32 q / 8 kv heads, d 128, "
                         "page 16, r 2, b 256, bf16 KV; each step appends one token per sequence "
                         "and builds the pages that filled"),
}


# HBM traffic of the scan kernel, from two rocprofv3 counter runs of
#   rocprofv3 --pmc FETCH_SIZE --kernel-include-regex 'locks|elementwise' -- \
#       python bench.py --workload W --second none --steps 8 --warmup 2 --no-dense \
#       --no-build --no-cpu-baseline --no-kivi-pass --copy-calib-mib 1024
# and the same with WRITE_SIZE (KiB per dispatch; per-workload files under profiles/).
# Each counter is divided by what it reads for the 1 GiB copy over 1 GiB, so the
# result is in bytes.  Valid only for the scan sources these hashes name.
SCAN_SOURCES = ("paper_2607_24555_amd/csrc/scan.hip", "paper_2607_24555_amd/csrc/locks_internal.h")
SCAN_TRAFFIC = {
    # workload: (sha256 of SCAN_SOURCES, FETCH_SIZE KiB, WRITE_SIZE KiB,
    #            copy FETCH factor, copy WRITE factor, profile file)
    "1m": ("d72bd2acddea2be2", 55126.2, 8985.9, 0.500016, 1.0, "profiles/scan_1m_hbm_counters.md"),
    "128k": ("d72bd2acddea2be2", 215269.2, 8618.9, 0.500016, 1.0, "profiles/scan_128k_hbm_counters.md"),
    "128k-r2": ("d72bd2acddea2be2", 86822.1, 8668.3, 0.500014, 1.0, "profiles/scan_128k-r2_hbm_counters.md"),
    "reasoning": ("d72bd2acddea2be2", 194797.6, 21323.1, 0.500014, 1.0, "profiles/scan_reasoning_hbm_counters.md"),
    "1m-B32": ("d72bd2acddea2be2", 33145.2, 4518.8, 0.500014, 1.0, "profiles/scan_1m-B32_hbm_counters.md"),
    "1m-B64": ("d72bd2acddea2be2", 21813.7, 2318.0, 0.500013, 1.0, "profiles/scan_1m-B64_hbm_counters.md"),
    "128k-B32": ("d72bd2acddea2be2", 127531.1, 4382.0, 0.500015, 1.0, "profiles/scan_128k-B32_hbm_counters.md"),
    "128k-B64": ("d72bd2acddea2be2", 84462.2, 2312.3, 0.500015, 1.0, "profiles/scan_128k-B64_hbm_counters.md"),
}


def scan_sources_sha():
    import hashlib
    h = hashlib.sha256()
    for f in SCAN_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def scan_traffic(workload):
    """Counted HBM bytes per scan launch, or None if not measured for the current
    scan sources."""
    t = SCAN_TRAFFIC.get(workload)
    if t is None or t[0] != scan_sources_sha():
        return None, None
    _, fetch_kib, write_kib, ff, fw, prof = t
    fetch, write = fetch_kib * 1024 / ff, write_kib * 1024 / fw
    return int(fetch + write), {"fetch_bytes": int(fetch), "write_bytes": int(write),
                                "copy_factor_fetch": ff, "copy_factor_write": fw,
                                "source_sha": t[0], "profile": prof}


def copy_calibration(mib, dev):
    """A plain copy of known size (reads and writes mib MiB) for counter scaling."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(4):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    del src, dst


def as_graphs(fns):
    """Capture each fn() (one per rotated copy) into its own HIP graph; the library
    allocates nothing and only enqueues on the current stream.  Returns a replay
    function of the step index."""
    import torch
    from paper_2607_24555_amd import locks as B
    B.init()   # the side stream exists before any capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for fn in fns:
            fn()
    torch.cuda.current_stream().wait_stream(side)
    graphs = []
    for fn in fns:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        graphs.append(g)
    torch.cuda.synchronize()
    return lambda i: graphs[i % len(graphs)].replay()


def timed(fn, n, sync):
    """Wall time and event time per call of n calls of fn(i) on torch's current stream."""
    import torch
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    sync()
    t0 = time.perf_counter()
    start.record()
    for i in range(n):
        fn(i)
    end.record()
    sync()
    t1 = time.perf_counter()
    return (t1 - t0) / n * 1e6, start.elapsed_time(end) / n * 1e3


def windows(fn, steps, sync, first=0):
    """The timing protocol.  WINDOWS clean windows of `steps` calls, each between
    two synchronisations, timed by the wall clock and by two HIP events; a window
    whose time per step lies more than CV_LIMIT from the median of the windows is
    timed again (three tries).  Then one dispersion window records a HIP event
    before every call and after the last, for the per-step mean and sd (the events
    between steps add a few microseconds each, so this window is not part of the
    value); if its sd / mean exceeds CV_LIMIT it is timed again (three tries).
    Returns the summary dict; 'ok' is False when a window was refused three times."""
    import torch
    i = first

    def clean():
        nonlocal i
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        sync()
        t0 = time.perf_counter()
        a.record()
        for _ in range(steps):
            fn(i)
            i += 1
        b.record()
        sync()
        t1 = time.perf_counter()
        return (t1 - t0) / steps * 1e6, a.elapsed_time(b) / steps * 1e3

    runs = [clean() for _ in range(WINDOWS)]
    refused, ok = 0, True
    for w in range(WINDOWS):
        for attempt in range(3):
            med = statistics.median(r[0] for r in runs)
            if abs(runs[w][0] - med) <= CV_LIMIT * med:
                break
            refused += 1
            runs[w] = clean()
        else:
            ok = False
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    for attempt in range(3):
        sync()
        for j in range(steps):
            evs[j].record()
            fn(i)
            i += 1
        evs[steps].record()
        sync()
        per = [evs[j].elapsed_time(evs[j + 1]) * 1e3 for j in range(steps)]
        pm = statistics.fmean(per)
        psd = statistics.pstdev(per) if len(per) > 1 else 0.0
        if psd <= CV_LIMIT * pm:
            break
        refused += 1
    else:
        ok = False
    walls = [r[0] for r in runs]
    mean = statistics.fmean(walls)
    return {"n": WINDOWS, "steps_each": steps, "per_step_us": [round(x, 2) for x in walls],
            "event_per_step_us": [round(r[1], 2) for r in runs],
            "mean_us": round(mean, 2), "sd_us": round(statistics.stdev(walls), 2),
            "dispersion_window": {"steps": steps, "mean_us": round(pm, 2), "sd_us": round(psd, 2),
                                  "cv": round(psd / pm, 4) if pm > 0 else None},
            "refused": refused, "ok": ok, "next_index": i}


def build_flops(B_, d, r):
    """Algorithmic flops of one page-head's build: centroid B d, Gram 2 B^2 d, a
    symmetric B x B eigendecomposition with vectors ~9 B^3 (tridiagonal reduction
    plus implicit QR), basis V = D^T U_r / sigma 2 d B r."""
    return B_ * d + 2 * B_ * B_ * d + 9 * B_ ** 3 + 2 * d * B_ * r


# ---------------------------------------------------------------- oracle leg

def oracle_unit(w, cfg, s, h):
    """The oracle's own records and its whole decode step for one (seq, KV head)."""
    from oracle import locks_oracle as O
    from paper_2607_24555_amd import locks as B
    from workloads import gather_unit
    k, v, q = gather_unit(w, s, h)
    basis = B.BASIS_NAMES[cfg.basis]
    rec = O.unit_summaries(k, cfg.rank, basis, cfg.page_size)
    return k, v, q, rec


def cpu_step(k, v, q, rec, cfg, min_s=10.0, max_reps=20):
    """The oracle's decode step (score every page, select, attend) on one full unit,
    repeated until min_s seconds have passed; BLAS threads = this process's CPUs."""
    from threadpoolctl import threadpool_limits
    from oracle import locks_oracle as O
    from paper_2607_24555_amd import locks as B
    cores = len(os.sched_getaffinity(0))
    basis = B.BASIS_NAMES[cfg.basis]
    with threadpool_limits(limits=cores):
        t0 = time.perf_counter()
        reps = 0
        while True:
            ref = O.decode_step(q, k, v, rec, cfg.rank, cfg.budget_tokens, basis,
                                cfg.page_size)
            reps += 1
            if time.perf_counter() - t0 > min_s or reps >= max_reps:
                break
        dt = (time.perf_counter() - t0) / reps
    return ref, dt, reps, cores


def parity_gate(ref, k, v, q, cfg, ids, sel, out, lse, s, h):
    """The timed step's outputs for unit (s, h) against the oracle's step on the same
    records: table by the gap rule (near ties: only pages within the score
    tolerance band of the cut may differ), page LSEs of the table, output against the
    oracle's attention over the GPU's table, output LSE.  Returns (ok, detail)."""
    import numpy as np
    from oracle import locks_oracle as O
    G = cfg.group
    L = k.shape[0]
    P = cfg.page_size
    n_c, n = L // P, -(-L // P)
    got = [int(x) for x in ids[s, h].tolist() if int(x) >= 0]
    hs = slice(h * G, (h + 1) * G)
    gsel = sel[s, hs].double().cpu().numpy()
    o = out[s, hs].double().cpu().numpy()
    l = lse[s, hs].double().cpu().numpy()
    det = {"unit": [s, h], "pages": n, "oracle_gap": ref["gap"] if math.isfinite(ref["gap"])
           else None}
    problems = []
    if got != sorted(set(got)) or len(got) != min(cfg.k, n) or (n and (got[0] != 0 or got[-1] != n - 1)):
        problems.append("malformed table")
    same = got == ref["ids"]
    det["table"] = "identical" if same else "differs"
    if not same:
        if ref["gap"] > GAP_TOL:
            problems.append("table differs above the gap tolerance")
        else:
            lm = ref["log_mbar"]
            cand = sorted(range(1, n - 1), key=lambda j: (-lm[j], j))
            cut = lm[cand[cfg.k - 3]]
            if any(not (0 < j < n - 1) or abs(lm[j] - cut) > 4 * LSE_TOL
                   for j in set(got) ^ set(ref["ids"])):
                problems.append("near-tie table differs outside the tolerance band")
    err = 0.0
    for t, j in enumerate(got):
        if j < n_c:
            err = max(err, float(np.max(np.abs(gsel[:, t] - ref["s_hat"][:, j]))))
        elif not np.isnan(gsel[:, t]).all():
            problems.append("page LSE of a page without summary is not NaN")
    det["max_sel_lse_err"] = err
    if err > LSE_TOL:
        problems.append("page LSE error")
    o_ref, l_ref = O.attend(q, k, v, got, P)
    rel = max(float(np.linalg.norm(o[g] - o_ref[g]) / max(np.linalg.norm(o_ref[g]), 1e-30))
              for g in range(G))
    det["max_rel_l2"] = rel
    det["max_lse_err"] = float(np.max(np.abs(l - l_ref)))
    if rel > OUT_TOL:
        problems.append("output rel-L2")
    if det["max_lse_err"] > LSE_TOL:
        problems.append("output LSE")
    det["ok"] = not problems
    if problems:
        det["problems"] = problems
    return det["ok"], det


# ---------------------------------------------------------------- one workload

def run_block(name, args, dev, with_oracle, rest):
    """Build, scan, fused step (timing protocol), dense baseline, KIVI pass and the
    oracle leg for one workload.  Returns the block's dict; rest['fail'] is set when
    the parity gate fails."""
    import torch
    from paper_2607_24555_amd import locks as B
    from workloads import make_workload

    wid, ov, desc = WORKLOADS[name]
    ov = dict(ov)
    basis = ov.pop("basis", B.LOCKS_BASIS_INT4)
    growing = name == "reasoning"
    if growing:   # room for every appended token: warm-up plus up to three tries per window
        ov["spare_pages"] = (args.warmup + 4 * WINDOWS * args.steps) // 16 + 2
    t_gen = time.perf_counter()
    w = make_workload(wid, seed=args.seed, device=dev, **ov)
    t_gen = time.perf_counter() - t_gen
    cfg = B.config_for(w.spec, w.num_blocks, w.max_pages)
    cfg.basis = basis
    q, pt, sl = w.q, w.page_table, w.seq_lens
    R = 1 if growing else max(1, args.copies)
    ks = [w.k_cache] + [w.k_cache.clone() for _ in range(R - 1)]
    vs = [w.v_cache] + [w.v_cache.clone() for _ in range(R - 1)]
    summ = [B.alloc_summaries(cfg, dev) for _ in range(R)]
    ws = B.alloc_workspace(cfg, dev)
    sync = torch.cuda.synchronize

    P = cfg.page_size
    n_pages = sum(math.ceil(L / P) for L in w.spec.seq_lens)
    complete_heads = sum(L // P for L in w.spec.seq_lens) * cfg.num_kv_heads
    payload = B.summary_payload_bytes_ex(cfg.rank, cfg.basis, cfg.page_size)
    stride = B.summary_stride(cfg.rank, cfg.basis, cfg.page_size)
    k_sel = min(cfg.k, max(math.ceil(L / P) for L in w.spec.seq_lens))
    kv_page = 2 * P * 128 * 2
    alg_scan = complete_heads * payload
    alg_attend = sum(min(cfg.k, math.ceil(L / P)) for L in w.spec.seq_lens) * \
        cfg.num_kv_heads * kv_page
    alg_step = alg_scan + alg_attend

    # ---- summary build (separately timed): every complete page, every copy
    build_us = None
    for i in range(R):
        B.build_summaries(cfg, ks[i], pt, sl, summ[i])
    sync()
    if not args.no_build:
        _, build_us = timed(lambda i: B.build_summaries(cfg, ks[i % R], pt, sl, summ[i % R]),
                            R, sync)
    kivi = None
    if args.kivi:
        stage = B.LOCKS_KIVI_PRE if args.kivi_stage == "pre" else B.LOCKS_KIVI_POST
        kivi = B.Kivi(args.kivi, 32, stage)
        # pages finalised before the timed steps: quantised, summaries from the keys
        # as written (POST) or rebuilt from the quantised keys (PRE)
        for i in range(R):
            B.kivi_quantize(cfg, kivi, ks[i], vs[i], pt, sl)
            if stage == B.LOCKS_KIVI_PRE:
                B.build_summaries(cfg, ks[i], pt, sl, summ[i])
        sync()

    # ---- the oracle's own records for the checked unit (seq 0, KV head 0) replace
    # the GPU-built ones in copy 0, so the timed steps of copy 0 run on them
    gate_unit = (0, 0)
    oracle = None
    if with_oracle and not growing and not args.kivi:
        t_or = time.perf_counter()
        k0, v0, q0, rec0 = oracle_unit(w, cfg, *gate_unit)
        n_c0 = k0.shape[0] // P
        blocks = pt[gate_unit[0], :n_c0].long()
        summ[0][blocks, gate_unit[1]] = torch.from_numpy(rec0).to(dev)
        sync()
        oracle = (k0, v0, q0, rec0, time.perf_counter() - t_or)

    # ---- scan alone (dominant kernel): roofline on its algorithmic bytes
    all_lse = torch.empty(cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq, device=dev)
    scans = [B.prepare_score_pages(cfg, q, summ[i], pt, sl, ws, all_lse) for i in range(R)]
    for i in range(args.warmup):
        scans[i % R]()
    _, scan_us = timed(lambda i: scans[i % R](), args.steps, sync)

    # ---- fused decode step: one prepared call and one set of outputs per copy
    outs = [B.alloc_select_outputs(cfg, dev) + B.alloc_attend_outputs(cfg, dev) for _ in range(R)]
    n_built = 0
    if not growing:
        prepared = [B.prepare_decode_step(cfg, q, ks[i], vs[i], pt, sl, summ[i], ws,
                                          out_ids=outs[i][0], out_sel_lse=outs[i][1],
                                          out=outs[i][2], out_lse=outs[i][3]) for i in range(R)]
        if args.graph:
            step = as_graphs(prepared)
        else:
            def step(i):
                prepared[i % R]()
    else:
        if args.graph:
            raise SystemExit("--graph replays fixed launches; the reasoning workload grows every step")
        # every step writes one new token per sequence into the paged cache (the
        # caller's KV write), bumps seq_lens and builds the pages that just filled
        T = args.warmup + 4 * WINDOWS * args.steps   # every window may be timed three times
        lens0 = torch.tensor(w.spec.seq_lens, dtype=torch.long)
        gen = torch.Generator(device=dev).manual_seed(args.seed + 7)
        new_k = torch.randn(T, cfg.num_seqs, cfg.num_kv_heads, 128, generator=gen, device=dev,
                            dtype=torch.float32).to(ks[0].dtype)
        new_v = torch.randn_like(new_k)
        pos = lens0[None, :] + torch.arange(T)[:, None]            # [T][S] token index
        if int((pos // 16).max()) >= cfg.max_pages_per_seq:
            raise SystemExit(f"{T} appended tokens overrun the spare pages of the page table")
        blk_at = pt.long().cpu().gather(1, (pos // 16).T).T         # [T][S] physical block
        if int(blk_at.min()) < 0:
            raise SystemExit(f"{T} appended tokens reach pages without a physical block")
        hk = torch.arange(cfg.num_kv_heads)
        flat = ((blk_at[:, :, None] * cfg.num_kv_heads + hk) * 16 + (pos % 16)[:, :, None])
        flat = flat.reshape(T, -1).to(dev)
        lists = []
        for t in range(T):
            full = ((pos[t] + 1) % 16 == 0).nonzero().flatten()
            lists.append(torch.stack([full, pos[t, full] // 16], 1).to(torch.int32).to(dev)
                         if len(full) else None)
        k_rows, v_rows = ks[0].view(-1, 128), vs[0].view(-1, 128)
        o = outs[0]
        if args.torch_kv_write:
            prepared = [B.prepare_decode_step(cfg, q, ks[0], vs[0], pt, sl, summ[0], ws,
                                              build_list=lists[t], out_ids=o[0], out_sel_lse=o[1],
                                              out=o[2], out_lse=o[3], kivi=kivi) for t in range(T)]
        else:   # the step writes the new token's K and V itself, beside the scan
            prepared = [B.prepare_decode_step(cfg, q, ks[0], vs[0], pt, sl, summ[0], ws,
                                              build_list=lists[t], out_ids=o[0], out_sel_lse=o[1],
                                              out=o[2], out_lse=o[3], kivi=kivi, k_new=new_k[t],
                                              v_new=new_v[t]) for t in range(T)]
        calls = [0]  # appended tokens so far: warm-up and timed steps continue one sequence

        def step(_i):
            t = calls[0]
            calls[0] += 1
            sl.add_(1)
            if args.torch_kv_write:
                k_rows.index_copy_(0, flat[t], new_k[t].view(-1, 128))
                v_rows.index_copy_(0, flat[t], new_v[t].view(-1, 128))
            prepared[t]()

    for i in range(args.warmup):
        step(i)
    win = windows(step, args.steps, sync, first=args.warmup)
    step_ev_us = statistics.fmean(win["event_per_step_us"])
    if growing:
        n_built = sum(0 if x is None else len(x)
                      for x in lists[args.warmup:args.warmup + WINDOWS * args.steps])
    step_us = win["mean_us"]

    block = {
        "workload": desc,
        "global_batch": cfg.num_seqs,
        "seq_len": int(max(w.spec.seq_lens)),
        "value_us": step_us,
        "windows": {k: v for k, v in win.items() if k != "next_index"},
        "step": {"alg_bytes": alg_step, "alg_GBps": round(alg_step / (step_us * 1e-6) / 1e9, 1),
                 "frac_of_peak": round(alg_step / (step_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                 "event_us": None if step_ev_us is None else round(step_ev_us, 2),
                 "summary_stride_bytes": stride,
                 "launch": "hip-graph replay" if args.graph else "eager",
                 "selected_pages_per_kv_head": k_sel,
                 "pages_built_inline": n_built if growing else None,
                 "includes_kv_append": growing,
                 "kv_append": (None if not growing else
                               "torch index_copy before the step" if args.torch_kv_write else
                               "inside the step (locks_decode_step_ex)")},
    }

    # ---- scan roofline
    scan_gbps = alg_scan / (scan_us * 1e-6) / 1e9
    traffic, traffic_detail = scan_traffic(name)
    block["roofline"] = {"bound": "hbm", "kernel": "scan_kernel (locks_score_pages)",
                         "achieved": round(scan_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": round(scan_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic,
                         "traffic_detail": traffic_detail,
                         "alg_bytes_per_launch": alg_scan, "unit_bytes": payload,
                         "units_per_launch": complete_heads, "avg_launch_us": round(scan_us, 2)}

    # ---- dense baseline on identical inputs
    if not args.no_dense:
        dout, dlse = B.alloc_attend_outputs(cfg, dev)
        dense = [B.prepare_dense_attend(cfg, q, ks[i], vs[i], pt, sl, ws, dout, dlse)
                 for i in range(R)]

        def dstep(i):
            dense[i % R]()

        for i in range(max(2, args.warmup // 2)):
            dstep(i)
        dense_us, _ = timed(dstep, max(4, args.steps // 4), sync)
        dense_bytes = n_pages * cfg.num_kv_heads * kv_page
        gbps = dense_bytes / (dense_us * 1e-6) / 1e9
        block["dense"] = {"us": round(dense_us, 2), "bytes": dense_bytes, "GBps": round(gbps, 1),
                          "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4),
                          "speedup_sparse_vs_dense": round(dense_us / step_us, 3)}

    # ---- build against both ceilings
    if build_us is not None:
        fl = build_flops(P, 128, cfg.rank) * complete_heads
        rd = complete_heads * P * 128 * 2
        wr = complete_heads * payload
        block["build"] = {
            "us": round(build_us, 1), "pages": complete_heads,
            "read_GBps": round(rd / (build_us * 1e-6) / 1e9, 1),
            "hbm_frac": round((rd + wr) / (build_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "flops_per_page_head": build_flops(P, 128, cfg.rank),
            "TFLOPs": round(fl / (build_us * 1e-6) / 1e12, 2),
            "valu_frac": round(fl / (build_us * 1e-6) / 1e12 / FP32_VALU_PEAK_TFLOPS, 4)}

    # ---- KIVI fake quantisation of every complete page (separately timed, last:
    # it rewrites the caches in place)
    if rest.get("kivi_pass") and P == 16:
        kp = B.Kivi(args.kivi or 4, 32, B.LOCKS_KIVI_POST)
        B.kivi_quantize(cfg, kp, ks[0], vs[0], pt, sl)
        _, kivi_us = timed(lambda i: B.kivi_quantize(cfg, kp, ks[i % R], vs[i % R], pt, sl),
                           max(R, 4), sync)
        kivi_bytes = complete_heads * P * 128 * 2 * 2 * 2   # K and V, read and written
        block["kivi_pass"] = {"us": round(kivi_us, 1), "pages": complete_heads,
                              "bits": args.kivi or 4, "v_group": 32, "bytes": kivi_bytes,
                              "GBps": round(kivi_bytes / (kivi_us * 1e-6) / 1e9, 1)}
    block["gen_s"] = round(t_gen, 1)

    # ---- oracle leg: parity of the timed step on the checked unit, CPU baseline
    if oracle is not None:
        k0, v0, q0, rec0, t_build = oracle
        ref, dt, reps, cores = cpu_step(k0, v0, q0, rec0, cfg,
                                        min_s=10.0 if rest.get("cpu_baseline") else 0.0)
        o = outs[0]
        ok, det = parity_gate(ref, k0, v0, q0, cfg, o[0], o[1], o[2], o[3], *gate_unit)
        det["outputs_of"] = "the last timed step on copy 0 (oracle records for this unit)"
        block["parity"] = det
        if not ok:
            rest["fail"] = True
        if rest.get("cpu_baseline"):
            units = cfg.num_seqs * cfg.num_kv_heads
            unit_pages = -(-k0.shape[0] // P)
            page_heads = n_pages * cfg.num_kv_heads
            scale = page_heads / unit_pages
            rest["cpu_baseline"] = {
                "value": round(dt * scale * 1e6, 1), "unit": "us", "cores": cores,
                "kind": "oracle",
                "sample": f"oracle decode step (score every page, select, attend) on the full "
                          f"unit (seq {gate_unit[0]}, KV head {gate_unit[1]}) of the {name} "
                          f"workload: {unit_pages} pages, G={cfg.group} heads, {reps} reps of "
                          f"{dt:.3f} s with BLAS on {cores} threads (einsum steps on one); "
                          f"scaled by page-heads x{scale:.2f} to the step's {page_heads} "
                          f"({units} units)",
                "unit_s": round(dt, 4)}
    return block


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the Locks decode step runs on one GPU; sharding across "
                                   "GPUs is not implemented",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch

    dev = torch.device("cuda:0")
    if args.copy_calib_mib > 0:
        copy_calibration(args.copy_calib_mib, dev)
    second = args.second if args.second is not None else ("128k" if args.workload == "1m" else "none")
    with_oracle = not args.no_cpu_baseline
    rest = {"cpu_baseline": with_oracle, "kivi_pass": not args.no_kivi_pass}
    main_block = run_block(args.workload, args, dev, with_oracle, rest)
    torch.cuda.empty_cache()
    blocks = {}
    if second != "none":
        rest2 = {"cpu_baseline": False, "kivi_pass": False}
        blocks[second] = run_block(second, args, dev, with_oracle, rest2)
        if rest2.get("fail"):
            rest["fail"] = True
    if rest.get("fail") or not main_block["windows"]["ok"]:
        print(json.dumps({"error": "parity gate failed or a timing window was refused three "
                                   "times; no value reported",
                          "parity": main_block.get("parity"),
                          "second_parity": {k: b.get("parity") for k, b in blocks.items()},
                          "windows": main_block["windows"]}), flush=True)
        sys.exit(1)
    res = {
        "metric": METRIC,
        "value": main_block["value_us"],
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_block["value_us"] / 1e3, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": main_block["workload"], "global_batch": main_block["global_batch"],
                   "seq_len": main_block["seq_len"],
                   "parallelism": "single-gpu", "copies_rotated": args.copies,
                   "kivi": None if not args.kivi else {"bits": args.kivi, "v_group": 32,
                                                       "stage": args.kivi_stage}},
    }
    res.update({k: v for k, v in main_block.items()
                if k not in ("workload", "value_us", "global_batch", "seq_len")})
    if with_oracle and "cpu_baseline" in rest and isinstance(rest["cpu_baseline"], dict):
        res["cpu_baseline"] = rest["cpu_baseline"]
    for k, b in blocks.items():
        res["at_" + k] = b
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
