#!/usr/bin/env python
"""Decode-step benchmark of the Locks sparse decode attention on one MI355X.

One step = the fused locks_decode_step (summary scan -> share-average combine and
top-k table -> sparse attention over the table) on the 1,048,576-token GLM-4-9B-
shaped workload (1 sequence, 32 query heads over 2 KV heads, d = 128, page 16,
r = 8, budget 2048 tokens, bf16 KV, synthetic inputs).  Inputs are resident in HBM
before timing; the step rotates over --copies independent copies of the KV cache
and summary store so that the 256 MB last-level cache cannot serve repeats.

Prints ONE JSON line.  `value` is the per-step latency in microseconds.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-step latency (µs) + achieved HBM GB/s vs peak at 128K/1M ctx, r=8"
HBM_PEAK_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--copies", type=int, default=3)
    ap.add_argument("--workload", choices=list(WORKLOADS), default="1m")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    "reasoning": (4, {}, "qwen3-4b-reasoning: 64 seq x U[8K,64K] tokens, 32 q / 8 kv heads, d 128, "
                         "page 16, r 2, b 256, bf16 KV; each step appends one token per sequence "
                         "and builds the pages that filled"),
}


# HBM traffic of the scan kernel, from two rocprofv3 counter runs of
#   rocprofv3 --pmc FETCH_SIZE --kernel-include-regex 'locks|elementwise' -- \
#       python bench.py --workload W --steps 4 --warmup 1 --no-dense --no-build \
#       --no-cpu-baseline --copy-calib-mib 1024
# and the same with WRITE_SIZE (KiB per dispatch; per-workload files under profiles/).
# Each counter is divided by what it reads for the 1 GiB copy over 1 GiB, so the
# result is in bytes.  Valid only for the scan sources these hashes name.
SCAN_SOURCES = ("paper_2607_24555_amd/csrc/scan.hip", "paper_2607_24555_amd/csrc/locks_internal.h")
SCAN_TRAFFIC = {
    # workload: (sha256 of SCAN_SOURCES, FETCH_SIZE KiB, WRITE_SIZE KiB,
    #            copy FETCH factor, copy WRITE factor, profile file)
    "1m": ("d263b7a576261335", 55610.2, 9468.7, 0.500015, 1.0, "profiles/scan_1m_hbm_counters.md"),
    "128k": ("d263b7a576261335", 215102.7, 8729.0, 0.500015, 1.0, "profiles/scan_128k_hbm_counters.md"),
    "128k-r2": ("d263b7a576261335", 86759.6, 8934.0, 0.500016, 1.0, "profiles/scan_128k-r2_hbm_counters.md"),
    "reasoning": ("d263b7a576261335", 194688.8, 22087.2, 0.500016, 1.0, "profiles/scan_reasoning_hbm_counters.md"),
    "32k": ("d263b7a576261335", 6774.7, 288.0, 0.500015, 1.0, "profiles/scan_32k_hbm_counters.md"),
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


def as_graphs(fn, n_copies):
    """Capture fn(i) for every rotated copy into its own HIP graph (the library
    allocates nothing and only enqueues on the current stream); returns a
    replay function with fn's signature."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(n_copies):
            fn(i)
    torch.cuda.current_stream().wait_stream(side)
    graphs = []
    for i in range(n_copies):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn(i)
        graphs.append(g)
    torch.cuda.synchronize()
    return lambda i: graphs[i % n_copies].replay()


def timed(fn, n, sync):
    """Wall time and summed event time of n calls of fn(i) on torch's current stream."""
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


def cpu_baseline(w, cfg, sample_pages):
    """The CPU oracle's decode step (score + select + attend) on a prefix of one
    (sequence, KV head) holding `sample_pages` complete pages, scaled to the whole
    step by page-heads.  BLAS limited to one thread."""
    from threadpoolctl import threadpool_limits

    from oracle import locks_oracle as O
    from paper_2607_24555_amd import locks as B
    from workloads import gather_unit

    k, v, q = gather_unit(w, 0, 0)
    L = min(k.shape[0], sample_pages * 16)
    k, v = k[:L], v[:L]
    basis = B.BASIS_NAMES[cfg.basis]
    rec = O.unit_summaries(k, cfg.rank, basis)           # build: not part of the step
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        reps = 0
        while True:
            O.decode_step(q, k, v, rec, cfg.rank, cfg.budget_tokens, basis)
            reps += 1
            if time.perf_counter() - t0 > 10.0 or reps >= 20:
                break
        dt = (time.perf_counter() - t0) / reps
    total_page_heads = sum(math.ceil(L_ / 16) for L_ in w.spec.seq_lens) * cfg.num_kv_heads
    scale = total_page_heads / (L // 16)
    return {"value": round(dt * scale * 1e6, 1), "unit": "us", "cores": 1, "kind": "oracle",
            "sample": f"oracle decode step on seq 0 / KV head 0 truncated to {L // 16} pages "
                      f"({L} tokens, G={cfg.group} heads), {reps} reps, {dt:.3f} s each, "
                      f"scaled x{scale:.1f} to the step's {total_page_heads} page-heads"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the Locks decode step runs on one GPU; sharding across "
                                   "GPUs is not implemented",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch

    from paper_2607_24555_amd import locks as B
    from workloads import make_workload

    dev = torch.device("cuda:0")
    if args.copy_calib_mib > 0:
        copy_calibration(args.copy_calib_mib, dev)
    wid, ov, desc = WORKLOADS[args.workload]
    ov = dict(ov)
    basis = ov.pop("basis", B.LOCKS_BASIS_INT4)
    t_gen = time.perf_counter()
    w = make_workload(wid, seed=args.seed, device=dev, **ov)
    t_gen = time.perf_counter() - t_gen
    cfg = B.config_for(w.spec, w.num_blocks, w.max_pages)
    cfg.basis = basis
    q, pt, sl = w.q, w.page_table, w.seq_lens
    growing = args.workload == "reasoning"
    R = 1 if growing else max(1, args.copies)
    ks = [w.k_cache] + [w.k_cache.clone() for _ in range(R - 1)]
    vs = [w.v_cache] + [w.v_cache.clone() for _ in range(R - 1)]
    summ = [B.alloc_summaries(cfg, dev) for _ in range(R)]
    ws = B.alloc_workspace(cfg, dev)
    sync = torch.cuda.synchronize

    n_pages = sum(math.ceil(L / 16) for L in w.spec.seq_lens)
    page_heads = n_pages * cfg.num_kv_heads
    complete_heads = sum(L // 16 for L in w.spec.seq_lens) * cfg.num_kv_heads
    payload = B.summary_payload_bytes_ex(cfg.rank, cfg.basis)
    stride = B.summary_stride(cfg.rank, cfg.basis)
    k_sel = min(cfg.k, max(math.ceil(L / 16) for L in w.spec.seq_lens))
    kv_page = 2 * 16 * 128 * 2
    alg_scan = complete_heads * payload
    alg_attend = sum(min(cfg.k, math.ceil(L / 16)) for L in w.spec.seq_lens) * \
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

    # ---- scan alone (dominant kernel): roofline on its algorithmic bytes
    all_lse = torch.empty(cfg.num_seqs, cfg.num_q_heads, cfg.max_pages_per_seq, device=dev)
    for i in range(args.warmup):
        B.score_pages(cfg, q, summ[i % R], pt, sl, ws, all_lse)
    _, scan_us = timed(lambda i: B.score_pages(cfg, q, summ[i % R], pt, sl, ws, all_lse),
                       args.steps, sync)

    # ---- fused decode step
    ids, sel = B.alloc_select_outputs(cfg, dev)
    out, lse = B.alloc_attend_outputs(cfg, dev)

    def step(i):
        B.decode_step(cfg, q, ks[i % R], vs[i % R], pt, sl, summ[i % R], ws, out_ids=ids,
                      out_sel_lse=sel, out=out, out_lse=lse)

    n_built = 0
    if growing:
        # every step writes one new token per sequence into the paged cache (the
        # caller's KV write), bumps seq_lens and builds the pages that just filled
        T = args.warmup + args.steps
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
        # flat row of (block, KV head, token slot) in the cache viewed as [rows][128]
        hk = torch.arange(cfg.num_kv_heads)
        flat = ((blk_at[:, :, None] * cfg.num_kv_heads + hk) * 16 + (pos % 16)[:, :, None])
        flat = flat.reshape(T, -1).to(dev)
        lists = []
        for t in range(T):
            full = ((pos[t] + 1) % 16 == 0).nonzero().flatten()
            lists.append(torch.stack([full, pos[t, full] // 16], 1).to(torch.int32).to(dev)
                         if len(full) else None)
        n_built = sum(0 if x is None else len(x) for x in lists[args.warmup:])
        k_rows, v_rows = ks[0].view(-1, 128), vs[0].view(-1, 128)

        calls = [0]  # appended tokens so far: warm-up and timed steps continue one sequence

        def step(_i):
            i = calls[0]
            calls[0] += 1
            sl.add_(1)
            if args.torch_kv_write:
                k_rows.index_copy_(0, flat[i], new_k[i].view(-1, 128))
                v_rows.index_copy_(0, flat[i], new_v[i].view(-1, 128))
                B.decode_step(cfg, q, ks[0], vs[0], pt, sl, summ[0], ws, build_list=lists[i],
                              out_ids=ids, out_sel_lse=sel, out=out, out_lse=lse, kivi=kivi)
            else:   # the step writes the new token's K and V itself, beside the scan
                B.decode_step(cfg, q, ks[0], vs[0], pt, sl, summ[0], ws, build_list=lists[i],
                              out_ids=ids, out_sel_lse=sel, out=out, out_lse=lse, kivi=kivi,
                              k_new=new_k[i], v_new=new_v[i])

    if growing and args.graph:
        raise SystemExit("--graph replays fixed launches; the reasoning workload grows every step")
    run = as_graphs(step, R) if args.graph else step
    for i in range(args.warmup):
        run(i)
    step_wall_us, step_ev_us = timed(run, args.steps, sync)

    # ---- dense baseline on identical inputs
    dense_us = None
    if not args.no_dense:
        dout, dlse = B.alloc_attend_outputs(cfg, dev)

        def dstep(i):
            B.dense_attend(cfg, q, ks[i % R], vs[i % R], pt, sl, ws, out=dout, out_lse=dlse)

        drun = as_graphs(dstep, R) if args.graph else dstep
        for i in range(max(2, args.warmup // 2)):
            drun(i)
        dense_us, _ = timed(drun, max(4, args.steps // 4), sync)

    # ---- KIVI fake quantisation of every complete page (separately timed, last:
    # it rewrites the caches in place)
    kivi_us = None
    if not args.no_kivi_pass:
        kp = B.Kivi(args.kivi or 4, 32, B.LOCKS_KIVI_POST)
        B.kivi_quantize(cfg, kp, ks[0], vs[0], pt, sl)
        _, kivi_us = timed(lambda i: B.kivi_quantize(cfg, kp, ks[i % R], vs[i % R], pt, sl),
                           max(R, 4), sync)
    kivi_bytes = complete_heads * 16 * 128 * 2 * 2 * 2   # K and V, read and written

    scan_gbps = alg_scan / (scan_us * 1e-6) / 1e9
    traffic, traffic_detail = scan_traffic(args.workload)
    res = {
        "metric": METRIC,
        "value": round(step_wall_us, 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_wall_us / 1e3, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": desc, "global_batch": cfg.num_seqs,
                   "seq_len": int(max(w.spec.seq_lens)), "parallelism": "single-gpu",
                   "summary_basis": B.BASIS_NAMES[cfg.basis], "copies_rotated": R,
                   "kivi": None if kivi is None else {"bits": kivi.bits, "v_group": kivi.v_group,
                                                      "stage": args.kivi_stage}},
        "roofline": {"bound": "hbm", "kernel": "scan_kernel (locks_score_pages)",
                     "achieved": round(scan_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(scan_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "traffic_detail": traffic_detail,
                     "alg_bytes_per_launch": alg_scan, "unit_bytes": payload,
                     "units_per_launch": complete_heads, "avg_launch_us": round(scan_us, 2)},
        "step": {"alg_bytes": alg_step, "alg_GBps": round(alg_step / (step_wall_us * 1e-6) / 1e9, 1),
                 "frac_of_peak": round(alg_step / (step_wall_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                 "event_us": round(step_ev_us, 2), "summary_stride_bytes": stride,
                 "launch": "hip-graph replay" if args.graph else "eager",
                 "selected_pages_per_kv_head": k_sel,
                 "pages_built_inline": n_built if growing else None,
                 "includes_kv_append": growing,
                 "kv_append": (None if not growing else
                               "torch index_copy before the step" if args.torch_kv_write else
                               "inside the step (locks_decode_step_ex)")},
        "dense": None if dense_us is None else {
            "us": round(dense_us, 2), "bytes": n_pages * cfg.num_kv_heads * kv_page,
            "GBps": round(n_pages * cfg.num_kv_heads * kv_page / (dense_us * 1e-6) / 1e9, 1),
            "speedup_sparse_vs_dense": round(dense_us / step_wall_us, 3)},
        "build": None if build_us is None else {
            "us": round(build_us, 1), "pages": complete_heads,
            "read_GBps": round(complete_heads * 16 * 128 * 2 / (build_us * 1e-6) / 1e9, 1)},
        "kivi_pass": None if kivi_us is None else {
            "us": round(kivi_us, 1), "pages": complete_heads, "bits": args.kivi or 4,
            "v_group": 32, "bytes": kivi_bytes,
            "GBps": round(kivi_bytes / (kivi_us * 1e-6) / 1e9, 1)},
        "gen_s": round(t_gen, 1),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, cfg, sample_pages=8192)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
