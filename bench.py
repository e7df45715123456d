"""Throughput of hierarchical transition-attended retrieval on one MI355X.

One step = one batch of queries through the whole retrieval path on the GPU:
coarse scoring and top-c selection (htam_retrieve_coarse), the bank stream
over the selected clusters' segments with softmax statistics and per-slot
top-k (htam_attend_transitions), and the final merge into the top-k memories
and their weights (htam_topk). Inputs (bank, queries) are resident in HBM
before the timed region; the bank build is offline and untimed.

The default workload is the largest that fits one GPU: 8,192 queries of
d = 2,048 against 16,384 clusters and 4,194,304 fp32 records (a 34 GB bank,
far beyond the last-level cache, so every step streams it from HBM). A bank
that would fit the 256 MB last-level cache is timed over copies of itself
that together exceed 1 GiB, one per step in turn (--no-rotate: one bank).
The bank also carries its keys in the tiled order that the bank stream reads
(htam_memory_tile) and, for fp32 banks, its coarse keys rounded to bf16
(htam_coarse_keys_bf16), both built with the bank, untimed (--no-tiled:
neither).

Prints one JSON line: queries/s for the workload (whole timed region), the
roofline position of the dominant kernel (the bank stream, HBM-bound),
measured with HIP events stamped at that kernel's start and end by its own
dispatch inside the timed region, the median step time and per-stage times
(coarse GEMM + selection, routing, stream, merges, final top-k; stage and
kernel events on every --event-every-th step: markers between calls cost
the small workloads a few microseconds per step), and the CPU oracle timed
on a seeded 256-query sample of the same workload on the host's cores.

Other paths (--path): prefix-aware coarse scoring, flat retrieval over every
record, and the online update (main + delta retrieval, compaction, feedback
statistics); each reports the roofline of the kernel it adds.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--path P] [--gpus 1]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "retrieval queries/sec at fixed bank size; % HBM roofline and % MFMA peak"
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
# the largest single-GPU workload: 8,192 queries, d = 2,048, 16,384 clusters,
# 4,194,304 fp32 records (34.4 GB, far beyond the 256 MB last-level cache, so
# every step streams the bank from HBM)
DEFAULT_WORKLOAD = "before_after_f32"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# Sources of the bank-stream kernels and their launch (counter figures of the
# stream stay valid while these are unchanged).
STREAM_SOURCES = ("dev.hpp", "internal.hpp", "stream.hpp", "stream_lds_bf16.hip",
                  "stream_lds_f32.hip", "stream_generic.hip", "fine.hip")


def kernel_source_sha256(names=None) -> str:
    """Hash of the library's device and host sources (all of them, or the
    named files): a changed kernel invalidates counter figures taken from an
    older build."""
    csrc = os.path.join(ROOT, "paper_2605_29734_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".hpp", ".cpp", ".h")) and (names is None or name in names):
            h.update(name.encode())
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()


def stream_kernel_traffic(workload: str):
    """Measured HBM bytes per launch of the bank-stream kernel (FETCH_SIZE +
    WRITE_SIZE, scaled by the same counters' reading for a plain copy of known
    size) from the committed rocprofv3 counter summary; None unless that
    summary was taken from the current sources of the stream kernels."""
    path = os.path.join(ROOT, "profiles", "fine_stream_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
        if rec.get("source_sha256") != kernel_source_sha256(STREAM_SOURCES):
            return None
        return rec.get("workloads", {}).get(workload, {}).get("bytes_per_launch")
    except (OSError, ValueError, AttributeError):
        return None


def copy_calibration(mib: int, launches: int = 5):
    """Plain streaming copies of known size, the reference reading for the
    FETCH_SIZE / WRITE_SIZE counters: each launch of the elementwise kernel
    reads ``mib`` MiB once and writes ``mib`` MiB once (a kernel, not a DMA
    transfer, so that the counters see it)."""
    import torch
    n = mib << 20
    src = torch.full((n // 4,), 1.0, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(launches):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": n, "launches": launches}), flush=True)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(spec, w, bank, target_s: float):
    """Time the CPU oracle on a seeded uniform sample of 256 of the workload's
    queries (all of them when there are fewer): coarse scores over every
    cluster, selection, and the fine stage over the selected segments. Rows
    are independent, so queries/s on the sample is the oracle's rate on the
    workload. Host copies of the touched segments are made before the clock
    starts."""
    import oracle
    cores = int(os.environ.get("OMP_NUM_THREADS") or len(os.sched_getaffinity(0)))
    q = w.queries.float().cpu().numpy()
    c = w.coarse_keys.float().cpu().numpy()
    off = bank.seg_offsets.cpu().numpy()
    tid = bank.transition_id.cpu().numpy()
    n_rows = min(spec.B, 256)
    rows = np.sort(np.random.default_rng(0).choice(spec.B, size=n_rows, replace=False))
    qh = oracle.round_bf16(q[rows]) if spec.compute == "bf16" else q[rows]
    ch = oracle.round_bf16(c) if spec.compute == "bf16" else c
    sel, _ = oracle.coarse(qh, ch, spec.top_c)
    touched = np.unique(sel)
    seg = {}
    for g in touched:                      # host copies of the touched segments, untimed
        a, b = int(off[g]), int(off[g + 1])
        seg[int(g)] = (a, bank.fine_keys[a:b].float().cpu().numpy())


    def fetch(a, b):
        g = int(np.searchsorted(off, a, side="right") - 1)
        s0, arr = seg[g]
        return arr[a - s0:b - s0]

    done, t0 = 0, time.perf_counter()
    while True:
        oracle.retrieve(q, c, off, spec.top_c, spec.top_k, spec.tau, spec.compute,
                        fetch_keys=fetch, transition_id=tid, rows=rows)
        done += rows.size
        el = time.perf_counter() - t0
        if el >= target_s:
            break
    return {"value": done / el, "unit": "queries/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{rows.size} of {spec.B} queries (seeded uniform subset) x "
                      f"{done // rows.size} passes ({el:.1f} s; coarse scores over all {spec.G} "
                      f"clusters, fine stage over the selected segments, fp64)"}


def bench_alt(args, spec, w, bank):
    """The flat path (htam_retrieve_flat: every record a candidate) or the
    prefix path (htam_retrieve_coarse_prefix, then the fine stage and the
    merge), timed like the hierarchical step. Roofline: the flat path is the
    dense B x N score GEMM (MFMA-bound; the whole step against the bf16 peak);
    the prefix path's added kernel is the grouped edge-score GEMM, which reads
    each used source node's edge slice once (HBM-bound at these shapes)."""
    import torch
    from paper_2605_29734_amd import htam, synth
    q = w.queries
    dev = q.device
    kc = htam.HTAM_KERNEL_COARSE
    mk = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    K, E = args.steps, max(1, args.event_every)
    if args.path == "flat":
        out = (torch.empty(spec.B, spec.top_k, dtype=torch.int32, device=dev),
               torch.empty(spec.B, spec.top_k, device=dev), torch.empty(spec.B, spec.top_k, device=dev),
               torch.empty(spec.B, device=dev), torch.empty(spec.B, device=dev),
               torch.empty(spec.B, dtype=torch.int32, device=dev))
        ws = htam._workspace(htam.lib.htam_retrieve_flat_workspace_size(
            htam.ctypes.byref(bank.struct), spec.B, spec.top_k), dev)

        def step(i, marks):
            marks[i][0].record()
            htam.htam_retrieve_flat(bank, q, spec.tau, spec.top_k, out=out, ws=ws)
    else:
        edges, prefix = synth.make_prefix(spec, w.coarse_keys, args.prefix_len, device=dev,
                                          seed=args.seed)
        r = htam.Retriever(bank, spec.B, spec.top_c, spec.top_k, spec.tau)
        wsp = htam._workspace(htam.lib.htam_retrieve_coarse_prefix_workspace_size(
            htam.ctypes.byref(bank.struct), spec.B, args.prefix_len, spec.top_c), dev)

        def step(i, marks):
            marks[i][0].record()
            htam.htam_retrieve_coarse_prefix(bank, edges, prefix, args.lam, q, spec.top_c,
                                             out=r.sel, ws=wsp)
            marks[i][1].record()
            htam.htam_attend_transitions(bank, q, r.sel[0], r.tau, r.k, out=r.slots, ws=r.ws_attend)
            htam.htam_topk(r.slots[2], r.slots[3], r.k, r.slots[0], r.slots[1], r.tau, out=r.rows,
                           sorted_lists=True)
    marks = [[mk(), mk()] for _ in range(K)] + [[mk()]]
    ev = [(mk(), mk()) for _ in range((K + E - 1) // E)]
    for a, b in ev:
        a.record()
        b.record()
    for i in range(args.warmup):
        step(0, marks)
    torch.cuda.synchronize()
    log(f"[bench] timing {K} steps ({args.path})")
    t0 = time.perf_counter()
    for i in range(K):
        if i % E == 0:
            htam.lib.htam_set_kernel_events(kc, ev[i // E][0].cuda_event, ev[i // E][1].cuda_event)
        elif i % E == 1:
            htam.lib.htam_set_kernel_events(kc, None, None)
        step(i, marks)
    marks[K][0].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    htam.lib.htam_set_kernel_events(kc, None, None)
    ms_total = marks[0][0].elapsed_time(marks[K][0])
    step_ms = [marks[i][0].elapsed_time(marks[i + 1][0]) for i in range(K)]
    t_kernel = float(np.mean([a.elapsed_time(b) for a, b in ev])) * 1e-3
    kb = bank.fine_keys.element_size()
    res = {
        "metric": METRIC, "value": spec.B * K / (ms_total * 1e-3), "unit": "queries/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": ms_total / K,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if spec.compute == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": spec.name, "path": args.path, "queries": spec.B, "d": spec.d,
                   "clusters": spec.G, "transitions": spec.N, "top_c": spec.top_c,
                   "top_k": spec.top_k, "tau": spec.tau, "key_storage": spec.storage,
                   "bank_bytes": int(spec.N * spec.d * kb)},
        "stages": {"step_ms_median": float(np.median(step_ms)), "step_ms_wall": wall / K * 1e3,
                   "source_sha256": kernel_source_sha256()},
    }
    if args.path == "flat":
        flops = 2.0 * spec.B * spec.N * spec.d
        t_step = ms_total / K * 1e-3
        res["roofline"] = {"bound": "mfma", "kernel": "flat retrieval step (score GEMM, "
                           "segmented top-k, merge)", "achieved": flops / t_step / 1e12,
                           "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                           "frac": flops / t_step / 1e12 / MFMA_BF16_PEAK_TFLOPS, "traffic": None,
                           "flops_per_step": flops}
        res["stages"]["score_gemm_ms_last_band"] = t_kernel * 1e3
    else:
        P = prefix.cpu().numpy()
        G = spec.G
        valid = np.cumprod((P >= 0) & (P < G), axis=1).astype(bool)
        n_pairs = int(valid.sum())
        n_src = int(np.unique(P[valid]).size)
        eb = edges.element_size()
        alg = n_src * G * spec.d * eb + spec.B * spec.d * q.element_size()
        res["roofline"] = {"bound": "hbm", "kernel": "prefix_gemm (edge scores)",
                           "achieved": alg / t_kernel / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": alg / t_kernel / 1e9 / HBM_PEAK_GBS, "traffic": None,
                           "alg_bytes_per_launch": alg, "launch_ms": t_kernel * 1e3}
        coarse_ms = [marks[i][0].elapsed_time(marks[i][1]) for i in range(K)]
        res["stages"].update({"prefix_coarse_stage_ms_median": float(np.median(coarse_ms)),
                              "prefix_pairs": n_pairs, "prefix_sources": n_src,
                              "prefix_edge_tflops": 2.0 * n_pairs * G * spec.d / t_kernel / 1e12,
                              "prefix_len_max": args.prefix_len, "lambda": args.lam})
    return res


def bench_update(args, spec, w):
    """The online update. The records are split in arrival order into a main
    bank and a delta bank of recent ones (--delta-frac); the timed step is
    retrieval over both banks (what queries see between compactions). Also
    timed: the compaction of the delta into the main bank (htam_memory_merge,
    HBM-bound: every key row read and written once, the roofline here), the
    feedback statistics of 2^20 step outcomes, and the rule-based direction
    scores over them."""
    import torch
    from paper_2605_29734_amd import htam
    q = w.queries
    dev = q.device
    n_main = int(spec.N * (1.0 - args.delta_frac))
    main = htam.build_bank(w.cluster_of[:n_main].contiguous(), w.keys_in[:n_main].contiguous(),
                           w.coarse_keys, spec.compute)
    delta = htam.build_bank(w.cluster_of[n_main:].contiguous(), w.keys_in[n_main:].contiguous(),
                            w.coarse_keys, spec.compute)
    delta.transition_id += n_main
    del w.keys_in
    torch.cuda.synchronize()
    mk = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    K = args.steps
    for _ in range(args.warmup):
        htam.retrieve_two_banks(main, delta, q, spec.top_c, spec.top_k, spec.tau)
    torch.cuda.synchronize()
    log(f"[bench] timing {K} steps (update: main + delta retrieval)")
    e0, e1 = mk(), mk()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(K):
        htam.retrieve_two_banks(main, delta, q, spec.top_c, spec.top_k, spec.tau)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = e0.elapsed_time(e1)
    # compaction
    merged = htam.htam_memory_merge(main, delta)
    torch.cuda.synchronize()
    reps = 5
    e0.record()
    for _ in range(reps):
        merged = htam.htam_memory_merge(main, delta)
    e1.record()
    torch.cuda.synchronize()
    t_merge = e0.elapsed_time(e1) / reps * 1e-3
    kb = main.fine_keys.element_size()
    merge_bytes = 2 * spec.N * (spec.d * kb + 4) + 16 * (spec.G + 1)
    # statistics: 2^20 outcomes over the bank's clusters (4 state buckets), then
    # scores for every query over prefixes of up to 5 directions
    G, NB, n_ev = min(spec.G, 1024), 4, 1 << 20
    gen = torch.Generator(device=dev).manual_seed(args.seed)
    src = torch.randint(-1, G, (n_ev,), dtype=torch.int32, device=dev, generator=gen)
    dst = torch.randint(0, G, (n_ev,), dtype=torch.int32, device=dev, generator=gen)
    bk = torch.randint(0, NB, (n_ev,), dtype=torch.int32, device=dev, generator=gen)
    feat = torch.rand(n_ev, htam.HTAM_FEEDBACK_FEATURES, device=dev, generator=gen)
    st = htam.empty_stats(G, NB, dev)
    htam.htam_feedback_update(st, src, dst, bk, feat)
    torch.cuda.synchronize()
    e0.record()
    htam.htam_feedback_update(st, src, dst, bk, feat)
    e1.record()
    torch.cuda.synchronize()
    t_fb = e0.elapsed_time(e1) * 1e-3
    P = torch.randint(-1, G, (spec.B, 5), dtype=torch.int32, device=dev, generator=gen)
    qb = torch.randint(0, NB, (spec.B,), dtype=torch.int32, device=dev, generator=gen)
    wv = torch.randn(htam.HTAM_STATS_WORDS, device=dev, generator=gen)
    S = htam.htam_transition_scores(st, P, qb, 0.5, wv, 8)
    torch.cuda.synchronize()
    e0.record()
    htam.htam_transition_scores(st, P, qb, 0.5, wv, 8, out=S)
    e1.record()
    torch.cuda.synchronize()
    t_ts = e0.elapsed_time(e1) * 1e-3
    achieved = merge_bytes / t_merge / 1e9
    return {
        "metric": METRIC, "value": spec.B * K / (ms_total * 1e-3), "unit": "queries/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": ms_total / K,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if spec.compute == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": spec.name, "path": "update", "queries": spec.B, "d": spec.d,
                   "clusters": spec.G, "transitions": spec.N, "delta_records": spec.N - n_main,
                   "top_c": spec.top_c, "top_k": spec.top_k, "tau": spec.tau,
                   "key_storage": spec.storage},
        "roofline": {"bound": "hbm", "kernel": "htam_memory_merge (compaction)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "alg_bytes_per_launch": merge_bytes, "launch_ms": t_merge * 1e3},
        "stages": {"step_ms_wall": wall / K * 1e3, "merge_ms": t_merge * 1e3,
                   "feedback_events_per_s": n_ev / t_fb, "feedback_ms_per_2^20_events": t_fb * 1e3,
                   "transition_scores_ms": t_ts * 1e3, "stats_clusters": G, "stats_buckets": NB,
                   "source_sha256": kernel_source_sha256()},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-rotate", action="store_true",
                    help="time one bank even when it fits the last-level cache")
    ap.add_argument("--no-tiled", action="store_true",
                    help="no prepared copies: the stream reads the row-major keys and the "
                         "coarse scoring rounds fp32 coarse keys on every call")
    ap.add_argument("--event-every", type=int, default=4, metavar="E",
                    help="stamp the kernel and stage timing events on every E-th timed step")
    ap.add_argument("--path", default="hierarchical",
                    choices=["hierarchical", "prefix", "flat", "update"],
                    help="hierarchical retrieval (default); the same with prefix-aware coarse "
                         "scoring; flat retrieval over every record; or the online update "
                         "(retrieval over a main and a delta bank, compaction, statistics)")
    ap.add_argument("--delta-frac", type=float, default=0.01,
                    help="update path: share of the records in the delta bank")
    ap.add_argument("--prefix-len", type=int, default=5, metavar="L",
                    help="prefix path: longest prefix (lengths uniform on 0..L)")
    ap.add_argument("--lam", type=float, default=0.5, help="prefix path: recency decay lambda")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run plain copies of MIB MiB (counter calibration) and exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU; runs over several GPUs are not supported "
              "(one process per GPU, each streaming its own shard of the clusters, is the "
              "intended split)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return

    import torch

    from paper_2605_29734_amd import htam, synth
    spec = synth.SPECS[args.workload]
    dev = torch.device("cuda:0")
    log(f"[bench] workload {spec.name}: generating on {dev}")
    w = synth.make(spec, device=dev, seed=args.seed)
    bank = None
    if args.path != "update":
        bank = htam.build_bank(w.cluster_of, w.keys_in, w.coarse_keys, spec.compute)
        torch.cuda.synchronize()
        del w.keys_in
    q = w.queries
    if args.path == "update":
        res = bench_update(args, spec, w)
        print(json.dumps(res), flush=True)
        return
    if args.path != "hierarchical":
        res = bench_alt(args, spec, w, bank)
        print(json.dumps(res), flush=True)
        return
    r = htam.Retriever(bank, spec.B, spec.top_c, spec.top_k, spec.tau)
    # A bank smaller than the last-level cache (256 MB Infinity Cache) would be
    # read from the cache on every step after the first: rotate over copies
    # of it that together exceed 1 GiB, so that each step reads its bank from
    # HBM (the workspaces fit any copy: same shapes).
    bank_bytes = bank.fine_keys.numel() * bank.fine_keys.element_size()
    n_copies = 1 if args.no_rotate else min(32, max(1, -(-(1 << 30) // max(bank_bytes, 1))))
    banks = [bank] + [htam.Bank(coarse_keys=bank.coarse_keys.clone(),
                                fine_keys=bank.fine_keys.clone(), seg_offsets=bank.seg_offsets,
                                transition_id=bank.transition_id, compute=bank.compute)
                      for _ in range(n_copies - 1)]
    if n_copies > 1:
        log(f"[bench] rotating over {n_copies} copies of the {bank_bytes / 2**20:.0f} MiB bank")
    # the copies built with the bank, untimed: the fine keys in the tiled
    # order of htam_memory_tile (the bank stream reads 1 KB of consecutive
    # bytes per load) and fp32 coarse keys rounded to bf16 once
    tiled = not args.no_tiled and spec.d % 32 == 0
    if not args.no_tiled:
        banks = [htam.prepared(b) for b in banks]
        torch.cuda.synchronize()
    r.bank = banks[0]
    log(f"[bench] warmup {args.warmup}")
    for i in range(max(args.warmup, n_copies)):
        r.bank = banks[i % n_copies]
        r.run(q)
    torch.cuda.synchronize()

    K = args.steps
    E = max(1, args.event_every)
    n_ev = (K + E - 1) // E              # timed steps i with i % E == 0
    mk = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    ev_s = [(mk(), mk()) for _ in range(n_ev)]
    ev_c = [(mk(), mk()) for _ in range(n_ev)]
    # per step: start, coarse done, attend done, end (= the next step's start)
    marks = [[mk() for _ in range(3)] for _ in range(K)] + [[mk()]]
    for a, b in ev_s + ev_c:        # materialise the events before handing them to the library
        a.record()
        b.record()
    torch.cuda.synchronize()
    lib, ks, kc = htam.lib, htam.HTAM_KERNEL_STREAM, htam.HTAM_KERNEL_COARSE
    log(f"[bench] timing {K} steps")
    t0 = time.perf_counter()
    for i in range(K):
        if i % E == 0:
            j = i // E
            lib.htam_set_kernel_events(ks, ev_s[j][0].cuda_event, ev_s[j][1].cuda_event)
            lib.htam_set_kernel_events(kc, ev_c[j][0].cuda_event, ev_c[j][1].cuda_event)
        elif i % E == 1:
            lib.htam_set_kernel_events(ks, None, None)
            lib.htam_set_kernel_events(kc, None, None)
        # stage boundaries on the stamped steps only: on the small workloads
        # every marker between calls shows in the step time
        stamped = i % E == 0
        bk = banks[i % n_copies]
        marks[i][0].record()
        htam.htam_retrieve_coarse(bk, q, r.c, out=r.sel, ws=r.ws_coarse)
        if stamped:
            marks[i][1].record()
        htam.htam_attend_transitions(bk, q, r.sel[0], r.tau, r.k, out=r.slots, ws=r.ws_attend)
        if stamped:
            marks[i][2].record()
        htam.htam_topk(r.slots[2], r.slots[3], r.k, r.slots[0], r.slots[1], r.tau, out=r.rows,
                       sorted_lists=True)
    marks[K][0].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    lib.htam_set_kernel_events(ks, None, None)
    lib.htam_set_kernel_events(kc, None, None)
    step_ms = [marks[i][0].elapsed_time(marks[i + 1][0]) for i in range(K)]
    ms_total = marks[0][0].elapsed_time(marks[K][0])
    ms_step = ms_total / K
    med = lambda xs: float(np.median(xs))        # noqa: E731
    st_steps = range(0, K, E)
    coarse_stage = [marks[i][0].elapsed_time(marks[i][1]) for i in st_steps]
    attend_stage = [marks[i][1].elapsed_time(marks[i][2]) for i in st_steps]
    topk_stage = [marks[i][2].elapsed_time(marks[i + 1][0]) for i in st_steps]
    stream_ms = [a.elapsed_time(b) for a, b in ev_s]
    gemm_ms = [a.elapsed_time(b) for a, b in ev_c]
    # on the stamped steps: routing = attend start -> stream start, merges =
    # stream end -> attend end
    route_ms = [marks[j * E][1].elapsed_time(ev_s[j][0]) for j in range(n_ev)]
    merge_ms = [ev_s[j][1].elapsed_time(marks[j * E][2]) for j in range(n_ev)]
    t_stream = sum(stream_ms) / n_ev * 1e-3
    t_coarse = sum(gemm_ms) / n_ev * 1e-3
    t_coarse_stage = med(coarse_stage) * 1e-3

    # algorithmic bytes of one bank-stream launch: every row of every selected
    # segment read once, plus the queries
    sel = r.sel[0].cpu().numpy()
    off = bank.seg_offsets.cpu().numpy()
    kb = bank.fine_keys.element_size()
    touched = np.unique(sel)
    rows_touched = int((off[touched + 1] - off[touched]).sum())
    alg_bytes = rows_touched * spec.d * kb + spec.B * spec.d * q.element_size()
    achieved = alg_bytes / t_stream / 1e9
    coarse_flops = 2.0 * spec.B * spec.G * spec.d
    pairs = int((off[sel + 1] - off[sel]).sum())
    tflops = lambda t: coarse_flops / t / 1e12    # noqa: E731

    res = {
        "metric": METRIC,
        "value": spec.B * K / (ms_total * 1e-3),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if spec.compute == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": spec.name, "queries": spec.B, "d": spec.d, "clusters": spec.G,
                   "transitions": spec.N, "top_c": spec.top_c, "top_k": spec.top_k,
                   "tau": spec.tau, "key_storage": spec.storage,
                   "bank_bytes": int(spec.N * spec.d * kb), "bank_copies": n_copies,
                   "tiled_keys": tiled,
                   "coarse_keys_bf16": banks[0].coarse_keys_bf16 is not None},
        "roofline": {"bound": "hbm", "kernel": "fine_stream", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": stream_kernel_traffic(spec.name),
                     "alg_bytes_per_launch": alg_bytes, "launch_ms": t_stream * 1e3},
        "stages": {"step_ms_median": med(step_ms), "step_ms_min": min(step_ms),
                   "step_ms_wall": wall / K * 1e3,
                   "coarse_stage_ms_median": med(coarse_stage),
                   "coarse_stage_mfma_frac": tflops(t_coarse_stage) / MFMA_BF16_PEAK_TFLOPS,
                   "coarse_gemm_ms": t_coarse * 1e3,
                   "coarse_gemm_mfma_frac": tflops(t_coarse) / MFMA_BF16_PEAK_TFLOPS,
                   "attend_stage_ms_median": med(attend_stage),
                   "route_ms_median": med(route_ms),
                   "fine_stream_ms": t_stream * 1e3,
                   "fine_stream_hbm_frac": achieved / HBM_PEAK_GBS,
                   "slot_merge_ms_median": med(merge_ms),
                   "final_topk_ms_median": med(topk_stage),
                   "scored_pairs_per_step": pairs,
                   "kernel_timed_steps": n_ev,
                   "source_sha256": kernel_source_sha256()},
    }
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline")
        res["cpu_baseline"] = cpu_baseline(spec, w, bank, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
