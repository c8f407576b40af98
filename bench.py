"""Benchmark of the WARP search path on one MI355X.

A step is one batched search (centroid filter GEMM, selection, plan, residual
scan, document fold, top-k) of the workload's whole query batch, with the
index and the queries already resident in HBM. Prints one JSON line. The
default workload is the full-scale one (8.8M passages, about 600M embeddings,
b = 2, 4,096 queries of 32 tokens, nprobe 32, k = 1000).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

METRIC = "queries/s, p50 query latency, scored embeddings/s (% of HBM peak BW)"
HBM_PEAK_GBS = 8000.0
FP16_MFMA_PEAK_TFLOPS = 2500.0  # dense fp16 matrix-core peak of the MI355X
INT8_MFMA_PEAK_TOPS = 5000.0
CSRC = os.path.join(ROOT, "paper_2501_17788_amd", "csrc")
TRAFFIC_TABLE = os.path.join(ROOT, "profiles", "traffic.md")


def csrc_hash() -> str:
    """Hash of the engine sources: counter figures are used only for the code they measured."""
    import hashlib

    h = hashlib.sha1()
    for name in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch (FETCH_SIZE x 2 + WRITE_SIZE x 1, calibrated on a copy kernel)
    recorded in profiles/traffic.md for these exact sources, else None."""
    try:
        rows = open(TRAFFIC_TABLE).read().splitlines()
    except OSError:
        return None
    h = csrc_hash()
    for line in rows:
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 5 and cells[0] == kernel and cells[1] == workload and cells[2] == h:
            try:
                return float(cells[3]) + float(cells[4])
            except ValueError:
                return None
    return None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model() -> str:
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True).stdout
        for line in out.splitlines():
            if line.startswith("Model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def host_threads() -> int:
    """Host threads for the generator and the oracle: the CPUs this process may run on, at
    most 16 (a one-GPU share of the host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def describe(wl) -> str:
    lens = (f"U[{int(wl.len_a)},{int(wl.len_b)}]" if wl.len_kind == "uniform"
            else f"lognormal mean {wl.len_a:g} cap {int(wl.len_b)}")
    return (f"{wl.name}: {wl.n_docs} docs ({lens} tokens), {wl.n_centroids} centroids, Zipf {wl.zipf_s}, "
            f"b={wl.nbits}, {wl.n_queries} queries x {wl.n_qtok} tokens, nprobe={wl.nprobe}, "
            f"t'={wl.t_prime}, k={wl.k}")


def recall_study(args) -> int:
    """The hyperparameter study of Section 4.6 on synthetic data: nRecall@k of the engine's top-k
    against exhaustive MaxSim over the uncompressed fp32 token vectors, as nprobe, t' and b vary,
    plus the rank of each query's target document. Prints a markdown table (and writes JSON)."""
    import torch

    import synth
    from paper_2501_17788_amd import Index, t_prime_policy

    base = synth.with_overrides(synth.WORKLOADS[args.workload], query_noise=args.query_noise)
    dev = torch.device("cuda:0")
    data = {}
    for b in (4, 2):
        t0 = time.time()
        data[b] = synth.make_index(synth.with_overrides(base, nbits=b), workers=min(16, host_threads()))
        log(f"recall: generated b={b} index in {time.time() - t0:.1f} s")
    ref = data[4]
    assert np.array_equal(ref.queries, data[2].queries)
    lens = ref.doc_lengths.astype(np.int64)
    n_docs, L = len(lens), int(lens.max())
    N = int(lens.sum())
    t0 = time.time()
    X = torch.from_numpy(synth.token_vectors(ref.workload, np.arange(N))).to(dev)
    log(f"recall: regenerated {N} token vectors in {time.time() - t0:.1f} s")
    # documents padded to L tokens; padding rows score -inf
    starts = np.zeros(n_docs + 1, np.int64)
    np.cumsum(lens, out=starts[1:])
    doc_of = np.repeat(np.arange(n_docs), lens)
    slot = torch.from_numpy(doc_of * L + (np.arange(N) - starts[doc_of])).to(dev)
    pad = torch.zeros(n_docs * L, 128, device=dev)
    pad[slot] = X
    del X
    valid = torch.zeros(n_docs * L, dtype=torch.bool, device=dev)
    valid[slot] = True
    valid = valid.view(n_docs, L, 1)
    Q = torch.from_numpy(ref.queries).to(dev)  # [nq, T, 128]
    nq, T = Q.shape[0], Q.shape[1]
    kmax = 100
    exh = []
    qc = max(1, 256 // T)
    for q0 in range(0, nq, qc):
        qq = Q[q0:q0 + qc].reshape(-1, 128)
        S = (pad @ qq.T).view(n_docs, L, -1).masked_fill(~valid, float("-inf")).amax(dim=1)
        scores = S.view(n_docs, -1, T).sum(dim=2)  # [n_docs, queries of the chunk]
        exh.append(torch.topk(scores.T, kmax, dim=1).indices.cpu().numpy())
    exh = np.concatenate(exh)
    log("recall: exhaustive MaxSim done")
    targets = ref.query_targets
    tp_policy = t_prime_policy(N)
    rows = []
    for b in (4, 2):
        ix = Index.from_synthetic(data[b])
        for nprobe in (1, 2, 4, 8, 16, 32, 64):
            log(f"recall: b={b} nprobe={nprobe}")
            for tp in sorted({1_000, 10_000, tp_policy, 100_000, 400_000}):
                ids = ix.search(data[b].queries, nprobe, tp, kmax)[0]
                r10 = np.mean([len(set(ids[i, :10]) & set(exh[i, :10])) / 10 for i in range(nq)])
                r100 = np.mean([len(set(ids[i]) & set(exh[i])) / 100 for i in range(nq)])
                s1 = float(np.mean(ids[:, 0] == targets))
                s10 = float(np.mean([targets[i] in ids[i, :10] for i in range(nq)]))
                rows.append({"b": b, "nprobe": nprobe, "t_prime": tp, "nrecall10": r10, "nrecall100": r100,
                             "target_at_1": s1, "target_in_10": s10})
        ix.close()
    ex1 = float(np.mean(exh[:, 0] == targets))
    print(f"| b | nprobe | t' | nRecall@10 | nRecall@100 | target at 1 | target in top 10 |")
    print("|---|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['b']} | {r['nprobe']} | {r['t_prime']:,} | {r['nrecall10']:.3f} | {r['nrecall100']:.3f} | "
              f"{r['target_at_1']:.3f} | {r['target_in_10']:.3f} |")
    print(f"\nquery noise {args.query_noise}: exhaustive MaxSim over the uncompressed vectors ranks the target "
          f"first for {ex1:.3f} of {nq} queries; t' policy value {tp_policy:,}")
    if args.recall_out:
        with open(args.recall_out, "w") as f:
            json.dump({"workload": describe(base), "rows": rows, "exhaustive_target_at_1": ex1,
                       "t_prime_policy": tp_policy}, f)
    return 0


def build_bench(args) -> int:
    """Index construction on the device (Section 4.1) for the workload's tokens: k-means on a passage
    sample proportional to sqrt(n_docs), assignment, quantiles, codes. Prints one JSON line."""
    import torch

    import synth
    import paper_2501_17788_amd as w

    wl = synth.with_overrides(synth.WORKLOADS[args.workload], nbits=args.build_nbits)
    data = synth.make_index(wl, with_queries=True, workers=min(16, host_threads()))
    lens = data.doc_lengths.astype(np.int64)
    N = int(lens.sum())
    t0 = time.time()
    X = torch.from_numpy(synth.token_vectors(wl, np.arange(N))).cuda()
    docs = torch.from_numpy(np.repeat(np.arange(len(lens)), lens).astype(np.int32)).cuda()
    log(f"build: {N} tokens regenerated in {time.time() - t0:.1f} s")
    sample = w.sample_passages(lens, c=16.0, seed=0)
    C0 = w.initial_centroids(X, sample, wl.n_centroids, seed=0)
    n_quant = min(N, 1 << 16)
    times = {}
    for it in (0, args.build_iterations):  # the difference isolates the k-means steps
        torch.cuda.synchronize()
        a = time.perf_counter()
        built = w.build_index(X, docs, len(lens), C0, sample, it, wl.nbits, n_quant)
        torch.cuda.synchronize()
        times[it] = time.perf_counter() - a
        log(f"build: {it} k-means steps: {times[it]:.2f} s")
    with w.Index.from_device(built["centroids"], built["offsets"], built["doc_ids"], built["codes"], wl.nbits,
                             built["weights"], len(lens)) as ix:
        ids = ix.search(data.queries, wl.nprobe, wl.t_prime, wl.k)[0]
    hit = float(np.mean(ids[:, 0] == data.query_targets))
    rec = {"mode": "index construction", "workload": describe(wl), "n_tokens": N, "n_centroids": wl.n_centroids,
           "sample_tokens": int(len(sample)), "iterations": args.build_iterations, "n_quant_tokens": n_quant,
           "seconds_total": times[args.build_iterations], "seconds_without_kmeans": times[0],
           "seconds_per_kmeans_step": (times[args.build_iterations] - times[0]) / max(1, args.build_iterations),
           "tokens_per_s_encode": N / times[0], "target_first_after_search": hit}
    print(json.dumps(rec), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    help="tiny, small, mid, long or full (default: full, the largest, at nprobe 32; "
                         "small for --recall-study and --build)")
    ap.add_argument("--nprobe", type=int, default=0, help="override the workload's nprobe (the full workload "
                                                            "is also measured at 16 and 64)")
    ap.add_argument("--latency-runs", type=int, default=200)
    ap.add_argument("--cpu-queries", type=int, default=2, help="queries the oracle runs on all host threads")
    ap.add_argument("--cpu1-tokens", type=int, default=4,
                    help="tokens of query 0 the oracle runs on one thread (scaled to a query)")
    ap.add_argument("--host-steps", type=int, default=2, help="batches through the blocking host-pointer call")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy a buffer of this size 3 times on the device (a kernel of "
                         "known traffic to scale HBM counters against)")
    ap.add_argument("--recall-study", action="store_true",
                    help="instead of the benchmark, run the nprobe / t' / b recall study (Section 4.6)")
    ap.add_argument("--recall-out", default="", help="JSON output of the recall study")
    ap.add_argument("--build", action="store_true", help="instead of the benchmark, time index construction")
    ap.add_argument("--build-iterations", type=int, default=8)
    ap.add_argument("--build-nbits", type=int, default=4)
    ap.add_argument("--query-noise", type=float, default=0.05,
                    help="recall study: per-component noise of the query tokens around their document's tokens")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the search path has no multi-GPU mode (--gpus {args.gpus} "
              f"requested). Run with --gpus 1.", file=sys.stderr)
        return 2

    if args.workload is None:
        args.workload = "small" if (args.recall_study or args.build) else "full"
    if args.recall_study:
        return recall_study(args)
    if args.build:
        return build_bench(args)

    import torch

    import synth
    from paper_2501_17788_amd import Index

    wl = synth.WORKLOADS[args.workload]
    if args.nprobe:
        wl = synth.with_overrides(wl, nprobe=args.nprobe)
    log(f"bench: generating {describe(wl)}")
    t0 = time.time()
    data = synth.make_index(wl, workers=min(16, host_threads()))
    log(f"bench: {data.n_embeddings} embeddings in {time.time() - t0:.1f} s")
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    t0 = time.time()
    ix = Index.from_synthetic(data)
    log(f"bench: index loaded in {time.time() - t0:.1f} s")
    q = torch.from_numpy(data.queries).to(dev)
    nq = wl.n_queries

    # scored embeddings per query (exact, from the engine's own counters) and the probed
    # clusters, from a debug search of the same batch
    dbg = ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k, bitmap=False)
    scored = dbg["n_scored"].astype(np.int64)
    row_bytes = 128 * wl.nbits // 8 + 4

    out = None
    for _ in range(args.warmup):
        out = ix.search_async(q, wl.nprobe, wl.t_prime, wl.k, out=out)
    ix.sync()
    log(f"bench: warmup done ({args.warmup} steps)")

    ix.set_timing(True)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        out = ix.search_async(q, wl.nprobe, wl.t_prime, wl.k, out=out)
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    ix.sync()  # settles the per-stage event timings
    stages = ix.stage_timings()
    ix.set_timing(False)
    elapsed = t_end - t_start
    ms_step = elapsed * 1e3 / args.steps
    qps = nq * args.steps / elapsed
    log(f"bench: {args.steps} steps in {elapsed:.3f} s -> {qps:.1f} queries/s")
    # the timed batch agrees with the debug run
    ids = out[0].cpu().numpy()
    same_as_debug = bool(np.array_equal(ids, dbg["ids"]))

    # the blocking host-pointer call: the host's query check and the host <-> device copies
    # of queries and results included (a few batches: not the headline figure)
    host_steps = max(1, min(args.steps, args.host_steps))
    ix.search(data.queries, wl.nprobe, wl.t_prime, wl.k)
    a = time.perf_counter()
    for _ in range(host_steps):
        ix.search(data.queries, wl.nprobe, wl.t_prime, wl.k)
    host_qps = nq * host_steps / (time.perf_counter() - a)
    log(f"bench: blocking host-pointer searches {host_qps:.1f} queries/s ({host_steps} batches)")

    # batch-1 latency
    lat = []
    q1 = [q[i:i + 1].contiguous() for i in range(min(nq, 16))]
    out1 = None
    for i in range(5):
        out1 = ix.search_async(q1[i % len(q1)], wl.nprobe, wl.t_prime, wl.k, out=out1)
    torch.cuda.synchronize()
    for i in range(args.latency_runs):
        a = time.perf_counter()
        out1 = ix.search_async(q1[i % len(q1)], wl.nprobe, wl.t_prime, wl.k, out=out1)
        torch.cuda.synchronize()
        lat.append((time.perf_counter() - a) * 1e3)
    p50, p99 = float(np.percentile(lat, 50)), float(np.percentile(lat, 99))
    log(f"bench: batch-1 latency p50 {p50:.3f} ms p99 {p99:.3f} ms")
    ix.close()

    # roofline of the dominant kernel: the residual scan
    scan_ms, scan_n = stages["scan"]
    scan_avg_s = scan_ms / 1e3 / max(scan_n, 1)
    launches_per_step = max(scan_n, 1) / args.steps
    pairs_per_launch = float(scored.sum()) / launches_per_step  # scored (token, embedding) pairs
    hbm_equiv = pairs_per_launch * row_bytes / scan_avg_s / 1e9  # 16b + 4 bytes per scored pair
    # distinct probed embeddings per launch: each probed cluster is read once per wave
    sizes = np.diff(data.offsets)
    waves = max(1, int(round(launches_per_step)))
    per_wave = -(-nq // waves)
    distinct = sum(int(sizes[np.unique(dbg["sel"][w0:w0 + per_wave])].sum()) for w0 in range(0, nq, per_wave))
    distinct_per_launch = distinct / waves  # waves taken as equal slices of the batch (an estimate)
    # a traffic row is keyed by the workload as configured (nprobe overrides get their own key)
    traffic_key = wl.name if wl.nprobe == synth.WORKLOADS[wl.name].nprobe else f"{wl.name}:nprobe{wl.nprobe}"
    traffic = measured_traffic("k_scan_mx", traffic_key)
    counted_gbs = None if traffic is None else traffic / scan_avg_s / 1e9
    roofline = {
        "bound": "hbm", "kernel": "k_scan_mx", "unit": "GB/s", "peak": HBM_PEAK_GBS,
        "achieved": counted_gbs, "frac": None if counted_gbs is None else counted_gbs / HBM_PEAK_GBS,
        "traffic": traffic, "avg_launch_ms": scan_avg_s * 1e3, "launches_per_step": launches_per_step,
        "basis": "HBM bytes per launch counted by rocprofv3 (FETCH_SIZE x 2 + WRITE_SIZE, calibrated on a "
                 "device copy; profiles/traffic.md, valid for these sources only) / average launch time "
                 "from HIP events on the search stream",
        "min_read": {"bytes_per_launch": distinct_per_launch * row_bytes,
                     "GBps": distinct_per_launch * row_bytes / scan_avg_s / 1e9,
                     "frac": distinct_per_launch * row_bytes / scan_avg_s / 1e9 / HBM_PEAK_GBS,
                     "what": "codes and document ids of every distinct probed embedding, read once per "
                             "launch (the least a cluster-major scan reads)"},
    }
    # matrix-core work of the scan: the method's 128 multiply-adds per scored pair, and the 9 int8
    # digit products per dimension that the exact kernel issues
    method_tops = pairs_per_launch * 2 * 128 / scan_avg_s / 1e12
    issued_tops = pairs_per_launch * 2 * 9 * 128 / scan_avg_s / 1e12
    scan_mfma = {"method_TOPs": method_tops, "method_frac_of_int8_peak": method_tops / INT8_MFMA_PEAK_TOPS,
                 "issued_TOPs": issued_tops, "issued_frac_of_int8_peak": issued_tops / INT8_MFMA_PEAK_TOPS,
                 "pairs_per_launch": pairs_per_launch, "peak": INT8_MFMA_PEAK_TOPS, "unit": "TOP/s"}
    gemm_ms, gemm_n = stages["filter_gemm"]
    gemm_flops = 2.0 * nq * wl.n_qtok * wl.n_centroids * 128 / (max(gemm_n, 1) / args.steps)
    gemm_tflops = gemm_flops / (gemm_ms / 1e3 / max(gemm_n, 1)) / 1e12 if gemm_n else None

    cpu, cpu1 = None, None
    if not args.no_cpu:
        import oracle

        threads = host_threads()
        # all host threads: whole queries (the tokens of a query in parallel when there are
        # fewer queries than threads), checked against the engine's results
        nc = min(args.cpu_queries, nq)
        log(f"bench: oracle on {nc} queries with {threads} threads")
        a = time.perf_counter()
        ref = oracle.search_index(data, queries=data.queries[:nc], threads=threads, debug=False)
        cpu_s = time.perf_counter() - a
        cpu = {"value": nc / cpu_s, "unit": "queries/s", "cores": threads, "kind": "oracle",
               "sample": f"first {nc} of the {nq} queries of the same workload "
                         f"({int(scored[:nc].sum())} scored embeddings), {cpu_s:.1f} s wall",
               "cpu_model": cpu_model(),
               "parity_ids": bool(np.array_equal(ref["ids"], dbg["ids"][:nc])),
               "parity_fixed_scores": bool(np.array_equal(ref["fixed"], dbg["fixed"][:nc]))}
        # one thread (the paper's setting): the first tokens of one query, scaled to a whole
        # query by embeddings scored
        nt1 = max(1, min(wl.n_qtok, args.cpu1_tokens))
        log(f"bench: oracle on 1 thread, query 0 restricted to its first {nt1} tokens")
        a = time.perf_counter()
        r1 = oracle.search_index(data, queries=data.queries[:1, :nt1], threads=1, debug=True)
        t1 = time.perf_counter() - a
        rate1 = float(r1["n_scored"][0]) / t1
        cpu1 = {"value": rate1 / float(scored.mean()), "unit": "queries/s", "cores": 1, "kind": "oracle",
                "scored_emb_per_s": rate1, "ms_per_query": float(scored.mean()) / rate1 * 1e3,
                "sample": f"query 0, first {nt1} of {wl.n_qtok} tokens ({int(r1['n_scored'][0])} scored "
                          f"embeddings, {t1:.1f} s); per-query figures scaled by the batch's mean "
                          f"{float(scored.mean()):.4g} scored embeddings per query",
                "paper_context": "the paper's WARP engine: 171.3 ms end to end per query on LoTTE Pooled "
                                 "(660M tokens, nprobe 32), one thread of a Xeon Gold 6132 at 2.6 GHz, "
                                 "query encoding included (Section 5)"}

    rec = {
        "metric": METRIC,
        "value": qps,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i32",
        "data": "synthetic",
        "config": {"workload": describe(wl), "n_embeddings": data.n_embeddings,
                   "scored_embeddings_per_query": float(scored.mean()), "batch": nq},
        "p50_ms_batch1": p50,
        "p99_ms_batch1": p99,
        "scored_emb_per_s": float(scored.sum()) * args.steps / elapsed,
        "hbm_frac_effective": float(scored.sum()) * args.steps * row_bytes / elapsed / (HBM_PEAK_GBS * 1e9),
        "stage_ms_per_step": {k: v[0] / args.steps for k, v in stages.items()},
        "roofline": roofline,
        "scan_mfma": scan_mfma,
        "scan_hbm_equivalent": {"bytes_per_scored_embedding": row_bytes, "GBps": hbm_equiv,
                                "frac_of_hbm_peak": hbm_equiv / HBM_PEAK_GBS,
                                "what": "scored pairs x (16b + 4) bytes: what a token-major scan would "
                                        "stream (not a roofline fraction for the cluster-major scan)"},
        "filter_gemm": {"TFLOPs": gemm_tflops, "flops_per_launch": gemm_flops,
                        "frac_of_fp16_peak": (gemm_tflops / FP16_MFMA_PEAK_TFLOPS) if gemm_tflops else None,
                        "issued_fp16_TFLOPs": 3 * gemm_tflops if gemm_tflops else None,
                        "peak": FP16_MFMA_PEAK_TFLOPS,
                        "what": "2 x M x N x 128 per launch; the kernel issues three fp16 products per "
                                "multiply-add (split operands)"},
        "host_api": {"value": host_qps, "unit": "queries/s", "batches": host_steps,
                     "what": "warp_search with host buffers: query check on the host, queries copied in, "
                             "ids, scores and counts copied out"},
        "cpu_baseline": cpu,
        "cpu_baseline_1thread": cpu1,
        "timed_batch_matches_debug_run": same_as_debug,
    }
    print(json.dumps(rec), flush=True)
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 18  # float32 elements
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: copied {args.copy_calibration_mib} MiB 3 times")
    return 0


if __name__ == "__main__":
    sys.exit(main())
