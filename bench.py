#!/usr/bin/env python3
"""Exact Top-20 hybrid retrieval throughput and PVS scan bandwidth on one MI355X.

Workload (default): the passage-scale configuration, N = 8,800,000 unit-norm
clustered vectors of d = 768 (4,096 centres, std 0.5) with a BM25 sparse
channel (vocab 30,000, Poisson(60) documents, Zipf(1.1) + topic mix), K = 20,
RRF k = 60, weights 1:1.  All inputs are seeded synthetic data; the index
(int8 codes, scales, norms, float32 rows) and the queries are resident in HBM
before a timed region starts.

One step = one eahr_topk call on a batch of queries: the PVS dense channel on
the GPU (threshold sampling, interval scan, rescoring, sort, certification)
plus PBM and weighted-RRF certification on the host, with depth doubling from
20 until the ordered Top-20 is fixed.  The headline is the batch of 256
queries (value = queries/s); batches of 1 (distinct queries of the 200-query
single-request set, one per step) and 64 are timed in the same run and
reported under ``per_batch``.

Kernel times come from HIP events the library records on its own stream
around each kernel class of every scan round, inside the timed region.
``kernels`` lists every class with its algorithmic bytes and rate:
  * scan variants: N (d + 12) + 8 N / 64 bytes per launch (codes, three
    per-row floats, visibility bits), independent of the batch;
  * rescore: (4 d + 12) bytes per row load (a float32 row and the three
    per-row floats its intervals are recomputed from; one load serves the
    adjacent records of one row) plus 16 bytes per candidate pair (its
    (row, query, integer dot) record) and 8 per certified pair (its key);
and ``roofline`` is the class with the most time in the headline batch
(HBM-bound: achieved GB/s against 8 TB/s), ``roofline_scan`` the dominant
scan variant.  ``traffic`` is filled from the committed PMC summary of that
kernel (FETCH_SIZE + WRITE_SIZE per launch, scaled by the same counters on a
plain device copy) when its source is unchanged since, else null.
``cpu_baseline`` times the CPU oracle (exhaustive float64 dense ranking, brute
force sparse ranking, exact complete-list RRF) on a few queries of the
headline batch and checks their Top-20.

``--copy-calibration MB`` only runs a device-to-device copy of MB MiB ten
times (the reference kernel for the PMC byte counters) and exits.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
T0 = time.time()


def log(msg: str) -> None:
    print(f"[bench {time.time() - T0:7.1f}s] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="passage")
    ap.add_argument("--batch", type=int, default=256, help="queries per eahr_topk call (headline)")
    ap.add_argument("--extra", default="1:200,64:3", help="extra batch:steps configurations")
    ap.add_argument("--n", type=int, default=None, help="override corpus rows (quick runs only)")
    ap.add_argument("--weights", default="1:1")
    ap.add_argument("--range-size", type=int, default=4096)
    ap.add_argument("--cpu-queries", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ablation", action="store_true",
                    help="skip the rank-generator ablation (global-scale scalar quantisation vs PVS)")
    ap.add_argument("--ablation-queries", type=int, default=20)
    ap.add_argument("--configs", default="weights21,sparse_gpu,mid,adv,temporal",
                    help="further configurations (comma-separated): weights21 (the passage batch at "
                         "weights 2:1), sparse_gpu (the passage batch, and every further workload, "
                         "again with PBM's posting work on the GPU), mid, adv, temporal; empty for none")
    ap.add_argument("--no-streams", action="store_true",
                    help="skip the controlled rank-stream experiment (host only)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MB")
    return ap.parse_args()


# committed PMC summaries: kernel class -> (file, sources whose hash it records)
SCAN_SOURCES = ["paper_2608_07152_amd/csrc/pvs_scan.hip", "paper_2608_07152_amd/csrc/pvs_device.h"]
RANK_SOURCES = ["paper_2608_07152_amd/csrc/pvs_rank.hip", "paper_2608_07152_amd/csrc/pvs_device.h"]
TRAFFIC_FILES = {
    "rescore": ("profiles/k_rescore_passage_b256_traffic.txt", RANK_SOURCES),
    "k_scan_mfma<8>": ("profiles/k_scan_mfma_r1_8tile_passage_b256_traffic.txt", SCAN_SOURCES),
    "k_scan_mfma<4>": ("profiles/k_scan_mfma_r1_4tile_passage_b256_traffic.txt", SCAN_SOURCES),
    "k_scan_gemv<1>": ("profiles/k_scan_gemv1_passage_b1_traffic.txt", SCAN_SOURCES),
}


def sources_sha(paths):
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_for(kernel):
    """HBM bytes per launch from the committed PMC summary, or None when
    there is none or the kernel's source changed since it was taken."""
    if kernel not in TRAFFIC_FILES:
        return None
    path, srcs = TRAFFIC_FILES[kernel]
    full = os.path.join(ROOT, path)
    if not os.path.exists(full):
        return None
    vals = {}
    with open(full) as f:
        for line in f:
            if ":" in line:
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != sources_sha(srcs) or "traffic_bytes_per_launch" not in vals:
        return None
    return float(vals["traffic_bytes_per_launch"])


def copy_calibration(mb):
    import torch
    n = mb * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(10):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "copies": 10}), flush=True)


def step_summary(eahr, prof, res, d, n_visible, bsz, steps, el, step_ms):
    """Throughput, kernel classes with their algorithmic bytes, and the
    per-query work counters of a timed series of eahr_topk calls."""
    import numpy as np
    # dominant scan kernel variant = most total scan time
    vms = prof["variant_ms"]
    v = max(range(len(vms)), key=lambda i: vms[i])
    launches = max(1, prof["variant_launches"][v])
    avg_ms = vms[v] / launches
    bpl = prof["variant_bytes"][v] / launches
    achieved = bpl / (avg_ms * 1e-3) / 1e9 if avg_ms > 0 else 0.0
    variants = {eahr.pvs_profile.VARIANTS[i]: {"ms": vms[i], "launches": prof["variant_launches"][i]}
                for i in range(len(vms)) if prof["variant_launches"][i]}
    # every kernel class with its algorithmic bytes
    kernels = {}
    for i, name in enumerate(eahr.pvs_profile.VARIANTS):
        if prof["variant_launches"][i]:
            ms, n = vms[i], prof["variant_launches"][i]
            kernels[name] = {"ms": ms, "launches": n, "bytes": prof["variant_bytes"][i],
                             "gbs": prof["variant_bytes"][i] / (ms * 1e-3) / 1e9 if ms > 0 else 0.0}
    if prof["scan_rounds"]:
        rb = (prof["rescore_row_reads"] * (4 * d + 12) + prof["rescore_rows"] * 16
              + prof["rescore_certified"] * 8)
        ms = prof["rescore_ms"]
        kernels["rescore"] = {"ms": ms, "launches": prof["scan_rounds"], "bytes": rb,
                              "gbs": rb / (ms * 1e-3) / 1e9 if ms > 0 else 0.0}
    dom = max(kernels, key=lambda k: kernels[k]["ms"])
    kernels["sort_pack"] = {"ms": prof["sort_ms"], "launches": prof["scan_rounds"]}
    kernels["sample_select"] = {"ms": prof["sample_ms"], "launches": prof["scan_rounds"]}
    stats = [s for r in res for s in r[3]]
    dd = np.array([s["dense_depth"] for s in stats])
    kms = prof["scan_ms"] + prof["sample_ms"] + prof["rescore_ms"] + prof["sort_ms"]
    return {
        "batch": bsz, "steps": steps, "queries_per_s": steps * bsz / el,
        "ms_per_step": el / steps * 1e3,
        "scan_kernel": eahr.pvs_profile.VARIANTS[v],
        "scan_gbs": achieved, "scan_frac": achieved / HBM_PEAK_GBS, "scan_avg_launch_ms": avg_ms,
        "scan_launches": launches, "scan_bytes_per_launch": bpl, "scan_variants": variants,
        "kernels": kernels, "dominant": dom,
        "kernel_ms": {"scan": prof["scan_ms"], "sample_select": prof["sample_ms"],
                      "rescore": prof["rescore_ms"], "sort_pack": prof["sort_ms"]},
        # share of the wall time the GPU spent in the dense channel's kernels
        "gpu_busy_frac": kms / (el * 1e3) if el > 0 else 0.0,
        "rescored_pairs": prof["rescore_rows"], "rescore_row_reads": prof["rescore_row_reads"],
        "host_ms": {"dense_calls": prof["host_dense_ms"], "sparse_rounds": prof["host_sparse_ms"],
                    "certify": prof["host_fuse_ms"]},
        "dense_depth": {"mean": float(dd.mean()), "median": float(np.median(dd)), "max": int(dd.max())},
        # per-call latency (per query when the batch is 1), Sec. 3.5 reports p50/p95/p99
        "latency_ms": {"p50": float(np.percentile(step_ms, 50)), "p95": float(np.percentile(step_ms, 95)),
                       "p99": float(np.percentile(step_ms, 99)), "max": float(np.max(step_ms))},
        # read ratio d_i / n_i: dense n_i = the visible rows; sparse only where the list was read to its end
        "dense_read_ratio": {"median": float(np.median(dd) / n_visible), "max": float(dd.max() / n_visible)},
        "sparse_exhausted": int(sum(s["sparse_len"] >= 0 for s in stats)),
        "sparse_depth_mean": float(np.mean([s["sparse_depth"] for s in stats])),
        # work counters of Sec. 3.5 per query (medians)
        "dense_f32_evals_median": float(np.median([s["dense_evals"] for s in stats])),
        "sparse_postings_median": float(np.median([s["sparse_postings"] for s in stats])),
        "sparse_scored_median": float(np.median([s["sparse_scored"] for s in stats])),
        "failed": int(sum(int(np.sum(r[2] != 0)) for r in res)),
    }


def cpu_host_info():
    """Usable host cores and the CPU model (the oracle baseline's machine)."""
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cores, model


def cpu_baseline(x, post, q, qs, K, wts, n_queries, visible=None):
    """Time the oracle (exhaustive float64 dense ranking streamed in 1M-row
    chunks, brute-force sparse scores, exact complete-list RRF) on the first
    n_queries of a batch; returns the Top-K lists, seconds and the threads the
    oracle's float64 products ran on."""
    import numpy as np
    from oracle import dense as odense
    from oracle import rrf as orrf
    from oracle import sparse as osparse
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = 1
    out = []
    t = time.perf_counter()
    step = 1 << 20
    ids = np.arange(len(x), dtype=np.int64)
    if visible is not None:
        ids = ids[visible]
    for b in range(n_queries):
        s64 = np.concatenate([odense.scores64(q[b], x[r:r + step]) for r in range(0, len(x), step)])
        dense_list = odense.rank_order(s64[ids], ids)
        S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, qs[b][0], qs[b][1], len(x),
                                  visible)
        sparse_list = osparse.sparse_ranking(S)
        out.append(orrf.rrf_topk([dense_list, sparse_list], list(wts), 60, K))
    el = time.perf_counter() - t
    return out, el, blas


def cpu_baseline_entry(n, el, threads, what):
    cores, model = cpu_host_info()
    return {"value": n / el, "unit": "queries/s", "cores": threads, "host_cores": cores,
            "cpu_model": model, "kind": "oracle", "seconds": el, "sample": what}


def bench_workload(name, eahr, torch, datagen, K, steps, warmup, cpu_queries, wts=(1, 1),
                   sparse_gpu=False):
    """One further configuration of the workload table: its own corpus,
    index and query batch (one eahr_topk call per step on all its queries),
    kernel rooflines, work counters, and the oracle on a few queries (timed
    as a CPU baseline and compared with the GPU's Top-K)."""
    import numpy as np
    t0 = time.perf_counter()
    w = datagen.workload(name)
    x, lab = datagen.corpus(w)
    q, qlab = datagen.queries(w)
    epochs = [(0, None)]
    if name == "temporal":
        steps_ = list(datagen.temporal_steps(w, w.n))
        x = np.concatenate([x] + [st.insert_rows for st in steps_])
        lab = np.concatenate([lab] + [st.insert_labels for st in steps_])
        docs = datagen.temporal_docs(w, lab, w.n)
    elif not w.adversarial:
        docs = datagen.sparse_docs(w, lab)
    idx = eahr.pvs_build(x[:w.n])
    if name == "temporal":
        vis = np.zeros(len(x), dtype=bool)
        vis[:w.n] = True
        epochs = [(0, vis.copy())]
        rows = w.n
        for st in steps_:
            eahr.pvs_delete(idx, st.delete_ids)
            eahr.pvs_insert(idx, st.insert_rows)
            vis[st.delete_ids] = False
            vis[rows:rows + len(st.insert_rows)] = True
            rows += len(st.insert_rows)
            epochs.append((eahr.pvs_snapshot(idx), vis.copy()))
    if w.adversarial:
        post, qs = datagen.adversarial_postings(w, x, q)
        posts = [post]
    elif name == "temporal":
        qs = datagen.sparse_queries(w, qlab)
        posts = [datagen.bm25_impacts(w, docs, v) for _, v in epochs]
    else:
        qs = datagen.sparse_queries(w, qlab)
        posts = [datagen.bm25_impacts(w, docs)]
    pbms = [eahr.pbm_build(p.term_ptr, p.doc, p.impact, len(x), 4096) for p in posts]
    qd = torch.from_numpy(q).cuda()
    torch.cuda.synchronize()
    log(f"{name}: set up in {time.perf_counter() - t0:.1f}s ({len(x)} rows, {len(q)} queries)")
    # temporal: warm up on S0, then one timed step per snapshot S1..S5
    runs = [(e, pbms[i]) for i, (e, _) in enumerate(epochs)] if name == "temporal" else None

    def call(i, sgen="pbm"):
        if runs is not None:
            e, pb = runs[i]
            return eahr.eahr_topk(idx, pb, qd, qs, K=K, w_dense=wts[0], w_sparse=wts[1], epoch=e,
                                  sparse_generator=sgen)
        return eahr.eahr_topk(idx, pbms[0], qd, qs, K=K, w_dense=wts[0], w_sparse=wts[1],
                              sparse_generator=sgen)

    if runs is not None:
        warm, timed = [0], list(range(1, len(runs)))
    else:
        warm, timed = [0] * warmup, [0] * steps
    for i in warm:
        call(i)
    eahr.pvs_profile_enable(True)
    torch.cuda.synchronize()
    t = time.perf_counter()
    res, step_ms = [], []
    for i in timed:
        ts = time.perf_counter()
        res.append(call(i))
        step_ms.append((time.perf_counter() - ts) * 1e3)
    torch.cuda.synchronize()
    el = time.perf_counter() - t
    prof = eahr.pvs_profile_read()
    eahr.pvs_profile_enable(False)
    n_vis = float(np.mean([eahr.pvs_info(idx, e)[2] for e, _ in (epochs[1:] if runs else epochs)]))
    out = step_summary(eahr, prof, res, w.d, n_vis, len(q), len(timed), el, step_ms)
    out["workload"] = (f"{name} N={w.n} d={w.d} centers={w.centers} queries={len(q)} K={K} k=60 "
                       f"weights={wts[0]}:{wts[1]}" + (" snapshots S1-S5 (one step each)"
                                                         if runs else ""))
    out["roofline"] = roofline_of(out["dominant"], out["kernels"][out["dominant"]])
    out["roofline_scan"] = roofline_of(out["scan_kernel"], out["kernels"][out["scan_kernel"]])
    log(f"{name}: {out['queries_per_s']:.1f} q/s, dominant {out['dominant']} "
        f"{out['roofline']['frac']:.2f} of HBM, scan {out['scan_kernel']} {out['scan_frac']:.2f}")
    if sparse_gpu:
        out["sparse_gpu"] = sparse_gpu_steps(eahr, torch, lambda i: call(i, "pbm_gpu"), warm, timed, res)
        log(f"{name}: PBM on the GPU {out['sparse_gpu']['queries_per_s']:.1f} q/s")
    if cpu_queries > 0:
        last_e, last_vis = (epochs[-1] if runs else epochs[0])
        post = posts[-1]
        want, cel, threads = cpu_baseline(x, post, q, qs, K, wts, cpu_queries, last_vis)
        ids, cnt, _, _ = res[-1]
        match = sum(list(ids[b, :cnt[b]]) == want[b] for b in range(cpu_queries))
        out["cpu_baseline"] = cpu_baseline_entry(
            cpu_queries, cel, threads,
            f"{cpu_queries} queries of the batch" + (" on snapshot S5" if runs else "")
            + " over every visible row (exhaustive fp64 dense sort, brute-force sparse, exact RRF)")
        out["oracle_check"] = {"queries": cpu_queries, "top20_equal": int(match)}
        log(f"{name}: cpu oracle {cel:.1f}s, {match}/{cpu_queries} Top-20 equal")
    for pb in pbms:
        eahr.pbm_free(pb)
    eahr.pvs_free(idx)
    del qd
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def roofline_of(name, k):
    """HBM roofline of one kernel class over the timed region."""
    launches = max(1, k["launches"])
    avg_ms = k["ms"] / launches
    bpl = k["bytes"] / launches
    achieved = bpl / (avg_ms * 1e-3) / 1e9 if avg_ms > 0 else 0.0
    return {"bound": "hbm", "kernel": name, "achieved": achieved, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic_for(name),
            "avg_launch_ms": avg_ms, "launches": k["launches"], "bytes_per_launch": bpl}


def query_set_for(w, batch):
    if w.name != "passage":
        return "default"
    return {64: "b64", 256: "b256"}.get(batch, "single")


def generator_ablation(eahr, torch, x, idx, pbm, qdev, sparse_q, w, K, wts, nq, batch):
    """Rank-generator ablation (Sec. 4.4, Table 4-1): the same eahr_topk with
    the dense generator replaced by global-scale scalar-quantisation intervals
    ("scalar") or by one exhaustive float32 scan ("scan"), or the sparse
    generator replaced by the complete exact sparse ranking
    ("sparse_complete").  Single requests
    are timed in paired rounds (generator order rotating, 1 warm-up + 3 runs
    each, median per query) and compared by the geometric mean of the
    per-query latency ratios; the batch is timed for 1 warm-up + 2 steps with
    PVS and scalar intervals (an exhaustive scan of a whole batch would keep
    8 bytes per row and query on the host).  f32 evaluations are the (query,
    row) pairs scored in float32 by each call."""
    import numpy as np
    log("ablation: building the global-scale index")
    t = time.perf_counter()
    gidx = eahr.pvs_build_quant(x, "global")
    torch.cuda.synchronize()
    log(f"ablation: global-scale index built in {time.perf_counter() - t:.1f}s")
    gens = {"pvs": (idx, "intervals", "pbm"), "scalar": (gidx, "intervals", "pbm"),
            "scan": (idx, "full_scan", "pbm"), "sparse_complete": (idx, "intervals", "complete")}

    def call(g, a, b):
        ix, gen, sgen = gens[g]
        eahr.pvs_profile_enable(True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r = eahr.eahr_topk(ix, pbm, a, b, K=K, w_dense=wts[0], w_sparse=wts[1], dense_generator=gen,
                           sparse_generator=sgen)
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        pairs = eahr.pvs_profile_read()["rescore_rows"]
        eahr.pvs_profile_enable(False)
        return el, pairs, r

    name1 = query_set_for(w, 1)
    qd, qs = qdev[name1], sparse_q[name1]
    nq = min(nq, qd.shape[0])
    names = list(gens)
    lat = {g: [] for g in gens}
    evals = {g: [] for g in gens}
    same = {g: 0 for g in gens}
    for i in range(nq):
        a, b = qd[i:i + 1], qs[i:i + 1]
        order = names[i % len(names):] + names[:i % len(names)]
        times = {g: [] for g in gens}
        ids = {}
        for rep in range(4):
            for g in order:
                el, pairs, r = call(g, a, b)
                if rep:
                    times[g].append(el)
                else:
                    evals[g].append(pairs)
                    ids[g] = r[0][0, :r[1][0]].tolist()
        for g in gens:
            same[g] += ids[g] == ids["pvs"]
            lat[g].append(float(np.median(times[g])))

    def gmean_ratio(g):
        return float(np.exp(np.mean(np.log(np.array(lat[g]) / np.array(lat["pvs"])))))

    def reduction(g):
        return 1.0 - float(np.median(evals["pvs"])) / max(1.0, float(np.median(evals[g])))

    single = {
        "queries": nq,
        "scalar_over_pvs_latency_gmean": gmean_ratio("scalar"),
        "scan_over_pvs_latency_gmean": gmean_ratio("scan"),
        "sparse_complete_over_pbm_latency_gmean": gmean_ratio("sparse_complete"),
        "median_ms": {g: float(np.median(lat[g]) * 1e3) for g in gens},
        "f32_evals_median": {g: float(np.median(evals[g])) for g in gens},
        "pvs_f32_evals_reduction_vs": {"scalar": reduction("scalar"), "scan": reduction("scan")},
        "topk_identical_to_pvs": {g: same[g] for g in ("scalar", "scan", "sparse_complete")},
    }
    log(f"ablation: single requests scalar/pvs = {single['scalar_over_pvs_latency_gmean']:.3f}, "
        f"scan/pvs = {single['scan_over_pvs_latency_gmean']:.3f}, "
        f"sparse complete/pbm = {single['sparse_complete_over_pbm_latency_gmean']:.3f}, f32 evals "
        + ", ".join(f"{g} {single['f32_evals_median'][g]:.0f}" for g in gens))
    nameb = query_set_for(w, batch)
    a, b = qdev[nameb][:batch], sparse_q[nameb][:batch]
    bt = {}
    for g in ("pvs", "scalar", "sparse_complete"):
        call(g, a, b)
        runs = [call(g, a, b) for _ in range(2)]
        bt[g] = {"ms_per_step": float(np.mean([r[0] for r in runs]) * 1e3),
                 "f32_evals_per_step": float(np.mean([r[1] for r in runs])),
                 "ids": runs[0][2][0]}
    batched = {
        "batch": batch,
        "scalar_over_pvs_latency": bt["scalar"]["ms_per_step"] / bt["pvs"]["ms_per_step"],
        "sparse_complete_over_pbm_latency": bt["sparse_complete"]["ms_per_step"] / bt["pvs"]["ms_per_step"],
        "ms_per_step": {g: bt[g]["ms_per_step"] for g in bt},
        "f32_evals_per_step": {g: bt[g]["f32_evals_per_step"] for g in bt},
        "topk_identical": bool(np.array_equal(bt["pvs"]["ids"], bt["scalar"]["ids"]) and
                               np.array_equal(bt["pvs"]["ids"], bt["sparse_complete"]["ids"])),
    }
    log(f"ablation: batch {batch} scalar/pvs = {batched['scalar_over_pvs_latency']:.3f}")
    eahr.pvs_free(gidx)
    torch.cuda.synchronize()
    return {"reference": "pvs",
            "alternatives": {"scalar": "scalar-quantisation intervals (one global scale)",
                             "scan": "exhaustive float32 scan, one sort per query",
                             "sparse_complete": "complete exact sparse ranking (PBM replaced)"},
            "single_requests": single, "batch": batched}


def controlled_streams(eahr, datagen, K=20, check_every=16):
    """The controlled rank streams of Sec. 3.4 through eahr_fuse_lists: 3
    sizes x 5 relationships x 3 seeds, both lists advancing together with a
    check every 16 ranks.  Per instance: the first checkpoint at which the
    ordered Top-20 is fixed, the read ratio (that depth / n) and whether a
    list was read to its end (Sec. 4.2 reports the same three)."""
    import numpy as np
    out = {}
    t0 = time.perf_counter()
    for rel in datagen.STREAM_RELATIONS:
        inst = []
        for n in datagen.STREAM_SIZES:
            for seed in datagen.STREAM_SEEDS:
                a, b = datagen.controlled_streams(rel, n, seed)
                t = time.perf_counter()
                _, st = eahr.eahr_fuse_lists(a, b, K=K, step=check_every)
                el = time.perf_counter() - t
                d = max(st["dense_depth"], st["sparse_depth"])
                inst.append({"n": n, "seed": seed, "first_resolved_depth": d, "read_ratio": d / n,
                             "exhausted": st["dense_status"] == eahr.LIST_EXHAUSTED
                             or st["sparse_status"] == eahr.LIST_EXHAUSTED,
                             "fuse_ms": el * 1e3})
        d = [i["first_resolved_depth"] for i in inst]
        r = [i["read_ratio"] for i in inst]
        out[rel] = {"median_depth": float(np.median(d)), "read_ratio_min": min(r), "read_ratio_max": max(r),
                    "exhausted": sum(i["exhausted"] for i in inst), "instances": inst}
        log(f"streams {rel}: median depth {np.median(d):.0f}, read ratio {min(r):.4f}-{max(r):.4f}, "
            f"exhausted {out[rel]['exhausted']}/{len(inst)}")
    out["seconds"] = time.perf_counter() - t0
    return out


def sparse_gpu_steps(eahr, torch, call, warm, timed, host_res):
    """The same steps with Posting Block-Max's posting work on the GPU
    (EAHR_SPARSE_PBM_GPU): queries/s, per-step time and whether every step's
    Top-K, counts and statuses equal the host generator's."""
    import numpy as np
    for i in warm:
        call(i)
    torch.cuda.synchronize()
    t = time.perf_counter()
    res, step_ms = [], []
    for i in timed:
        ts = time.perf_counter()
        res.append(call(i))
        step_ms.append((time.perf_counter() - ts) * 1e3)
    torch.cuda.synchronize()
    el = time.perf_counter() - t
    nq = sum(len(r[1]) for r in res)
    same = all(np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and np.array_equal(a[2], b[2])
               for a, b in zip(res, host_res))
    postings = [float(np.mean([s["sparse_postings"] for s in r[3]])) for r in res]
    return {"queries_per_s": nq / el, "ms_per_step": float(np.mean(step_ms)),
            "topk_equal_to_host_generator": bool(same),
            "sparse_postings_mean": float(np.mean(postings))}


def sparse_only_compare(eahr, torch, pbm, qs, K, steps):
    """The sparse channel alone (weights 0:1, the Top-K of the exact sparse
    ranking) over one batch, with the host generator and with the GPU one:
    queries/s of each and whether their Top-K agree."""
    import numpy as np
    out = {}
    ref = None
    for gen in ("pbm", "pbm_gpu"):
        eahr.eahr_topk(None, pbm, None, qs, K=K, w_dense=0, w_sparse=1, sparse_generator=gen)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(steps):
            r = eahr.eahr_topk(None, pbm, None, qs, K=K, w_dense=0, w_sparse=1, sparse_generator=gen)
        torch.cuda.synchronize()
        out[gen + "_queries_per_s"] = steps * len(qs) / (time.perf_counter() - t)
        if ref is None:
            ref = r
        else:
            out["topk_equal"] = bool(np.array_equal(ref[0], r[0]) and np.array_equal(ref[1], r[1]))
    log(f"sparse only: host {out['pbm_queries_per_s']:.0f} q/s, GPU {out['pbm_gpu_queries_per_s']:.0f} q/s")
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU; --gpus N with N > 1 is not supported",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    import numpy as np
    import torch

    from paper_2608_07152_amd import datagen, eahr

    eahr.load()
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    wts = tuple(int(v) for v in args.weights.split(":"))
    K = 20
    over = {"n": args.n} if args.n else {}
    w = datagen.workload(args.workload, **over)
    log(f"workload {w.name}: n={w.n} d={w.d} centers={w.centers}")
    x, lab = datagen.corpus(w)
    log("dense corpus generated")
    configs = [(args.batch, args.steps, args.warmup)]
    for item in filter(None, args.extra.split(",")):
        bsz, st = (int(v) for v in item.split(":"))
        configs.append((bsz, st, 1))
    qsets = {}
    for bsz, steps, _ in configs:
        name = query_set_for(w, bsz)
        if name not in qsets:
            cnt = datagen.QUERY_SETS[w.name][name][1]
            qsets[name] = datagen.queries(w, name, count=max(cnt, bsz))
    if w.adversarial:
        post = None
    else:
        docs = datagen.sparse_docs(w, lab)
        log(f"sparse documents generated: {len(docs.doc)} postings")
        post = datagen.bm25_impacts(w, docs)
        del docs
    sparse_q = {}
    for name, (q, qlab) in qsets.items():
        if w.adversarial:
            post_a, sq = datagen.adversarial_postings(w, x, q)
            post = post_a
        else:
            sq = datagen.sparse_queries(w, qlab, datagen.query_set_offset(w, name))
        sparse_q[name] = sq
    log("sparse impacts computed")
    idx = eahr.pvs_build(x)
    torch.cuda.synchronize()
    log("pvs index built")
    pbm = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, args.range_size)
    log("pbm index built")
    qdev = {name: torch.from_numpy(q).cuda() for name, (q, _) in qsets.items()}
    torch.cuda.synchronize()

    def run_config(bsz, steps, warmup, weights=None, sgen="pbm"):
        wts_ = weights or wts
        name = query_set_for(w, bsz)
        qd, qs = qdev[name], sparse_q[name]
        pool = qd.shape[0]

        def batch_at(i):
            s = (i * bsz) % pool
            if s + bsz > pool:
                s = 0
            return qd[s:s + bsz], qs[s:s + bsz]

        for i in range(warmup):
            a, b = batch_at(i)
            eahr.eahr_topk(idx, pbm, a, b, K=K, w_dense=wts_[0], w_sparse=wts_[1], sparse_generator=sgen)
        eahr.pvs_profile_enable(True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        res = []
        step_ms = []
        for i in range(steps):
            a, b = batch_at(warmup + i)
            t_step = time.perf_counter()   # eahr_topk returns host results: the step is complete
            res.append(eahr.eahr_topk(idx, pbm, a, b, K=K, w_dense=wts_[0], w_sparse=wts_[1],
                                      sparse_generator=sgen))
            step_ms.append((time.perf_counter() - t_step) * 1e3)
        torch.cuda.synchronize()
        el = time.perf_counter() - t
        prof = eahr.pvs_profile_read()
        eahr.pvs_profile_enable(False)
        out = step_summary(eahr, prof, res, w.d, w.n, bsz, steps, el, step_ms)
        log(f"batch {bsz}: {out['queries_per_s']:.1f} q/s, scan {out['scan_gbs']:.0f} GB/s")
        return out, res

    head, head_res = run_config(*configs[0])
    per_batch = [head]
    for cfg in configs[1:]:
        per_batch.append(run_config(*cfg)[0])

    ablation = None
    if not args.no_ablation:
        ablation = generator_ablation(eahr, torch, x, idx, pbm, qdev, sparse_q, w, K, wts,
                                      args.ablation_queries, args.batch)
    cfg_names = [c for c in args.configs.split(",") if c]
    further = {}
    if "weights21" in cfg_names and w.name == "passage":
        o, r21 = run_config(args.batch, args.steps, args.warmup, weights=(2, 1))
        o["workload"] = f"passage N={w.n} d={w.d} batch={args.batch} K={K} k=60 weights=2:1"
        o["roofline"] = roofline_of(o["dominant"], o["kernels"][o["dominant"]])
        o["roofline_scan"] = roofline_of(o["scan_kernel"], o["kernels"][o["scan_kernel"]])
        if not args.no_cpu_baseline:
            name = query_set_for(w, args.batch)
            want, cel, threads = cpu_baseline(x, post, qsets[name][0], sparse_q[name], K, (2, 1), 1)
            ids, cnt, _, _ = r21[0]
            o["cpu_baseline"] = cpu_baseline_entry(1, cel, threads, "1 query of the batch over the full corpus")
            o["oracle_check"] = {"queries": 1, "top20_equal": int(list(ids[0, :cnt[0]]) == want[0])}
        further["passage_2to1"] = o
    if "sparse_gpu" in cfg_names:
        # the headline batch with Posting Block-Max's posting work on the GPU
        o, rg = run_config(args.batch, args.steps, args.warmup, sgen="pbm_gpu")
        o["workload"] = (f"passage N={w.n} d={w.d} batch={args.batch} K={K} k=60 weights={wts[0]}:{wts[1]} "
                         f"sparse=PBM on the GPU")
        o["roofline"] = roofline_of(o["dominant"], o["kernels"][o["dominant"]])
        o["roofline_scan"] = roofline_of(o["scan_kernel"], o["kernels"][o["scan_kernel"]])
        o["topk_equal_to_host_generator"] = bool(all(
            np.array_equal(a[0], b[0]) and np.array_equal(a[2], b[2]) for a, b in zip(rg, head_res)))
        o["sparse_only"] = sparse_only_compare(eahr, torch, pbm, sparse_q[query_set_for(w, args.batch)][:args.batch],
                                               K, args.steps)
        further["passage_sparse_gpu"] = o

    line = {
        "metric": "exact Top-20 EAHR queries/s at 8.8Mx768 (PVS scan HBM GB/s in roofline)",
        "value": head["queries_per_s"],
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8+f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name} N={w.n} d={w.d} batch={args.batch} K={K} k=60 "
                               f"weights={wts[0]}:{wts[1]}",
                   "global_batch": args.batch, "parallelism": "single GPU"},
        "roofline": roofline_of(head["dominant"], head["kernels"][head["dominant"]]),
        "roofline_scan": roofline_of(head["scan_kernel"], head["kernels"][head["scan_kernel"]]),
        "per_batch": per_batch,
    }
    if ablation is not None:
        line["ablation"] = ablation
    if not args.no_streams:
        line["controlled_streams"] = controlled_streams(eahr, datagen)
    if not args.no_cpu_baseline:
        bsz = configs[0][0]
        name = query_set_for(w, bsz)
        q = qsets[name][0]
        qs = sparse_q[name]
        nqc = min(args.cpu_queries, bsz)
        log(f"cpu oracle on {nqc} queries")
        want, cel, threads = cpu_baseline(x, post, q, qs, K, wts, nqc)
        ids, cnt, _, _ = head_res[0]
        match = sum(list(ids[b, :cnt[b]]) == want[b] for b in range(nqc))
        line["cpu_baseline"] = cpu_baseline_entry(
            nqc, cel, threads, f"{nqc} queries of the headline batch over the full corpus "
                               f"(exhaustive fp64 dense sort, brute-force sparse, exact RRF)")
        line["oracle_check"] = {"queries": nqc, "top20_equal": int(match)}
        log(f"cpu oracle {cel:.1f}s, {match}/{nqc} Top-20 equal")
    others = [c for c in cfg_names if c in ("mid", "adv", "temporal")]
    if others:
        # the passage data is no longer needed
        eahr.pvs_free(idx)
        eahr.pbm_free(pbm)
        del x, post, qdev
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        for c in others:
            st = {"mid": (args.steps, args.warmup), "adv": (2, 1), "temporal": (5, 1)}[c]
            further[c] = bench_workload(c, eahr, torch, datagen, K, st[0], st[1],
                                        0 if args.no_cpu_baseline else 1,
                                        sparse_gpu="sparse_gpu" in cfg_names)
    if further:
        line["configs"] = further
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
