#!/usr/bin/env python3
"""Benchmark of the GPU query path on one MI355X.

One step = one chimera_search over the workload's whole query batch (probe,
candidate walk, refinement, residual scoring, top-k), with the index and the
queries already resident in HBM.  Prints ONE JSON line:

  value            whole-job QPS over the timed steps
  p50/p95/p99      end-to-end latency at nq=1 (H2D of Q, search, D2H)
  stages_ms        per-stage device time per step (HIP events on the search stream)
  roofline         the dominant kernel against its roofline
  cpu_baseline     the CPU oracle on a bounded sample of the same queries
  recall_at_k      against exact MaxSim (Chamfer, Def. 1) on raw tokens,
                   brute force in fp64 on the GPU for a sample of queries
  collab           the CPU-GPU collaborative scoring (Alg. 3) on the same
                   batch: QPS with chunks and with one chunk, the number of
                   full-precision scores per query, recall@k

The default workload is the 100k-document corpus (256 queries x 32 tokens,
nprobe 4, ncand 4096, k 10); ``--workload`` selects another.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "QPS at fixed recall@k (batch) + p50 latency nq=1; code-scan HBM GB/s"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
STAGES = ["round", "probe", "walk", "select", "score", "topk"]
KERNEL_OF_STAGE = {"probe": "k_probe", "walk": "k_cand_walk", "select": "k_select", "score": "k_residual_score",
                   "topk": "k_topk", "round": "k_round_queries"}
SOURCE_OF_STAGE = {"probe": "k_probe.hip", "walk": "k_prune.hip", "select": "k_prune.hip",
                   "score": "k_score.hip", "topk": "k_score.hip", "round": "k_probe.hip"}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def describe(w) -> str:
    lens = {0: f"exactly {w.len_lo} tokens", 1: f"lognormal length mean {w.len_mean:g} in [{w.len_lo},{w.len_hi}]",
            2: f"uniform length in [{w.len_lo},{w.len_hi}]"}[w.len_kind]
    pop = "uniform" if w.pop_kind == 0 else f"Zipf({w.zipf_s:g})"
    return (f"{w.name}: {w.ndocs:,} docs ({lens}), dim {w.dim}, {w.ncent:,} {pop} centroids, {w.nbits}-bit residual "
            f"codes; {w.nq} queries x {w.Tq} tokens; nprobe {w.nprobe}, ncand {w.ncand}, k {w.k}")


def build_corpus_index(w, threads):
    import numpy as np
    import synth
    from paper_2608_23553_amd import build_index
    corpus = synth.Corpus(w.corpus_spec(), nthreads=threads)

    passes = [0]

    def chunks():
        step = 50_000
        passes[0] += 1
        for d0 in range(0, w.ndocs, step):
            d1 = min(w.ndocs, d0 + step)
            k, cl = corpus.tokens(d0, d1)
            yield synth.k_to_bf16_bits(k), cl, corpus.lengths[d0:d1]
            if (d0 // step) % 20 == 19:
                log(f"index build pass {passes[0]}/2: {d1}/{w.ndocs} docs")

    t = time.perf_counter()
    b = build_index(synth.k_to_bf16_bits(corpus.centroids_k), w.nbits, chunks)
    log(f"index built on host in {time.perf_counter() - t:.1f}s: {b.info()}")
    return corpus, b


def exact_topk_gpu(q_k, corpus, k, device):
    """Exact Chamfer top-k (score desc, id asc) over raw grid tokens; fp64 on
    the GPU (every product and sum is exact), chunked over tokens."""
    import numpy as np
    import torch
    import synth
    nd = corpus.spec.ndocs
    Q = torch.from_numpy(q_k.astype(np.float64) / 2048.0).to(device)  # [nq, Tq, d]
    nq, Tq, _ = Q.shape
    F = torch.empty((nq, nd), dtype=torch.float64, device=device)
    # chunks of whole documents, ~8 GB of fp64 scores each; a chunk's
    # documents are finished inside it
    step = max(100, int(1e9 // (nq * Tq * 70)))
    t_log = time.perf_counter()
    for d0 in range(0, nd, step):
        d1 = min(nd, d0 + step)
        tk, _ = corpus.tokens(d0, d1)
        T = torch.from_numpy(tk.astype(np.float64) / 2048.0).to(device)  # [rows, d]
        lens = torch.from_numpy(corpus.lengths[d0:d1].astype(np.int64)).to(device)
        doc = torch.repeat_interleave(torch.arange(d1 - d0, device=device), lens)
        S = torch.matmul(Q.reshape(nq * Tq, -1), T.T).reshape(nq, Tq, -1)
        best = torch.full((nq, Tq, d1 - d0), -float("inf"), dtype=torch.float64, device=device)
        best.scatter_reduce_(2, doc.view(1, 1, -1).expand(nq, Tq, -1), S, reduce="amax", include_self=True)
        F[:, d0:d1] = best.sum(dim=1)  # exact
        if time.perf_counter() - t_log > 20:
            log(f"exact MaxSim reference: {d1}/{nd} docs")
            t_log = time.perf_counter()
    order = torch.sort(F, dim=1, descending=True, stable=True).indices[:, :k]
    return order.cpu().numpy()


def source_sha(name):
    p = os.path.join(ROOT, "paper_2608_23553_amd", "csrc", name)
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def measured_traffic(stage, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source; else None."""
    p = os.path.join(ROOT, "profiles", f"traffic_{KERNEL_OF_STAGE[stage]}_{workload}.json")
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if d.get("source_sha256_16") != source_sha(SOURCE_OF_STAGE[stage]):
        return None
    return d.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="100k")
    ap.add_argument("--nq", type=int, default=0, help="override the batch size")
    ap.add_argument("--ncand", type=int, default=0, help="override the documents kept by the refinement")
    ap.add_argument("--refine", choices=["centroid", "token"], default="centroid",
                    help="refinement score: probed centroids' (chimera_search) or retrieved tokens' decoded "
                         "scores (chimera_search_refine)")
    ap.add_argument("--latency-iters", type=int, default=300)
    ap.add_argument("--recall-queries", type=int, default=64)
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU-oracle sample duration")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kfb", type=int, default=0, help="full-precision budget of the collaborative scoring "
                                                         "(default 4 k)")
    ap.add_argument("--chunks", type=int, default=4, help="chunks of the collaborative scoring")
    ap.add_argument("--no-collab", action="store_true", help="skip the collaborative-scoring measurement")
    ap.add_argument("--profile", action="store_true", help="warmup + timed steps only (for rocprofv3)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (calibrates rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_each_way": src.numel() * 4, "copies": 3}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only: the whole index is resident in one "
                                   "GPU's HBM and no multi-GPU path exists; run with --gpus 1"}))
        sys.exit(2)
    os.environ["CHIMERA_STAGE_TIMING"] = "1"

    import numpy as np
    import torch
    import synth
    from paper_2608_23553_amd import ChimeraError  # noqa: F401

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    dev = torch.device("cuda:0")
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 8)
    w = synth.WORKLOADS[args.workload]
    if args.nq:
        w = w.scaled(nq=args.nq)
    if args.ncand:
        w = w.scaled(ncand=args.ncand)
    from paper_2608_23553_amd import chimera as _ch
    rmode = _ch.REFINE_TOKEN if args.refine == "token" else _ch.REFINE_CENTROID
    corpus, builder = build_corpus_index(w, threads)
    idx = builder.upload(0)
    info = idx.info()
    q_k, q_src = corpus.queries(w.nq, w.Tq)
    Q = torch.from_numpy(synth.k_to_bf16_bits(q_k).view(np.int16)).to(dev).view(torch.bfloat16)
    ids = torch.empty((w.nq, w.k), dtype=torch.int32, device=dev)
    scores = torch.empty((w.nq, w.k), dtype=torch.float32, device=dev)

    # ---- timed region: K whole-batch searches
    for _ in range(args.warmup):
        idx.search(Q, w.nprobe, w.ncand, w.k, out=(ids, scores), refine=rmode)
    torch.cuda.synchronize()
    idx.stage_times()  # clear warm-up events
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        idx.search(Q, w.nprobe, w.ncand, w.k, out=(ids, scores), refine=rmode)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st = idx.stage_times()
    elapsed = t1 - t0
    qps = w.nq * args.steps / elapsed
    nsub = max(1, int(round(st[6])))
    stage_ms = {s: float(st[i]) / args.steps for i, s in enumerate(STAGES)}
    launches = nsub  # launches of each kernel over the timed steps
    log(f"{args.steps} steps in {elapsed:.3f}s: {qps:.0f} QPS; stages ms/step {stage_ms}")
    if args.profile:
        print(json.dumps({"metric": METRIC, "value": qps, "profile_only": True}))
        return

    # ---- algorithmic work of one step, from the stage taps and host copies
    log("counting the step's algorithmic work")
    ci, _ = idx.probe(Q, w.nprobe)
    cand, _, nval = idx.prune(Q, w.nprobe, w.ncand, refine=rmode)
    torch.cuda.synchronize()
    sec = builder.sections()
    lens = np.diff(sec["doc_off"])
    ci = ci.cpu().numpy()
    list_len = np.diff(sec["ivf_off"])
    entries = int(list_len[ci].sum())  # every probed (token, centroid) list, as the paper counts them
    # what the walk reads: each rank's distinct centroids once per query, except
    # the dense lists (up to 64 lists holding more than ndocs/16 docs, longest
    # first, ties to the lower id), which it applies from 8-byte per-doc masks
    dense_c = np.nonzero(list_len * 16 > w.ndocs)[0]
    dense_c = dense_c[np.lexsort((dense_c, -list_len[dense_c]))][:64]
    walked_len = list_len.copy()
    walked_len[dense_c] = 0
    walked = sum(int(walked_len[np.unique(ci[q, :, r])].sum()) for q in range(w.nq) for r in range(w.nprobe))
    walk_bytes = 4.0 * walked + (8.0 if len(dense_c) else 0.0) * w.nq * w.ndocs + 4.0 * w.nq * w.ndocs
    if rmode == _ch.REFINE_TOKEN:
        # every token of every probed list: its id, its document and its code
        tok_len = np.bincount(sec["cid"], minlength=w.ncent)
        walked = int(tok_len[ci].sum())
        walk_bytes = (8.0 + 16 * w.nbits) * walked + 4.0 * w.nq * w.ndocs
    cand, nval = cand.cpu().numpy(), nval.cpu().numpy()
    scored_tokens = int(sum(lens[cand[q, :nval[q]]].sum() for q in range(w.nq)))
    code_bytes_tok = 16 * w.nbits + 4
    work = {
        "probe": ("mfma", 2.0 * w.nq * w.Tq * w.ncent * 128, BF16_PEAK_TFLOPS, "TFLOP/s"),
        "walk": ("hbm", walk_bytes, HBM_PEAK_GBS, "GB/s"),
        "select": ("hbm", 8.0 * w.nq * w.ndocs, HBM_PEAK_GBS, "GB/s"),
        "score": ("hbm", float(code_bytes_tok * scored_tokens), HBM_PEAK_GBS, "GB/s"),
        "topk": ("hbm", 8.0 * int(nval.sum()), HBM_PEAK_GBS, "GB/s"),
        "round": ("hbm", 2.0 * 2 * w.nq * w.Tq * 128, HBM_PEAK_GBS, "GB/s"),
    }
    dominant = max(STAGES, key=lambda s: stage_ms[s])
    bound, amount, peak, unit = work[dominant]
    per_launch_s = stage_ms[dominant] * args.steps / launches / 1e3
    per_launch_amount = amount * args.steps / launches
    achieved = per_launch_amount / per_launch_s / (1e12 if unit == "TFLOP/s" else 1e9)
    # the committed counter summary describes the default configuration only
    default_cfg = not (args.nq or args.ncand or args.refine != "centroid")
    traffic = measured_traffic(dominant, w.name) if default_cfg else None
    roofline = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
                "traffic": traffic, "kernel": KERNEL_OF_STAGE[dominant],
                "per_launch": {"algorithmic": per_launch_amount, "ms": per_launch_s * 1e3}}
    score_gbs = work["score"][1] / (stage_ms["score"] / 1e3) / 1e9
    probe_tflops = work["probe"][1] / (stage_ms["probe"] / 1e3) / 1e12

    # ---- latency at nq=1 (H2D of the query, search, D2H of the results)
    log("latency at nq=1")
    nlat = args.latency_iters
    lq, _ = corpus.queries(nlat, w.Tq, query_seed=99)
    host_q = torch.from_numpy(synth.k_to_bf16_bits(lq).view(np.int16)).view(torch.bfloat16).pin_memory()
    dq = torch.empty((1, w.Tq, 128), dtype=torch.bfloat16, device=dev)
    o_ids = torch.empty((1, w.k), dtype=torch.int32, device=dev)
    o_sc = torch.empty((1, w.k), dtype=torch.float32, device=dev)
    h_ids = torch.empty((1, w.k), dtype=torch.int32).pin_memory()
    h_sc = torch.empty((1, w.k), dtype=torch.float32).pin_memory()
    for i in range(5):
        idx.search(dq.copy_(host_q[i:i + 1]), w.nprobe, w.ncand, w.k, out=(o_ids, o_sc), refine=rmode)
    torch.cuda.synchronize()
    idx.stage_times()
    lat = []
    for i in range(nlat):
        s = time.perf_counter()
        dq.copy_(host_q[i:i + 1], non_blocking=True)
        idx.search(dq, w.nprobe, w.ncand, w.k, out=(o_ids, o_sc), refine=rmode)
        h_ids.copy_(o_ids, non_blocking=True)
        h_sc.copy_(o_sc, non_blocking=True)
        torch.cuda.synchronize()
        lat.append((time.perf_counter() - s) * 1e3)
    lat = np.array(lat)
    lat_stage = idx.stage_times()
    lat_stage_ms = {s: float(lat_stage[i]) / nlat for i, s in enumerate(STAGES)}

    # ---- QPS at smaller batches (the same index and queries, resident in HBM)
    log("QPS at smaller batches")
    qps_by_batch = {}
    for nb in sorted({1, 8, 32, 128, w.nq}):
        if nb > w.nq:
            continue
        reps = max(3, min(50, int(2048 // nb)))
        bi = torch.empty((nb, w.k), dtype=torch.int32, device=dev)
        bs = torch.empty((nb, w.k), dtype=torch.float32, device=dev)
        idx.search(Q[:nb], w.nprobe, w.ncand, w.k, out=(bi, bs), refine=rmode)
        torch.cuda.synchronize()
        s = time.perf_counter()
        for _ in range(reps):
            idx.search(Q[:nb], w.nprobe, w.ncand, w.k, out=(bi, bs), refine=rmode)
        torch.cuda.synchronize()
        qps_by_batch[str(nb)] = nb * reps / (time.perf_counter() - s)
    idx.stage_times()  # drop these searches' events
    log(f"QPS by batch: {qps_by_batch}")

    # ---- recall@k against exact MaxSim
    log("recall against exact MaxSim")
    nr = min(args.recall_queries, w.nq)
    truth = exact_topk_gpu(q_k[:nr], corpus, w.k, dev)
    got = ids[:nr].cpu().numpy()
    recall = float(np.mean([len(set(got[i]) & set(truth[i])) / w.k for i in range(nr)]))
    src_first = float(np.mean(got[:, 0] == q_src[:nr]))

    # ---- CPU-GPU collaborative scoring (Alg. 3): the GPU path's candidates
    # re-ranked on the host from the full-precision tokens, chunk by chunk
    collab = None
    fb_bytes = info["ntokens"] * 2 * 128
    if not args.no_collab and fb_bytes <= 32 * 2**30:
        kfb = args.kfb or 4 * w.k
        log(f"collaborative scoring: kfb {kfb}, {args.chunks} chunks, {threads} host threads")
        tk, _ = corpus.tokens()
        fb = synth.k_to_bf16_bits(tk)
        del tk
        idx.attach_fullbit(fb)  # the index keeps its own grid copy
        del fb
        runs = {}
        for c in (args.chunks, 1):
            idx.search_collab(Q, w.nprobe, w.ncand, kfb, c, w.k, nthreads=threads)  # warm-up
            reps, s = 3, time.perf_counter()
            for _ in range(reps):
                cids, _, nfull = idx.search_collab(Q, w.nprobe, w.ncand, kfb, c, w.k, nthreads=threads)
            runs[c] = (w.nq * reps / (time.perf_counter() - s), cids, nfull)
            log(f"  chunks {c}: {runs[c][0]:.0f} QPS, full-precision scores per query "
                f"mean {nfull.mean():.2f} max {nfull.max()}")
        idx.attach_fullbit(None)
        qc, cids, nfull = runs[args.chunks]
        collab = {"qps": qc, "qps_one_chunk": runs[1][0], "kfb": kfb, "chunks": args.chunks, "host_threads": threads,
                  "k_hat_full_bit_mean": float(nfull.mean()), "k_hat_full_bit_max": int(nfull.max()),
                  "recall_at_k": float(np.mean([len(set(cids[i]) & set(truth[i])) / w.k for i in range(nr)])),
                  "recall_queries": nr}
    elif not args.no_collab:
        collab = {"skipped": f"the full-precision host store would take {fb_bytes / 2**30:.0f} GiB"}

    # ---- CPU baseline: the oracle, untouched, on a bounded sample
    log("CPU baseline")
    cpu = None
    # the oracle keeps every raw token (256 B) and its unpacked codes (128 B)
    oracle_bytes = info["ntokens"] * (2 * 128 + 128)
    if not args.no_cpu_baseline and oracle_bytes > 64 * 2**30:
        log(f"CPU baseline skipped: the oracle's in-memory index would take {oracle_bytes / 2**30:.0f} GiB")
        cpu = {"value": None, "kind": "oracle",
               "skipped": f"the oracle's in-memory index needs {oracle_bytes / 2**30:.0f} GiB of host memory"}
    elif not args.no_cpu_baseline:
        import oracle
        tk, cl = corpus.tokens()
        oi = oracle.OracleIndex(corpus.centroids_k, corpus.doc_off, cl, w.nbits, tok_k=tk)
        del tk
        probe_n = min(w.nq, max(1, threads))  # one query per thread
        s = time.perf_counter()
        oi.search(q_k[:probe_n], w.nprobe, w.ncand, w.k, nthreads=threads, refine=args.refine == "token")
        t_probe = time.perf_counter() - s
        n_cpu = int(min(w.nq, max(probe_n, probe_n * args.cpu_seconds / max(t_probe, 1e-3) // probe_n * probe_n)))
        s = time.perf_counter()
        ref = oi.search(q_k[:n_cpu], w.nprobe, w.ncand, w.k, nthreads=threads, refine=args.refine == "token")
        t_cpu = time.perf_counter() - s
        agree = bool(np.array_equal(ref["ids"], ids[:n_cpu].cpu().numpy()))
        cpu = {"value": n_cpu / t_cpu, "unit": "queries/s", "cores": threads, "kind": "oracle",
               "sample": f"first {n_cpu} of the {w.nq} benchmark queries, whole path (probe, candidates, F', "
                         f"top-ncand, document scores, top-k), {threads} threads over queries, {t_cpu:.1f}s",
               "ids_match_gpu": agree}

    out = {
        "metric": METRIC, "value": qps, "unit": "queries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": describe(w), "ndocs": w.ndocs, "ntokens": info["ntokens"], "ncent": w.ncent,
                   "nbits": w.nbits, "nq": w.nq, "Tq": w.Tq, "nprobe": w.nprobe, "ncand": w.ncand, "k": w.k,
                   "refine": args.refine,
                   "index_device_bytes": info["device_bytes"]},
        "recall_at_k": recall, "recall_queries": nr, "source_doc_top1": src_first, "qps_by_batch": qps_by_batch,
        "p50_ms_nq1": float(np.percentile(lat, 50)), "p95_ms_nq1": float(np.percentile(lat, 95)),
        "p99_ms_nq1": float(np.percentile(lat, 99)), "nq1_stages_ms": lat_stage_ms,
        "code_scan_GBps": score_gbs, "probe_TFLOPs": probe_tflops, "stages_ms": stage_ms,
        "work_per_step": {"posting_entries": entries, "posting_entries_walked": walked, "scored_tokens": scored_tokens,
                          "candidates": int(nval.sum())},
        "roofline": roofline, "cpu_baseline": cpu, "collab": collab,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
