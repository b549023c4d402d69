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
                   batch, when its host store fits: QPS with chunks and with
                   one chunk, full-precision scores per query, recall@k

The default workload is the 8.8M-document corpus with MS MARCO's shape (4,096
queries x 32 tokens, nprobe 16, ncand 16,384, k 100); ``--workload`` selects
another.  The corpus is generated on the host in two passes over document
chunks: the first feeds the builder's residual histogram, the exact-Chamfer
reference on the GPU and the oracle's view of the corpus (for the CPU
baseline); the second feeds the builder's codes.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "QPS at fixed recall@k (batch) + p50 latency nq=1; code-scan HBM GB/s"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
STAGES = ["round", "probe", "walk", "select", "score", "topk"]
RABITQ_SEED = 20260
KERNEL_OF_STAGE = {"probe": "k_probe", "walk": "k_cand_walk", "select": "k_select", "score": "k_residual_score",
                   "topk": "k_topk", "round": "k_round_queries"}
SOURCE_OF_STAGE = {"probe": "k_probe.hip", "walk": "k_prune.hip", "select": "k_prune.hip",
                   "score": "k_score.hip", "topk": "k_score.hip", "round": "k_probe.hip"}


def host_memory_fits(nbytes: int, cap: float = 240 * 2**30):
    """Whether a host allocation of nbytes fits beside this process: under
    the available memory with 16 GiB to spare, and under cap in total."""
    rss = avail = 0
    try:
        with open("/proc/self/status") as f:
            for line in f:
                if line.startswith("VmRSS:"):
                    rss = int(line.split()[1]) * 1024
        with open("/proc/meminfo") as f:
            for line in f:
                if line.startswith("MemAvailable:"):
                    avail = int(line.split()[1]) * 1024
    except OSError:
        return False, "host memory unknown"
    log(f"host memory: {rss / 2**30:.1f} GiB in use, {avail / 2**30:.0f} GiB available, {nbytes / 2**30:.1f} GiB wanted")
    if nbytes + 16 * 2**30 > avail or nbytes + rss > cap:
        return False, (f"the full-precision host store would take {nbytes / 2**30:.0f} GiB beside "
                       f"{rss / 2**30:.0f} GiB in use ({avail / 2**30:.0f} GiB available)")
    return True, ""


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def describe(w) -> str:
    lens = {0: f"exactly {w.len_lo} tokens", 1: f"lognormal length mean {w.len_mean:g} in [{w.len_lo},{w.len_hi}]",
            2: f"uniform length in [{w.len_lo},{w.len_hi}]"}[w.len_kind]
    pop = "uniform" if w.pop_kind == 0 else f"Zipf({w.zipf_s:g})"
    return (f"{w.name}: {w.ndocs:,} docs ({lens}), dim {w.dim}, {w.ncent:,} {pop} centroids, {w.nbits}-bit residual "
            f"codes; {w.nq} queries x {w.Tq} tokens; nprobe {w.nprobe}, ncand {w.ncand}, k {w.k}")


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


# --------------------------------------------------------------- recall reference
def chamfer_block(Qf, T, lens):
    """Exact Chamfer scores F[q, v] = sum_j max_{t in v} <Q_j, t> (Def. 1) of a
    block of documents.  Qf [nq, Tq, d] float64, T [rows, d] float64 holding
    the documents' tokens back to back, lens [n] int64 (host).  Every value is
    a grid value, so each product and sum is exact in float64 and F is exact.
    Documents of one length are scored together, so no padding enters a max."""
    import numpy as np
    import torch
    nq, Tq, d = Qf.shape
    lens = np.asarray(lens, dtype=np.int64)
    off = np.zeros(len(lens) + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    F = torch.empty((nq, len(lens)), dtype=torch.float64, device=Qf.device)
    A = Qf.reshape(nq * Tq, d)
    tile_rows = 1 << 18
    for L in np.unique(lens):
        docs = np.nonzero(lens == L)[0]
        per = max(1, tile_rows // int(L))
        for i in range(0, len(docs), per):
            dt = docs[i:i + per]
            rows = (off[dt][:, None] + np.arange(L)[None, :]).reshape(-1)
            S = A @ T[torch.from_numpy(rows).to(T.device)].T  # [nq*Tq, nt*L]
            F[:, torch.from_numpy(dt).to(T.device)] = S.view(nq, Tq, len(dt), int(L)).amax(dim=3).sum(dim=1)
    return F


def topk_ids(F, k):
    """The k best documents of each row by (score desc, id asc)."""
    import torch
    return torch.sort(F, dim=1, descending=True, stable=True).indices[:, :k]


class ExactReference:
    """Exact Chamfer scores of the recall queries over the whole corpus,
    accumulated chunk by chunk on the device as the corpus is generated."""

    def __init__(self, q_k, ndocs, device):
        import numpy as np
        import torch
        self.Qf = torch.from_numpy(q_k.astype(np.float64) / 2048.0).to(device)
        self.F = torch.empty((q_k.shape[0], ndocs), dtype=torch.float64, device=device)
        self.device = device

    def feed(self, k_chunk, lens, d0):
        import torch
        T = torch.from_numpy(k_chunk).to(self.device).to(torch.float64).mul_(1.0 / 2048.0)
        self.F[:, d0:d0 + len(lens)] = chamfer_block(self.Qf, T, lens)

    def topk(self, k):
        return topk_ids(self.F, k).cpu().numpy()


# --------------------------------------------------------------- CPU baseline
class OracleView:
    """The CPU baseline's oracle: its own quantiser (residual histogram) and
    assignment, accumulated from the same generated chunks; documents are
    regenerated when a query scores them (oracle.search_streamed)."""

    def __init__(self, corpus, threads):
        import numpy as np
        from concurrent.futures import ThreadPoolExecutor
        self.corpus, self.threads = corpus, threads
        self.hist = np.zeros(8193, dtype=np.int64)
        self.cid = np.empty(corpus.ntok, dtype=np.int32)
        self.pool = ThreadPoolExecutor(max_workers=threads)

    def feed(self, k_chunk, cl, d0, d1):
        import numpy as np
        import oracle
        c = self.corpus
        n = len(cl)
        cuts = np.linspace(0, n, self.threads + 1).astype(np.int64)
        parts = self.pool.map(lambda i: oracle.residual_hist(k_chunk[cuts[i]:cuts[i + 1]], cl[cuts[i]:cuts[i + 1]],
                                                             c.centroids_k), range(self.threads))
        self.hist += np.sum(list(parts), axis=0)
        self.cid[c.doc_off[d0]:c.doc_off[d1]] = cl

    def run(self, w, q_k, gpu_ids, seconds):
        """Whole queries in batches of one per thread until `seconds` pass."""
        import numpy as np
        import oracle
        import synth
        t = time.perf_counter()
        oi = oracle.OracleIndex(self.corpus.centroids_k, self.corpus.doc_off, self.cid, w.nbits, hist=self.hist,
                                with_codes=False)
        log(f"CPU baseline: oracle view built in {time.perf_counter() - t:.1f}s")
        regen = synth.Corpus(w.corpus_spec(), nthreads=1)  # one thread per query

        lat = []

        def one(qi):
            t1 = time.perf_counter()
            r = oracle.search_streamed(oi, q_k[qi], w.nprobe, w.ncand, w.k, regen.docs_tokens)
            lat.append(time.perf_counter() - t1)
            return r

        done, agree = 0, True
        t0 = time.perf_counter()
        while done < w.nq and time.perf_counter() - t0 < seconds:
            batch = list(range(done, min(w.nq, done + self.threads)))
            for qi, ref in zip(batch, self.pool.map(one, batch)):
                m = len(ref["ids"])
                agree &= bool(np.array_equal(ref["ids"], gpu_ids[qi, :m]))
            done += len(batch)
            log(f"CPU baseline: {done} queries in {time.perf_counter() - t0:.1f}s")
        t_cpu = time.perf_counter() - t0
        self.pool.shutdown()
        return {"value": done / t_cpu, "unit": "queries/s", "cores": self.threads, "kind": "oracle",
                "cpu_model": cpu_model(), "s_per_query_one_thread": float(np.median(lat)) if lat else None,
                "sample": f"first {done} of the {w.nq} benchmark queries, whole path (probe, candidates, F', "
                          f"top-ncand, document scores, top-k), {self.threads} threads, one query each, "
                          f"{t_cpu:.1f}s",
                "ids_match_gpu": agree}


# --------------------------------------------------------------- index build
def build(w, corpus, threads, ref, view, docs_per_chunk, rabitq_signs=None):
    """Two passes over the corpus; returns the product builder."""
    import synth
    from paper_2608_23553_amd import Builder
    b = Builder(synth.k_to_bf16_bits(corpus.centroids_k), w.nbits)
    if rabitq_signs is not None:
        b.rabitq(rabitq_signs)
    nd = w.ndocs
    t, t_log = time.perf_counter(), time.perf_counter()
    for d0 in range(0, nd, docs_per_chunk):
        d1 = min(nd, d0 + docs_per_chunk)
        k, bf, cl = corpus.tokens_ex(d0, d1, want_k=ref is not None or view is not None)
        b.add_residuals(bf, cl)
        if ref is not None:
            ref.feed(k, corpus.lengths[d0:d1], d0)
        if view is not None:
            view.feed(k, cl, d0, d1)
        if time.perf_counter() - t_log > 15 or d1 == nd:
            log(f"pass 1 (residuals, reference, oracle view): {d1}/{nd} docs, {time.perf_counter() - t:.0f}s")
            t_log = time.perf_counter()
    b.freeze()
    b.reserve(nd, corpus.ntok)
    for d0 in range(0, nd, docs_per_chunk):
        d1 = min(nd, d0 + docs_per_chunk)
        _, bf, cl = corpus.tokens_ex(d0, d1, want_k=False)
        b.add_docs(bf, cl, corpus.lengths[d0:d1])
        if time.perf_counter() - t_log > 15 or d1 == nd:
            log(f"pass 2 (codes): {d1}/{nd} docs, {time.perf_counter() - t:.0f}s")
            t_log = time.perf_counter()
    log(f"index built on host in {time.perf_counter() - t:.1f}s: {b.info()}")
    return b


def source_sha(name):
    p = os.path.join(ROOT, "paper_2608_23553_amd", "csrc", name)
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def measured_traffic(stage, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel and host source; else None."""
    p = os.path.join(ROOT, "profiles", f"traffic_{KERNEL_OF_STAGE[stage]}_{workload}.json")
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if d.get("source_sha256_16") != source_sha(SOURCE_OF_STAGE[stage]):
        return None
    # the host code sizes the sub-batches, and with them what one launch covers
    if "host_sha256_16" in d and d["host_sha256_16"] != source_sha("api.cpp"):
        return None
    return d.get("hbm_bytes_per_launch")


CHIMERA_MAX_NCAND = 1 << 20


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="8.8m")
    ap.add_argument("--nq", type=int, default=0, help="override the batch size")
    ap.add_argument("--ncand", type=int, default=0, help="override the documents kept by the refinement")
    ap.add_argument("--nprobe", type=int, default=0, help="override the centroids probed per query token")
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
    ap.add_argument("--delete-frac", type=float, default=0.0,
                    help="finally delete this seeded fraction of the documents and time searches with the deletion "
                         "bitmap, the compaction, and searches after it")
    ap.add_argument("--rabitq", action="store_true",
                    help="also encode RaBitQ codes (B = 4) and measure the 1-bit GPU scoring and the 4-bit host "
                         "re-rank (the encoder takes about 50 us per token per host thread)")
    ap.add_argument("--no-recall-sweep", action="store_true",
                    help="skip the QPS / recall sweep over larger nprobe and ncand")
    ap.add_argument("--docs-per-chunk", type=int, default=100_000, help="documents per generated chunk")
    ap.add_argument("--profile", action="store_true",
                    help="warmup + timed steps only (for rocprofv3): no reference, oracle or extra legs")
    ap.add_argument("--save-index", default="", help="also write the built index to this file")
    ap.add_argument("--load-index", default="",
                    help="load the index from this file (chimera_index_load) instead of building it; "
                         "only with --profile")
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
    if args.load_index and not args.profile:
        print(json.dumps({"error": "--load-index is for --profile runs (the reference and the oracle view are "
                                   "built from the generated corpus)"}))
        sys.exit(2)
    os.environ["CHIMERA_STAGE_TIMING"] = "1"

    import numpy as np
    import torch
    import synth
    from paper_2608_23553_amd import Index
    from paper_2608_23553_amd import chimera as _ch

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    dev = torch.device("cuda:0")
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 8)
    w = synth.WORKLOADS[args.workload]
    for key in ("nq", "ncand", "nprobe"):
        if getattr(args, key):
            w = w.scaled(**{key: getattr(args, key)})
    rmode = _ch.REFINE_TOKEN if args.refine == "token" else _ch.REFINE_CENTROID
    log(f"workload {describe(w)}; {threads} host threads ({cpu_model()})")
    corpus = synth.Corpus(w.corpus_spec(), nthreads=threads)
    q_k, q_src = corpus.queries(w.nq, w.Tq)
    nr = min(args.recall_queries, w.nq)
    ref = view = builder = None
    if args.load_index:
        t = time.perf_counter()
        idx = Index.load(args.load_index, 0)
        log(f"index loaded in {time.perf_counter() - t:.1f}s")
    else:
        if not args.profile:
            ref = ExactReference(q_k[:nr], w.ndocs, dev)
            if not args.no_cpu_baseline:
                view = OracleView(corpus, threads)
        builder = build(w, corpus, threads, ref, view, args.docs_per_chunk,
                        rabitq_signs=synth.rotation_signs(RABITQ_SEED) if args.rabitq else None)
        if args.save_index:
            t = time.perf_counter()
            builder.save(args.save_index)
            log(f"index saved in {time.perf_counter() - t:.1f}s")
        t = time.perf_counter()
        idx = builder.upload(0)
        log(f"index uploaded in {time.perf_counter() - t:.1f}s")
    info = idx.info()
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
        print(json.dumps({"metric": METRIC, "value": qps, "profile_only": True, "stages_ms": stage_ms}), flush=True)
        return

    # ---- algorithmic work of one step, from the stage taps and host copies
    log("counting the step's algorithmic work")
    ci, _ = idx.probe(Q, w.nprobe)
    cand, _, nval = idx.prune(Q, w.nprobe, w.ncand, refine=rmode)
    torch.cuda.synchronize()
    sec = builder.sections(("doc_off", "ivf_off") + (("cid",) if rmode == _ch.REFINE_TOKEN else ()))
    builder.close()
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
    del sec
    cand, nval = cand.cpu().numpy(), nval.cpu().numpy()
    scored_tokens = int(sum(lens[cand[q, :nval[q]]].sum() for q in range(w.nq)))
    code_bytes_tok = 16 * w.nbits + 4
    work = {
        "probe": ("mfma", 2.0 * w.nq * w.Tq * w.ncent * 128, BF16_PEAK_TFLOPS, "TFLOP/s"),
        "walk": ("hbm", walk_bytes, HBM_PEAK_GBS, "GB/s"),
        "select": ("hbm", 4.0 * w.nq * w.ndocs, HBM_PEAK_GBS, "GB/s"),  # one read of F'
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
    default_cfg = not (args.nq or args.ncand or args.nprobe or args.refine != "centroid")
    traffic = measured_traffic(dominant, w.name) if default_cfg else None
    roofline = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
                "traffic": traffic, "kernel": KERNEL_OF_STAGE[dominant],
                "per_launch": {"algorithmic": per_launch_amount, "ms": per_launch_s * 1e3, "launches_per_step":
                               launches / args.steps}}
    stage_rooflines = {}
    for s in STAGES:
        bd, am, pk, un = work[s]
        if stage_ms[s] > 0:
            a = am / (stage_ms[s] / 1e3) / (1e12 if un == "TFLOP/s" else 1e9)
            stage_rooflines[s] = {"bound": bd, "achieved": a, "unit": un, "frac": a / pk}
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
    for nb in sorted({1, 8, 32, 128, 512, w.nq}):
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

    # ---- recall@k against exact MaxSim (reference accumulated during the build)
    truth = ref.topk(w.k)
    got = ids[:nr].cpu().numpy()
    recall = float(np.mean([len(set(got[i]) & set(truth[i])) / w.k for i in range(nr)]))
    src_first = float(np.mean(got[:, 0] == q_src[:nr]))
    del ref

    # ---- QPS at fixed recall@k: the same batch with more probed centroids
    # and more kept candidates, each timed over 2 whole-batch searches
    sweep, qps_at = None, None
    if not args.no_recall_sweep:
        sweep = [{"path": "gpu", "nprobe": w.nprobe, "ncand": w.ncand, "qps": qps, "recall_at_k": recall}]
        si = torch.empty_like(ids)
        ss = torch.empty_like(scores)
        for mp, mc in ((2, 1), (2, 2), (4, 2), (4, 4)):
            npb, nc = min(64, w.nprobe * mp, w.ncent), min(w.ncand * mc, CHIMERA_MAX_NCAND, w.ndocs)
            if any(e["nprobe"] == npb and e["ncand"] == nc for e in sweep):
                continue
            try:
                idx.search(Q, npb, nc, w.k, out=(si, ss), refine=rmode)
            except _ch.ChimeraError as e:  # e.g. a walk state beyond the LDS (Tq x nprobe)
                sweep.append({"path": "gpu", "nprobe": npb, "ncand": nc, "error": str(e)})
                log(f"sweep nprobe {npb} ncand {nc}: {e}")
                continue
            torch.cuda.synchronize()
            s0 = time.perf_counter()
            for _ in range(2):
                idx.search(Q, npb, nc, w.k, out=(si, ss), refine=rmode)
            torch.cuda.synchronize()
            q_s = 2 * w.nq / (time.perf_counter() - s0)
            g = si[:nr].cpu().numpy()
            r = float(np.mean([len(set(g[i]) & set(truth[i])) / w.k for i in range(nr)]))
            sweep.append({"path": "gpu", "nprobe": npb, "ncand": nc, "qps": q_s, "recall_at_k": r})
            log(f"sweep nprobe {npb} ncand {nc}: {q_s:.0f} QPS, recall@{w.k} {r:.3f}")
        if len(sweep) > 1 and any("qps" in e for e in sweep[1:]):
            idx.stage_times()  # drop these searches' events
        qps_at = {str(t): max((e["qps"] for e in sweep if e.get("recall_at_k", 0) >= t), default=None)
                  for t in (0.8, 0.9, 0.95)}

    # ---- RaBitQ codes (Sec. 2.2, Sec. 3.1): the same candidates scored on
    # the GPU from the 1-bit codes (no S^T table), then re-ranked on the host
    # from the 4-bit codes (Alg. 3)
    rabitq = None
    if args.rabitq and info.get("rabitq", True):
        log("RaBitQ: 1-bit GPU scoring")
        for _ in range(args.warmup):
            idx.search_rabitq(Q, w.nprobe, w.ncand, w.k, out=(ids, scores))
        torch.cuda.synchronize()
        idx.stage_times()
        s = time.perf_counter()
        for _ in range(args.steps):
            idx.search_rabitq(Q, w.nprobe, w.ncand, w.k, out=(ids, scores))
        torch.cuda.synchronize()
        el = time.perf_counter() - s
        rst = idx.stage_times()
        r_stage = {sname: float(rst[i]) / args.steps for i, sname in enumerate(STAGES)}
        rq_scan = 20.0 * scored_tokens  # 16 B of sign bits and a 4 B factor per scored token
        got = ids[:nr].cpu().numpy()
        rabitq = {"qps": w.nq * args.steps / el, "stages_ms": r_stage,
                  "recall_at_k": float(np.mean([len(set(got[i]) & set(truth[i])) / w.k for i in range(nr)])),
                  "score_roofline": {"bound": "hbm", "achieved": rq_scan / (r_stage["score"] / 1e3) / 1e9,
                                     "unit": "GB/s", "frac": rq_scan / (r_stage["score"] / 1e3) / 1e9 / HBM_PEAK_GBS,
                                     "bytes_per_token": 20}}
        log(f"  {rabitq['qps']:.0f} QPS, recall@{w.k} {rabitq['recall_at_k']:.3f}, stages {r_stage}")
        kfb = args.kfb or 4 * w.k
        idx.search_collab_rabitq(Q, w.nprobe, w.ncand, kfb, args.chunks, w.k, nthreads=threads)  # warm-up
        reps, s = 3, time.perf_counter()
        for _ in range(reps):
            cids, _, nfull = idx.search_collab_rabitq(Q, w.nprobe, w.ncand, kfb, args.chunks, w.k, nthreads=threads)
        rabitq["collab"] = {"qps": w.nq * reps / (time.perf_counter() - s), "kfb": kfb, "chunks": args.chunks,
                            "k_hat_full_bit_mean": float(nfull.mean()),
                            "recall_at_k": float(np.mean([len(set(cids[i]) & set(truth[i])) / w.k
                                                          for i in range(nr)]))}
        log(f"  4-bit host re-rank: {rabitq['collab']['qps']:.0f} QPS, "
            f"recall@{w.k} {rabitq['collab']['recall_at_k']:.3f}")

    # ---- CPU-GPU collaborative scoring (Alg. 3): the GPU path's candidates
    # re-ranked on the host from the full-precision tokens, chunk by chunk.
    # The store is generated and attached in ranges of documents, so the
    # process holds it once (150 GB at 8.8M)
    collab = None
    fb_bytes = info["ntokens"] * 2 * 128
    fits, why = host_memory_fits(fb_bytes)
    if not args.no_collab and fits:
        kfb = args.kfb or 4 * w.k
        log(f"collaborative scoring: kfb {kfb}, {args.chunks} chunks, {threads} host threads; "
            f"attaching a {fb_bytes / 2**30:.1f} GiB full-precision store")
        t_att = time.perf_counter()
        step_docs = max(1, int(2**32 // (256 * 180)))  # at most 4 GiB of tokens per range
        for d0 in range(0, w.ndocs, step_docs):
            d1 = min(w.ndocs, d0 + step_docs)
            _, fb, _ = corpus.tokens_ex(d0, d1, want_k=False, want_cluster=False)
            idx.attach_fullbit_range(fb, int(corpus.doc_off[d0]))  # the index keeps its own grid copy
            del fb
        log(f"  attached in {time.perf_counter() - t_att:.1f}s")
        runs = {}
        for c in (args.chunks, 1):
            idx.search_collab(Q, w.nprobe, w.ncand, kfb, c, w.k, nthreads=threads)  # warm-up
            reps, s = 3, time.perf_counter()
            for _ in range(reps):
                cids, _, nfull = idx.search_collab(Q, w.nprobe, w.ncand, kfb, c, w.k, nthreads=threads)
            runs[c] = (w.nq * reps / (time.perf_counter() - s), cids, nfull)
            log(f"  chunks {c}: {runs[c][0]:.0f} QPS, full-precision scores per query "
                f"mean {nfull.mean():.2f} max {nfull.max()}")
        qc, cids, nfull = runs[args.chunks]
        collab = {"qps": qc, "qps_one_chunk": runs[1][0], "kfb": kfb, "chunks": args.chunks, "host_threads": threads,
                  "k_hat_full_bit_mean": float(nfull.mean()), "k_hat_full_bit_max": int(nfull.max()),
                  "recall_at_k": float(np.mean([len(set(cids[i]) & set(truth[i])) / w.k for i in range(nr)])),
                  "recall_queries": nr}
        log(f"  recall@{w.k} {collab['recall_at_k']:.3f}")
        if sweep is not None:
            sweep.append({"path": "collaborative", "nprobe": w.nprobe, "ncand": w.ncand, "kfb": kfb,
                          "chunks": args.chunks, "qps": qc, "recall_at_k": collab["recall_at_k"]})
            # a smaller full-precision budget (the paper's backward tuning,
            # Sec. 3.2): the fastest configuration that holds each target wins
            if not args.kfb and 2 * w.k < kfb:
                k2 = 2 * w.k
                idx.search_collab(Q, w.nprobe, w.ncand, k2, args.chunks, w.k, nthreads=threads)
                reps, s = 3, time.perf_counter()
                for _ in range(reps):
                    cids2, _, _ = idx.search_collab(Q, w.nprobe, w.ncand, k2, args.chunks, w.k, nthreads=threads)
                q2 = w.nq * reps / (time.perf_counter() - s)
                r2 = float(np.mean([len(set(cids2[i]) & set(truth[i])) / w.k for i in range(nr)]))
                sweep.append({"path": "collaborative", "nprobe": w.nprobe, "ncand": w.ncand, "kfb": k2,
                              "chunks": args.chunks, "qps": q2, "recall_at_k": r2})
                log(f"  kfb {k2}: {q2:.0f} QPS, recall@{w.k} {r2:.3f}")
            qps_at = {str(t): max((e["qps"] for e in sweep if e.get("recall_at_k", 0) >= t), default=None)
                      for t in (0.8, 0.9, 0.95)}
        idx.attach_fullbit(None)
    elif not args.no_collab:
        collab = {"skipped": why}

    # ---- CPU baseline: the oracle, untouched, on a bounded sample
    cpu = None
    if view is not None:
        log("CPU baseline")
        cpu = view.run(w, q_k, ids.cpu().numpy(), args.cpu_seconds)

    # ---- updates (Sec. 3.3): deletions through the bitmap, then compaction
    updates = None
    if args.delete_frac > 0:
        gone = np.nonzero(np.random.default_rng(5).random(w.ndocs) < args.delete_frac)[0]
        idx.delete(gone)

        def timed():
            idx.search(Q, w.nprobe, w.ncand, w.k, out=(ids, scores), refine=rmode)
            torch.cuda.synchronize()
            s0 = time.perf_counter()
            for _ in range(args.steps):
                idx.search(Q, w.nprobe, w.ncand, w.k, out=(ids, scores), refine=rmode)
            torch.cuda.synchronize()
            return w.nq * args.steps / (time.perf_counter() - s0)

        q_del = timed()
        got = ids.cpu().numpy()
        assert not np.isin(got[got >= 0], gone).any(), "a deleted document was returned"
        s0 = time.perf_counter()
        idx.compact()
        t_compact = time.perf_counter() - s0
        q_cmp = timed()
        idx.stage_times()
        updates = {"deleted_docs": int(len(gone)), "qps_with_bitmap": q_del, "compact_s": t_compact,
                   "qps_after_compact": q_cmp, "qps_before": qps}
        log(f"updates: {len(gone)} documents deleted: {q_del:.0f} QPS with the bitmap, compaction "
            f"{t_compact:.1f}s, {q_cmp:.0f} QPS after it (before: {qps:.0f})")

    out = {
        "metric": METRIC, "value": qps, "unit": "queries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": describe(w), "ndocs": w.ndocs, "ntokens": info["ntokens"], "ncent": w.ncent,
                   "nbits": w.nbits, "nq": w.nq, "Tq": w.Tq, "nprobe": w.nprobe, "ncand": w.ncand, "k": w.k,
                   "refine": args.refine,
                   "index_device_bytes": info["device_bytes"]},
        "recall_at_k": recall, "recall_queries": nr, "source_doc_top1": src_first, "qps_by_batch": qps_by_batch,
        "recall_sweep": sweep, "qps_at_recall": qps_at,
        "p50_ms_nq1": float(np.percentile(lat, 50)), "p95_ms_nq1": float(np.percentile(lat, 95)),
        "p99_ms_nq1": float(np.percentile(lat, 99)), "nq1_stages_ms": lat_stage_ms,
        "code_scan_GBps": score_gbs, "probe_TFLOPs": probe_tflops, "stages_ms": stage_ms,
        "stage_rooflines": stage_rooflines,
        "work_per_step": {"posting_entries": entries, "posting_entries_walked": walked, "scored_tokens": scored_tokens,
                          "candidates": int(nval.sum())},
        "roofline": roofline, "cpu_baseline": cpu, "collab": collab, "rabitq": rabitq, "updates": updates,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
