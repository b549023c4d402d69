"""Full-size workloads for the GPU parity tests: the product index and the
oracle's view of the same corpus, built from one stream of generated chunks,
and the oracle's search on a few sampled queries.

The oracle never holds the codes of the whole corpus here.  It keeps the
assignment, its own quantiser (from a residual histogram accumulated over
the same chunks the product builder reads) and the posting lists, and
regenerates the tokens of a query's top-ncand documents to score them
(oracle.search_streamed, which composes the stage functions exactly as the
oracle's own search does; pinned by test_search_composes_stage_definitions
and test_sampled_oracle_equals_full_oracle)."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
import synth
from paper_2608_23553_amd import Builder


def host_threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 8)


def hist_parallel(pool, nthreads, k, cl, cent_k):
    """oracle.residual_hist of one chunk, split over threads (a sum of
    per-slice histograms)."""
    n = len(cl)
    cuts = np.linspace(0, n, nthreads + 1).astype(np.int64)
    parts = pool.map(lambda i: oracle.residual_hist(k[cuts[i]:cuts[i + 1]], cl[cuts[i]:cuts[i + 1]], cent_k),
                     range(nthreads))
    return np.sum(list(parts), axis=0)


def build_both(w, nthreads=0, docs_per_chunk=50_000, say=print):
    """Product Builder and OracleIndex (without codes) for workload w."""
    nthreads = nthreads or host_threads()
    c = synth.Corpus(w.corpus_spec(), nthreads=nthreads)
    b = Builder(synth.k_to_bf16_bits(c.centroids_k), w.nbits)
    hist = np.zeros(8193, dtype=np.int64)
    cid = np.empty(c.ntok, dtype=np.int32)
    nd = w.ndocs
    with ThreadPoolExecutor(max_workers=nthreads) as pool:
        for d0 in range(0, nd, docs_per_chunk):  # pass 1: residuals, histogram, assignment
            d1 = min(nd, d0 + docs_per_chunk)
            k, bf, cl = c.tokens_ex(d0, d1)
            b.add_residuals(bf, cl)
            hist += hist_parallel(pool, nthreads, k, cl, c.centroids_k)
            cid[c.doc_off[d0]:c.doc_off[d1]] = cl
            if d0 % (20 * docs_per_chunk) == 0:
                say(f"pass 1: {d1}/{nd} docs")
    b.freeze()
    b.reserve(nd, c.ntok)
    for d0 in range(0, nd, docs_per_chunk):  # pass 2: codes
        d1 = min(nd, d0 + docs_per_chunk)
        _, bf, cl = c.tokens_ex(d0, d1, want_k=False)
        b.add_docs(bf, cl, c.lengths[d0:d1])
        if d0 % (20 * docs_per_chunk) == 0:
            say(f"pass 2: {d1}/{nd} docs")
    say("pass 2 done; oracle index")
    oi = oracle.OracleIndex(c.centroids_k, c.doc_off, cid, w.nbits, hist=hist, with_codes=False)
    return c, b, oi


def oracle_search_one(c, oi, q_k, nprobe, ncand, k):
    """The oracle's search of one query [Tq, dim], stage by stage."""
    def docs_tokens(ids):
        return c.docs_tokens(ids)
    return oracle.search_streamed(oi, q_k, nprobe, ncand, k, docs_tokens)
