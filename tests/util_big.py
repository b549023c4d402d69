"""Full-size workloads for the GPU parity tests: the product index and the
oracle's view of the same corpus, built from one stream of generated chunks,
and the oracle's search on a few sampled queries.

The oracle never holds the codes of the whole corpus here.  It keeps the
assignment, its own quantiser (from a residual histogram accumulated over
the same chunks the product builder reads) and the posting lists, and
regenerates the tokens of a query's top-ncand documents to score them.  The
stage functions are composed exactly as the oracle's own search composes
them (pinned by test_search_composes_stage_definitions)."""
import numpy as np

import oracle
import synth
from paper_2608_23553_amd import Builder


def build_both(w, nthreads=0, docs_per_chunk=50_000, say=print):
    """Product Builder and OracleIndex (without codes) for workload w."""
    c = synth.Corpus(w.corpus_spec(), nthreads=nthreads)
    b = Builder(synth.k_to_bf16_bits(c.centroids_k), w.nbits)
    hist = np.zeros(8193, dtype=np.int64)
    cid = np.empty(c.ntok, dtype=np.int32)
    nd = w.ndocs
    for d0 in range(0, nd, docs_per_chunk):  # pass 1: residuals, histogram, assignment
        d1 = min(nd, d0 + docs_per_chunk)
        k, cl = c.tokens(d0, d1)
        b.add_residuals(synth.k_to_bf16_bits(k), cl)
        oracle.residual_hist(k, cl, c.centroids_k, hist)
        cid[c.doc_off[d0]:c.doc_off[d1]] = cl
        if d0 % (20 * docs_per_chunk) == 0:
            say(f"pass 1: {d1}/{nd} docs")
    b.freeze()
    for d0 in range(0, nd, docs_per_chunk):  # pass 2: codes
        d1 = min(nd, d0 + docs_per_chunk)
        k, cl = c.tokens(d0, d1)
        b.add_docs(synth.k_to_bf16_bits(k), cl, c.lengths[d0:d1])
        if d0 % (20 * docs_per_chunk) == 0:
            say(f"pass 2: {d1}/{nd} docs")
    oi = oracle.OracleIndex(c.centroids_k, c.doc_off, cid, w.nbits, hist=hist, with_codes=False)
    return c, b, oi


def oracle_search_one(c, oi, q_k, nprobe, ncand, k):
    """The oracle's search of one query [Tq, dim], stage by stage."""
    S = oracle.centroid_scores(q_k, c.centroids_k)
    ci, ck = oracle.probe(S, nprobe)
    docs, fp = oracle.partial_scores(S, ci, oi.ivf_off, oi.ivf_doc, oi.ndocs)
    r, rk = oracle.topk(docs, fp, ncand)
    tk, cl, begin = c.docs_tokens(r.astype(np.int64))
    codes = oracle.encode(tk, cl, oi.cent_k, oi.cut_k, oi.nbits)
    fh = oracle.doc_scores(S, q_k, oi.w_k, begin, c.lengths[r].astype(np.int32), cl, codes)
    ids, keys = oracle.topk(r, fh, k)
    return dict(cent_ids=ci, cent_keys=ck, cand=r, cand_keys=rk, ids=ids, keys=keys,
                scores=oracle.keys_to_scores(keys))
