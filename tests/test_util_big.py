"""The full-size helpers on a small corpus: the oracle's view built from the
chunk stream, and its per-query search with regenerated documents, equal the
oracle's own all-in-memory index and search."""
import numpy as np

import oracle
import synth
from util_big import build_both, oracle_search_one


def test_sampled_oracle_equals_full_oracle():
    for name, nd in (("1m", 3000), ("2m-long", 400)):
        w = synth.WORKLOADS[name].scaled(ndocs=nd)
        c, b, oi = build_both(w, docs_per_chunk=700, say=lambda *a: None)
        b.close()
        k, cl = c.tokens()
        full = oracle.OracleIndex(c.centroids_k, c.doc_off, cl, w.nbits, tok_k=k)
        assert np.array_equal(oi.cut_k, full.cut_k) and np.array_equal(oi.w_k, full.w_k)
        q, _ = c.queries(4, w.Tq, query_seed=11)
        ncand, kk = min(w.ncand, nd // 3), min(w.k, nd // 10)
        ref = full.search(q, w.nprobe, ncand, kk)
        for qi in range(4):
            got = oracle_search_one(c, oi, q[qi], w.nprobe, ncand, kk)
            assert np.array_equal(got["cent_ids"], ref["cent_ids"][qi])
            assert np.array_equal(got["cent_keys"], ref["cent_keys"][qi])
            n = ref["n_cand"][qi]
            assert np.array_equal(got["cand"], ref["cand"][qi, :n])
            assert np.array_equal(got["cand_keys"], ref["cand_keys"][qi, :n])
            assert np.array_equal(got["ids"], ref["ids"][qi, :len(got["ids"])])
            assert np.array_equal(got["keys"], ref["keys"][qi, :len(got["ids"])])
