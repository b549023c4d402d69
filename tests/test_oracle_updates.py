"""Pins of the oracle's search with a deletion bitmap (Sec. 3.3, handling
updates): skipping deleted documents during retrieval must give what the
unmodified search gives on the same corpus with those documents emptied (no
tokens, so in no posting list), under the same quantiser.  That second route
runs the oracle's whole C search (orc_search), which knows nothing of
deletions."""
import numpy as np
import pytest

import oracle
from util_corpus import corpus, oracle_index


def _emptied(w, c, k, cl, deleted, hist):
    """OracleIndex of the corpus with the deleted documents' tokens removed."""
    lens = np.diff(c.doc_off)
    keep_tok = np.repeat(~deleted, lens)
    new_lens = np.where(deleted, 0, lens)
    doc_off = np.concatenate([[0], np.cumsum(new_lens)]).astype(np.int64)
    return oracle.OracleIndex(c.centroids_k, doc_off, cl[keep_tok], w.nbits, tok_k=k[keep_tok], hist=hist)


@pytest.mark.parametrize("name,ndocs,frac", [("tiny", None, 0.15), ("100k", 3000, 0.3)])
@pytest.mark.parametrize("refine", [False, True])
def test_deleted_search_equals_search_of_the_emptied_corpus(name, ndocs, frac, refine):
    w, c, k, cl = corpus(name, ndocs)
    oi = oracle_index(name, ndocs)
    q, src = c.queries(min(w.nq, 12), w.Tq, query_seed=5)
    rng = np.random.default_rng(41)
    deleted = rng.random(w.ndocs) < frac
    deleted[src] = True  # every query's source document is gone
    ncand, nprobe, kk = min(w.ncand, w.ndocs // 3), w.nprobe, min(w.k, 50)
    got = oracle.search_deleted(oi, q, nprobe, ncand, kk, deleted, refine=refine)
    ref = _emptied(w, c, k, cl, deleted, oi.hist).search(q, nprobe, ncand, kk, refine=refine)
    assert np.array_equal(got["ids"], ref["ids"])
    assert np.array_equal(got["keys"], ref["keys"])
    hit = got["ids"][got["ids"] >= 0]
    assert not deleted[hit].any()
    # and without deletions it is the plain search
    none = oracle.search_deleted(oi, q, nprobe, ncand, kk, np.zeros(w.ndocs, bool), refine=refine)
    plain = oi.search(q, nprobe, ncand, kk, refine=refine)
    assert np.array_equal(none["ids"], plain["ids"]) and np.array_equal(none["keys"], plain["keys"])


def test_deleting_every_document_leaves_no_result():
    w, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(3, w.Tq)
    got = oracle.search_deleted(oi, q, w.nprobe, w.ncand, w.k, np.ones(w.ndocs, bool))
    assert (got["ids"] == -1).all() and np.isneginf(got["scores"]).all()
