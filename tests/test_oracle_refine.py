"""Oracle pins for refinement from the retrieved tokens' decoded scores: F'
of Sec. 3.2 (candidate refinement, Alg. 2) with each token retrieved through a
probed list scored by its own approximation (centroid score plus decoded
residual), as document scoring scores it."""
import numpy as np

import oracle
from util_corpus import corpus, oracle_index, rand_grid


def test_token_lists_match_sets():
    rng = np.random.default_rng(30)
    ncent, ntok = 17, 500
    cid = rng.integers(0, ncent, ntok).astype(np.int32)
    cid[:5] = 3  # one crowded list; some centroids stay empty
    off, tok = oracle.ivf_tokens(cid, ncent)
    assert off[0] == 0 and off[-1] == ntok
    for c in range(ncent):
        assert tok[off[c]:off[c + 1]].tolist() == np.nonzero(cid == c)[0].tolist()


def test_token_docs():
    doc_off = np.array([0, 3, 3, 7, 8], np.int64)
    assert oracle.token_docs(doc_off).tolist() == [0, 0, 0, 2, 2, 2, 2, 3]


def _brute_force(S, ci, q, w, cid, codes, doc_off):
    """The definition written out per (document, query token)."""
    ndocs = doc_off.shape[0] - 1
    Tq = S.shape[0]
    docs, fp = [], []
    for v in range(ndocs):
        total, hit = 0, False
        for j in range(Tq):
            best = None
            for t in range(doc_off[v], doc_off[v + 1]):
                if cid[t] in ci[j]:
                    s = int(S[j, cid[t]]) + int(np.dot(q[j].astype(np.int64), w[codes[t]].astype(np.int64)))
                    best = s if best is None else max(best, s)
            if best is not None:
                total += best
                hit = True
        if hit:
            docs.append(v)
            fp.append(total)
    return np.array(docs, np.int32), np.array(fp, np.int64)


def test_refined_fprime_matches_definition():
    rng = np.random.default_rng(31)
    ncent, dim, Tq, nprobe, B = 20, 16, 5, 3, 4
    doc_off = np.concatenate([[0], np.cumsum(rng.integers(0, 7, 30))]).astype(np.int64)  # some empty docs
    ntok = int(doc_off[-1])
    cid = rng.integers(0, ncent, ntok).astype(np.int32)
    codes = rng.integers(0, B, (ntok, dim)).astype(np.uint8)
    w = rng.integers(-300, 300, B).astype(np.int32)
    q = rng.integers(-2048, 2048, (Tq, dim)).astype(np.int16)
    S = rng.integers(-(1 << 22), 1 << 22, (Tq, ncent)).astype(np.int64)  # negative scores included
    ci = np.stack([rng.permutation(ncent)[:nprobe] for _ in range(Tq)]).astype(np.int32)
    off, tok = oracle.ivf_tokens(cid, ncent)
    tdoc = oracle.token_docs(doc_off)
    d, fp = oracle.partial_scores_res(S, ci, q, w, off, tok, tdoc, codes, doc_off.shape[0] - 1)
    bd, bfp = _brute_force(S, ci, q, w, cid, codes, doc_off)
    assert np.array_equal(d, bd) and np.array_equal(fp, bfp)


def test_zero_weights_reduce_to_centroid_only_fprime():
    """With every bucket weight 0 a retrieved token scores as its centroid, so
    the refined F' is the centroid-only F' (pinned in test_oracle_prune)."""
    w_, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(3, 32)
    off, tok, tdoc = oi.token_lists()
    zero = np.zeros_like(oi.w_k)
    for qi in range(3):
        S = oracle.centroid_scores(q[qi], c.centroids_k)
        ci, _ = oracle.probe(S, 3)
        d0, f0 = oracle.partial_scores(S, ci, oi.ivf_off, oi.ivf_doc, w_.ndocs)
        d1, f1 = oracle.partial_scores_res(S, ci, q[qi], zero, off, tok, tdoc, oi.codes, w_.ndocs)
        assert np.array_equal(d0, d1) and np.array_equal(f0, f1)


def test_all_centroids_probed_gives_complete_document_scores():
    """Probing every centroid retrieves every token, so the refined F' of each
    document is its complete score from document scoring (pinned against
    brute force on the dequantised vectors)."""
    w_, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(2, 32)
    off, tok, tdoc = oi.token_lists()
    lens = np.diff(c.doc_off).astype(np.int32)
    for qi in range(2):
        S = oracle.centroid_scores(q[qi], c.centroids_k)
        ci, _ = oracle.probe(S, w_.ncent)
        d, fp = oracle.partial_scores_res(S, ci, q[qi], oi.w_k, off, tok, tdoc, oi.codes, w_.ndocs)
        assert np.array_equal(d, np.arange(w_.ndocs, dtype=np.int32))
        full = oracle.doc_scores(S, q[qi], oi.w_k, c.doc_off[:-1], lens, cl, oi.codes)
        assert np.array_equal(fp, full)


def test_refined_search_composes_stage_definitions():
    w_, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, src = c.queries(3, 32)
    off, tok, tdoc = oi.token_lists()
    out = oi.search(q, w_.nprobe, w_.ncand, w_.k, refine=True)
    pr = oi.prune(q, w_.nprobe, w_.ncand, refine=True)
    for qi in range(3):
        S = oracle.centroid_scores(q[qi], c.centroids_k)
        ci, ck = oracle.probe(S, w_.nprobe)
        d, fp = oracle.partial_scores_res(S, ci, q[qi], oi.w_k, off, tok, tdoc, oi.codes, w_.ndocs)
        r, rk = oracle.topk(d, fp, w_.ncand)
        for o in (out, pr):
            assert np.array_equal(o["cand"][qi, :len(r)], r) and o["n_cand"][qi] == len(r)
            assert np.array_equal(o["cand_keys"][qi, :len(r)], rk)
        fh = oracle.doc_scores(S, q[qi], oi.w_k, c.doc_off[r], np.diff(c.doc_off)[r].astype(np.int32), cl, oi.codes)
        ids, keys = oracle.topk(r, fh, w_.k)
        assert np.array_equal(out["ids"][qi], ids) and np.array_equal(out["keys"][qi], keys)
        assert out["ids"][qi, 0] == src[qi]


def test_refined_fprime_negative_maximum_is_kept():
    """A (document, query token) pair whose retrieved tokens all score below 0
    adds that negative maximum, not 0."""
    rng = np.random.default_rng(32)
    dim = 8
    doc_off = np.array([0, 2, 4], np.int64)
    cid = np.array([0, 1, 1, 2], np.int32)
    codes = np.zeros((4, dim), np.uint8)
    w = np.array([0, 0, 0, 0], np.int32)
    q = rand_grid(rng, (1, dim))
    S = np.array([[-50, -7, 30]], np.int64)
    ci = np.array([[0, 1]], np.int32)
    off, tok = oracle.ivf_tokens(cid, 3)
    d, fp = oracle.partial_scores_res(S, ci, q, w, off, tok, oracle.token_docs(doc_off), codes, 2)
    assert d.tolist() == [0, 1] and fp.tolist() == [-7, -7]
