"""Oracle pins: posting lists, candidate set S, partial score F' (Sec. 3.2
candidate generation and refinement), top-ncand."""
import itertools

import numpy as np
import pytest

import oracle
from util_corpus import oracle_index, corpus, rand_grid


def _toy_corpus(rng, ndocs=40, ncent=12, lo=1, hi=6):
    lens = rng.integers(lo, hi + 1, size=ndocs)
    doc_off = np.zeros(ndocs + 1, np.int64)
    doc_off[1:] = np.cumsum(lens)
    cid = rng.integers(0, ncent, size=doc_off[-1]).astype(np.int32)
    return doc_off, cid


def _brute_fprime(S, cent_ids, doc_off, cid):
    """F' written from the definition, one doc at a time (pure Python)."""
    Tq, nprobe = cent_ids.shape
    out = {}
    for v in range(len(doc_off) - 1):
        toks = set(cid[doc_off[v]:doc_off[v + 1]].tolist())
        hit_any = False
        total = 0
        for j in range(Tq):
            vals = [S[j, c] for c in cent_ids[j] if c in toks]
            if vals:
                hit_any = True
                total += max(vals)
        if hit_any:
            out[v] = total
    return out


def test_ivf_lists_match_sets():
    rng = np.random.default_rng(4)
    doc_off, cid = _toy_corpus(rng)
    off, docs = oracle.ivf_docs(cid, doc_off, 12)
    for c in range(12):
        ref = sorted({v for v in range(40) if c in cid[doc_off[v]:doc_off[v + 1]]})
        assert docs[off[c]:off[c + 1]].tolist() == ref


def test_candidates_and_fprime_match_definition():
    rng = np.random.default_rng(5)
    for trial in range(20):
        doc_off, cid = _toy_corpus(rng)
        off, docs = oracle.ivf_docs(cid, doc_off, 12)
        Tq, nprobe = 5, int(rng.integers(1, 6))
        S = rng.integers(-30, 30, size=(Tq, 12)).astype(np.int64)   # negatives and ties
        cent_ids, _ = oracle.probe(S, nprobe)
        ref = _brute_fprime(S, cent_ids, doc_off, cid)
        cand = oracle.candidates(cent_ids, off, docs, 40)
        assert cand.tolist() == sorted(ref)
        d, fp = oracle.partial_scores(S, cent_ids, off, docs, 40)
        assert d.tolist() == sorted(ref)
        assert fp.tolist() == [ref[v] for v in sorted(ref)]


def test_fprime_negative_maximum_is_kept():
    """Hand-built case (F' definition, not the init-0 of Alg. 2): a doc whose
    only retrieved token scores -5 gets F' = -5 for that query token."""
    doc_off = np.array([0, 2, 3], np.int64)        # doc0: tokens in c0, c1 ; doc1: token in c2
    cid = np.array([0, 1, 2], np.int32)
    off, docs = oracle.ivf_docs(cid, doc_off, 3)
    S = np.array([[9, -5, -7],                     # j=0 probes c0 (9) and c1 (-5)
                  [-5, -9, -1]], np.int64)         # j=1 probes c2 (-1) and c0 (-5)
    cent_ids = np.array([[0, 1], [2, 0]], np.int32)
    d, fp = oracle.partial_scores(S, cent_ids, off, docs, 2)
    # doc0: j0 max(9, -5) = 9 ; j1 only c0 hits -> -5 ; F' = 4
    # doc1: j0 no hit -> 0 ; j1 c2 -> -1 ; F' = -1
    assert d.tolist() == [0, 1] and fp.tolist() == [4, -1]


def test_token_level_lists_give_same_fprime():
    rng = np.random.default_rng(6)
    doc_off, cid = _toy_corpus(rng, ndocs=30)
    off, docs = oracle.ivf_docs(cid, doc_off, 12)
    S = rng.integers(-20, 40, size=(4, 12)).astype(np.int64)
    cent_ids, _ = oracle.probe(S, 3)
    tok2doc = np.repeat(np.arange(30), np.diff(doc_off))
    # token-level walk: every token of every probed list, atomic-max style
    M = {}
    for j in range(4):
        for c in cent_ids[j]:
            for t in np.nonzero(cid == c)[0]:
                key = (tok2doc[t], j)
                M[key] = max(M.get(key, -10**18), S[j, c])
    ref = {}
    for (v, j), s in M.items():
        ref[v] = ref.get(v, 0) + s
    d, fp = oracle.partial_scores(S, cent_ids, off, docs, 30)
    assert dict(zip(d.tolist(), fp.tolist())) == ref


def test_all_centroids_probed_gives_whole_corpus_and_full_interaction():
    w, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(2, 32)
    S = oracle.centroid_scores(q[0], c.centroids_k)
    cent_ids, _ = oracle.probe(S, w.ncent)
    cand = oracle.candidates(cent_ids, oi.ivf_off, oi.ivf_doc, w.ndocs)
    assert np.array_equal(cand, np.arange(w.ndocs))
    d, fp = oracle.partial_scores(S, cent_ids, oi.ivf_off, oi.ivf_doc, w.ndocs)
    # full centroid interaction: sum_j max_t S[j, cid(t)]
    full = np.array([S[:, cl[c.doc_off[v]:c.doc_off[v + 1]]].max(axis=1).sum() for v in range(w.ndocs)])
    assert np.array_equal(fp, full)


def test_fprime_monotone_in_nprobe_for_nonnegative_scores():
    rng = np.random.default_rng(7)
    doc_off, cid = _toy_corpus(rng)
    off, docs = oracle.ivf_docs(cid, doc_off, 12)
    S = rng.integers(0, 50, size=(4, 12)).astype(np.int64)
    prev = np.zeros(40, np.int64)
    for nprobe in range(1, 13):
        cent_ids, _ = oracle.probe(S, nprobe)
        d, fp = oracle.partial_scores(S, cent_ids, off, docs, 40)
        cur = np.zeros(40, np.int64)
        cur[d] = fp
        assert np.all(cur >= prev)
        prev = cur


def test_topk_matches_lexsort_with_ties():
    rng = np.random.default_rng(8)
    ids = rng.permutation(5000).astype(np.int32)
    keys = rng.integers(0, 20, size=5000).astype(np.int64)
    for k in (1, 7, 256, 5000, 6000):
        oi, ok = oracle.topk(ids, keys, k)
        order = np.lexsort((ids, -keys))[:k]
        assert np.array_equal(oi, ids[order]) and np.array_equal(ok, keys[order])
