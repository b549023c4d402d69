"""Oracle pins for the CPU-GPU collaborative document scoring (Sec. 4,
document scoring; Alg. 3): the non-concurrent special case, the complete
special case, the paper's worst-case count of full-precision scores, the
no-extra-work case, the accuracy guarantee against the non-concurrent
strategy, and an end-to-end case on the tiny corpus against brute force."""
import numpy as np
import pytest

import oracle
from util_corpus import corpus, oracle_index


def _inputs(rng, n, distinct=True):
    ids = np.sort(rng.choice(10 * n, n, replace=False)).astype(np.int32)
    approx = rng.permutation(n).astype(np.int64) if distinct else rng.integers(0, 5, n).astype(np.int64)
    exact = {int(d): int(v) for d, v in zip(ids, rng.integers(-1000, 1000, n))}
    return ids, approx, exact


def _top(pairs, m):
    """The m best (key, id) pairs by key desc, id asc."""
    return sorted(pairs, key=lambda kv: (-kv[0], kv[1]))[:m]


@pytest.mark.parametrize("distinct", [True, False])
def test_one_chunk_is_the_non_concurrent_strategy(distinct):
    """c = 1: full-precision scores for exactly the top-kfb by F^, then the
    top-k of those (the strategy the paper improves on)."""
    rng = np.random.default_rng(40)
    n, kfb, k = 50, 12, 5
    ids, approx, exact = _inputs(rng, n, distinct)
    got_ids, got_keys, nf = oracle.collaborative_scoring(ids, approx, exact.__getitem__, n, kfb, 1, k)
    chosen = [d for _, d in _top(list(zip(approx.tolist(), ids.tolist())), kfb)]
    want = _top([(exact[d], d) for d in chosen], k)
    assert nf == kfb
    assert got_ids.tolist() == [d for _, d in want] and got_keys.tolist() == [v for v, _ in want]


@pytest.mark.parametrize("chunks", [1, 3, 7])
def test_budget_covering_every_candidate_scores_all(chunks):
    rng = np.random.default_rng(41)
    n, k = 40, 6
    ids, approx, exact = _inputs(rng, n)
    got_ids, got_keys, nf = oracle.collaborative_scoring(ids, approx, exact.__getitem__, n, n, chunks, k)
    want = _top([(v, d) for d, v in exact.items()], k)
    assert nf == n
    assert got_ids.tolist() == [d for _, d in want]


@pytest.mark.parametrize("chunks,kfb", [(4, 8), (2, 6), (8, 16)])
def test_increasing_scores_reach_the_papers_worst_case(chunks, kfb):
    """F^ increasing along S_refine, every chunk at least kfb long: each chunk
    puts only new documents in the top, so the count is
    sum_i (i/c) kfb = (c+1)/2 kfb (Sec. 4, when c divides kfb)."""
    n = chunks * kfb
    ids = np.arange(n, dtype=np.int32)
    approx = np.arange(n, dtype=np.int64)
    _, _, nf = oracle.collaborative_scoring(ids, approx, lambda d: d, n, kfb, chunks, 1)
    assert nf == (chunks + 1) * kfb // 2


def test_quota_rounds_up_when_chunks_do_not_divide_kfb():
    """c = 3, kfb = 4, increasing F^: the quotas after each chunk are
    ceil(4/3), ceil(8/3), 4 = 2, 3, 4 new documents (the reading of i/c kfb
    for a fractional value), 9 in all."""
    n = 12
    _, _, nf = oracle.collaborative_scoring(np.arange(n, dtype=np.int32), np.arange(n, dtype=np.int64),
                                            lambda d: d, n, 4, 3, 1)
    assert nf == 9


@pytest.mark.parametrize("chunks", [2, 4, 5])
def test_decreasing_scores_need_no_extra_work(chunks):
    """F^ decreasing along S_refine: the top after chunk i contains the top
    after chunk i-1, so exactly kfb documents get full-precision scores."""
    n, kfb = 60, 10
    ids = np.arange(n, dtype=np.int32)
    approx = np.arange(n, 0, -1).astype(np.int64)
    _, _, nf = oracle.collaborative_scoring(ids, approx, lambda d: -d, n, kfb, chunks, 3)
    assert nf == kfb


def test_never_worse_than_the_non_concurrent_strategy():
    """The scored set contains the top-kfb by F^ (the last chunk scores it),
    so the r-th returned full-precision key is never below that of c = 1."""
    rng = np.random.default_rng(42)
    for _ in range(30):
        n = int(rng.integers(5, 80))
        ids, approx, exact = _inputs(rng, n, distinct=bool(rng.integers(0, 2)))
        kfb = int(rng.integers(1, n + 1))
        k = int(rng.integers(1, kfb + 1))
        chunks = int(rng.integers(1, 9))
        _, base, nf1 = oracle.collaborative_scoring(ids, approx, exact.__getitem__, n, kfb, 1, k)
        _, keys, nf = oracle.collaborative_scoring(ids, approx, exact.__getitem__, n, kfb, chunks, k)
        assert np.all(keys >= base) and nf >= nf1 == kfb


def test_chunks_follow_ncand_not_the_kept_count():
    """Chunk bounds come from ncand; with fewer kept documents the last
    chunks are short or empty and only what was seen is ranked."""
    ids = np.array([3, 8, 9], np.int32)
    approx = np.array([1, 3, 2], np.int64)
    # ncand 8, 4 chunks: positions 0-1 | 2 | (empty) | (empty); kfb 2
    _, _, nf = oracle.collaborative_scoring(ids, approx, lambda d: d, 8, 2, 4, 1)
    # after chunk 0 the top 1 of {3, 8} is 8; after chunk 1 the top 1 of
    # {3, 8, 9} is 8; then the top 2 is {8, 9}
    assert nf == 2


def test_identity_full_scores_give_the_approximate_top_k():
    """With the full-precision score equal to F^ the answer is the top-k by
    F^, which the oracle's search computes independently (orc_search)."""
    w, c, k_, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(4, 32)
    ref = oi.search(q, w.nprobe, w.ncand, w.k)
    pr = oi.prune(q, w.nprobe, w.ncand)
    lens = np.diff(c.doc_off)
    for qi in range(4):
        r = np.sort(pr["cand"][qi, :pr["n_cand"][qi]]).astype(np.int32)
        S = oracle.centroid_scores(q[qi], c.centroids_k)
        fh = oracle.doc_scores(S, q[qi], oi.w_k, c.doc_off[r], lens[r].astype(np.int32), cl, oi.codes)
        f = dict(zip(r.tolist(), fh.tolist()))
        ids, keys, _ = oracle.collaborative_scoring(r, fh, f.__getitem__, w.ncand, 2 * w.k, 3, w.k)
        assert np.array_equal(ids, ref["ids"][qi]) and np.array_equal(keys, ref["keys"][qi])


def test_tiny_end_to_end_against_brute_force():
    """kfb = ncand: every kept document is scored exactly, so the answer is the
    exact Chamfer top-k over the kept set, computed here by brute force in
    float64 over the grid values."""
    w, c, k_, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, src = c.queries(3, 32)
    out = oi.search_collab(q, k_, w.nprobe, w.ncand, w.ncand, 4, w.k)
    pr = oi.prune(q, w.nprobe, w.ncand)
    for qi in range(3):
        kept = pr["cand"][qi, :pr["n_cand"][qi]]
        brute = []
        for d in kept:
            D = k_[c.doc_off[d]:c.doc_off[d + 1]].astype(np.float64)
            brute.append((int(round((q[qi].astype(np.float64) @ D.T).max(axis=1).sum())), int(d)))
        want = _top(brute, w.k)
        assert out["ids"][qi].tolist() == [d for _, d in want]
        assert out["keys"][qi].tolist() == [v for v, _ in want]
        assert out["n_full"][qi] == len(kept)
        assert out["ids"][qi, 0] == src[qi]
