"""Oracle pins: residual quantiser, codes, packing, complete document scores
(Sec. 3.2 document scoring; Chamfer, Def. 1), exact MaxSim, whole path."""
import numpy as np
import pytest

import oracle
from util_corpus import corpus, oracle_index, rand_grid


def test_histogram_quantiles_match_sorted_array():
    rng = np.random.default_rng(10)
    ncent, ntok = 50, 400
    cent = rand_grid(rng, (ncent, 128))
    cid = rng.integers(0, ncent, ntok).astype(np.int32)
    tok = (cent[cid].astype(np.int32) + rng.integers(-90, 90, (ntok, 128))).clip(-2048, 2048).astype(np.int16)
    hist = oracle.residual_hist(tok, cid, cent)
    r = np.sort((tok.astype(np.int64) - cent[cid]).ravel())
    n = r.size
    assert hist.sum() == n
    for nbits in (2, 4):
        B = 1 << nbits
        cut, w = oracle.quantizer(hist, nbits)
        assert cut.tolist() == [int(r[min(i * n // B, n - 1)]) for i in range(1, B)]
        mids = [int(r[min((2 * u + 1) * n // (2 * B), n - 1)]) for u in range(B)]
        assert w.tolist() == [oracle.grid_k(m / 2048.0) for m in mids]


def test_encode_is_count_of_cutoffs_below():
    rng = np.random.default_rng(11)
    cent = rand_grid(rng, (8, 128))
    cid = rng.integers(0, 8, 64).astype(np.int32)
    tok = (cent[cid].astype(np.int32) + rng.integers(-40, 40, (64, 128))).astype(np.int16)
    cut = np.array([-20, -3, -3, 0, 5, 5, 9, 15, 18, 22, 25, 30, 31, 33, 36], np.int32)
    codes = oracle.encode(tok, cid, cent, cut, 4)
    r = tok.astype(np.int64) - cent[cid]
    # searchsorted(side="left") counts cutoffs strictly below r
    assert np.array_equal(codes, np.searchsorted(cut, r, side="left"))


def test_value_on_cutoff_goes_to_lower_bucket():
    cent = np.zeros((1, 128), np.int16)
    tok = np.zeros((1, 128), np.int16)
    tok[0, :5] = [-7, -6, 0, 1, 2]
    codes = oracle.encode(tok, np.zeros(1, np.int32), cent, np.array([-6, 0, 1], np.int32), 2)
    assert codes[0, :5].tolist() == [0, 0, 1, 2, 3]


def test_pack_layout_and_round_trip():
    codes2 = np.tile(np.array([0, 1, 2, 3], np.uint8), 32)[None, :]
    p2 = oracle.pack(codes2, 2)
    assert p2.shape == (1, 32) and np.all(p2 == 0b11100100)     # dim 4i+s at bits [2s, 2s+1]
    codes4 = np.tile(np.array([3, 12], np.uint8), 64)[None, :]
    p4 = oracle.pack(codes4, 4)
    assert p4.shape == (1, 64) and np.all(p4 == 0xC3)            # dim 2i low nibble, 2i+1 high
    rng = np.random.default_rng(12)
    for nbits in (2, 4):
        c = rng.integers(0, 1 << nbits, (33, 128)).astype(np.uint8)
        assert np.array_equal(oracle.unpack(oracle.pack(c, nbits), 128, nbits), c)


def test_zero_residuals_give_zero_weights_and_centroid_only_scores():
    rng = np.random.default_rng(13)
    ncent, ndocs = 40, 25
    cent = rand_grid(rng, (ncent, 128))
    lens = rng.integers(1, 7, ndocs)
    doc_off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    cid = rng.integers(0, ncent, doc_off[-1]).astype(np.int32)
    tok = cent[cid].copy()                                  # tokens equal to their centroids
    oi = oracle.OracleIndex(cent, doc_off, cid, 2, tok_k=tok)
    assert np.all(oi.w_k == 0) and np.all(oi.cut_k == 0)
    q = rand_grid(rng, (3, 6, 128))
    S = oracle.centroid_scores(q[0], cent)
    fh = oracle.doc_scores(S, q[0], oi.w_k, doc_off[:-1], lens, cid, oi.codes)
    ref = [S[:, cid[doc_off[v]:doc_off[v + 1]]].max(axis=1).sum() for v in range(ndocs)]
    assert fh.tolist() == ref


def test_doc_scores_equal_brute_force_on_dequantised_vectors():
    w, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(3, 32)
    docs = np.array([0, 5, 999, 123])
    lens = np.diff(c.doc_off)[docs].astype(np.int32)
    for qi in range(3):
        S = oracle.centroid_scores(q[qi], c.centroids_k)
        fh = oracle.doc_scores(S, q[qi], oi.w_k, c.doc_off[docs], lens, cl, oi.codes)
        deq = c.centroids_k[cl].astype(np.float64) + oi.w_k[oi.codes].astype(np.float64)  # exact, k units
        qq = q[qi].astype(np.float64)
        for i, v in enumerate(docs):
            sc = qq @ deq[c.doc_off[v]:c.doc_off[v + 1]].T          # exact in fp64
            assert fh[i] == int(sc.max(axis=1).sum())


def test_exact_chamfer_against_fp64_matmul():
    w, c, k, cl = corpus("tiny")
    q, _ = c.queries(2, 32)
    F = oracle.exact_chamfer(q[1], k[: c.doc_off[50]], c.doc_off[:51])
    for v in (0, 17, 49):
        sc = q[1].astype(np.float64) @ k[c.doc_off[v]:c.doc_off[v + 1]].T.astype(np.float64)
        assert F[v] == int(sc.max(axis=1).sum())


def test_exhaustive_mode_equals_brute_force_chamfer_on_dequantised():
    """nprobe = ncent and ncand >= ndocs: the path's top-k is brute-force
    Chamfer over the dequantised vectors, keys bit-exact."""
    w, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(4, 32)
    out = oi.search(q, nprobe=w.ncent, ncand=w.ndocs, k=20)
    deq = c.centroids_k[cl].astype(np.float64) + oi.w_k[oi.codes].astype(np.float64)
    for qi in range(4):
        sc = q[qi].astype(np.float64) @ deq.T
        F = np.array([sc[:, c.doc_off[v]:c.doc_off[v + 1]].max(axis=1).sum() for v in range(w.ndocs)])
        order = np.lexsort((np.arange(w.ndocs), -F))[:20]
        assert np.array_equal(out["ids"][qi], order)
        assert np.array_equal(out["keys"][qi], F[order].astype(np.int64))
        assert out["n_sq"][qi] == w.ndocs


def test_search_composes_stage_definitions():
    w, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, _ = c.queries(3, 32)
    out = oi.search(q, w.nprobe, w.ncand, w.k)
    for qi in range(3):
        S = oracle.centroid_scores(q[qi], c.centroids_k)
        ci, ck = oracle.probe(S, w.nprobe)
        assert np.array_equal(out["cent_ids"][qi], ci) and np.array_equal(out["cent_keys"][qi], ck)
        d, fp = oracle.partial_scores(S, ci, oi.ivf_off, oi.ivf_doc, w.ndocs)
        r, rk = oracle.topk(d, fp, w.ncand)
        assert np.array_equal(out["cand"][qi, :len(r)], r) and out["n_cand"][qi] == len(r)
        fh = oracle.doc_scores(S, q[qi], oi.w_k, c.doc_off[r], np.diff(c.doc_off)[r].astype(np.int32), cl, oi.codes)
        ids, keys = oracle.topk(r, fh, w.k)
        assert np.array_equal(out["ids"][qi], ids) and np.array_equal(out["keys"][qi], keys)


def test_key_to_score_single_rounding():
    """The score is the key's value rounded once to fp32.  The comparison is
    made in float64 against that fp32 value: a Python float compared with an
    np.float32 is first cast to fp32, which would let an unrounded result
    pass."""
    for key in (0, 1, -1, 2**24 + 1, 2**27 + 3, -(2**26) - 5, 123456789):
        want = float(np.float32(key) * np.float32(2.0 ** -22))
        assert oracle.key_to_score(key) == want
    assert oracle.key_to_score(2**24 + 1) == 4.0  # 2^24 + 1 is not an fp32 value


def test_synthetic_clusters_are_nearest_centroid():
    """The generator records the centroid a token was drawn around; at noise
    0.05 it is the nearest centroid (the IVF assignment, Sec. 2.3)."""
    w, c, k, cl = corpus("tiny")
    assert np.array_equal(oracle.assign(k, c.centroids_k), cl)


def test_source_document_ranks_first():
    w, c, k, cl = corpus("tiny")
    oi = oracle_index("tiny")
    q, src = c.queries(w.nq, w.Tq)
    out = oi.search(q, w.nprobe, w.ncand, w.k)
    assert np.mean(out["ids"][:, 0] == src) >= 0.9


@pytest.mark.slow
def test_synthetic_clusters_are_nearest_centroid_100k_sample():
    import synth
    w = synth.WORKLOADS["100k"]
    c = synth.Corpus(w.corpus_spec())
    rng = np.random.default_rng(14)
    docs = rng.choice(w.ndocs, 40, replace=False)
    k, cl, _ = c.docs_tokens(docs)
    assert np.array_equal(oracle.assign(k, c.centroids_k), cl)
