"""The benchmark's recall reference (exact Chamfer in float64 with torch,
grouped by document length) against the oracle's exact Chamfer (int64 keys),
and its top-k order against the oracle's tie rule."""
import dataclasses

import numpy as np
import torch

import bench
import oracle
import synth


def test_chamfer_block_equals_oracle_exact_chamfer():
    w = synth.WORKLOADS["100k"].scaled(ndocs=300)  # lognormal lengths: many length groups
    c = synth.Corpus(w.corpus_spec())
    k, _ = c.tokens()
    q, _ = c.queries(5, w.Tq, query_seed=3)
    Qf = torch.from_numpy(q.astype(np.float64) / 2048.0)
    T = torch.from_numpy(k.astype(np.float64) / 2048.0)
    F = bench.chamfer_block(Qf, T, c.lengths).numpy()
    for qi in range(len(q)):
        keys = oracle.exact_chamfer(q[qi], k, c.doc_off)
        # the reference is exact: its scores are the oracle's keys times 2^-22
        assert np.array_equal(F[qi] * 2.0 ** 22, keys.astype(np.float64))


def test_exact_reference_chunked_feed_equals_whole():
    w = synth.WORKLOADS["tiny"].scaled(ndocs=200)
    c = synth.Corpus(w.corpus_spec())
    k, _ = c.tokens()
    q, _ = c.queries(3, w.Tq)
    ref = bench.ExactReference(q, w.ndocs, "cpu")
    for d0 in range(0, w.ndocs, 64):  # chunks as the build feeds them
        d1 = min(w.ndocs, d0 + 64)
        ref.feed(k[c.doc_off[d0]:c.doc_off[d1]], c.lengths[d0:d1], d0)
    for qi in range(len(q)):
        keys = oracle.exact_chamfer(q[qi], k, c.doc_off)
        assert np.array_equal(ref.F[qi].numpy() * 2.0 ** 22, keys.astype(np.float64))
        ids, _ = oracle.topk(np.arange(w.ndocs, dtype=np.int32), keys, 10)
        assert np.array_equal(ref.topk(10)[qi], ids)


def test_topk_ids_breaks_ties_by_lowest_id():
    F = torch.tensor([[1.0, 3.0, 3.0, 2.0, 3.0]], dtype=torch.float64)
    assert bench.topk_ids(F, 4).tolist() == [[1, 2, 4, 3]]


def test_cpu_baseline_leg_matches_in_memory_oracle():
    """The bench's CPU baseline (quantiser fed chunk by chunk, documents
    regenerated per query) returns the in-memory oracle's top-k ids, and
    reports its per-query latency on one thread."""
    w = synth.WORKLOADS["100k"].scaled(ndocs=400)
    c = synth.Corpus(w.corpus_spec())
    k, cl = c.tokens()
    view = bench.OracleView(c, threads=2)
    for d0 in range(0, w.ndocs, 150):  # chunks as the build feeds them
        d1 = min(w.ndocs, d0 + 150)
        a, b = c.doc_off[d0], c.doc_off[d1]
        view.feed(k[a:b], cl[a:b], d0, d1)
    q, _ = c.queries(4, w.Tq, query_seed=5)
    oi = oracle.OracleIndex(c.centroids_k, c.doc_off, cl, w.nbits, tok_k=k)
    ref = oi.search(q, w.nprobe, min(w.ncand, w.ndocs), w.k)
    wq = dataclasses.replace(w, nq=4, ncand=min(w.ncand, w.ndocs))
    out = view.run(wq, q, ref["ids"], seconds=60)
    assert out["ids_match_gpu"] is True
    assert out["cores"] == 2 and out["value"] > 0
    assert out["s_per_query_one_thread"] > 0
    bad = ref["ids"].copy()
    bad[0, [0, 1]] = bad[0, [1, 0]]  # a swapped pair in the order must be seen
    view2 = bench.OracleView(c, threads=2)
    view2.hist, view2.cid = view.hist, view.cid
    assert view2.run(wq, q, bad, seconds=60)["ids_match_gpu"] is False
