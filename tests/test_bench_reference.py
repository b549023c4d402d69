"""The benchmark's recall reference (exact Chamfer in float64 with torch,
grouped by document length) against the oracle's exact Chamfer (int64 keys),
and its top-k order against the oracle's tie rule."""
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
