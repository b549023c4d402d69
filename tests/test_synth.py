"""The shared input generator: counter-based RNG, grid membership, recipe shape."""
import numpy as np
import pytest

import synth
from synth import WORKLOADS


def _splitmix64_seq(seed, n):
    # SplitMix64 as published (Steele, Lea & Flood 2014), written out here
    out, x = [], seed
    M = (1 << 64) - 1
    for _ in range(n):
        x = (x + 0x9E3779B97F4A7C15) & M
        z = x
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
        out.append(z ^ (z >> 31))
    return out


def test_splitmix64_known_values():
    # first output from state 0 is the widely quoted 0xE220A8397B1DCDAF
    assert synth.splitmix64_at(0, 0) == 0xE220A8397B1DCDAF
    ref = _splitmix64_seq(12345, 8)
    assert [synth.splitmix64_at(12345, i) for i in range(8)] == ref


def test_to_grid_examples():
    assert synth.to_grid(0.0) == 0.0
    assert synth.to_grid(1.0) == 1.0
    assert synth.to_grid(0.5 / 2048) == 0.0          # tie -> even (0)
    assert synth.to_grid(1.5 / 2048) == 2.0 / 2048   # tie -> even (2)
    assert synth.to_grid(0.0625 + 1e-9) == 0.0625
    # above 2^-4 the spacing is the bf16 spacing: 2^-4..2^-3 -> 2^-11
    assert synth.to_grid(0.1 + 0.2 / 2048) == round(0.1 * 2048) / 2048


@pytest.mark.parametrize("name", ["tiny", "100k", "1m", "2m-long"])
def test_corpus_shapes(name):
    w = WORKLOADS[name].scaled(ndocs=2000)
    c = synth.Corpus(w.corpus_spec())
    assert c.centroids_k.shape == (w.ncent, 128)
    assert c.lengths.min() >= w.len_lo and c.lengths.max() <= w.len_hi
    k, cl = c.tokens(0, 50)
    assert k.shape[0] == c.doc_off[50]
    assert cl.min() >= 0 and cl.max() < w.ncent
    # every component is a bf16 value on the 2^-11 grid
    bits = synth.k_to_bf16_bits(k)
    assert bits.dtype == np.uint16
    n = np.linalg.norm(k / 2048.0, axis=1)
    assert np.all(np.abs(n - 1) < 0.01)


def test_doc_ranges_are_independent():
    w = WORKLOADS["100k"].scaled(ndocs=300)
    c = synth.Corpus(w.corpus_spec())
    k_all, cl_all = c.tokens(0, 300)
    k_mid, cl_mid = c.tokens(100, 140)
    a, b = c.doc_off[100], c.doc_off[140]
    assert np.array_equal(k_all[a:b], k_mid) and np.array_equal(cl_all[a:b], cl_mid)
    k_l, cl_l, beg = c.docs_tokens(np.array([7, 250, 7]))
    assert np.array_equal(k_l[beg[1]:beg[1] + c.lengths[250]], k_all[c.doc_off[250]:c.doc_off[251]])
    assert np.array_equal(k_l[beg[2]:], k_all[c.doc_off[7]:c.doc_off[8]])


def test_queries_deterministic_and_seeded():
    w = WORKLOADS["tiny"]
    c = synth.Corpus(w.corpus_spec())
    q1, s1 = c.queries(8, 32)
    q2, s2 = c.queries(8, 32)
    q3, _ = c.queries(8, 32, query_seed=1)
    q4, s4 = c.queries(4, 32, q0=4)
    assert np.array_equal(q1, q2) and np.array_equal(s1, s2)
    assert not np.array_equal(q1, q3)
    assert np.array_equal(q1[4:], q4) and np.array_equal(s1[4:], s4)


def test_lognormal_length_mean():
    w = WORKLOADS["1m"].scaled(ndocs=200_000)
    c = synth.Corpus(w.corpus_spec())
    # sigma 0.5 lognormal, mean 70, clipped to [8,180]: clipped mean ~69.4
    assert 68.5 < c.lengths.mean() < 70.3


def test_zipf_popularity_head():
    w = WORKLOADS["1m"].scaled(ndocs=20_000)
    c = synth.Corpus(w.corpus_spec())
    _, cl = c.tokens(want_k=False)
    share = np.bincount(cl, minlength=w.ncent).max() / cl.size
    # Zipf(1.1) over 65,536 ranks: the head rank holds ~13.7% of the mass
    assert 0.12 < share < 0.155


def test_docs_tokens_equals_per_range_generation():
    c = synth.Corpus(synth.WORKLOADS["tiny"].corpus_spec())
    docs = np.array([7, 999, 0, 7, 512], dtype=np.int64)
    k, cl, begin = c.docs_tokens(docs)
    for i, d in enumerate(docs):
        kk, cc = c.tokens(int(d), int(d) + 1)
        rows = slice(int(begin[i]), int(begin[i]) + len(cc))
        assert np.array_equal(k[rows], kk) and np.array_equal(cl[rows], cc)
