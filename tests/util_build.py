"""Test helpers that build product indexes from synthetic corpora (host side)."""
import functools

import numpy as np

import synth
from paper_2608_23553_amd import build_index


def chunk_factory(corpus, docs_per_chunk=20_000):
    """Callable yielding (tokens_bf16, cids, doc_lens) chunks in doc order."""
    def gen():
        nd = corpus.spec.ndocs
        for d0 in range(0, nd, docs_per_chunk):
            d1 = min(nd, d0 + docs_per_chunk)
            k, cl = corpus.tokens(d0, d1)
            yield synth.k_to_bf16_bits(k), cl, corpus.lengths[d0:d1]
    return gen


def product_builder(corpus, nbits, docs_per_chunk=20_000, rabitq_signs=None):
    return build_index(synth.k_to_bf16_bits(corpus.centroids_k), nbits, chunk_factory(corpus, docs_per_chunk),
                       rabitq_signs=rabitq_signs)
