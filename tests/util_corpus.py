"""Shared test helpers: cached small corpora and oracle indexes (CPU only)."""
import functools

import numpy as np

import oracle
import synth
from synth import WORKLOADS


@functools.lru_cache(maxsize=None)
def corpus(name: str, ndocs: int | None = None):
    w = WORKLOADS[name]
    if ndocs is not None:
        w = w.scaled(ndocs=ndocs)
    c = synth.Corpus(w.corpus_spec())
    k, cl = c.tokens()
    return w, c, k, cl


@functools.lru_cache(maxsize=None)
def oracle_index(name: str, ndocs: int | None = None):
    w, c, k, cl = corpus(name, ndocs)
    return oracle.OracleIndex(c.centroids_k, c.doc_off, cl, w.nbits, tok_k=k)


def rand_grid(rng, shape, scale=1.0):
    """Random grid vectors (unit rows, scaled) as int16 grid integers."""
    x = rng.standard_normal(shape)
    x /= np.linalg.norm(x, axis=-1, keepdims=True)
    x *= scale
    return oracle.grid_f32(x.astype(np.float32))
