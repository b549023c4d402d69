"""Seeded synthetic multi-vector corpora: the shared input generator.

This package only produces inputs (centroids, document tokens with the
centroid each was drawn around, document lengths, queries).  It holds none of
the retrieval method's arithmetic, and both the CPU oracle and the GPU library
consume what it generates.  The C source (``synth.c``) documents the recipe
and the counter-based random number generator.

Vector components are returned as int16 grid integers ``k`` (value
``k / 2048``); :func:`k_to_bf16_bits` and :func:`k_to_f32` convert them,
exactly, to the storage types the GPU library accepts.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

from .configs import WORKLOADS, Workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

LEN_FIXED, LEN_LOGNORMAL, LEN_UNIFORM = 0, 1, 2
POP_UNIFORM, POP_ZIPF = 0, 1


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("ndocs", ctypes.c_int64),
        ("ncent", ctypes.c_int32),
        ("dim", ctypes.c_int32),
        ("len_kind", ctypes.c_int32),
        ("len_lo", ctypes.c_int32),
        ("len_hi", ctypes.c_int32),
        ("len_mean", ctypes.c_double),
        ("len_sigma", ctypes.c_double),
        ("pop_kind", ctypes.c_int32),
        ("zipf_s", ctypes.c_double),
        ("tok_sigma", ctypes.c_double),
        ("q_sigma", ctypes.c_double),
    ]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build() (make -C synth)")
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    lib.synth_create.argtypes = [ctypes.POINTER(_Cfg)]
    lib.synth_create.restype = P
    lib.synth_free.argtypes = [P]
    lib.synth_centroids.argtypes = [P]
    lib.synth_centroids.restype = ctypes.POINTER(ctypes.c_int16)
    lib.synth_doc_lengths.argtypes = [P, ctypes.c_int64, ctypes.c_int64, P]
    lib.synth_doc_tokens.argtypes = [P, ctypes.c_int64, ctypes.c_int64, P, P, P, P, ctypes.c_int]
    lib.synth_doc_tokens_ex.argtypes = [P, ctypes.c_int64, ctypes.c_int64, P, P, P, P, P, ctypes.c_int]
    lib.synth_docs_tokens.argtypes = [P, P, ctypes.c_int64, P, P, P, ctypes.c_int]
    lib.synth_queries.argtypes = [P, ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                  P, P, ctypes.c_int]
    lib.synth_splitmix64_at.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
    lib.synth_splitmix64_at.restype = ctypes.c_uint64
    lib.synth_to_grid.argtypes = [ctypes.c_double]
    lib.synth_to_grid.restype = ctypes.c_double
    _lib = lib
    return lib


def _ptr(a: np.ndarray | None):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


@dataclass
class CorpusSpec:
    seed: int
    ndocs: int
    ncent: int
    dim: int = 128
    len_kind: int = LEN_FIXED
    len_lo: int = 32
    len_hi: int = 32
    len_mean: float = 0.0
    len_sigma: float = 0.5
    pop_kind: int = POP_UNIFORM
    zipf_s: float = 1.1
    tok_sigma: float = 0.05
    q_sigma: float = 0.1


class Corpus:
    """A generated corpus.  Tokens are produced on demand, per doc range."""

    def __init__(self, spec: CorpusSpec, nthreads: int = 0):
        self.spec = spec
        self.nthreads = nthreads
        lib = _load()
        cfg = _Cfg(spec.seed, spec.ndocs, spec.ncent, spec.dim, spec.len_kind, spec.len_lo, spec.len_hi,
                   spec.len_mean, spec.len_sigma, spec.pop_kind, spec.zipf_s, spec.tok_sigma, spec.q_sigma)
        self._ctx = lib.synth_create(ctypes.byref(cfg))
        if not self._ctx:
            raise ValueError(f"bad corpus spec {spec}")
        cp = lib.synth_centroids(self._ctx)
        self.centroids_k = np.ctypeslib.as_array(cp, shape=(spec.ncent, spec.dim)).copy()
        self.lengths = np.empty(spec.ndocs, dtype=np.int32)
        if spec.ndocs:
            lib.synth_doc_lengths(self._ctx, 0, spec.ndocs, _ptr(self.lengths))
        self.doc_off = np.zeros(spec.ndocs + 1, dtype=np.int64)
        np.cumsum(self.lengths, out=self.doc_off[1:])
        self.ntok = int(self.doc_off[-1])

    def __del__(self):
        ctx = getattr(self, "_ctx", None)
        if ctx and _lib is not None:
            _lib.synth_free(ctx)
            self._ctx = None

    @property
    def dim(self) -> int:
        return self.spec.dim

    def tokens(self, d0: int = 0, d1: int | None = None, want_k: bool = True):
        """Tokens of docs [d0, d1): (k int16 [rows, dim] or None, cluster int32 [rows])."""
        if d1 is None:
            d1 = self.spec.ndocs
        base = self.doc_off[d0]
        rows = int(self.doc_off[d1] - base)
        off = np.ascontiguousarray(self.doc_off[d0:d1] - base)
        lens = np.ascontiguousarray(self.lengths[d0:d1])
        k = np.empty((rows, self.dim), dtype=np.int16) if want_k else None
        cl = np.empty(rows, dtype=np.int32)
        _lib.synth_doc_tokens(self._ctx, d0, d1, _ptr(off), _ptr(lens), _ptr(k), _ptr(cl), self.nthreads)
        return k, cl

    def tokens_ex(self, d0: int = 0, d1: int | None = None, want_k: bool = True, want_bf16: bool = True,
                  want_cluster: bool = True):
        """Tokens of docs [d0, d1) in one generation: (k int16 [rows, dim],
        bf16 bit patterns uint16 [rows, dim], cluster int32 [rows]); an output
        not asked for is None."""
        if d1 is None:
            d1 = self.spec.ndocs
        base = self.doc_off[d0]
        rows = int(self.doc_off[d1] - base)
        off = np.ascontiguousarray(self.doc_off[d0:d1] - base)
        lens = np.ascontiguousarray(self.lengths[d0:d1])
        k = np.empty((rows, self.dim), dtype=np.int16) if want_k else None
        b = np.empty((rows, self.dim), dtype=np.uint16) if want_bf16 else None
        cl = np.empty(rows, dtype=np.int32) if want_cluster else None
        _lib.synth_doc_tokens_ex(self._ctx, d0, d1, _ptr(off), _ptr(lens), _ptr(k), _ptr(b), _ptr(cl),
                                 self.nthreads)
        return k, b, cl

    def docs_tokens(self, docs: np.ndarray):
        """Tokens of an arbitrary list of docs, concatenated in list order.

        Returns (k [rows, dim], cluster [rows], begin [len(docs)]) where begin
        indexes the first row of each listed doc."""
        docs = np.asarray(docs, dtype=np.int64)
        lens = self.lengths[docs].astype(np.int64)
        begin = np.zeros(len(docs), dtype=np.int64)
        if len(docs):
            np.cumsum(lens[:-1], out=begin[1:])
        rows = int(lens.sum())
        k = np.empty((rows, self.dim), dtype=np.int16)
        cl = np.empty(rows, dtype=np.int32)
        _lib.synth_docs_tokens(self._ctx, _ptr(docs), len(docs), _ptr(begin), _ptr(k), _ptr(cl), self.nthreads)
        return k, cl, begin

    def queries(self, nq: int, Tq: int, query_seed: int = 0, q0: int = 0):
        """Queries [q0, q0+nq): (k int16 [nq, Tq, dim], source doc int64 [nq])."""
        k = np.empty((nq, Tq, self.dim), dtype=np.int16)
        src = np.empty(nq, dtype=np.int64)
        _lib.synth_queries(self._ctx, query_seed, q0, q0 + nq, Tq, _ptr(k), _ptr(src), self.nthreads)
        return k, src


def k_to_f32(k: np.ndarray) -> np.ndarray:
    """Grid integers -> float32 values (exact)."""
    return k.astype(np.float32) * np.float32(1.0 / 2048.0)


def k_to_bf16_bits(k: np.ndarray) -> np.ndarray:
    """Grid integers -> bf16 bit patterns (exact: every grid value is a bf16)."""
    f = k_to_f32(k)
    bits = f.view(np.uint32)
    if np.any(bits & 0xFFFF):
        raise ValueError("value not representable in bf16")
    return (bits >> 16).astype(np.uint16)


def rotation_signs(seed: int, dim: int = 128) -> np.ndarray:
    """Random signs (int8 +-1 [dim]) of a RaBitQ rotation, seeded."""
    return np.where(np.random.default_rng(seed).random(dim) < 0.5, -1, 1).astype(np.int8)


def splitmix64_at(state: int, n: int) -> int:
    return int(_load().synth_splitmix64_at(state, n))


def to_grid(x: float) -> float:
    return float(_load().synth_to_grid(x))
