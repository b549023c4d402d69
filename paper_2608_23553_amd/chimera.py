"""Thin ctypes binding of ``libchimera.so`` (see ``include/chimera.h``).

Argument marshalling only: every step of the query path runs in the HIP
library.  Device buffers and streams come from PyTorch (ROCm); host buffers
for the index builder are numpy arrays.  If the library is missing the import
of this module still works, but every call raises ``RuntimeError``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Callable, Iterable, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libchimera.so")

OK, E_INVAL, E_NOMEM, E_IO, E_FORMAT, E_DEVICE, E_UNSUPPORTED, E_BUSY = range(8)
F32, BF16 = 0, 1
REFINE_CENTROID, REFINE_TOKEN = 0, 1
_ERR_NAMES = {1: "INVAL", 2: "NOMEM", 3: "IO", 4: "FORMAT", 5: "DEVICE", 6: "UNSUPPORTED", 7: "BUSY"}

_lib = None


class ChimeraError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"chimera error {_ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


class _Info(ctypes.Structure):
    _fields_ = [("ndocs", ctypes.c_int64), ("ntokens", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("ncent", ctypes.c_int32), ("dim", ctypes.c_int32), ("nbits", ctypes.c_int32),
                ("max_doc_len", ctypes.c_int32), ("device_bytes", ctypes.c_int64), ("device", ctypes.c_int32),
                ("q_norm_limit", ctypes.c_double), ("ndeleted", ctypes.c_int64)]


def lib():
    """Loads libchimera.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, INT = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int
    sig = {
        "chimera_last_error": ([], ctypes.c_char_p),
        "chimera_builder_create": ([P, I32, I32, I32, P], INT),
        "chimera_builder_add_residuals": ([P, P, P, I64], INT),
        "chimera_builder_freeze_quantizer": ([P], INT),
        "chimera_builder_add_docs": ([P, P, P, P, I64], INT),
        "chimera_builder_reserve": ([P, I64, I64], INT),
        "chimera_builder_rabitq": ([P, P], INT),
        "chimera_builder_rabitq_sections": ([P, P, P, P, P], INT),
        "chimera_builder_quantizer": ([P, P, P], INT),
        "chimera_builder_save": ([P, ctypes.c_char_p], INT),
        "chimera_builder_upload": ([P, INT, P], INT),
        "chimera_builder_sections": ([P, P, P, P, P, P], INT),
        "chimera_builder_info": ([P, P], INT),
        "chimera_builder_free": ([P], None),
        "chimera_index_load": ([ctypes.c_char_p, INT, P], INT),
        "chimera_index_free": ([P], None),
        "chimera_index_info_get": ([P, P], INT),
        "chimera_index_delete": ([P, P, I64], INT),
        "chimera_index_compact": ([P], INT),
        "chimera_search": ([P, P, INT, I64, I32, I32, I32, I32, I32, P, P, P], INT),
        "chimera_search_refine": ([P, P, INT, I64, I32, I32, I32, I32, I32, I32, P, P, P], INT),
        "chimera_search_noalloc": ([P, P, INT, I64, I32, I32, I32, I32, I32, P, P, P], INT),
        "chimera_search_rabitq": ([P, P, INT, I64, I32, I32, I32, I32, I32, P, P, P], INT),
        "chimera_probe": ([P, P, INT, I64, I32, I32, I32, P, P, P], INT),
        "chimera_candidates": ([P, P, INT, I64, I32, I32, I32, P, P, I64, P], INT),
        "chimera_prune": ([P, P, INT, I64, I32, I32, I32, I32, P, P, P, P], INT),
        "chimera_prune_refine": ([P, P, INT, I64, I32, I32, I32, I32, I32, P, P, P, P], INT),
        "chimera_stage_times": ([P, P], INT),
        "chimera_fullbit_attach": ([P, P, I64], INT),
        "chimera_fullbit_attach_range": ([P, P, I64, I64], INT),
        "chimera_search_collab": ([P, P, INT, I64, I32, I32, I32, I32, I32, I32, I32, P, P, P, I32, P], INT),
        "chimera_search_collab_rabitq": ([P, P, INT, I64, I32, I32, I32, I32, I32, I32, I32, P, P, P, I32, P],
                                         INT),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def last_error() -> str:
    return lib().chimera_last_error().decode()


def _check(rc: int):
    if rc != OK:
        raise ChimeraError(rc, last_error())


def _np(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


def _info(st: _Info) -> dict:
    return {k: getattr(st, k) for k, _ in _Info._fields_}


# --------------------------------------------------------------- builder
class Builder:
    """Offline index builder (host only).  Two passes over the same stream of
    tokens in document order: add_residuals(...) for all tokens, freeze(),
    then add_docs(...) for all documents."""

    def __init__(self, centroids_bf16: np.ndarray, nbits: int):
        c = np.ascontiguousarray(centroids_bf16, dtype=np.uint16)
        h = ctypes.c_void_p()
        _check(lib().chimera_builder_create(_np(c), c.shape[0], c.shape[1], nbits, ctypes.byref(h)))
        self._h = h
        self.ncent, self.dim, self.nbits = c.shape[0], c.shape[1], nbits

    def __del__(self):
        self.close()

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.chimera_builder_free(self._h)
            self._h = None

    def _rows(self, t: np.ndarray, c: np.ndarray, n: int):
        """The library reads n rows of tokens and cids: check the arrays
        hold exactly that many."""
        if c.shape != (n,):
            raise ValueError(f"cids must be [{n}], got {list(c.shape)}")
        if t.shape != (n, self.dim):
            raise ValueError(f"tokens must be [{n}, {self.dim}], got {list(t.shape)}")

    def add_residuals(self, tokens_bf16: np.ndarray, cids: np.ndarray):
        t = np.ascontiguousarray(tokens_bf16, dtype=np.uint16)
        c = np.ascontiguousarray(cids, dtype=np.int32)
        if c.ndim != 1:
            raise ValueError(f"cids must be [ntok], got {list(c.shape)}")
        self._rows(t, c, c.shape[0])
        _check(lib().chimera_builder_add_residuals(self._h, _np(t), _np(c), c.shape[0]))

    def freeze(self):
        _check(lib().chimera_builder_freeze_quantizer(self._h))

    def add_docs(self, tokens_bf16: np.ndarray, cids: np.ndarray, doc_lens: np.ndarray):
        t = np.ascontiguousarray(tokens_bf16, dtype=np.uint16)
        c = np.ascontiguousarray(cids, dtype=np.int32)
        l = np.ascontiguousarray(doc_lens, dtype=np.int32)
        if l.ndim != 1:
            raise ValueError("doc_lens must be [ndocs]")
        self._rows(t, c, int(l.astype(np.int64).sum()))
        _check(lib().chimera_builder_add_docs(self._h, _np(t), _np(c), _np(l), l.shape[0]))

    def reserve(self, ndocs: int, ntok: int):
        _check(lib().chimera_builder_reserve(self._h, ndocs, ntok))

    def rabitq(self, signs: np.ndarray):
        """chimera_builder_rabitq: also encode the tokens with RaBitQ under
        the rotation H diag(signs) (signs int8 [dim] of +-1)."""
        s = np.ascontiguousarray(signs, dtype=np.int8)
        if s.shape != (self.dim,):
            raise ValueError(f"signs must be [{self.dim}], got {list(s.shape)}")
        _check(lib().chimera_builder_rabitq(self._h, _np(s)))

    def quantizer(self) -> Tuple[np.ndarray, np.ndarray]:
        B = 1 << self.nbits
        cut = np.empty(B - 1, np.int32)
        w = np.empty(B, np.uint16)
        _check(lib().chimera_builder_quantizer(self._h, _np(cut), _np(w)))
        return cut, w

    def info(self) -> dict:
        st = _Info()
        _check(lib().chimera_builder_info(self._h, ctypes.byref(st)))
        return _info(st)

    def rabitq_sections(self) -> dict:
        """Host copies of the RaBitQ sections (chimera_builder_rabitq_sections)."""
        n = self.info()["ntokens"]
        out = dict(bits1=np.empty((n, self.dim // 8), np.uint8), g1=np.empty(n, np.float32),
                   codes4=np.empty((n, self.dim // 2), np.uint8), g4=np.empty(n, np.float32))
        _check(lib().chimera_builder_rabitq_sections(self._h, _np(out["bits1"]), _np(out["g1"]), _np(out["codes4"]),
                                                     _np(out["g4"])))
        return out

    def sections(self, which=("doc_off", "cid", "codes", "ivf_off", "ivf_doc")) -> dict:
        """Host copies of the built sections named in `which`."""
        inf = self.info()
        shapes = dict(doc_off=((inf["ndocs"] + 1,), np.int64), cid=((inf["ntokens"],), np.int32),
                      codes=((inf["ntokens"], self.dim * self.nbits // 8), np.uint8),
                      ivf_off=((self.ncent + 1,), np.int64), ivf_doc=((inf["nnz"],), np.int32))
        out = {n: np.empty(*shapes[n]) for n in which}
        _check(lib().chimera_builder_sections(self._h, *(_np(out.get(n)) for n in
                                                        ("doc_off", "cid", "codes", "ivf_off", "ivf_doc"))))
        return out

    def save(self, path: str):
        _check(lib().chimera_builder_save(self._h, path.encode()))

    def upload(self, device: int = 0) -> "Index":
        h = ctypes.c_void_p()
        _check(lib().chimera_builder_upload(self._h, device, ctypes.byref(h)))
        return Index(h)


def build_index(centroids_bf16: np.ndarray, nbits: int,
                chunks: Callable[[], Iterable[Tuple[np.ndarray, np.ndarray, np.ndarray]]],
                rabitq_signs: np.ndarray | None = None) -> Builder:
    """Two-pass streaming build.  ``chunks()`` must yield the same sequence of
    (tokens_bf16 [rows,dim], cids [rows], doc_lens [ndocs_chunk]) each time it
    is called, covering every document in order.  rabitq_signs: also encode
    RaBitQ codes (Builder.rabitq)."""
    b = Builder(centroids_bf16, nbits)
    if rabitq_signs is not None:
        b.rabitq(rabitq_signs)
    for tok, cid, _ in chunks():
        b.add_residuals(tok, cid)
    b.freeze()
    for tok, cid, lens in chunks():
        b.add_docs(tok, cid, lens)
    return b


# ----------------------------------------------------------------- index
def _stream_ptr(stream) -> ctypes.c_void_p:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _q_args(Q):
    import torch
    if not Q.is_cuda:
        raise ValueError("Q must be a device tensor")
    if Q.dim() != 3:
        raise ValueError("Q must be [nq, Tq, d]")
    Q = Q.contiguous()
    if Q.dtype == torch.float32:
        dt = F32
    elif Q.dtype == torch.bfloat16:
        dt = BF16
    else:
        raise ValueError("Q must be float32 or bfloat16")
    return Q, dt


class Index:
    """A device-resident index (owns its HBM); see ``chimera_index_load``."""

    def __init__(self, handle: ctypes.c_void_p):
        self._h = handle
        self._info = self.info()

    @classmethod
    def load(cls, path: str, device: int = 0) -> "Index":
        h = ctypes.c_void_p()
        _check(lib().chimera_index_load(path.encode(), device, ctypes.byref(h)))
        return cls(h)

    def close(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.chimera_index_free(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def info(self) -> dict:
        st = _Info()
        _check(lib().chimera_index_info_get(self._h, ctypes.byref(st)))
        return _info(st)

    def delete(self, doc_ids):
        """chimera_index_delete: later searches skip these documents."""
        ids = np.ascontiguousarray(np.asarray(doc_ids, dtype=np.int64).ravel())
        _check(lib().chimera_index_delete(self._h, _np(ids), ids.size))
        self._info = self.info()

    def compact(self):
        """chimera_index_compact: drops the deleted documents' tokens and
        posting entries from the device index (ids unchanged)."""
        _check(lib().chimera_index_compact(self._h))
        self._info = self.info()

    def _q(self, Q):
        """Q as the library takes it, on the index's own GPU (the library
        receives a bare device pointer and cannot check that)."""
        Q, dt = _q_args(Q)
        if Q.device.index != self._info["device"]:
            raise ValueError(f"Q is on {Q.device}, the index on cuda:{self._info['device']}")
        return Q, dt

    @property
    def device(self):
        import torch
        return torch.device("cuda", self._info["device"])

    def search(self, Q, nprobe: int, ncand: int, k: int, out=None, stream=None, refine: int = REFINE_CENTROID):
        """Top-k (ids int32 [nq,k], scores float32 [nq,k]) for queries Q [nq,Tq,d].
        refine: REFINE_CENTROID (chimera_search) or REFINE_TOKEN
        (chimera_search_refine)."""
        import torch
        Q, dt = self._q(Q)
        nq, Tq, d = Q.shape
        if out is None:
            ids = torch.empty((nq, k), dtype=torch.int32, device=Q.device)
            scores = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
        else:
            ids, scores = out
            for t, dtype, name in ((ids, torch.int32, "ids"), (scores, torch.float32, "scores")):
                if tuple(t.shape) != (nq, k) or t.dtype != dtype or t.device != Q.device or not t.is_contiguous():
                    raise ValueError(f"out {name} must be a contiguous {dtype} tensor [{nq}, {k}] on {Q.device}")
        if refine == REFINE_CENTROID:
            _check(lib().chimera_search(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe, ncand, k,
                                        ctypes.c_void_p(ids.data_ptr()), ctypes.c_void_p(scores.data_ptr()),
                                        _stream_ptr(stream)))
        else:
            _check(lib().chimera_search_refine(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe, ncand,
                                               k, refine, ctypes.c_void_p(ids.data_ptr()),
                                               ctypes.c_void_p(scores.data_ptr()), _stream_ptr(stream)))
        return ids, scores

    def search_rabitq(self, Q, nprobe: int, ncand: int, k: int, out=None, stream=None):
        """chimera_search_rabitq: step 4 scored from the RaBitQ 1-bit codes."""
        import torch
        Q, dt = self._q(Q)
        nq, Tq, d = Q.shape
        if out is None:
            ids = torch.empty((nq, k), dtype=torch.int32, device=Q.device)
            scores = torch.empty((nq, k), dtype=torch.float32, device=Q.device)
        else:
            ids, scores = out
        _check(lib().chimera_search_rabitq(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe, ncand, k,
                                           ctypes.c_void_p(ids.data_ptr()), ctypes.c_void_p(scores.data_ptr()),
                                           _stream_ptr(stream)))
        return ids, scores

    def attach_fullbit(self, tokens_bf16):
        """Attaches the full-precision store: host uint16 [ntok, d] bf16 bits
        in the index's token order (chimera_fullbit_attach, which keeps its own
        grid-integer copy).  None drops it."""
        if tokens_bf16 is None:
            _check(lib().chimera_fullbit_attach(self._h, None, 0))
            return
        a = np.ascontiguousarray(tokens_bf16, dtype=np.uint16)
        dim = self._info["dim"]
        if a.ndim != 2 or a.shape[1] != dim:
            raise ValueError(f"tokens must be [ntok, {dim}], got {list(a.shape)}")
        _check(lib().chimera_fullbit_attach(self._h, _np(a), a.shape[0]))

    def attach_fullbit_range(self, tokens_bf16, t0: int):
        """Tokens t0 .. t0+n-1 of the full-precision store (chimera_fullbit_attach_range):
        host uint16 [n, d] bf16 bits; t0 = 0 starts a new store, later ranges
        follow on."""
        a = np.ascontiguousarray(tokens_bf16, dtype=np.uint16)
        dim = self._info["dim"]
        if a.ndim != 2 or a.shape[1] != dim:
            raise ValueError(f"tokens must be [n, {dim}], got {list(a.shape)}")
        _check(lib().chimera_fullbit_attach_range(self._h, _np(a), t0, a.shape[0]))

    def search_collab(self, Q, nprobe: int, ncand: int, kfb: int, chunks: int, k: int, nthreads: int = 0,
                      stream=None):
        """CPU-GPU collaborative scoring (chimera_search_collab): host numpy
        (ids int32 [nq,k], scores float32 [nq,k], n_full int32 [nq])."""
        Q, dt = self._q(Q)
        nq, Tq, d = Q.shape
        ids = np.empty((nq, k), dtype=np.int32)
        scores = np.empty((nq, k), dtype=np.float32)
        n_full = np.empty(nq, dtype=np.int32)
        _check(lib().chimera_search_collab(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe, ncand, kfb,
                                           chunks, k, _np(ids), _np(scores), _np(n_full), nthreads,
                                           _stream_ptr(stream)))
        return ids, scores, n_full

    def search_collab_rabitq(self, Q, nprobe: int, ncand: int, kfb: int, chunks: int, k: int, nthreads: int = 0,
                             stream=None):
        """chimera_search_collab_rabitq: GPU 1-bit RaBitQ scores, host 4-bit
        RaBitQ scores (host numpy ids, scores, n_full)."""
        Q, dt = self._q(Q)
        nq, Tq, d = Q.shape
        ids = np.empty((nq, k), dtype=np.int32)
        scores = np.empty((nq, k), dtype=np.float32)
        n_full = np.empty(nq, dtype=np.int32)
        _check(lib().chimera_search_collab_rabitq(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe,
                                                  ncand, kfb, chunks, k, _np(ids), _np(scores), _np(n_full),
                                                  nthreads, _stream_ptr(stream)))
        return ids, scores, n_full

    def search_raw(self, q_ptr: int, q_dtype: int, nq: int, Tq: int, d: int, nprobe: int, ncand: int, k: int,
                   ids_ptr: int, scores_ptr: int, stream_ptr: int) -> int:
        """Direct call with raw pointers; returns the status code."""
        return lib().chimera_search(self._h, ctypes.c_void_p(q_ptr), q_dtype, nq, Tq, d, nprobe, ncand, k,
                                    ctypes.c_void_p(ids_ptr), ctypes.c_void_p(scores_ptr), ctypes.c_void_p(stream_ptr))

    def probe(self, Q, nprobe: int, stream=None):
        import torch
        Q, dt = self._q(Q)
        nq, Tq, d = Q.shape
        ids = torch.empty((nq, Tq, nprobe), dtype=torch.int32, device=Q.device)
        keys = torch.empty((nq, Tq, nprobe), dtype=torch.int32, device=Q.device)
        _check(lib().chimera_probe(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe,
                                   ctypes.c_void_p(ids.data_ptr()), ctypes.c_void_p(keys.data_ptr()),
                                   _stream_ptr(stream)))
        return ids, keys

    def candidates(self, Q, nprobe: int, capacity: int | None = None, stream=None):
        import torch
        Q, dt = self._q(Q)
        nq, Tq, d = Q.shape
        if capacity is None:
            capacity = nq * self._info["ndocs"]
        offsets = torch.empty(nq + 1, dtype=torch.int64, device=Q.device)
        doc_ids = torch.empty(max(capacity, 1), dtype=torch.int32, device=Q.device)
        _check(lib().chimera_candidates(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe,
                                        ctypes.c_void_p(offsets.data_ptr()), ctypes.c_void_p(doc_ids.data_ptr()),
                                        capacity, _stream_ptr(stream)))
        return offsets, doc_ids

    def prune(self, Q, nprobe: int, ncand: int, stream=None, refine: int = REFINE_CENTROID):
        import torch
        Q, dt = self._q(Q)
        nq, Tq, d = Q.shape
        nc = min(ncand, self._info["ndocs"])
        cand = torch.empty((nq, nc), dtype=torch.int32, device=Q.device)
        keys = torch.empty((nq, nc), dtype=torch.int32, device=Q.device)
        nval = torch.empty(nq, dtype=torch.int32, device=Q.device)
        if refine == REFINE_CENTROID:
            _check(lib().chimera_prune(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe, ncand,
                                       ctypes.c_void_p(cand.data_ptr()), ctypes.c_void_p(keys.data_ptr()),
                                       ctypes.c_void_p(nval.data_ptr()), _stream_ptr(stream)))
        else:
            _check(lib().chimera_prune_refine(self._h, ctypes.c_void_p(Q.data_ptr()), dt, nq, Tq, d, nprobe, ncand,
                                              refine, ctypes.c_void_p(cand.data_ptr()),
                                              ctypes.c_void_p(keys.data_ptr()), ctypes.c_void_p(nval.data_ptr()),
                                              _stream_ptr(stream)))
        return cand, keys, nval

    def stage_times(self) -> np.ndarray:
        """[round, probe, walk, select, score, topk] ms summed since the last
        call, then the number of sub-batches (see chimera_stage_times)."""
        ms = np.zeros(7, np.float32)
        _check(lib().chimera_stage_times(self._h, _np(ms)))
        return ms
