"""CPU oracle of the GPU query path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the GPU library
(``paper_2608_23553_amd``); both consume the seeded inputs from ``synth``.

All arithmetic is exact int64 on grid integers (``oracle.h`` explains the
convention); this module only marshals numpy arrays into ``liboracle.so``.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

KEY_SCALE = 2.0 ** -22  # one key unit


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build() (make -C oracle)")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "orc_grid_k": ([ctypes.c_double], I32),
        "orc_grid_f32": ([P, I64, P], None),
        "orc_grid_bf16": ([P, I64, P], None),
        "orc_assign": ([P, I64, P, I32, I32, P, ctypes.c_int], None),
        "orc_ivf_docs": ([P, P, I64, I32, P, P], I64),
        "orc_ivf_tokens": ([P, I64, I32, P, P], None),
        "orc_residual_hist": ([P, P, I64, P, I32, P], None),
        "orc_quantizer": ([P, ctypes.c_int, P, P], ctypes.c_int),
        "orc_encode": ([P, P, I64, P, I32, P, ctypes.c_int, P], None),
        "orc_pack": ([P, I64, I32, ctypes.c_int, P], None),
        "orc_unpack": ([P, I64, I32, ctypes.c_int, P], None),
        "orc_centroid_scores": ([P, I32, P, I32, I32, P], None),
        "orc_probe": ([P, I32, I32, I32, P, P], None),
        "orc_candidates": ([P, I32, I32, P, P, I64, P], I64),
        "orc_partial_scores": ([P, P, I32, I32, I32, P, P, I64, P, P], I64),
        "orc_partial_scores_res": ([P, P, I32, I32, I32, P, I32, P, P, P, P, P, I64, P, P], I64),
        "orc_topk": ([P, P, I64, I64, P, P], I64),
        "orc_doc_scores": ([P, I32, I32, P, I32, P, I64, P, P, P, P, P], None),
        "orc_key_to_score": ([I64], ctypes.c_float),
        "orc_exact_chamfer": ([P, I32, I32, P, P, I64, P], None),
        "orc_search": ([P, I32, I32, P, I64, P, P, P, P, P, P, I64, I32, I32, I32, I32,
                        P, P, P, P, P, P, P, P, ctypes.c_int, P, P, P, ctypes.c_int], ctypes.c_int),
        "orc_prune_batch": ([P, I32, I32, I64, P, P, P, I64, I32, I32, I32, P, P, P, P, P, P,
                             ctypes.c_int, P, P, P, P, P, ctypes.c_int], ctypes.c_int),
        "orc_rabitq_rotate": ([P, I64, I32, P, P], None),
        "orc_rabitq_quantize": ([P, I64, I32, ctypes.c_int, P, P], None),
        "orc_rabitq_encode": ([P, I64, I32, P, ctypes.c_int, P, P, P], None),
        "orc_rabitq_pack1": ([P, I64, I32, ctypes.c_int, P], None),
        "orc_lut_ip": ([P, P, I32], I64),
        "orc_rabitq_doc_scores": ([P, I32, I32, P, ctypes.c_int, ctypes.c_int, I64, P, P, P, P, P], None),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _p(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------ grid
def grid_k(x: float) -> int:
    return int(_load().orc_grid_k(float(x)))


def grid_f32(x) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, dtype=np.int16)
    _load().orc_grid_f32(_p(x), x.size, _p(out))
    return out


def grid_bf16(bits) -> np.ndarray:
    bits = _c(bits, np.uint16)
    out = np.empty(bits.shape, dtype=np.int16)
    _load().orc_grid_bf16(_p(bits), bits.size, _p(out))
    return out


# ------------------------------------------------------- index building
def assign(tok_k, cent_k, nthreads: int = 0) -> np.ndarray:
    tok_k, cent_k = _c(tok_k, np.int16), _c(cent_k, np.int16)
    out = np.empty(tok_k.shape[0], dtype=np.int32)
    _load().orc_assign(_p(tok_k), tok_k.shape[0], _p(cent_k), cent_k.shape[0], cent_k.shape[1], _p(out), nthreads)
    return out


def ivf_docs(cid, doc_off, ncent: int):
    cid, doc_off = _c(cid, np.int32), _c(doc_off, np.int64)
    ndocs = doc_off.shape[0] - 1
    off = np.empty(ncent + 1, dtype=np.int64)
    nnz = _load().orc_ivf_docs(_p(cid), _p(doc_off), ndocs, ncent, _p(off), None)
    docs = np.empty(max(nnz, 1), dtype=np.int32)
    _load().orc_ivf_docs(_p(cid), _p(doc_off), ndocs, ncent, _p(off), _p(docs))
    return off, docs[:nnz]


def ivf_tokens(cid, ncent: int):
    """Token-level lists: (tok_off [ncent+1], ivf_tok [ntok]), tokens ascending."""
    cid = _c(cid, np.int32)
    off = np.empty(ncent + 1, dtype=np.int64)
    tok = np.empty(max(cid.shape[0], 1), dtype=np.int32)
    _load().orc_ivf_tokens(_p(cid), cid.shape[0], ncent, _p(off), _p(tok))
    return off, tok[:cid.shape[0]]


def token_docs(doc_off) -> np.ndarray:
    """Document of every token (doc_off [ndocs+1])."""
    doc_off = _c(doc_off, np.int64)
    return np.repeat(np.arange(doc_off.shape[0] - 1, dtype=np.int32), np.diff(doc_off))


def residual_hist(tok_k, cid, cent_k, hist=None) -> np.ndarray:
    tok_k, cid, cent_k = _c(tok_k, np.int16), _c(cid, np.int32), _c(cent_k, np.int16)
    if hist is None:
        hist = np.zeros(8193, dtype=np.int64)
    _load().orc_residual_hist(_p(tok_k), _p(cid), cid.shape[0], _p(cent_k), cent_k.shape[1], _p(hist))
    return hist


def quantizer(hist, nbits: int):
    hist = _c(hist, np.int64)
    B = 1 << nbits
    cut = np.empty(B - 1, dtype=np.int32)
    w = np.empty(B, dtype=np.int32)
    if _load().orc_quantizer(_p(hist), nbits, _p(cut), _p(w)) != 0:
        raise ValueError("empty residual histogram")
    return cut, w


def encode(tok_k, cid, cent_k, cut_k, nbits: int) -> np.ndarray:
    tok_k, cid, cent_k, cut_k = _c(tok_k, np.int16), _c(cid, np.int32), _c(cent_k, np.int16), _c(cut_k, np.int32)
    out = np.empty(tok_k.shape, dtype=np.uint8)
    _load().orc_encode(_p(tok_k), _p(cid), cid.shape[0], _p(cent_k), cent_k.shape[1], _p(cut_k), nbits, _p(out))
    return out


def pack(codes, nbits: int) -> np.ndarray:
    codes = _c(codes, np.uint8)
    ntok, dim = codes.shape
    out = np.empty((ntok, dim * nbits // 8), dtype=np.uint8)
    _load().orc_pack(_p(codes), ntok, dim, nbits, _p(out))
    return out


def unpack(packed, dim: int, nbits: int) -> np.ndarray:
    packed = _c(packed, np.uint8)
    ntok = packed.shape[0]
    out = np.empty((ntok, dim), dtype=np.uint8)
    _load().orc_unpack(_p(packed), ntok, dim, nbits, _p(out))
    return out


# ----------------------------------------------------------- query path
def centroid_scores(q_k, cent_k) -> np.ndarray:
    q_k, cent_k = _c(q_k, np.int16), _c(cent_k, np.int16)
    Tq, dim = q_k.shape
    S = np.empty((Tq, cent_k.shape[0]), dtype=np.int64)
    _load().orc_centroid_scores(_p(q_k), Tq, _p(cent_k), cent_k.shape[0], dim, _p(S))
    return S


def probe(S, nprobe: int):
    S = _c(S, np.int64)
    Tq, ncent = S.shape
    ids = np.empty((Tq, nprobe), dtype=np.int32)
    keys = np.empty((Tq, nprobe), dtype=np.int64)
    _load().orc_probe(_p(S), Tq, ncent, nprobe, _p(ids), _p(keys))
    return ids, keys


def candidates(cent_ids, ivf_off, ivf_doc, ndocs: int) -> np.ndarray:
    cent_ids = _c(cent_ids, np.int32)
    Tq, nprobe = cent_ids.shape
    out = np.empty(max(ndocs, 1), dtype=np.int32)
    n = _load().orc_candidates(_p(cent_ids), Tq, nprobe, _p(_c(ivf_off, np.int64)), _p(_c(ivf_doc, np.int32)),
                               ndocs, _p(out))
    return out[:n].copy()


def partial_scores(S, cent_ids, ivf_off, ivf_doc, ndocs: int):
    S, cent_ids = _c(S, np.int64), _c(cent_ids, np.int32)
    Tq, ncent = S.shape
    nprobe = cent_ids.shape[1]
    docs = np.empty(max(ndocs, 1), dtype=np.int32)
    fp = np.empty(max(ndocs, 1), dtype=np.int64)
    n = _load().orc_partial_scores(_p(S), _p(cent_ids), Tq, ncent, nprobe, _p(_c(ivf_off, np.int64)),
                                   _p(_c(ivf_doc, np.int32)), ndocs, _p(docs), _p(fp))
    return docs[:n].copy(), fp[:n].copy()


def partial_scores_res(S, cent_ids, q_k, w_k, tok_off, ivf_tok, tok_doc, codes, ndocs: int):
    """F' from the retrieved tokens' decoded scores (see orc_partial_scores_res)."""
    S, cent_ids, q_k, w_k = _c(S, np.int64), _c(cent_ids, np.int32), _c(q_k, np.int16), _c(w_k, np.int32)
    tok_off, ivf_tok, tok_doc = _c(tok_off, np.int64), _c(ivf_tok, np.int32), _c(tok_doc, np.int32)
    codes = _c(codes, np.uint8)
    Tq, ncent = S.shape
    nprobe = cent_ids.shape[1]
    docs = np.empty(max(ndocs, 1), dtype=np.int32)
    fp = np.empty(max(ndocs, 1), dtype=np.int64)
    n = _load().orc_partial_scores_res(_p(S), _p(cent_ids), Tq, ncent, nprobe, _p(q_k), q_k.shape[1], _p(w_k),
                                       _p(tok_off), _p(ivf_tok), _p(tok_doc), _p(codes), ndocs, _p(docs), _p(fp))
    return docs[:n].copy(), fp[:n].copy()


def topk(ids, keys, k: int):
    ids, keys = _c(ids, np.int32), _c(keys, np.int64)
    n = ids.shape[0]
    oi = np.empty(max(min(k, n), 1), dtype=np.int32)
    ok = np.empty(max(min(k, n), 1), dtype=np.int64)
    m = _load().orc_topk(_p(ids), _p(keys), n, k, _p(oi), _p(ok))
    return oi[:m].copy(), ok[:m].copy()


def doc_scores(S, q_k, w_k, tok_begin, tok_len, cid, codes) -> np.ndarray:
    S, q_k, w_k = _c(S, np.int64), _c(q_k, np.int16), _c(w_k, np.int32)
    tok_begin, tok_len = _c(tok_begin, np.int64), _c(tok_len, np.int32)
    cid, codes = _c(cid, np.int32), _c(codes, np.uint8)
    Tq, ncent = S.shape
    n = tok_begin.shape[0]
    out = np.empty(max(n, 1), dtype=np.int64)
    _load().orc_doc_scores(_p(S), Tq, ncent, _p(q_k), q_k.shape[1], _p(w_k), n, _p(tok_begin), _p(tok_len),
                           _p(cid), _p(codes), _p(out))
    return out[:n].copy()


def key_to_score(key: int) -> float:
    return float(_load().orc_key_to_score(int(key)))


def keys_to_scores(keys) -> np.ndarray:
    """Vector form of the key -> fp32 score rule (single rounding, then 2^-22)."""
    keys = np.asarray(keys, dtype=np.int64)
    out = np.array([key_to_score(int(x)) for x in keys.ravel()], dtype=np.float32).reshape(keys.shape)
    out[keys == np.iinfo(np.int64).min] = -np.inf
    return out


def exact_chamfer(q_k, tok_k, doc_off) -> np.ndarray:
    q_k, tok_k, doc_off = _c(q_k, np.int16), _c(tok_k, np.int16), _c(doc_off, np.int64)
    Tq, dim = q_k.shape
    ndocs = doc_off.shape[0] - 1
    F = np.empty(max(ndocs, 1), dtype=np.int64)
    _load().orc_exact_chamfer(_p(q_k), Tq, dim, _p(tok_k), _p(doc_off), ndocs, _p(F))
    return F[:ndocs].copy()


def collaborative_scoring(refine_ids, approx_keys, exact_key, ncand: int, kfb: int, chunks: int, k: int):
    """CPU-GPU collaborative document scoring (Sec. 4, document scoring;
    Alg. 3) for one query, written from the algorithm's steps.

    refine_ids  S_refine, in the order it is cut into chunks (ascending
                document id: the paper leaves the order open)
    approx_keys the GPU-side complete scores F^ of those documents (keys)
    exact_key   doc -> full-precision score key
    Chunk i (0-based) holds positions floor(i ncand / chunks) ..
    floor((i+1) ncand / chunks) - 1 of S_refine.  After chunk i every document
    seen so far that ranks among the first ceil((i+1) kfb / chunks) by
    (F^ desc, id asc) gets a full-precision score if it has none.  Returns the
    k best scored documents by (F desc, id asc) as (ids, keys) padded with
    (-1, INT64_MIN), and the number of full-precision scores computed."""
    n = len(refine_ids)
    seen = []
    full = {}
    for i in range(chunks):
        lo, hi = i * ncand // chunks, (i + 1) * ncand // chunks
        seen.extend(range(lo, min(hi, n)))
        quota = min(-(-(i + 1) * kfb // chunks), len(seen))
        ranked = sorted(seen, key=lambda u: (-int(approx_keys[u]), int(refine_ids[u])))
        for u in ranked[:quota]:
            d = int(refine_ids[u])
            if d not in full:
                full[d] = int(exact_key(d))
    best = sorted(full.items(), key=lambda kv: (-kv[1], kv[0]))[:k]
    ids = np.full(k, -1, np.int32)
    keys = np.full(k, np.iinfo(np.int64).min, np.int64)
    for r, (d, key) in enumerate(best):
        ids[r], keys[r] = d, key
    return ids, keys, len(full)


def search_streamed(oi, q_k, nprobe: int, ncand: int, k: int, docs_tokens):
    """The oracle's search of one query q_k [Tq, dim] on an OracleIndex built
    without codes: the stages composed as orc_search composes them, with the
    kept documents' tokens supplied by docs_tokens(ids int64) -> (tok_k
    [rows, dim], cid [rows], begin [len(ids)]) and encoded here (for corpora
    whose tokens do not fit in memory; regenerated by the caller)."""
    S = centroid_scores(q_k, oi.cent_k)
    ci, ck = probe(S, nprobe)
    docs, fp = partial_scores(S, ci, oi.ivf_off, oi.ivf_doc, oi.ndocs)
    r, rk = topk(docs, fp, ncand)
    tk, cl, begin = docs_tokens(r.astype(np.int64))
    codes = encode(tk, cl, oi.cent_k, oi.cut_k, oi.nbits)
    lens = np.diff(oi.doc_off)[r].astype(np.int32)
    fh = doc_scores(S, q_k, oi.w_k, begin, lens, cl, codes)
    ids, keys = topk(r, fh, k)
    return dict(cent_ids=ci, cent_keys=ck, cand=r, cand_keys=rk, ids=ids, keys=keys, scores=keys_to_scores(keys))


def search_deleted(oi, q_k, nprobe: int, ncand: int, k: int, deleted, refine: bool = False):
    """The search with a deletion bitmap (Sec. 3.3, handling updates): the
    stages composed as orc_search composes them, with the deleted documents
    (deleted: bool [ndocs]) dropped from S_Q before the top-ncand.  q_k
    [nq, Tq, dim]; ids padded with -1 and keys with INT64_MIN past the hits."""
    q_k = _c(q_k, np.int16)
    deleted = np.asarray(deleted, dtype=bool)
    nq = q_k.shape[0]
    ids = np.full((nq, k), -1, np.int32)
    keys = np.full((nq, k), np.iinfo(np.int64).min, np.int64)
    lens = np.diff(oi.doc_off)
    rf, off, tok, tdoc = oi._refine_args(refine)
    for qi in range(nq):
        S = centroid_scores(q_k[qi], oi.cent_k)
        ci, _ = probe(S, nprobe)
        if rf:
            docs, fp = partial_scores_res(S, ci, q_k[qi], oi.w_k, off, tok, tdoc, oi.codes, oi.ndocs)
        else:
            docs, fp = partial_scores(S, ci, oi.ivf_off, oi.ivf_doc, oi.ndocs)
        keep = ~deleted[docs]
        r, _ = topk(docs[keep], fp[keep], ncand)
        fh = doc_scores(S, q_k[qi], oi.w_k, oi.doc_off[r], lens[r].astype(np.int32), oi.cid, oi.codes)
        i, kk = topk(r, fh, k)
        ids[qi, :len(i)], keys[qi, :len(i)] = i, kk
    return dict(ids=ids, keys=keys, scores=keys_to_scores(keys))


# ------------------------------------------------------- RaBitQ (Sec. 2.2, 3.1, 4.1)
def rabitq_rotate(x_k, signs) -> np.ndarray:
    """xp = H diag(s) x per row (orc_rabitq_rotate), int64."""
    x_k, signs = _c(np.atleast_2d(x_k), np.int16), _c(signs, np.int8)
    n, D = x_k.shape
    out = np.empty((n, D), np.int64)
    _load().orc_rabitq_rotate(_p(x_k), n, D, _p(signs), _p(out))
    return out


def rabitq_quantize(xp, B: int):
    """Nearest codewords of the rows of xp: (codes uint8 [n, D], az int64 [n])."""
    xp = _c(np.atleast_2d(xp), np.int64)
    n, D = xp.shape
    codes = np.empty((n, D), np.uint8)
    az = np.empty(max(n, 1), np.int64)
    _load().orc_rabitq_quantize(_p(xp), n, D, B, _p(codes), _p(az))
    return codes, az[:n]


def rabitq_encode(x_k, signs, B: int):
    """(codes uint8 [n, D], gB float32 [n], g1 float32 [n]) of grid tokens."""
    x_k, signs = _c(np.atleast_2d(x_k), np.int16), _c(signs, np.int8)
    n, D = x_k.shape
    codes = np.empty((n, D), np.uint8)
    gB = np.empty(max(n, 1), np.float32)
    g1 = np.empty(max(n, 1), np.float32)
    _load().orc_rabitq_encode(_p(x_k), n, D, _p(signs), B, _p(codes), _p(gB), _p(g1))
    return codes, gB[:n], g1[:n]


def rabitq_pack1(codes, B: int) -> np.ndarray:
    codes = _c(np.atleast_2d(codes), np.uint8)
    n, D = codes.shape
    out = np.empty((n, D // 8), np.uint8)
    _load().orc_rabitq_pack1(_p(codes), n, D, B, _p(out))
    return out


def lut_ip(xq, bits) -> int:
    xq, bits = _c(xq, np.int64), _c(bits, np.uint8)
    return int(_load().orc_lut_ip(_p(xq), _p(bits), xq.shape[0]))


def rabitq_doc_scores(q_k, signs, B: int, bits: int, tok_begin, tok_len, codes, g) -> np.ndarray:
    q_k, signs = _c(q_k, np.int16), _c(signs, np.int8)
    tok_begin, tok_len = _c(tok_begin, np.int64), _c(tok_len, np.int32)
    codes, g = _c(codes, np.uint8), _c(g, np.float32)
    Tq, D = q_k.shape
    n = tok_begin.shape[0]
    out = np.empty(max(n, 1), np.int64)
    _load().orc_rabitq_doc_scores(_p(q_k), Tq, D, _p(signs), B, bits, n, _p(tok_begin), _p(tok_len), _p(codes),
                                  _p(g), _p(out))
    return out[:n].copy()


def search_rabitq(oi, q_k, nprobe: int, ncand: int, k: int, signs, B: int, codes, g1):
    """The search with the document scores of the 1-bit RaBitQ part (Sec.
    3.2 document scoring on the GPU): probe, candidates, F' and top-ncand as
    orc_search, then F^ from rabitq_doc_scores (bits 1) and the top-k.  codes
    [ntok, D] are the B-bit codes of every token, g1 their 1-bit factors."""
    q_k = _c(q_k, np.int16)
    nq = q_k.shape[0]
    ids = np.full((nq, k), -1, np.int32)
    keys = np.full((nq, k), np.iinfo(np.int64).min, np.int64)
    lens = np.diff(oi.doc_off)
    for qi in range(nq):
        S = centroid_scores(q_k[qi], oi.cent_k)
        ci, _ = probe(S, nprobe)
        docs, fp = partial_scores(S, ci, oi.ivf_off, oi.ivf_doc, oi.ndocs)
        r, _ = topk(docs, fp, ncand)
        fh = rabitq_doc_scores(q_k[qi], signs, B, 1, oi.doc_off[r], lens[r].astype(np.int32), codes, g1)
        i, kk = topk(r, fh, k)
        ids[qi, :len(i)], keys[qi, :len(i)] = i, kk
    return dict(ids=ids, keys=keys, scores=keys_to_scores(keys))


def search_collab_rabitq(oi, q_k, nprobe: int, ncand: int, kfb: int, chunks: int, k: int, signs, B: int,
                         codes, g1, gB):
    """Alg. 3 with the paper's code split (Sec. 3.1): steps 1-3 as orc_search,
    the GPU-side score of each kept document from the 1-bit part of its
    RaBitQ codes and the CPU-side score from the whole B-bit codes
    (rabitq_doc_scores with bits 1 and bits B), through
    collaborative_scoring."""
    q_k = _c(q_k, np.int16)
    nq = q_k.shape[0]
    nc = min(ncand, oi.ndocs)
    pr = oi.prune(q_k, nprobe, nc)
    out = dict(ids=np.empty((nq, k), np.int32), keys=np.empty((nq, k), np.int64), n_full=np.empty(nq, np.int64))
    lens = np.diff(oi.doc_off)
    for qi in range(nq):
        r = np.sort(pr["cand"][qi, :pr["n_cand"][qi]]).astype(np.int32)
        fh = rabitq_doc_scores(q_k[qi], signs, B, 1, oi.doc_off[r], lens[r].astype(np.int32), codes, g1)

        def full(d, q=q_k[qi]):
            return rabitq_doc_scores(q, signs, B, B, oi.doc_off[d:d + 1], lens[d:d + 1].astype(np.int32), codes,
                                     gB)[0]

        ids, keys, nf = collaborative_scoring(r, fh, full, nc, kfb, chunks, k)
        out["ids"][qi], out["keys"][qi], out["n_full"][qi] = ids, keys, nf
    out["scores"] = keys_to_scores(out["keys"])
    return out


# ------------------------------------------------------- oracle index
class OracleIndex:
    """The oracle's own view of a corpus: assignment given by the corpus,
    quantiser, codes and posting lists computed here from raw grid tokens."""

    def __init__(self, cent_k, doc_off, cid, nbits: int, tok_k=None, hist=None, with_codes=True):
        self.cent_k = _c(cent_k, np.int16)
        self.doc_off = _c(doc_off, np.int64)
        self.cid = _c(cid, np.int32)
        self.nbits = nbits
        self.ncent, self.dim = self.cent_k.shape
        self.ndocs = self.doc_off.shape[0] - 1
        if hist is None:
            hist = residual_hist(tok_k, self.cid, self.cent_k)
        self.hist = hist
        self.cut_k, self.w_k = quantizer(hist, nbits)
        self.codes = encode(tok_k, self.cid, self.cent_k, self.cut_k, nbits) if with_codes else None
        self.ivf_off, self.ivf_doc = ivf_docs(self.cid, self.doc_off, self.ncent)
        self._tok = None

    def token_lists(self):
        """(tok_off, ivf_tok, tok_doc), built on first use (refine 1 only)."""
        if self._tok is None:
            off, tok = ivf_tokens(self.cid, self.ncent)
            self._tok = (off, tok, token_docs(self.doc_off))
        return self._tok

    def _refine_args(self, refine: bool):
        if not refine:
            return 0, None, None, None
        if self.codes is None:
            raise ValueError("refine mode scores retrieved tokens from their codes; build with codes")
        off, tok, tdoc = self.token_lists()
        return 1, off, tok, tdoc

    def search(self, q_k, nprobe: int, ncand: int, k: int, nthreads: int = 0, refine: bool = False):
        """Full path for queries q_k [nq, Tq, dim]; returns a dict of arrays.
        refine: F' from the retrieved tokens' decoded scores instead of the
        probed centroids' (orc_partial_scores_res)."""
        q_k = _c(q_k, np.int16)
        nq, Tq, dim = q_k.shape
        out = dict(
            cent_ids=np.empty((nq, Tq, nprobe), np.int32), cent_keys=np.empty((nq, Tq, nprobe), np.int64),
            n_sq=np.empty(nq, np.int64), cand=np.full((nq, ncand), -1, np.int32),
            cand_keys=np.zeros((nq, ncand), np.int64), n_cand=np.empty(nq, np.int64),
            ids=np.empty((nq, k), np.int32), keys=np.empty((nq, k), np.int64))
        rf, off, tok, tdoc = self._refine_args(refine)
        _load().orc_search(_p(self.cent_k), self.ncent, dim, _p(self.doc_off), self.ndocs, _p(self.cid),
                           _p(self.codes), _p(self.w_k), _p(self.ivf_off), _p(self.ivf_doc), _p(q_k), nq, Tq,
                           nprobe, ncand, k, _p(out["cent_ids"]), _p(out["cent_keys"]), _p(out["n_sq"]),
                           _p(out["cand"]), _p(out["cand_keys"]), _p(out["n_cand"]), _p(out["ids"]),
                           _p(out["keys"]), rf, _p(off), _p(tok), _p(tdoc), nthreads)
        out["scores"] = keys_to_scores(out["keys"])
        return out

    def search_collab(self, q_k, tok_k, nprobe: int, ncand: int, kfb: int, chunks: int, k: int):
        """Steps 1-3 of the search, then Alg. 3 (collaborative_scoring) with
        F^ from the residual codes (doc_scores) and the full-precision score
        the exact Chamfer score of the grid tokens tok_k [ntok, dim]."""
        q_k = _c(q_k, np.int16)
        tok_k = _c(tok_k, np.int16)
        nq = q_k.shape[0]
        nc = min(ncand, self.ndocs)
        pr = self.prune(q_k, nprobe, nc)
        out = dict(ids=np.empty((nq, k), np.int32), keys=np.empty((nq, k), np.int64),
                   n_full=np.empty(nq, np.int64))
        lens = np.diff(self.doc_off)
        for qi in range(nq):
            r = np.sort(pr["cand"][qi, :pr["n_cand"][qi]]).astype(np.int32)
            S = centroid_scores(q_k[qi], self.cent_k)
            fh = doc_scores(S, q_k[qi], self.w_k, self.doc_off[r], lens[r].astype(np.int32), self.cid, self.codes)

            def exact(d, q=q_k[qi]):
                b, e = int(self.doc_off[d]), int(self.doc_off[d + 1])
                return exact_chamfer(q, tok_k[b:e], np.array([0, e - b], np.int64))[0]

            ids, keys, nf = collaborative_scoring(r, fh, exact, nc, kfb, chunks, k)
            out["ids"][qi], out["keys"][qi], out["n_full"][qi] = ids, keys, nf
        out["scores"] = keys_to_scores(out["keys"])
        return out

    def prune(self, q_k, nprobe: int, ncand: int, nthreads: int = 0, refine: bool = False):
        q_k = _c(q_k, np.int16)
        nq, Tq, dim = q_k.shape
        out = dict(
            cent_ids=np.empty((nq, Tq, nprobe), np.int32), cent_keys=np.empty((nq, Tq, nprobe), np.int64),
            n_sq=np.empty(nq, np.int64), cand=np.full((nq, ncand), -1, np.int32),
            cand_keys=np.zeros((nq, ncand), np.int64), n_cand=np.empty(nq, np.int64))
        rf, off, tok, tdoc = self._refine_args(refine)
        _load().orc_prune_batch(_p(self.cent_k), self.ncent, dim, self.ndocs, _p(self.ivf_off), _p(self.ivf_doc),
                                _p(q_k), nq, Tq, nprobe, ncand, _p(out["cent_ids"]), _p(out["cent_keys"]),
                                _p(out["n_sq"]), _p(out["cand"]), _p(out["cand_keys"]), _p(out["n_cand"]),
                                rf, _p(self.w_k) if rf else None, _p(self.codes) if rf else None, _p(off), _p(tok),
                                _p(tdoc), nthreads)
        return out
