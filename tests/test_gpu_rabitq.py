"""chimera_search_rabitq on the GPU against oracle.search_rabitq, element by
element: steps 1-3 as chimera_search, then document scores from the RaBitQ
1-bit codes (bit-exact keys), on the Tiny, 100k and 2M-long recipes, across
sub-batches, and after deletions and compaction."""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2608_23553_amd import ChimeraError, chimera
from util_build import product_builder
from util_gpu import q_tensor, say, setup

pytestmark = pytest.mark.gpu


def _rq_index(name, ndocs=None, seed=17, with_g4=False):
    w, c, k, cl, oi, _ = setup(name, ndocs)
    signs = synth.rotation_signs(seed)
    idx = product_builder(c, w.nbits, rabitq_signs=signs).upload(0)
    codes, g4, g1 = oracle.rabitq_encode(k, signs, 4)
    if with_g4:
        return w, c, k, oi, idx, signs, codes, g1, g4
    return w, c, k, oi, idx, signs, codes, g1


def check_rq(idx, oi, q, nprobe, ncand, k, signs, codes, g1, label, dtype="bf16"):
    say("rabitq search", label, q.shape, nprobe, ncand, k, dtype)
    ids, scores = idx.search_rabitq(q_tensor(q, dtype), nprobe, ncand, k)
    torch.cuda.synchronize()
    ref = oracle.search_rabitq(oi, q, nprobe, ncand, k, signs, 4, codes, g1)
    gi, gs = ids.cpu().numpy(), scores.cpu().numpy()
    bad = np.nonzero((gi != ref["ids"]).any(axis=1))[0]
    assert bad.size == 0, f"{label}: ids differ for queries {bad[:8]}: gpu {gi[bad[0]][:6]} oracle {ref['ids'][bad[0]][:6]}"
    assert np.array_equal(gs, ref["scores"]), f"{label}: scores differ"
    return gi, gs


@pytest.mark.parametrize("name,ndocs,nq", [("tiny", None, 16), ("100k", 6000, 12)])
def test_rabitq_search_matches_the_oracle(name, ndocs, nq):
    w, c, k, oi, idx, signs, codes, g1 = _rq_index(name, ndocs)
    q, src = c.queries(nq, w.Tq, query_seed=8)
    nc, kk = min(w.ncand, w.ndocs // 3), min(w.k, 50)
    gi, _ = check_rq(idx, oi, q, w.nprobe, nc, kk, signs, codes, g1, name)
    check_rq(idx, oi, q[:3], w.nprobe, nc, kk, signs, codes, g1, name + " f32", "f32")
    # the 1-bit scores still find the query's source document
    assert np.mean(gi[:, 0] == src) >= 0.5
    idx.close()


def test_rabitq_search_tq64_long_documents():
    """The 2M-long recipe (64 query tokens: two row blocks, documents of 128
    to 512 tokens) on its first 500 documents."""
    w, c, k, oi, idx, signs, codes, g1 = _rq_index("2m-long", 500)
    q, _ = c.queries(3, w.Tq, query_seed=4)
    check_rq(idx, oi, q, w.nprobe, 200, 50, signs, codes, g1, "2m-long 500 docs")
    idx.close()


def test_rabitq_search_in_sub_batches_and_after_compaction():
    w, c, k, oi, idx, signs, codes, g1 = _rq_index("100k", 6000, seed=23)
    q, src = c.queries(40, w.Tq, query_seed=12)
    nc, kk = 800, 20
    old = os.environ.get("CHIMERA_SCRATCH_MB")
    os.environ["CHIMERA_SCRATCH_MB"] = "16"
    try:
        check_rq(idx, oi, q, w.nprobe, nc, kk, signs, codes, g1, "16 MB scratch")
    finally:
        if old is None:
            os.environ.pop("CHIMERA_SCRATCH_MB")
        else:
            os.environ["CHIMERA_SCRATCH_MB"] = old
    deleted = np.zeros(w.ndocs, bool)
    deleted[src] = True
    deleted[np.random.default_rng(5).choice(w.ndocs, 900, replace=False)] = True
    idx.delete(np.nonzero(deleted)[0])
    lens = np.diff(c.doc_off)
    keep_tok = np.repeat(~deleted, lens)
    doc_off = np.concatenate([[0], np.cumsum(np.where(deleted, 0, lens))]).astype(np.int64)
    oe = oracle.OracleIndex(c.centroids_k, doc_off, oi.cid[keep_tok], w.nbits, tok_k=k[keep_tok], hist=oi.hist)
    for label in ("deleted", "compacted"):
        if label == "compacted":
            idx.compact()
        gi, _ = check_rq(idx, oe, q, w.nprobe, nc, kk, signs, codes[keep_tok], g1[keep_tok], label)
        assert not deleted[gi[gi >= 0]].any()
    idx.close()


def test_rabitq_search_needs_rabitq_codes():
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(2, w.Tq)
    with pytest.raises(ChimeraError) as e:
        idx.search_rabitq(q_tensor(q, "bf16"), w.nprobe, w.ncand, w.k)
    assert e.value.code == chimera.E_UNSUPPORTED


@pytest.mark.parametrize("kfb_mult,chunks,isa", [(2, 1, None), (3, 4, None), (3, 4, "avx2"), (2, 3, "plain")])
def test_rabitq_collab_search(kfb_mult, chunks, isa, monkeypatch):
    """Alg. 3 with the code split: GPU 1-bit scores chunk by chunk, host
    scores from the 4-bit codes, with each host instruction set's dot
    products (capped by CHIMERA_COLLAB_ISA)."""
    if isa:
        monkeypatch.setenv("CHIMERA_COLLAB_ISA", isa)
    w, c, k, oi, idx, signs, codes, g1, g4 = _rq_index("tiny", with_g4=True)
    q, src = c.queries(8, w.Tq, query_seed=21)
    say("rabitq collab", kfb_mult, chunks)
    gi, gs, gn = idx.search_collab_rabitq(q_tensor(q, "bf16"), w.nprobe, w.ncand, kfb_mult * w.k, chunks, w.k)
    ref = oracle.search_collab_rabitq(oi, q, w.nprobe, w.ncand, kfb_mult * w.k, chunks, w.k, signs, 4, codes, g1, g4)
    assert np.array_equal(gi, ref["ids"])
    assert np.array_equal(gs, ref["scores"])
    assert np.array_equal(gn, ref["n_full"])
    assert np.mean(gi[:, 0] == src) >= 0.8
    idx.close()
