"""Deletions on the GPU (Sec. 3.3, handling updates): a deletion bitmap over
document ids that retrieval skips, and compaction.  Searches after
chimera_index_delete, and again after chimera_index_compact, are compared
element by element with oracle.search_deleted, and the collaborative path
with the oracle's index of the same corpus with the deleted documents
emptied (the equivalence the CPU pins establish)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2608_23553_amd import ChimeraError, chimera
from util_build import product_builder
from util_gpu import q_tensor, say, setup

pytestmark = pytest.mark.gpu


def check_deleted(idx, oi, q, nprobe, ncand, k, deleted, label, refine=False):
    say("search with deletions", label, q.shape, nprobe, ncand, k, "refine" if refine else "")
    ids, scores = idx.search(q_tensor(q, "bf16"), nprobe, ncand, k,
                             refine=chimera.REFINE_TOKEN if refine else chimera.REFINE_CENTROID)
    torch.cuda.synchronize()
    ref = oracle.search_deleted(oi, q, nprobe, ncand, k, deleted, refine=refine)
    gi, gs = ids.cpu().numpy(), scores.cpu().numpy()
    bad = np.nonzero((gi != ref["ids"]).any(axis=1))[0]
    assert bad.size == 0, f"{label}: ids differ for queries {bad[:8]}"
    assert np.array_equal(gs, ref["scores"]), f"{label}: scores differ"
    assert not deleted[gi[gi >= 0]].any()
    return gi, gs


def _emptied_oracle(w, c, k, cl, deleted, hist):
    lens = np.diff(c.doc_off)
    keep_tok = np.repeat(~deleted, lens)
    doc_off = np.concatenate([[0], np.cumsum(np.where(deleted, 0, lens))]).astype(np.int64)
    return oracle.OracleIndex(c.centroids_k, doc_off, cl[keep_tok], w.nbits, tok_k=k[keep_tok], hist=hist), k[keep_tok]


@pytest.mark.parametrize("name,ndocs", [("tiny", None), ("100k", 6000)])
def test_delete_then_compact(name, ndocs):
    w, c, k, cl, oi, _ = setup(name, ndocs)
    idx = product_builder(c, w.nbits).upload(0)  # its own index: this test changes it
    q, src = c.queries(min(w.nq, 16), w.Tq, query_seed=3)
    nprobe, ncand, kk = w.nprobe, min(w.ncand, w.ndocs // 3), min(w.k, 50)
    rng = np.random.default_rng(7)
    pick = rng.choice(w.ndocs, w.ndocs // 5, replace=False)
    ids_del = np.concatenate([pick, src, src[:3]])  # repeats are allowed
    deleted = np.zeros(w.ndocs, bool)
    deleted[ids_del] = True
    before = idx.info()
    say("delete", int(deleted.sum()), "of", w.ndocs)
    idx.delete(ids_del)
    assert idx.info()["ndeleted"] == int(deleted.sum())
    idx.delete(src)  # already deleted: no change
    assert idx.info()["ndeleted"] == int(deleted.sum())
    res = {}
    for refine in (False, True):
        res[refine] = check_deleted(idx, oi, q, nprobe, ncand, kk, deleted, f"{name} deleted", refine)
    # the candidate set tap: S_Q without the deleted documents
    off, docs = idx.candidates(q_tensor(q, "bf16"), nprobe)
    torch.cuda.synchronize()
    off, docs = off.cpu().numpy(), docs.cpu().numpy()
    for qi in range(len(q)):
        ci = oi.search(q[qi:qi + 1], nprobe, ncand, kk)["cent_ids"][0]
        sq = oracle.candidates(ci, oi.ivf_off, oi.ivf_doc, w.ndocs)
        assert np.array_equal(docs[off[qi]:off[qi + 1]], sq[~deleted[sq]])
    # out-of-range ids change nothing
    for bad in ([w.ndocs], [-1], [0, w.ndocs + 5]):
        with pytest.raises(ChimeraError) as e:
            idx.delete(np.array(bad, np.int64))
        assert e.value.code == chimera.E_INVAL
    assert idx.info()["ndeleted"] == int(deleted.sum())
    say("compact")
    idx.compact()
    after = idx.info()
    lens = np.diff(c.doc_off)
    assert after["ntokens"] == before["ntokens"] - int(lens[deleted].sum())
    assert after["nnz"] < before["nnz"] and after["ndocs"] == before["ndocs"]
    assert after["device_bytes"] < before["device_bytes"]
    for refine in (False, True):
        gi, gs = check_deleted(idx, oi, q, nprobe, ncand, kk, deleted, f"{name} compacted", refine)
        assert np.array_equal(gi, res[refine][0]) and np.array_equal(gs, res[refine][1])
    idx.close()


def test_collab_search_with_deletions_and_compaction():
    """The full-precision host store follows the compaction."""
    w, c, k, cl, oi, _ = setup("tiny")
    idx = product_builder(c, w.nbits).upload(0)
    idx.attach_fullbit(synth.k_to_bf16_bits(k))
    q, src = c.queries(6, w.Tq, query_seed=11)
    deleted = np.zeros(w.ndocs, bool)
    deleted[src] = True
    deleted[np.random.default_rng(3).choice(w.ndocs, w.ndocs // 4, replace=False)] = True
    idx.delete(np.nonzero(deleted)[0])
    oe, ke = _emptied_oracle(w, c, k, cl, deleted, oi.hist)
    ref = oe.search_collab(q, ke, w.nprobe, w.ncand, 2 * w.k, 3, w.k)
    for label in ("deleted", "compacted"):
        if label == "compacted":
            idx.compact()
        say("collab", label)
        gi, gs, gn = idx.search_collab(q_tensor(q, "bf16"), w.nprobe, w.ncand, 2 * w.k, 3, w.k)
        assert np.array_equal(gi, ref["ids"]), label
        assert np.array_equal(gs, ref["scores"]), label
        assert np.array_equal(gn, ref["n_full"]), label
    idx.close()
