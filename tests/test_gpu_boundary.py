"""The C ABI's edges on the GPU, each against the oracle: an index written to
a file and loaded back, the largest k, the bound on query norms for exact
scores and its on-request check, all-zero queries (massive ties in every
top-k), searches split into several sub-batches, and the knobs of the 8.8M
and 2M-long workloads on reduced document counts."""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2608_23553_amd import ChimeraError, Index, chimera
from util_build import product_builder
from util_gpu import check_search, q_tensor, say, setup

pytestmark = pytest.mark.gpu


class env:
    """Sets environment variables for the duration of a with-block."""

    def __init__(self, **kv):
        self.kv, self.old = kv, {}

    def __enter__(self):
        for k, v in self.kv.items():
            self.old[k] = os.environ.get(k)
            os.environ[k] = v

    def __exit__(self, *a):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


@pytest.mark.parametrize("name,ndocs", [("tiny", None), ("2m-long", 600)])
def test_index_file_roundtrip_search(name, ndocs, tmp_path):
    """chimera_builder_save -> chimera_index_load -> search, against the oracle."""
    w, c, k, cl, oi, idx = setup(name, ndocs)
    b = product_builder(c, w.nbits)
    path = str(tmp_path / "index.chim")
    b.save(path)
    say("load", path, os.path.getsize(path), "bytes")
    loaded = Index.load(path, 0)
    a, l = idx.info(), loaded.info()
    for key in ("ndocs", "ntokens", "nnz", "ncent", "dim", "nbits", "max_doc_len", "device_bytes", "q_norm_limit"):
        assert a[key] == l[key], key
    q, _ = c.queries(6, w.Tq, query_seed=4)
    check_search(loaded, oi, q, w.nprobe, min(w.ncand, w.ndocs // 2), min(w.k, 100), "bf16", f"{name} loaded")
    loaded.close()


@pytest.mark.parametrize("name,ndocs,nq", [("tiny", None, 3), ("100k", 12_000, 2)])
def test_largest_k(name, ndocs, nq):
    """k = CHIMERA_MAX_K = 8192: the final top-k with 64 KiB of dynamic LDS
    (on tiny most of the rows are padding)."""
    w, c, k, cl, oi, idx = setup(name, ndocs)
    q, _ = c.queries(nq, w.Tq, query_seed=9)
    check_search(idx, oi, q, 8, 8192, 8192, "bf16", f"{name} k=8192")


def _norm(qk):
    return np.sqrt((qk.astype(np.float64) ** 2).sum(axis=-1)) / 2048.0


def test_query_norm_limit_matches_its_definition():
    """q_norm_limit = 4 / (max_c ||c|| + sqrt(dim) * max_u |w_u|), computed
    here from the index's own sections."""
    w, c, k, cl, oi, idx = setup("tiny")
    cmax = np.sqrt((c.centroids_k.astype(np.int64) ** 2).sum(axis=1).max()) / 2048.0
    wmax = np.abs(oi.w_k).max() / 2048.0
    lim = idx.info()["q_norm_limit"]
    assert abs(lim - 4.0 / (cmax + np.sqrt(128) * wmax)) < 1e-6 * lim
    assert lim > 2.0  # unit queries are well inside it


def _scaled_query(c, w, factor):
    """A tiny query whose token 0 is scaled by factor (then rounded onto the grid)."""
    q, _ = c.queries(2, w.Tq, query_seed=17)
    x = q.astype(np.float64) / 2048.0
    x[0, 0] *= factor
    return oracle.grid_f32(x.astype(np.float32))


def test_query_at_the_norm_limit_is_exact_and_beyond_it_is_refused():
    w, c, k, cl, oi, idx0 = setup("tiny")
    with env(CHIMERA_CHECK_QUERIES="1"):
        idx = product_builder(c, w.nbits).upload(0)
    lim = idx.info()["q_norm_limit"]
    q1 = c.queries(2, w.Tq, query_seed=17)[0]
    base = _norm(q1)[0, 0]
    below = _scaled_query(c, w, lim / base * (1 - 2e-3))
    assert _norm(below)[0, 0] < lim
    say("query token of norm", _norm(below)[0, 0], "limit", lim)
    # just below the limit: scores exact, so equal to the oracle's
    check_search(idx, oi, below, w.nprobe, w.ncand, w.k, "bf16", "tiny at the norm limit")
    check_search(idx, oi, below, w.nprobe, w.ncand, w.k, "f32", "tiny at the norm limit (f32)")
    above = _scaled_query(c, w, lim / base * (1 + 2e-3))
    assert _norm(above)[0, 0] >= lim
    for bad, label in ((above, "above the limit"), (None, "NaN")):
        if bad is None:
            Q = torch.from_numpy(q1.astype(np.float32) / 2048.0).cuda()
            Q[1, 5, 3] = float("nan")
        else:
            Q = q_tensor(bad, "f32")
        ids = torch.full((2, w.k), 7, dtype=torch.int32, device="cuda")
        sc = torch.full((2, w.k), 3.0, device="cuda")
        say("refused query:", label)
        with pytest.raises(ChimeraError) as e:
            idx.search(Q, w.nprobe, w.ncand, w.k, out=(ids, sc))
        assert e.value.code == chimera.E_INVAL
        assert ("query 0 token 0" if bad is not None else "query 1 token 5") in str(e.value)
        for tap in (lambda: idx.probe(Q, w.nprobe), lambda: idx.prune(Q, w.nprobe, w.ncand)):
            with pytest.raises(ChimeraError):
                tap()
        torch.cuda.synchronize()
        assert torch.all(ids == 7) and torch.all(sc == 3.0)
    # without the check the same index serves ordinary queries as before
    q, _ = c.queries(4, w.Tq)
    check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", "tiny, check on")
    idx.close()


@pytest.mark.parametrize("nq", [1, 5])
def test_all_zero_queries(nq):
    """Every centroid scores 0: the probe keeps the lowest ids, every
    candidate has F' = 0, and the refinement keeps the lowest document ids
    (at 100k with fewer than 128 queries the select is split over chunks and
    its per-chunk lists overflow, so it falls back to re-reading F')."""
    w, c, k, cl, oi, idx = setup("100k")
    q = np.zeros((nq, w.Tq, 128), np.int16)
    check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", f"100k all-zero nq={nq}")
    cand, ckeys, nval = idx.prune(q_tensor(q, "bf16"), w.nprobe, w.ncand)
    torch.cuda.synchronize()
    ref = oi.prune(q, w.nprobe, w.ncand)
    for qi in range(nq):
        n = ref["n_cand"][qi]
        assert nval[qi].item() == n
        assert np.array_equal(cand[qi, :n].cpu().numpy(), np.sort(ref["cand"][qi, :n]))


def test_search_split_into_sub_batches():
    """A 32 MB scratch budget splits a 100k search of 48 queries into about
    four sub-batches (each query needs ~2.5 MB: its S^T table and F'); the
    result is the oracle's and the one-pass result."""
    w, c, k, cl, oi, idx = setup("100k")
    q, _ = c.queries(48, w.Tq, query_seed=23)
    one = [t.cpu().numpy() for t in idx.search(q_tensor(q, "bf16"), w.nprobe, w.ncand, w.k)]
    with env(CHIMERA_SCRATCH_MB="32"):
        gi, gs, _ = check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", "100k, 32 MB scratch")
    assert np.array_equal(gi, one[0]) and np.array_equal(gs, one[1])


def test_sub_batches_shrink_when_the_arena_does_not_fit():
    """A device that cannot hold the arena (forced from the host: an arena
    above CHIMERA_SCRATCH_DEVICE_MB is refused as out of memory) halves the
    sub-batches until it fits, with the one-pass result; a single query that
    does not fit is E_NOMEM, and the index works again afterwards."""
    w, c, k, cl, oi, cached = setup("100k")
    q, _ = c.queries(48, w.Tq, query_seed=29)
    Q = q_tensor(q, "bf16")
    one = [t.cpu().numpy() for t in cached.search(Q, w.nprobe, w.ncand, w.k)]
    idx = product_builder(c, w.nbits).upload(0)  # a fresh index: no arena yet
    try:
        with env(CHIMERA_SCRATCH_DEVICE_MB="1"):  # less than one query's ~2.5 MB
            with pytest.raises(ChimeraError) as e:
                idx.search(Q, w.nprobe, w.ncand, w.k)
            assert e.value.code == chimera.E_NOMEM
        with env(CHIMERA_SCRATCH_DEVICE_MB="8"):  # 48 -> 24 -> 12 -> 6 -> 3 -> 2 queries per pass
            gi, gs, _ = check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", "100k, 8 MB device cap")
        assert np.array_equal(gi, one[0]) and np.array_equal(gs, one[1])
        ids, scores = idx.search(Q, w.nprobe, w.ncand, w.k)  # no cap: one pass
        assert np.array_equal(ids.cpu().numpy(), one[0]) and np.array_equal(scores.cpu().numpy(), one[1])
    finally:
        idx.close()


def test_batch_too_large_for_one_scorer_launch():
    """5,400 queries with every one of 100,000 documents kept would need more
    than 2^32 work-items in one scorer launch; the batch runs in sub-batches
    of at most 2^28 (query, candidate) pairs, with each query's result that
    of a search on its own (and the oracle's)."""
    w, c, k, cl, oi, idx = setup("100k")
    nq, ncand = 5400, w.ndocs
    q, _ = c.queries(nq, w.Tq, query_seed=31)
    ids, scores = idx.search(q_tensor(q, "bf16"), w.nprobe, ncand, w.k)
    ids, scores = ids.cpu().numpy(), scores.cpu().numpy()
    sample = [0, 1799, 1800, 3599, 3600, 5399]  # ends of the 3 equal sub-batches
    si, ss = idx.search(q_tensor(q[sample], "bf16"), w.nprobe, ncand, w.k)
    assert np.array_equal(ids[sample], si.cpu().numpy()) and np.array_equal(scores[sample], ss.cpu().numpy())
    ref = oi.search(q[-1:], w.nprobe, ncand, w.k)
    assert np.array_equal(ids[-1:], ref["ids"]) and np.array_equal(scores[-1:], ref["scores"])


def test_8_8m_knobs_on_60k_docs():
    """The 8.8M workload's recipe and knobs (262,144 Zipf(1.1) centroids,
    nprobe 16, ncand 16,384, k 100) on its first 60,000 documents."""
    w, c, k, cl, oi, idx = setup("8.8m", 60_000)
    q, _ = c.queries(6, w.Tq, query_seed=2)
    check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", "8.8m recipe, 60k docs")


def test_2m_long_knobs_on_40k_docs():
    """The 2M-long workload's knobs (4-bit codes, 64 query tokens, nprobe 32,
    ncand 32,768, k 1,000) on its first 40,000 documents."""
    w, c, k, cl, oi, idx = setup("2m-long", 40_000)
    q, _ = c.queries(3, w.Tq, query_seed=2)
    check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", "2m-long recipe, 40k docs")
