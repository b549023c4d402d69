"""GPU path against the CPU oracle, element by element (ids bit-exact,
scores bit-exact: keys are exact on the value grid, so the 1e-3 relative
tolerance is never needed).  Every call goes through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2608_23553_amd import ChimeraError, chimera
from util_gpu import check_search, q_tensor, say, setup

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------- tiny
def test_tiny_full_search_f32():
    w, c, k, cl, oi, idx = setup("tiny")
    q, src = c.queries(w.nq, w.Tq)
    gi, _, _ = check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "f32", "tiny")
    assert np.mean(gi[:, 0] == src) >= 0.9


def test_tiny_stage_taps():
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(w.nq, w.Tq)
    Q = q_tensor(q, "f32")
    say("probe tap tiny")
    ci, ck = idx.probe(Q, w.nprobe)
    say("candidates tap tiny")
    off, docs = idx.candidates(Q, w.nprobe)
    say("prune tap tiny")
    cand, ckeys, nval = idx.prune(Q, w.nprobe, w.ncand)
    torch.cuda.synchronize()
    ci, ck, off, docs = ci.cpu().numpy(), ck.cpu().numpy(), off.cpu().numpy(), docs.cpu().numpy()
    cand, ckeys, nval = cand.cpu().numpy(), ckeys.cpu().numpy(), nval.cpu().numpy()
    ref = oi.search(q, w.nprobe, w.ncand, w.k)
    assert np.array_equal(ci, ref["cent_ids"])
    assert np.array_equal(ck.astype(np.int64), ref["cent_keys"])
    for qi in range(w.nq):
        sq = oracle.candidates(ref["cent_ids"][qi], oi.ivf_off, oi.ivf_doc, w.ndocs)
        assert np.array_equal(docs[off[qi]:off[qi + 1]], sq)
        n = ref["n_cand"][qi]
        assert nval[qi] == n
        order = np.argsort(ref["cand"][qi, :n])
        assert np.array_equal(cand[qi, :n], ref["cand"][qi, :n][order])
        assert np.array_equal(ckeys[qi, :n].astype(np.int64), ref["cand_keys"][qi, :n][order])
        assert np.all(cand[qi, n:] == -1)


@pytest.mark.parametrize("Tq", [1, 7, 31, 33, 64])
def test_tiny_ragged_query_lengths(Tq):
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(5, Tq, query_seed=Tq)
    check_search(idx, oi, q, 3, 100, 10, "bf16", f"tiny Tq={Tq}")


@pytest.mark.parametrize("nprobe,ncand,k", [(1, 1, 1), (64, 1000, 1000), (2, 5000, 200), (8, 300, 300),
                                            (16, 700, 50), (17, 999, 33)])
def test_tiny_knob_extremes(nprobe, ncand, k):
    w, c, k_, cl, oi, idx = setup("tiny")
    q, _ = c.queries(6, 32, query_seed=7)
    gi, gs, ref = check_search(idx, oi, q, nprobe, ncand, k, "bf16", f"tiny np={nprobe} nc={ncand} k={k}")
    if k > ref["n_cand"].min():
        assert (gi == -1).any() and np.isneginf(gs).any()


def test_tiny_off_grid_queries_are_rounded_like_the_oracle():
    w, c, k, cl, oi, idx = setup("tiny")
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 32, 128)).astype(np.float32)
    x /= np.linalg.norm(x, axis=-1, keepdims=True)
    qk = oracle.grid_f32(x)
    say("off-grid f32 queries")
    ids, scores = idx.search(torch.from_numpy(x).cuda(), 4, 256, 10)
    torch.cuda.synchronize()
    ref = oi.search(qk, 4, 256, 10)
    assert np.array_equal(ids.cpu().numpy(), ref["ids"]) and np.array_equal(scores.cpu().numpy(), ref["scores"])


def test_tiny_determinism_and_batch_split_invariance():
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(12, 32, query_seed=11)
    Q = q_tensor(q, "bf16")
    say("determinism tiny")
    a = [t.cpu().numpy() for t in idx.search(Q, 4, 256, 10)]
    b = [t.cpu().numpy() for t in idx.search(Q, 4, 256, 10)]
    parts = [idx.search(Q[i:i + 1], 4, 256, 10) for i in range(12)]
    one = np.concatenate([p[0].cpu().numpy() for p in parts])
    one_s = np.concatenate([p[1].cpu().numpy() for p in parts])
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert np.array_equal(a[0], one) and np.array_equal(a[1], one_s)


def test_tiny_other_stream_and_nq0():
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(3, 32)
    s = torch.cuda.Stream()
    say("side stream")
    with torch.cuda.stream(s):
        ids, scores = idx.search(q_tensor(q, "f32"), 2, 256, 10, stream=s)
    s.synchronize()
    ref = oi.search(q, 2, 256, 10)
    assert np.array_equal(ids.cpu().numpy(), ref["ids"])
    empty = torch.empty((0, 32, 128), device="cuda")
    ids0, sc0 = idx.search(empty, 2, 256, 10)
    assert ids0.shape == (0, 10)


def test_validation_leaves_outputs_untouched():
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(2, 32)
    Q = q_tensor(q, "f32")
    ids = torch.full((2, 10), 7, dtype=torch.int32, device="cuda")
    sc = torch.full((2, 10), 3.0, device="cuda")
    L = chimera.lib()
    h = idx._h
    cases = [  # (args, expected code)
        (dict(d=64), chimera.E_INVAL), (dict(Tq=0), chimera.E_INVAL), (dict(Tq=65), chimera.E_UNSUPPORTED),
        (dict(nprobe=0), chimera.E_INVAL), (dict(nprobe=1025), chimera.E_INVAL),
        (dict(nprobe=65), chimera.E_UNSUPPORTED), (dict(k=0), chimera.E_INVAL), (dict(k=20, ncand=10), chimera.E_INVAL),
        (dict(q_dtype=5), chimera.E_INVAL), (dict(nq=-1), chimera.E_INVAL), (dict(k=9000, ncand=9000), chimera.E_UNSUPPORTED),
        (dict(Tq=64, nprobe=64), chimera.E_UNSUPPORTED),  # beyond the candidate walk's local memory
    ]
    for over, code in cases:
        a = dict(q_dtype=chimera.F32, nq=2, Tq=32, d=128, nprobe=2, ncand=256, k=10)
        a.update(over)
        rc = L.chimera_search(h, Q.data_ptr(), a["q_dtype"], a["nq"], a["Tq"], a["d"], a["nprobe"], a["ncand"],
                              a["k"], ids.data_ptr(), sc.data_ptr(), None)
        assert rc == code, (over, rc, chimera.last_error())
    torch.cuda.synchronize()
    assert torch.all(ids == 7) and torch.all(sc == 3.0)


def test_mfma_exact_on_adversarial_grid_values():
    """Probe keys are the exact integer S for inputs with large L1 norm
    (all components equal magnitude, signs matched to one centroid)."""
    w, c, k, cl, oi, idx = setup("tiny")
    cent = c.centroids_k
    q = np.zeros((1, 32, 128), np.int16)
    rng = np.random.default_rng(5)
    for j in range(32):
        sgn = np.sign(cent[rng.integers(0, w.ncent)]).astype(np.int64)
        sgn[sgn == 0] = 1
        mag = rng.choice([181, 180, 177, 176])  # ~1/sqrt(128) on the grid (bf16-exact values)
        q[0, j] = (sgn * mag).astype(np.int16)
    say("adversarial probe")
    ci, ck = idx.probe(q_tensor(q, "bf16"), 16)
    torch.cuda.synchronize()
    S = oracle.centroid_scores(q[0], cent)
    ids, keys = oracle.probe(S, 16)
    assert np.array_equal(ci.cpu().numpy()[0], ids) and np.array_equal(ck.cpu().numpy()[0].astype(np.int64), keys)


# ------------------------------------------------------------ 4-bit, Tq 64
def test_long_doc_4bit_small():
    w, c, k, cl, oi, idx = setup("2m-long", ndocs=800)
    q, _ = c.queries(6, w.Tq)
    check_search(idx, oi, q, w.nprobe, 2048, 200, "bf16", "2m-long recipe, 800 docs")


# ----------------------------------------------------------------- 100k
def test_100k_full_search():
    w, c, k, cl, oi, idx = setup("100k")
    q, src = c.queries(w.nq, w.Tq)
    gi, _, _ = check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", "100k")
    assert np.mean(gi[:, 0] == src) >= 0.9


@pytest.mark.parametrize("nprobe", [3, 8, 16])
def test_100k_probe_long_lane_streams(nprobe):
    """2048 queries in one probe launch: every lane of the probe sees 2048
    centroid keys, so lists of 4 and 8 pass from the sorting networks to key
    by key insertion part way; sampled rows against the oracle."""
    w, c, k, cl, oi, idx = setup("100k")
    q, _ = c.queries(2048, w.Tq, query_seed=11)
    say("probe 2048 queries", nprobe)
    ci, ck = idx.probe(q_tensor(q, "bf16"), nprobe)
    torch.cuda.synchronize()
    ci, ck = ci.cpu().numpy(), ck.cpu().numpy()
    for qi in (0, 1, 777, 1024, 1500, 2047):
        ids, keys = oracle.probe(oracle.centroid_scores(q[qi], c.centroids_k), nprobe)
        assert np.array_equal(ci[qi], ids), f"q{qi}: centroid ids differ"
        assert np.array_equal(ck[qi].astype(np.int64), keys), f"q{qi}: centroid keys differ"


def test_100k_prune_tap():
    w, c, k, cl, oi, idx = setup("100k")
    q, _ = c.queries(32, w.Tq, query_seed=3)
    say("prune tap 100k")
    cand, ckeys, nval = idx.prune(q_tensor(q, "bf16"), w.nprobe, w.ncand)
    torch.cuda.synchronize()
    ref = oi.prune(q, w.nprobe, w.ncand)
    cand, ckeys, nval = cand.cpu().numpy(), ckeys.cpu().numpy(), nval.cpu().numpy()
    for qi in range(32):
        n = ref["n_cand"][qi]
        assert nval[qi] == n
        order = np.argsort(ref["cand"][qi, :n])
        assert np.array_equal(cand[qi, :n], ref["cand"][qi, :n][order])
        assert np.array_equal(ckeys[qi, :n].astype(np.int64), ref["cand_keys"][qi, :n][order])


# ------------------------------------------- refinement from token scores
# F' from each retrieved token's decoded score (chimera_search_refine /
# chimera_prune_refine with CHIMERA_REFINE_TOKEN) against the oracle's
# orc_partial_scores_res, then the same document scoring and top-k.
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_refine_token_search(dtype):
    w, c, k, cl, oi, idx = setup("tiny")
    q, src = c.queries(w.nq, w.Tq)
    gi, _, _ = check_search(idx, oi, q, w.nprobe, w.ncand, w.k, dtype, "tiny refine", refine=True)
    assert np.mean(gi[:, 0] == src) >= 0.9


def test_tiny_refine_token_prune_tap():
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(w.nq, w.Tq, query_seed=5)
    say("prune tap tiny refine")
    cand, ckeys, nval = idx.prune(q_tensor(q, "bf16"), w.nprobe, w.ncand, refine=chimera.REFINE_TOKEN)
    torch.cuda.synchronize()
    cand, ckeys, nval = cand.cpu().numpy(), ckeys.cpu().numpy(), nval.cpu().numpy()
    ref = oi.prune(q, w.nprobe, w.ncand, refine=True)
    for qi in range(w.nq):
        n = ref["n_cand"][qi]
        assert nval[qi] == n
        order = np.argsort(ref["cand"][qi, :n])
        assert np.array_equal(cand[qi, :n], ref["cand"][qi, :n][order])
        assert np.array_equal(ckeys[qi, :n].astype(np.int64), ref["cand_keys"][qi, :n][order])
        assert np.all(cand[qi, n:] == -1)


@pytest.mark.parametrize("Tq", [1, 7, 33, 64])
def test_tiny_refine_token_ragged_query_lengths(Tq):
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(4, Tq, query_seed=40 + Tq)
    check_search(idx, oi, q, 3, 100, 10, "bf16", f"tiny refine Tq={Tq}", refine=True)


@pytest.mark.parametrize("nprobe,ncand,k", [(1, 1, 1), (64, 1000, 1000), (17, 999, 33)])
def test_tiny_refine_token_knob_extremes(nprobe, ncand, k):
    w, c, k_, cl, oi, idx = setup("tiny")
    q, _ = c.queries(4, 32, query_seed=8)
    check_search(idx, oi, q, nprobe, ncand, k, "bf16", f"tiny refine np={nprobe} nc={ncand} k={k}", refine=True)


def test_refine_token_long_doc_4bit_small():
    w, c, k, cl, oi, idx = setup("2m-long", ndocs=800)
    q, _ = c.queries(4, w.Tq)
    check_search(idx, oi, q, w.nprobe, 2048, 200, "bf16", "2m-long recipe refine, 800 docs", refine=True)


def test_refine_token_rejects_bad_mode_and_oversized_state():
    w, c, k, cl, oi, idx = setup("tiny")
    L = chimera.lib()
    Q = q_tensor(c.queries(2, 64)[0], "bf16")
    ids = torch.empty((2, 10), dtype=torch.int32, device="cuda")
    sc = torch.empty((2, 10), dtype=torch.float32, device="cuda")
    rc = L.chimera_search_refine(idx._h, Q.data_ptr(), chimera.BF16, 2, 64, 128, 2, 256, 10, 7, ids.data_ptr(),
                                 sc.data_ptr(), None)
    assert rc == chimera.E_INVAL
    rc = L.chimera_search_refine(idx._h, Q.data_ptr(), chimera.BF16, 2, 64, 128, 64, 256, 10, chimera.REFINE_TOKEN,
                                 ids.data_ptr(), sc.data_ptr(), None)
    assert rc == chimera.E_UNSUPPORTED


def test_100k_refine_token_search_and_prune_tap():
    w, c, k, cl, oi, idx = setup("100k")
    q, src = c.queries(64, w.Tq, query_seed=21)
    gi, _, _ = check_search(idx, oi, q, w.nprobe, w.ncand, w.k, "bf16", "100k refine", refine=True)
    assert np.mean(gi[:, 0] == src) >= 0.9
    cand, ckeys, nval = idx.prune(q_tensor(q[:16], "bf16"), w.nprobe, w.ncand, refine=chimera.REFINE_TOKEN)
    torch.cuda.synchronize()
    cand, ckeys, nval = cand.cpu().numpy(), ckeys.cpu().numpy(), nval.cpu().numpy()
    ref = oi.prune(q[:16], w.nprobe, w.ncand, refine=True)
    for qi in range(16):
        n = ref["n_cand"][qi]
        assert nval[qi] == n
        order = np.argsort(ref["cand"][qi, :n])
        assert np.array_equal(cand[qi, :n], ref["cand"][qi, :n][order])
        assert np.array_equal(ckeys[qi, :n].astype(np.int64), ref["cand_keys"][qi, :n][order])


@pytest.mark.parametrize("refine", [False, True])
def test_zipf_small_hot_lists(refine):
    """The 1M recipe (Zipf(1.1) centroids) at 3,000 documents: the hot
    centroids' lists hold a large share of every range, so the centroid-only
    walk applies them from the per-document masks and the token refinement
    walks them with whole waves."""
    w, c, k, cl, oi, idx = setup("1m", ndocs=3000)
    q, _ = c.queries(6, w.Tq, query_seed=13)
    check_search(idx, oi, q, w.nprobe, 500, 50, "bf16", f"1m recipe, 3000 docs, refine={refine}", refine=refine)


def test_many_dense_groups_per_rank():
    """64 centroids, each in far more than 1/16 of the documents, so all are
    dense lists: with nprobe 16 a rank's 32 query tokens fall in up to 29
    dense groups (more than 5 is checked here on the host), all applied from
    the documents' masks in one rank step; with nprobe 2 and queries whose
    tokens share centroids, a rank has a few groups of several tokens."""
    w, c, k, cl, oi, idx = setup("tiny", ndocs=2000, ncent=64)
    q, _ = c.queries(6, 32, query_seed=17)
    docs_per_list = np.array([len(np.unique(np.repeat(np.arange(w.ndocs), c.lengths)[cl == e])) for e in range(64)])
    assert np.all(docs_per_list * 16 > w.ndocs)
    most = max(len(np.unique(ids[:, r])) for ids in
               (np.asarray(oracle.probe(oracle.centroid_scores(qq, c.centroids_k), 16)[0]) for qq in q)
               for r in range(16))
    assert most > 5, most
    check_search(idx, oi, q, 16, 400, 20, "bf16", "64 dense centroids, nprobe 16")
    q2 = np.repeat(q[:, :4], 8, axis=1)  # 4 distinct tokens, each 8 times
    check_search(idx, oi, q2, 2, 400, 20, "bf16", "64 dense centroids, nprobe 2, shared tokens")


# ------------------------------------------------------ degenerate queries
def test_binding_checks_out_tensors():
    """Caller-supplied outputs are written by the kernels through bare
    pointers: the binding refuses a wrong shape, dtype, device or layout, and
    a correct pair gives the same answer as the binding's own outputs."""
    w, c, k_, cl, oi, idx = setup("tiny")
    q, _ = c.queries(3, 32)
    Q = q_tensor(q, "bf16")
    nq, k = 3, w.k
    dev = Q.device
    good_i = torch.empty((nq, k), dtype=torch.int32, device=dev)
    good_s = torch.empty((nq, k), dtype=torch.float32, device=dev)
    bad = [(torch.empty((nq, k - 1), dtype=torch.int32, device=dev), good_s),
           (good_i, torch.empty((nq + 1, k), dtype=torch.float32, device=dev)),
           (torch.empty((nq, k), dtype=torch.int64, device=dev), good_s),
           (good_i, torch.empty((nq, k), dtype=torch.bfloat16, device=dev)),
           (torch.empty((nq, k), dtype=torch.int32), good_s),
           (torch.empty((k, nq), dtype=torch.int32, device=dev).t(), good_s)]
    for o in bad:
        with pytest.raises(ValueError):
            idx.search(Q, w.nprobe, w.ncand, k, out=o)
    with pytest.raises(ValueError):
        idx.search(Q.cpu(), w.nprobe, w.ncand, k)
    ri, rs = idx.search(Q, w.nprobe, w.ncand, k)
    idx.search(Q, w.nprobe, w.ncand, k, out=(good_i, good_s))
    torch.cuda.synchronize()
    assert torch.equal(ri, good_i) and torch.equal(rs, good_s)


@pytest.mark.parametrize("refine", [False, True])
def test_tiny_zero_queries_break_every_tie_by_lowest_id(refine):
    """All-zero queries: every centroid and document score is 0, so the
    probe, the refinement select and the top-k are decided by the lowest-id
    rules alone."""
    w, c, k, cl, oi, idx = setup("tiny")
    q = np.zeros((3, 32, 128), np.int16)
    gi, gs, ref = check_search(idx, oi, q, 4, 300, 20, "bf16", f"tiny zero queries refine={refine}", refine=refine)
    assert np.all(gs == 0.0)
    assert np.all(np.diff(gi, axis=1) > 0)  # ascending ids among equal scores


@pytest.mark.parametrize("refine", [False, True])
def test_tiny_repeated_query_token(refine):
    """All 32 tokens of a query equal: at every rank they probe one centroid,
    so the walk shares one list among the whole query."""
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(4, 32, query_seed=17)
    q = np.repeat(q[:, :1, :], 32, axis=1)
    check_search(idx, oi, q, 3, 200, 10, "bf16", f"tiny repeated token refine={refine}", refine=refine)


@pytest.mark.parametrize("refine", [False, True])
def test_tiny_negated_queries(refine):
    """Negated queries (q -> -q): the probe turns to the centroids facing away
    from every source document, so the candidates and answers share nothing
    with the queries' own documents."""
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(4, 32, query_seed=18)
    check_search(idx, oi, (-q.astype(np.int32)).astype(np.int16), 2, 256, 10, "bf16",
                 f"tiny negated refine={refine}", refine=refine)


# ------------------------------------- CPU-GPU collaborative scoring (Alg. 3)
def check_collab(name, idx, oi, k_, qk, nprobe, ncand, kfb, chunks, k, nthreads=0):
    say("collab", name, qk.shape, nprobe, ncand, kfb, chunks, k)
    gi, gs, gn = idx.search_collab(q_tensor(qk, "bf16"), nprobe, ncand, kfb, chunks, k, nthreads=nthreads)
    ref = oi.search_collab(qk, k_, nprobe, ncand, kfb, chunks, k)
    assert np.array_equal(gi, ref["ids"]), f"{name}: ids differ"
    assert np.array_equal(gs, ref["scores"]), f"{name}: scores differ"
    assert np.array_equal(gn, ref["n_full"]), f"{name}: full-precision counts differ"
    return gi, gs, gn


@pytest.mark.parametrize("kfb_mult,chunks", [(1, 1), (2, 3), (4, 4), (3, 64)])
def test_tiny_collab_search(kfb_mult, chunks):
    w, c, k_, cl, oi, idx = setup("tiny")
    idx.attach_fullbit(synth.k_to_bf16_bits(k_))
    q, src = c.queries(8, 32)
    gi, _, gn = check_collab("tiny", idx, oi, k_, q, w.nprobe, w.ncand, kfb_mult * w.k, chunks, w.k)
    assert np.all(gi[:, 0] == src)
    assert np.all(gn >= min(kfb_mult * w.k, w.ncand))


def test_tiny_collab_edges():
    """More chunks than candidates (empty chunks), a budget above ncand, k =
    kfb, one host thread, and a query batch split into sub-batches."""
    w, c, k_, cl, oi, idx = setup("tiny")
    idx.attach_fullbit(synth.k_to_bf16_bits(k_))
    q, _ = c.queries(5, 32)
    check_collab("tiny ncand 5, 8 chunks", idx, oi, k_, q, w.nprobe, 5, 5, 8, 3)
    check_collab("tiny kfb > ncand", idx, oi, k_, q, w.nprobe, 20, 50, 3, 20)
    check_collab("tiny one thread", idx, oi, k_, q, w.nprobe, w.ncand, 30, 4, w.k, nthreads=1)
    check_collab("tiny ragged Tq", idx, oi, k_, q[:, :7], w.nprobe, w.ncand, 30, 4, w.k)


@pytest.mark.parametrize("isa", ["plain", "avx2", "vnni"])
def test_tiny_collab_each_host_instruction_set(isa, monkeypatch):
    """The host half's kernels for each instruction set (capped by
    CHIMERA_COLLAB_ISA; a host without it runs the next one down)."""
    w, c, k_, cl, oi, idx = setup("tiny")
    idx.attach_fullbit(synth.k_to_bf16_bits(k_))
    monkeypatch.setenv("CHIMERA_COLLAB_ISA", isa)
    q, _ = c.queries(6, 32)
    check_collab(f"tiny {isa}", idx, oi, k_, q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    check_collab(f"tiny {isa} Tq 19", idx, oi, k_, q[:, :19], w.nprobe, w.ncand, 3 * w.k, 3, w.k)


def test_collab_long_doc_4bit_64_query_tokens():
    """4-bit codes and 64 query tokens: the two-column-block scorer run chunk
    by chunk, and the host kernels' 64-token query layout."""
    w, c, k_, cl, oi, idx = setup("2m-long", ndocs=800)
    idx.attach_fullbit(synth.k_to_bf16_bits(k_))
    q, src = c.queries(4, w.Tq)
    gi, _, _ = check_collab("2m-long recipe, 800 docs", idx, oi, k_, q, w.nprobe, 512, 300, 4, 200)
    assert np.all(gi[:, 0] == src)


def test_collab_rejects_bad_arguments():
    w, c, k_, cl, oi, idx = setup("tiny")
    q, _ = c.queries(2, 32)
    Q = q_tensor(q, "bf16")
    idx.attach_fullbit(None)
    with pytest.raises(ChimeraError) as e:
        idx.search_collab(Q, w.nprobe, w.ncand, 20, 2, w.k)
    assert e.value.code == chimera.E_INVAL
    with pytest.raises(ChimeraError):
        idx.attach_fullbit(synth.k_to_bf16_bits(k_)[:-1])
    idx.attach_fullbit(synth.k_to_bf16_bits(k_))
    for kfb, chunks, k in [(5, 2, 10), (20, 0, 10), (20, 65, 10)]:
        with pytest.raises(ChimeraError) as e:
            idx.search_collab(Q, w.nprobe, w.ncand, kfb, chunks, k)
        assert e.value.code == chimera.E_INVAL


def test_collab_store_out_of_range_is_refused():
    """A store value that is not finite or lies outside [-1, 1] (the
    builder's rule, which bounds the host's 32-bit dot products) is refused:
    attach names the first such token and keeps the copy it had; a wrong
    width is refused before the library reads the array."""
    w, c, k_, cl, oi, idx = setup("tiny")
    good = synth.k_to_bf16_bits(k_)
    idx.attach_fullbit(good)
    q, _ = c.queries(3, 32)
    before = check_collab("tiny before", idx, oi, k_, q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    for bad in [1.0078125, -2.0, float("inf"), float("nan")]:
        b = good.copy()
        b[[123, 4567], 7] = np.array([bad], np.float32).view(np.uint32)[0] >> 16
        with pytest.raises(ChimeraError) as e:
            idx.attach_fullbit(b)
        assert e.value.code == chimera.E_INVAL and "token 123 " in str(e.value)
    with pytest.raises(ValueError):
        idx.attach_fullbit(good[:, :64])
    after = idx.search_collab(q_tensor(q, "bf16"), w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    for x, y in zip(before, after):
        assert np.array_equal(x, y)


def test_collab_store_attached_in_ranges():
    """The store attached range by range gives the same results as the whole
    array at once; an incomplete store, a range that does not follow on, and
    a range past the end are refused; a bad value names its global token and
    the range can be sent again; t0 = 0 starts over."""
    w, c, k_, cl, oi, idx = setup("tiny")
    good = synth.k_to_bf16_bits(k_)
    q, _ = c.queries(4, 32)
    Q = q_tensor(q, "bf16")
    idx.attach_fullbit(good)
    whole = check_collab("tiny whole store", idx, oi, k_, q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    n = good.shape[0]
    cuts = [0, 1, 700, 700, 5000, n - 3, n]
    idx.attach_fullbit_range(good[:cuts[1]], 0)
    with pytest.raises(ChimeraError) as e:
        idx.search_collab(Q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    assert e.value.code == chimera.E_INVAL and "incomplete" in str(e.value)
    with pytest.raises(ChimeraError) as e:
        idx.attach_fullbit_range(good[5:9], 5)  # does not follow on
    assert e.value.code == chimera.E_INVAL
    for a, b in zip(cuts[1:-1], cuts[2:]):
        if b == cuts[-2]:
            bad = good[a:b].copy()
            bad[17, 3] = np.array([2.0], np.float32).view(np.uint32)[0] >> 16
            with pytest.raises(ChimeraError) as e:
                idx.attach_fullbit_range(bad, a)
            assert e.value.code == chimera.E_INVAL and f"token {a + 17} " in str(e.value)
        idx.attach_fullbit_range(good[a:b], a)
    with pytest.raises(ChimeraError):
        idx.attach_fullbit_range(good[:1], n)  # past the end
    ranged = idx.search_collab(Q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    for x, y in zip(whole, ranged):
        assert np.array_equal(x, y)
    # starting over drops the complete store
    idx.attach_fullbit_range(good[:10], 0)
    with pytest.raises(ChimeraError):
        idx.search_collab(Q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    idx.attach_fullbit_range(good[10:], 10)
    again = idx.search_collab(Q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    for x, y in zip(whole, again):
        assert np.array_equal(x, y)


def test_collab_query_out_of_range_is_refused():
    """A query component outside [-2, 2] (no query token of L2 norm <= 2 has
    one) is refused with the lowest such query named; a component of exactly
    2 is taken and scored exactly; the index keeps working after the error."""
    w, c, k_, cl, oi, idx = setup("tiny")
    idx.attach_fullbit(synth.k_to_bf16_bits(k_))
    q, _ = c.queries(4, 32)
    bad = q.copy()
    bad[1, 5, 7] = 3 * 2048
    bad[3, 0, 0] = -3 * 2048
    with pytest.raises(ChimeraError) as e:
        idx.search_collab(q_tensor(bad, "bf16"), w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    assert e.value.code == chimera.E_INVAL and "query 1 " in str(e.value)
    edge = q.copy()
    edge[2, 3] = 0
    edge[2, 3, 9] = 2 * 2048  # a token of norm exactly 2
    check_collab("tiny component 2", idx, oi, k_, edge, w.nprobe, w.ncand, 3 * w.k, 3, w.k)
    check_collab("tiny after the error", idx, oi, k_, q, w.nprobe, w.ncand, 3 * w.k, 3, w.k)


def test_100k_collab_search(monkeypatch):
    w, c, k_, cl, oi, idx = setup("100k")
    idx.attach_fullbit(synth.k_to_bf16_bits(k_))
    q, src = c.queries(8, 32)
    gi, gs, gn = check_collab("100k", idx, oi, k_, q, w.nprobe, w.ncand, 100, 4, w.k)
    assert np.all(gi[:, 0] == src)
    say("100k collab full-precision scores per query", gn.tolist())
    # a 16 MB scratch budget runs the 8 queries as sub-batches of 4, each
    # writing its own rows of the host outputs
    monkeypatch.setenv("CHIMERA_SCRATCH_MB", "16")
    si, ss, sn = idx.search_collab(q_tensor(q, "bf16"), w.nprobe, w.ncand, 100, 4, w.k)
    assert np.array_equal(si, gi) and np.array_equal(ss, gs) and np.array_equal(sn, gn)
