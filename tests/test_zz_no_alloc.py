"""chimera_search_noalloc (the search whose scratch is the library's fixed
device array) against chimera_search on the same inputs, through the C ABI:
two calls in a row, the second with a smaller batch, ids and scores
bit-exact."""
import numpy as np
import pytest
import torch

from paper_2608_23553_amd import chimera
from util_gpu import q_tensor, say, setup

pytestmark = pytest.mark.gpu


def _noalloc(idx, Q, nprobe, ncand, k):
    nq, Tq, d = Q.shape
    ids = torch.full((nq, k), -7, dtype=torch.int32, device="cuda")
    scores = torch.full((nq, k), 5.0, dtype=torch.float32, device="cuda")
    rc = chimera.lib().chimera_search_noalloc(idx._h, Q.data_ptr(), chimera.BF16, nq, Tq, d, nprobe, ncand, k,
                                              ids.data_ptr(), scores.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert rc == chimera.OK, chimera.last_error()
    return ids, scores


@pytest.mark.parametrize("name,sizes", [("100k", (230, 37)), ("tiny", (16, 3))])
def test_noalloc_equals_search(name, sizes):
    w, c, k, cl, oi, idx = setup(name)
    for call, nq in enumerate(sizes):  # the second call is smaller and reuses the array
        q, _ = c.queries(nq, w.Tq, query_seed=31 + call)
        Q = q_tensor(q, "bf16")
        say("noalloc", name, nq)
        ids, scores = _noalloc(idx, Q, w.nprobe, w.ncand, w.k)
        ref_ids, ref_scores = idx.search(Q, w.nprobe, w.ncand, w.k)
        torch.cuda.synchronize()
        assert torch.equal(ids, ref_ids), f"{name} call {call}: ids differ"
        assert torch.equal(scores, ref_scores), f"{name} call {call}: scores differ"
        # the oracle too, on a few queries
        ref = oi.search(q[:4], w.nprobe, w.ncand, w.k)
        assert np.array_equal(ids[:4].cpu().numpy(), ref["ids"])
        assert np.array_equal(scores[:4].cpu().numpy(), ref["scores"])


def test_noalloc_validation_leaves_outputs_untouched():
    w, c, k, cl, oi, idx = setup("tiny")
    q, _ = c.queries(2, w.Tq)
    Q = q_tensor(q, "bf16")
    ids = torch.full((2, 10), 7, dtype=torch.int32, device="cuda")
    sc = torch.full((2, 10), 3.0, device="cuda")
    L = chimera.lib()
    for nprobe, ncand, kk, code in ((0, 256, 10, chimera.E_INVAL), (2, 5, 10, chimera.E_INVAL),
                                    (65, 256, 10, chimera.E_UNSUPPORTED)):
        rc = L.chimera_search_noalloc(idx._h, Q.data_ptr(), chimera.BF16, 2, w.Tq, 128, nprobe, ncand, kk,
                                      ids.data_ptr(), sc.data_ptr(), None)
        assert rc == code, chimera.last_error()
    torch.cuda.synchronize()
    assert torch.all(ids == 7) and torch.all(sc == 3.0)
