"""The generator's cluster labels are the IVF assignment (Sec. 2.3: each
token is assigned to the centroid of largest inner product, ties to the
lower id) on samples of over a million tokens of each large workload.

The check is independent of both the generator and the oracle: an fp32 GEMM
in torch on the CPU, exact here because every operand is a multiple of 2^-11
and every partial sum of t . c is bounded by |t| |c| < 4 (Cauchy-Schwarz on
any subset of the coordinates), so each one is a multiple of 2^-22 that fp32
holds exactly, in any summation order.  The oracle's own assignment is then
compared with it on a subsample."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.slow

CHUNK = 1024  # tokens per GEMM


def _sample(w, want_tokens: int, seed: int):
    """Random documents of the workload (seeded, without replacement) until
    want_tokens tokens: their grid integers and generator labels."""
    c = synth.Corpus(w.corpus_spec())
    rng = np.random.default_rng(seed)
    order = rng.permutation(w.ndocs)
    lens = c.lengths.astype(np.int64)
    need = int(np.searchsorted(np.cumsum(lens[order]), want_tokens)) + 1
    docs = np.sort(order[:need])
    k, cl, _ = c.docs_tokens(docs)
    return c, k, cl


def _largest_ip(k: np.ndarray, cent_k: np.ndarray, lab: np.ndarray):
    """Asserts, per token, that lab is the first index of the largest t . c."""
    tk2 = int((k.astype(np.int64) ** 2).sum(axis=1).max())
    ck2 = int((cent_k.astype(np.int64) ** 2).sum(axis=1).max())
    # |t| |c| < 4 in grid units: tk2 * ck2 < (4 * 2048^2)^2
    assert tk2 * ck2 < (4 * 2048**2) ** 2
    torch.set_float32_matmul_precision("highest")
    C = torch.from_numpy(cent_k.astype(np.float32) / 2048.0)
    S = torch.empty((CHUNK, C.shape[0]), dtype=torch.float32)
    ties = 0
    for t0 in range(0, len(k), CHUNK):
        n = min(CHUNK, len(k) - t0)
        T = torch.from_numpy(k[t0:t0 + n].astype(np.float32) / 2048.0)
        s = S[:n]
        torch.matmul(T, C.T, out=s)
        rows = torch.arange(n)
        lt = torch.from_numpy(lab[t0:t0 + n].astype(np.int64))
        top = s.amax(dim=1)
        own = s[rows, lt].clone()
        bad = torch.nonzero(own != top).flatten()
        assert len(bad) == 0, f"token {t0 + int(bad[0])}: label {int(lt[bad[0]])} is not the largest inner product"
        s[rows, lt] = -torch.inf
        second = s.amax(dim=1)
        for r in torch.nonzero(second == top).flatten().tolist():  # exact ties: the label must be the lowest id
            ties += 1
            others = torch.nonzero(s[r] == top[r]).flatten()
            assert int(others.min()) > int(lt[r]), f"token {t0 + r}: a lower centroid id ties with the label"
    return ties


@pytest.mark.parametrize("name,seed", [("1m", 31), ("8.8m", 32), ("2m-long", 33)])
def test_labels_are_the_largest_inner_product_on_a_million_tokens(name, seed):
    w = synth.WORKLOADS[name]
    c, k, cl = _sample(w, 1_000_000, seed)
    assert len(k) >= 1_000_000
    _largest_ip(k, c.centroids_k, cl)
    # the oracle's assignment agrees on a subsample (its cost is ntok * ncent)
    rng = np.random.default_rng(seed + 100)
    sub = rng.choice(len(k), 2_000_000_000 // (w.ncent * 128) + 1, replace=False)
    assert np.array_equal(oracle.assign(k[sub], c.centroids_k), cl[sub])
