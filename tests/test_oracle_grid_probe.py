"""Oracle pins: value grid, centroid scores, top-nprobe (Sec. 2.3 IVF probe;
Sec. 3.2 candidate generation)."""
import numpy as np
import pytest
import torch

import oracle
from util_corpus import rand_grid


def test_grid_examples_and_ties():
    q = 1.0 / 2048
    assert oracle.grid_k(0.0) == 0
    assert oracle.grid_k(0.5 * q) == 0 and oracle.grid_k(1.5 * q) == 2 and oracle.grid_k(2.5 * q) == 2
    assert oracle.grid_k(-1.5 * q) == -2
    assert oracle.grid_k(1.0) == 2048 and oracle.grid_k(-1.0) == -2048
    assert oracle.grid_k(0.0625) == 128
    # [2^-3, 2^-2): bf16 spacing 2^-10 -> even multiples of 2^-11 only
    assert oracle.grid_k(0.125 + 1.0 * q) == 256      # tie between 256 and 258 -> 256 (even mantissa)
    assert oracle.grid_k(0.125 + 3.0 * q) == 260      # tie between 258 and 260 -> 260


def test_grid_matches_library_bf16_rounding():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(200_000) * 0.2).astype(np.float32)
    k = oracle.grid_f32(x).astype(np.float64)
    big = np.abs(x) >= 0.0625
    # |x| >= 2^-4: the grid is bf16 round-to-nearest-even (torch's conversion)
    ref_big = torch.from_numpy(x[big]).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(k[big] / 2048.0, ref_big)
    # |x| < 2^-4: nearest multiple of 2^-11, ties to even (numpy's rint)
    ref_small = np.rint(x[~big].astype(np.float64) * 2048.0)
    assert np.array_equal(k[~big], ref_small)
    # idempotent and bf16-representable
    assert np.array_equal(oracle.grid_f32((k / 2048.0).astype(np.float32)), k.astype(np.int16))
    bits = oracle.grid_bf16(torch.from_numpy((k / 2048.0).astype(np.float32)).to(torch.bfloat16)
                            .view(torch.int16).numpy().view(np.uint16))
    assert np.array_equal(bits, k.astype(np.int16))


def test_grid_bf16_rounds_off_grid_values():
    """bf16 inputs below 2^-4 in magnitude lie between grid points: each reads
    as the nearest multiple of 2^-11, ties to even (numpy's rint on the exact
    value); from 2^-4 up every bf16 value is on the grid already."""
    rng = np.random.default_rng(20)
    x = np.concatenate([rng.standard_normal(100_000) * 0.02, rng.standard_normal(20_000) * 0.3,
                        (np.arange(-64, 65) + 0.5) / 2048]).astype(np.float32)
    bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    v = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert np.any(v * 2048 != np.rint(v * 2048))  # off-grid inputs are present
    assert np.array_equal(oracle.grid_bf16(bits).astype(np.float64), np.rint(v * 2048))


def test_centroid_scores_exact_against_fp64_matmul():
    rng = np.random.default_rng(1)
    cent = rand_grid(rng, (300, 128))
    q = rand_grid(rng, (7, 128))
    S = oracle.centroid_scores(q, cent)
    # grid products and their sums are exact in fp64 -> matmul gives the key
    ref = (q.astype(np.float64) / 2048) @ (cent.astype(np.float64) / 2048).T * 2.0 ** 22
    assert np.array_equal(S.astype(np.float64), ref)
    # transposition / sign / index mistakes would break this known case
    assert S[3, 17] == int(np.dot(q[3].astype(np.int64), cent[17].astype(np.int64)))


@pytest.mark.parametrize("nprobe", [1, 2, 5, 16, 300])
def test_probe_matches_lexsort(nprobe):
    rng = np.random.default_rng(2)
    S = rng.integers(-50, 50, size=(9, 300)).astype(np.int64)  # many ties
    ids, keys = oracle.probe(S, nprobe)
    for j in range(S.shape[0]):
        order = np.lexsort((np.arange(300), -S[j]))[:nprobe]
        assert np.array_equal(ids[j], order)
        assert np.array_equal(keys[j], S[j, order])


def test_probe_ties_go_to_lowest_id_and_self_ranks_first():
    rng = np.random.default_rng(3)
    cent = rand_grid(rng, (64, 128))
    cent[40] = cent[7]   # duplicate rows: equal scores everywhere
    cent[50] = cent[7]
    q = cent[[7, 12]].copy()
    S = oracle.centroid_scores(q, cent)
    ids, keys = oracle.probe(S, 4)
    assert list(ids[0][:3]) == [7, 40, 50]        # query == centroid 7: itself first, dups by id
    assert keys[0][0] == keys[0][1] == keys[0][2]
    assert ids[1][0] == 12
