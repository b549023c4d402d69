"""Pins of the oracle's RaBitQ codes (Sec. 2.2, Eqs. 2-6 with B bits; Sec.
3.1, the 1-bit most significant part; Sec. 4.1, the LUT binary inner
product), each against something other than the oracle itself: scipy's
Hadamard matrix, brute force over every codeword on small dimensions, the
paper's equations evaluated literally in float64, a direct dot product, and
the exact Chamfer score that fine codes must approach."""
import itertools
from fractions import Fraction

import numpy as np
import pytest
import scipy.linalg

import oracle
from util_corpus import corpus, rand_grid


def _signs(rng, D):
    return np.where(rng.random(D) < 0.5, -1, 1).astype(np.int8)


@pytest.mark.parametrize("D", [4, 16, 128])
def test_rotation_is_hadamard_times_signs(D):
    rng = np.random.default_rng(D)
    s = _signs(rng, D)
    x = rng.integers(-2048, 2048, (5, D)).astype(np.int16)
    H = scipy.linalg.hadamard(D).astype(np.int64)
    want = (H @ np.diag(s.astype(np.int64)) @ x.astype(np.int64).T).T
    got = oracle.rabitq_rotate(x, s)
    assert np.array_equal(got, want)
    # orthogonal up to the factor sqrt(D): <Pa, Pb> = D <a, b>
    a, b = x[0].astype(np.int64), x[1].astype(np.int64)
    assert int(got[0] @ got[1]) == D * int(a @ b)


def _brute(xp, B):
    """Every codeword: the code of largest <xp, y>/|y|, ties to smallest |y|,
    then to the larger code (a zero coordinate takes y = +1/2)."""
    D = len(xp)
    half = (1 << B) - 1
    best = None
    for code in itertools.product(range(1 << B), repeat=D):
        z = [2 * c - half for c in code]  # 2y
        A = sum(int(a) * b for a, b in zip(xp, z))
        if A <= 0:
            continue
        N = sum(b * b for b in z)
        key = (Fraction(A * A, N), -N, code)
        if best is None or key > best[0]:
            best = (key, code, A)
    return np.array(best[1], np.uint8), best[2]


@pytest.mark.parametrize("D,B", [(4, 1), (4, 2), (4, 3), (4, 4), (8, 1), (8, 2), (16, 1)])
def test_quantizer_is_the_nearest_codeword(D, B):
    rng = np.random.default_rng(100 * D + B)
    rows = [rng.integers(-40, 41, D) for _ in range(6)]
    rows.append(np.array([3, -3, 3, 0] * (D // 4)))          # equal magnitudes and zeros
    rows.append(np.array([5, 10, -15, 20] * (D // 4)))       # commensurate steps
    rows.append(np.array([1] + [0] * (D - 1)))
    if D * B > 12:  # keep brute force to 4096 codewords for the larger cases
        rows = rows[:3] + rows[6:]
    for xp in rows:
        if D * B > 16:
            continue
        codes, az = oracle.rabitq_quantize(np.array(xp, np.int64)[None, :], B)
        want, A = _brute(xp, B)
        assert np.array_equal(codes[0], want), (xp, codes[0], want)
        assert az[0] == A


def test_msb_is_the_sign_of_the_rotated_token():
    rng = np.random.default_rng(9)
    s = _signs(rng, 128)
    x = rand_grid(rng, (50, 128))
    for B in (2, 4):
        codes, _, _ = oracle.rabitq_encode(x, s, B)
        xp = oracle.rabitq_rotate(x, s)
        assert np.array_equal(codes >> (B - 1) == 1, xp >= 0)


def _literal_estimate(q_k, o_k, s, code, B, bits):
    """<q_r, o_r> estimated by Eqs. 2-6 in float64, with P = H diag(s)/sqrt(D)."""
    D = len(o_k)
    P = scipy.linalg.hadamard(D) @ np.diag(s.astype(np.float64)) / np.sqrt(D)
    q_r, o_r = q_k / 2048.0, o_k / 2048.0
    q, o = q_r / np.linalg.norm(q_r), o_r / np.linalg.norm(o_r)          # Eq. 2
    q_p, o_p = P @ q, P @ o
    if bits == 1:
        ob, Bb = (code >> (B - 1)).astype(np.float64), 1
    else:
        ob, Bb = code.astype(np.float64), B
    y = ob - (2 ** Bb - 1) / 2                                          # y = o_b - (2^B-1)/2
    obar = y / np.linalg.norm(y)                                        # Eq. 4's codeword
    ip_eq6 = (q_p @ ob - (2 ** Bb - 1) / 2 * q_p.sum()) / np.linalg.norm(y)   # Eq. 6
    assert abs(ip_eq6 - q_p @ obar) < 1e-12
    return np.linalg.norm(q_r) * np.linalg.norm(o_r) * ip_eq6 / (o_p @ obar)  # Eqs. 3 and 5


@pytest.mark.parametrize("B,bits", [(4, 4), (4, 1), (2, 2), (2, 1)])
def test_estimate_follows_equations_2_to_6(B, bits):
    rng = np.random.default_rng(B * 10 + bits)
    s = _signs(rng, 128)
    o = rand_grid(rng, (20, 128))
    q = rand_grid(rng, (20, 128))
    codes, gB, g1 = oracle.rabitq_encode(o, s, B)
    g = g1 if bits == 1 else gB
    for t in range(20):
        f = oracle.rabitq_doc_scores(q[t:t + 1], s, B, bits, np.array([t]), np.array([1], np.int32), codes, g)[0]
        lit = _literal_estimate(q[t].astype(np.float64), o[t].astype(np.float64), s, codes[t], B, bits)
        assert abs(f * 2.0 ** -22 - lit) <= 2.0 ** -22 + 2e-6 * abs(lit), (t, f * 2.0 ** -22, lit)


def test_lut_inner_product_is_the_binary_dot_product():
    rng = np.random.default_rng(4)
    for _ in range(20):
        xq = rng.integers(-30000, 30000, 128).astype(np.int64)
        code = rng.integers(0, 16, (1, 128)).astype(np.uint8)
        bits = oracle.rabitq_pack1(code, 4)[0]
        b = (code[0] >> 3).astype(np.int64)
        assert oracle.lut_ip(xq, bits) == int(xq @ b)
        # the packing: bit i of the token in byte i / 8, bit i % 8
        assert np.array_equal(np.unpackbits(bits, bitorder="little"), b.astype(np.uint8))


def test_fine_codes_approach_the_exact_chamfer_score():
    """With B = 8 the estimate is within ~1e-3 of every inner product, so
    the document scores approach the exact Chamfer scores; 1-bit scores are
    far coarser but still track them."""
    w, c, k, cl = corpus("tiny")
    rng = np.random.default_rng(2)
    s = _signs(rng, 128)
    q, _ = c.queries(4, w.Tq)
    lens = np.diff(c.doc_off)
    docs = np.arange(40)
    for B, bits, tol in ((8, 8, 0.01), (4, 4, 0.06), (4, 1, 0.5)):
        codes, gB, g1 = oracle.rabitq_encode(k, s, B)
        g = g1 if bits == 1 else gB
        errs = []
        for qi in range(len(q)):
            f = oracle.rabitq_doc_scores(q[qi], s, B, bits, c.doc_off[docs], lens[docs].astype(np.int32), codes, g)
            ex = oracle.exact_chamfer(q[qi], k, c.doc_off)[docs]
            errs.append(np.abs(f - ex) * 2.0 ** -22 / w.Tq)
        assert np.mean(errs) < tol, (B, bits, np.mean(errs))


def test_collab_with_full_budget_is_the_top_k_of_4bit_scores():
    """kfb = ncand with one chunk scores every kept document from its 4-bit
    codes, so Alg. 3 returns the top-k of those scores; the 1-bit scores only
    order the work."""
    w, c, k, cl = corpus("tiny")
    from util_corpus import oracle_index
    oi = oracle_index("tiny")
    s = _signs(np.random.default_rng(6), 128)
    codes, g4, g1 = oracle.rabitq_encode(k, s, 4)
    q, _ = c.queries(4, w.Tq)
    nc = 40
    out = oracle.search_collab_rabitq(oi, q, w.nprobe, nc, nc, 1, w.k, s, 4, codes, g1, g4)
    pr = oi.prune(q, w.nprobe, nc)
    lens = np.diff(c.doc_off)
    for qi in range(len(q)):
        r = np.sort(pr["cand"][qi, :pr["n_cand"][qi]]).astype(np.int32)
        f4 = oracle.rabitq_doc_scores(q[qi], s, 4, 4, c.doc_off[r], lens[r].astype(np.int32), codes, g4)
        ids, keys = oracle.topk(r, f4, w.k)
        assert np.array_equal(out["ids"][qi, :len(ids)], ids) and np.array_equal(out["keys"][qi, :len(ids)], keys)
        assert out["n_full"][qi] == len(r)
