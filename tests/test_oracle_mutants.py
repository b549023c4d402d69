"""Planted mistakes in the oracle, on the CPU: each mutant replaces one oracle
function by a wrapper around it that makes a plausible mistake (a tie broken
the wrong way, a dropped term, a flipped sign, a shifted index, a transposed
operand), and at least one of the named pins must then fail.  This checks
that the pins bind the oracle, not only that the oracle passes them.

The wrappers change what the real function receives or returns; none
re-implements the method, and every input they pass stays within the
arrays the oracle reads.  Cached corpora and oracle indexes are built
before any mutant is active, so no mutant leaks into another test."""
import math

import numpy as np
import pytest

import oracle
import test_oracle_collab as PC
import test_oracle_grid_probe as PG
import test_oracle_prune as PP
import test_oracle_quant_score as PQ
import test_oracle_refine as PR
from util_corpus import corpus, oracle_index

REAL = {name: getattr(oracle, name) for name in (
    "grid_k", "grid_f32", "centroid_scores", "probe", "candidates", "partial_scores", "topk", "encode",
    "quantizer", "pack", "doc_scores", "exact_chamfer", "key_to_score", "collaborative_scoring", "ivf_docs",
    "partial_scores_res", "ivf_tokens", "token_docs", "grid_bf16", "assign", "residual_hist", "unpack")}


# ----------------------------------------------------------------- grid
def grid_k_ties_away(x):
    """Halfway cases rounded away from zero instead of to even."""
    if abs(x) >= 0.0625:
        return REAL["grid_k"](x)
    return int(math.copysign(math.floor(abs(x) * 2048 + 0.5), x))


def grid_k_truncates(x):
    return int(x * 2048)


def grid_f32_no_bf16(x):
    """Every value rounded to a multiple of 2^-11, never to bf16 first."""
    return np.rint(np.asarray(x, np.float64) * 2048).astype(np.int16)


# ---------------------------------------------------- centroid scores, probe
def cs_negated(q, c):
    return -REAL["centroid_scores"](q, c)


def cs_drops_last_dim(q, c):
    return REAL["centroid_scores"](np.ascontiguousarray(q[..., :-1]), np.ascontiguousarray(c[:, :-1]))


def cs_shifted_centroid(q, c):
    return np.roll(REAL["centroid_scores"](q, c), 1, axis=1)


def probe_ties_highest_id(S, nprobe):
    ncent = S.shape[1]
    ids, keys = REAL["probe"](np.ascontiguousarray(S[:, ::-1]), nprobe)
    return (ncent - 1 - ids).astype(np.int32), keys


def probe_lowest_scores(S, nprobe):
    ids, keys = REAL["probe"](-np.asarray(S), nprobe)
    return ids, -keys


# --------------------------------------------------- candidates, F', top-k
def cand_drops_last_probe(cent_ids, ivf_off, ivf_doc, ndocs):
    ci = np.ascontiguousarray(cent_ids[:, :-1]) if cent_ids.shape[1] > 1 else cent_ids
    return REAL["candidates"](ci, ivf_off, ivf_doc, ndocs)


def fp_init_zero(S, cent_ids, ivf_off, ivf_doc, ndocs):
    """The per-token maximum starts at 0, so a negative maximum is lost."""
    return REAL["partial_scores"](np.maximum(S, 0), cent_ids, ivf_off, ivf_doc, ndocs)


def fp_drops_last_query_token(S, cent_ids, ivf_off, ivf_doc, ndocs):
    return REAL["partial_scores"](np.ascontiguousarray(S[:-1]), np.ascontiguousarray(cent_ids[:-1]), ivf_off,
                                  ivf_doc, ndocs)


def fp_first_probe_only(S, cent_ids, ivf_off, ivf_doc, ndocs):
    return REAL["partial_scores"](S, np.ascontiguousarray(cent_ids[:, :1]), ivf_off, ivf_doc, ndocs)


def topk_ties_highest_id(ids, keys, k):
    oi, ok = REAL["topk"](-np.asarray(ids, np.int64), keys, k)
    return (-oi).astype(np.int32), ok


def topk_ascending(ids, keys, k):
    oi, ok = REAL["topk"](ids, -np.asarray(keys, np.int64), k)
    return oi, -ok


# ------------------------------------------------------ quantiser, codes
def encode_cutoff_to_upper(tok, cid, cent, cut, nbits):
    """A residual equal to a cutoff goes to the upper bucket (<= for <)."""
    return REAL["encode"](tok, cid, cent, np.asarray(cut, np.int64) - 1, nbits)


def quantizer_weights_at_cutoffs(hist, nbits):
    cut, w = REAL["quantizer"](hist, nbits)
    w = w.copy()
    w[:-1] = [oracle.grid_k(x / 2048.0) for x in cut]
    return cut, w


def quantizer_cutoff_off_by_one(hist, nbits):
    cut, w = REAL["quantizer"](hist, nbits)
    return cut + 1, w


def pack_reversed_in_byte(codes, nbits):
    codes = np.asarray(codes, np.uint8)
    per = 8 // nbits
    r = codes.reshape(codes.shape[0], -1, per)[:, :, ::-1].reshape(codes.shape)
    return REAL["pack"](np.ascontiguousarray(r), nbits)


# ------------------------------------------------------- document scores
def ds_no_centroid_term(S, q, w, b, n, cid, codes):
    return REAL["doc_scores"](np.zeros_like(S), q, w, b, n, cid, codes)


def ds_no_residual_term(S, q, w, b, n, cid, codes):
    return REAL["doc_scores"](S, q, np.zeros_like(w), b, n, cid, codes)


def ds_residual_negated(S, q, w, b, n, cid, codes):
    return REAL["doc_scores"](S, q, -np.asarray(w), b, n, cid, codes)


def ds_window_shifted(S, q, w, b, n, cid, codes):
    """Each document's tokens read from one place early (the previous
    document's last token in, its own last token out); shifting later would
    read past the last document."""
    return REAL["doc_scores"](S, q, w, np.maximum(np.asarray(b) - 1, 0), n, cid, codes)


def chamfer_transposed(q, tok, doc_off):
    """Max over query tokens for each document token, summed over the
    document: the two sides of MaxSim swapped."""
    out = np.empty(len(doc_off) - 1, np.int64)
    for v in range(len(doc_off) - 1):
        out[v] = REAL["exact_chamfer"](tok[doc_off[v]:doc_off[v + 1]], q, np.array([0, len(q)], np.int64))[0]
    return out


def key_scale_2_21(key):
    return float(np.float32(key) * np.float32(2.0 ** -21))


def key_no_f32_rounding(key):
    return float(key) * 2.0 ** -22


# -------------------------------------------------- collaborative scoring
def collab_ignores_chunks(ids, approx, exact, ncand, kfb, chunks, k):
    return REAL["collaborative_scoring"](ids, approx, exact, ncand, kfb, 1, k)


def collab_budget_short(ids, approx, exact, ncand, kfb, chunks, k):
    return REAL["collaborative_scoring"](ids, approx, exact, ncand, max(kfb - 1, 1), chunks, k)


def collab_ranks_by_exact(ids, approx, exact, ncand, kfb, chunks, k):
    return REAL["collaborative_scoring"](ids, np.array([exact(int(d)) for d in ids], np.int64), exact, ncand, kfb,
                                         chunks, k)


def collab_returns_approx(ids, approx, exact, ncand, kfb, chunks, k):
    a = {int(d): int(x) for d, x in zip(ids, approx)}
    return REAL["collaborative_scoring"](ids, approx, a.__getitem__, ncand, kfb, chunks, k)


# ---------------------------------------------------------- posting lists
def ivf_one_entry_per_token(cid, doc_off, ncent):
    off, tok = oracle.ivf_tokens(cid, ncent)
    return off, oracle.token_docs(doc_off)[tok]


# ------------------------------------------ refinement from token scores
def pres_no_residual(S, ci, q, w, off, tok, tdoc, codes, ndocs):
    return REAL["partial_scores_res"](S, ci, q, np.zeros_like(w), off, tok, tdoc, codes, ndocs)


def pres_residual_negated(S, ci, q, w, off, tok, tdoc, codes, ndocs):
    return REAL["partial_scores_res"](S, ci, q, -np.asarray(w), off, tok, tdoc, codes, ndocs)


def pres_no_centroid_term(S, ci, q, w, off, tok, tdoc, codes, ndocs):
    return REAL["partial_scores_res"](np.zeros_like(S), ci, q, w, off, tok, tdoc, codes, ndocs)


def pres_first_probe_only(S, ci, q, w, off, tok, tdoc, codes, ndocs):
    return REAL["partial_scores_res"](S, np.ascontiguousarray(ci[:, :1]), q, w, off, tok, tdoc, codes, ndocs)


def pres_token_to_next_doc(S, ci, q, w, off, tok, tdoc, codes, ndocs):
    return REAL["partial_scores_res"](S, ci, q, w, off, tok, np.minimum(np.asarray(tdoc) + 1, ndocs - 1), codes,
                                      ndocs)


def ivf_tokens_descending(cid, ncent):
    off, tok = REAL["ivf_tokens"](cid, ncent)
    tok = tok.copy()
    for c in range(ncent):
        tok[off[c]:off[c + 1]] = tok[off[c]:off[c + 1]][::-1]
    return off, tok


def token_docs_off_by_one(doc_off):
    doc_off = np.asarray(doc_off, np.int64)
    return np.repeat(np.arange(1, doc_off.shape[0], dtype=np.int32), np.diff(doc_off))


# -------------------------------------------------- reading and building
def grid_bf16_floor(bits):
    """Off-grid bf16 values floored to the grid instead of rounded."""
    v = (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.floor(v * 2048).astype(np.int16)


def assign_farthest(tok, cent, nthreads=0):
    return REAL["assign"](tok, -np.asarray(cent, np.int16), nthreads)


def residual_hist_negated(tok, cid, cent, hist=None):
    """Residuals taken as centroid minus token."""
    h = REAL["residual_hist"](tok, cid, cent)[::-1].copy()
    if hist is not None:
        hist += h
        return hist
    return h


def unpack_reversed_in_byte(packed, dim, nbits):
    c = REAL["unpack"](packed, dim, nbits)
    per = 8 // nbits
    return np.ascontiguousarray(c.reshape(c.shape[0], -1, per)[:, :, ::-1].reshape(c.shape))


# ------------------------------------------------- the oracle index's search
REAL_SEARCH = oracle.OracleIndex.search


def search_ncand_short(self, q_k, nprobe, ncand, k, nthreads=0, refine=False):
    return REAL_SEARCH(self, q_k, nprobe, max(ncand - 1, 1), k, nthreads, refine)


def search_ignores_refine(self, q_k, nprobe, ncand, k, nthreads=0, refine=False):
    return REAL_SEARCH(self, q_k, nprobe, ncand, k, nthreads, False)


MUTANTS = [
    ("grid_k", grid_k_ties_away, [PG.test_grid_examples_and_ties]),
    ("grid_k", grid_k_truncates, [PG.test_grid_examples_and_ties]),
    ("grid_f32", grid_f32_no_bf16, [PG.test_grid_matches_library_bf16_rounding]),
    ("centroid_scores", cs_negated, [PG.test_centroid_scores_exact_against_fp64_matmul]),
    ("centroid_scores", cs_drops_last_dim, [PG.test_centroid_scores_exact_against_fp64_matmul]),
    ("centroid_scores", cs_shifted_centroid, [PG.test_centroid_scores_exact_against_fp64_matmul]),
    ("probe", probe_ties_highest_id, [lambda: PG.test_probe_matches_lexsort(5),
                                      PG.test_probe_ties_go_to_lowest_id_and_self_ranks_first]),
    ("probe", probe_lowest_scores, [lambda: PG.test_probe_matches_lexsort(5)]),
    ("candidates", cand_drops_last_probe, [PP.test_candidates_and_fprime_match_definition]),
    ("partial_scores", fp_init_zero, [PP.test_fprime_negative_maximum_is_kept]),
    ("partial_scores", fp_drops_last_query_token, [PP.test_candidates_and_fprime_match_definition]),
    ("partial_scores", fp_first_probe_only, [PP.test_candidates_and_fprime_match_definition]),
    ("topk", topk_ties_highest_id, [PP.test_topk_matches_lexsort_with_ties]),
    ("topk", topk_ascending, [PP.test_topk_matches_lexsort_with_ties]),
    ("encode", encode_cutoff_to_upper, [PQ.test_value_on_cutoff_goes_to_lower_bucket,
                                        PQ.test_encode_is_count_of_cutoffs_below]),
    ("quantizer", quantizer_weights_at_cutoffs, [PQ.test_histogram_quantiles_match_sorted_array]),
    ("quantizer", quantizer_cutoff_off_by_one, [PQ.test_histogram_quantiles_match_sorted_array]),
    ("pack", pack_reversed_in_byte, [PQ.test_pack_layout_and_round_trip]),
    ("doc_scores", ds_no_centroid_term, [PQ.test_doc_scores_equal_brute_force_on_dequantised_vectors]),
    ("doc_scores", ds_no_residual_term, [PQ.test_doc_scores_equal_brute_force_on_dequantised_vectors]),
    ("doc_scores", ds_residual_negated, [PQ.test_doc_scores_equal_brute_force_on_dequantised_vectors]),
    ("doc_scores", ds_window_shifted, [PQ.test_doc_scores_equal_brute_force_on_dequantised_vectors]),
    ("exact_chamfer", chamfer_transposed, [PQ.test_exact_chamfer_against_fp64_matmul]),
    ("key_to_score", key_scale_2_21, [PQ.test_key_to_score_single_rounding]),
    ("key_to_score", key_no_f32_rounding, [PQ.test_key_to_score_single_rounding]),
    ("collaborative_scoring", collab_ignores_chunks, [lambda: PC.test_increasing_scores_reach_the_papers_worst_case(4, 8)]),
    ("collaborative_scoring", collab_budget_short, [lambda: PC.test_one_chunk_is_the_non_concurrent_strategy(True)]),
    ("collaborative_scoring", collab_ranks_by_exact, [lambda: PC.test_one_chunk_is_the_non_concurrent_strategy(True)]),
    ("collaborative_scoring", collab_returns_approx, [lambda: PC.test_one_chunk_is_the_non_concurrent_strategy(True)]),
    ("ivf_docs", ivf_one_entry_per_token, [PP.test_ivf_lists_match_sets]),
    ("partial_scores_res", pres_no_residual, [PR.test_refined_fprime_matches_definition]),
    ("partial_scores_res", pres_residual_negated, [PR.test_refined_fprime_matches_definition]),
    ("partial_scores_res", pres_no_centroid_term, [PR.test_refined_fprime_matches_definition,
                                                   PR.test_refined_fprime_negative_maximum_is_kept]),
    ("partial_scores_res", pres_first_probe_only, [PR.test_refined_fprime_matches_definition]),
    ("partial_scores_res", pres_token_to_next_doc, [PR.test_refined_fprime_matches_definition]),
    ("ivf_tokens", ivf_tokens_descending, [PR.test_token_lists_match_sets]),
    ("token_docs", token_docs_off_by_one, [PR.test_token_docs]),
    ("grid_bf16", grid_bf16_floor, [PG.test_grid_bf16_rounds_off_grid_values]),
    ("assign", assign_farthest, [PQ.test_synthetic_clusters_are_nearest_centroid]),
    ("residual_hist", residual_hist_negated, [PQ.test_histogram_quantiles_match_sorted_array]),
    ("unpack", unpack_reversed_in_byte, [PQ.test_pack_layout_and_round_trip]),
    ("OracleIndex.search", search_ncand_short, [PQ.test_search_composes_stage_definitions]),
    ("OracleIndex.search", search_ignores_refine, [PR.test_refined_search_composes_stage_definitions]),
]


@pytest.fixture(scope="module", autouse=True)
def _caches_built_unmutated():
    corpus("tiny")
    oracle_index("tiny").token_lists()


@pytest.mark.parametrize("target,mutant,pins", MUTANTS, ids=[m[1].__name__ for m in MUTANTS])
def test_pins_catch_planted_mistake(target, mutant, pins, monkeypatch):
    for pin in pins:  # the pins hold for the oracle as it is
        pin()
    owner, name = (oracle.OracleIndex, target.split(".")[1]) if "." in target else (oracle, target)
    monkeypatch.setattr(owner, name, mutant)
    caught = 0
    for pin in pins:
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught > 0, f"no pin caught {mutant.__name__} in oracle.{target}"
