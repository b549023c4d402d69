"""GPU path against the oracle at the full sizes of the larger workloads, in
the launch configuration the benchmark times: the whole query batch in one
search call; sampled queries are checked element by element (centroid ids
and keys, the top-ncand candidates and their F' keys, the top-k ids and
scores, all bit-exact).

Each workload's corpus is generated and indexed on the host first (two
passes over ~70M to ~640M tokens).  CHIMERA_SKIP_BIG (comma-separated names,
or all) skips workloads for quick runs."""
import gc
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor, as_completed

import numpy as np
import pytest
import torch

import synth
from util_big import build_both, oracle_search_one

pytestmark = pytest.mark.gpu

_SKIP = {s.strip() for s in os.environ.get("CHIMERA_SKIP_BIG", "").split(",") if s.strip()}


_capsys = None


def say(*a):
    """A progress line that reaches the terminal as each step ends, past
    pytest's output capture: these tests run for minutes."""
    if _capsys is not None:
        with _capsys.disabled():
            print("[gpu-big]", *a, flush=True)
    else:
        print("[gpu-big]", *a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("name", ["1m", "2m-long", "8.8m"])
def test_full_size_sampled_parity(name, capsys):
    global _capsys
    _capsys = capsys
    if name in _SKIP or "all" in _SKIP:
        pytest.skip(f"full-size {name} workload skipped by CHIMERA_SKIP_BIG")
    w = synth.WORKLOADS[name]
    t0 = time.time()
    say(f"{name}: building product index and oracle view")
    c, b, oi = build_both(w, say=lambda *a: say(name, *a))
    say(f"{name}: built in {time.time() - t0:.0f}s: {b.info()}")
    idx = b.upload(0)
    b.close()
    q_k, _ = c.queries(w.nq, w.Tq)
    Q = torch.from_numpy(synth.k_to_bf16_bits(q_k).view(np.int16)).cuda().view(torch.bfloat16)
    say(f"{name}: GPU search of {w.nq} queries")
    ids, scores = idx.search(Q, w.nprobe, w.ncand, w.k)
    ci, ck = idx.probe(Q, w.nprobe)
    cand, ckeys, nval = idx.prune(Q, w.nprobe, w.ncand)
    torch.cuda.synchronize()
    ids, scores = ids.cpu().numpy(), scores.cpu().numpy()
    ci, ck = ci.cpu().numpy(), ck.cpu().numpy()
    cand, ckeys, nval = cand.cpu().numpy(), ckeys.cpu().numpy(), nval.cpu().numpy()

    # spread over the batch, with the first and last query of each of three
    # equal sub-batches (the split a 4096-query 8.8M batch runs in)
    b3 = -(-w.nq // 3)
    sample = sorted({0, 1, b3 - 1, b3, w.nq // 2, 2 * b3 - 1, 2 * b3, w.nq - 1})
    say(f"{name}: oracle on queries {sample}")
    with ThreadPoolExecutor(max_workers=len(sample)) as ex:
        futs = {ex.submit(oracle_search_one, c, oi, q_k[qi], w.nprobe, w.ncand, w.k): qi for qi in sample}
        got = {}
        for f in as_completed(futs):
            got[futs[f]] = f.result()
            say(f"{name}: oracle query {futs[f]} done ({time.time() - t0:.0f}s)")
    refs = [got[qi] for qi in sample]
    for qi, ref in zip(sample, refs):
        say(f"{name}: query {qi}")
        assert np.array_equal(ci[qi], ref["cent_ids"]), f"{name} q{qi}: centroid ids differ"
        assert np.array_equal(ck[qi].astype(np.int64), ref["cent_keys"]), f"{name} q{qi}: centroid keys differ"
        n = len(ref["cand"])
        assert nval[qi] == n, f"{name} q{qi}: {nval[qi]} candidates, oracle {n}"
        order = np.argsort(ref["cand"])
        assert np.array_equal(cand[qi, :n], ref["cand"][order]), f"{name} q{qi}: candidates differ"
        assert np.array_equal(ckeys[qi, :n].astype(np.int64), ref["cand_keys"][order]), f"{name} q{qi}: F' differs"
        m = len(ref["ids"])
        assert np.array_equal(ids[qi, :m], ref["ids"]), f"{name} q{qi}: top-k ids differ"
        assert np.array_equal(scores[qi, :m], ref["scores"]), f"{name} q{qi}: scores differ"
        assert np.all(ids[qi, m:] == -1)
    idx.close()
    del idx, oi, c
    gc.collect()
