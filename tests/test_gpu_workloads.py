"""Parity on the larger synthetic workloads, at full size (run on an MI355X).

The whole query batch goes through the engine in one call, as in the benchmark;
the oracle then checks sampled queries element by element: top-k ids, fixed-point
scores and counts from that batch, and probed centroids, missing-similarity
estimates, candidate sets and embeddings scored from a debug search of the same
queries. The float scores of the sampled queries' returned documents are also
checked against the fp64 explicit-decompression score (1e-4 relative), with
selection and m_i recomputed independently in numpy.

Each workload index is generated once per module (mid 9 s, long 31 s, full 69 s
with 16 processes); the oracle runs the tokens of one query in parallel.
"""
from __future__ import annotations

import os
import time

import numpy as np
import pytest

import oracle
import synth
from helpers import check_real_valued, index_arrays

pytestmark = pytest.mark.gpu

THREADS = min(16, len(os.sched_getaffinity(0)))


def say(*a):
    print(*a, flush=True)


_cache: dict = {}


def workload(name):
    if name not in _cache:
        _cache.clear()
        t0 = time.time()
        say(f"[{name}] generating")
        _cache[name] = synth.make_index(synth.WORKLOADS[name], workers=THREADS,
                                        progress=lambda m: say(f"[{name}] {m} ({time.time() - t0:.0f} s)"))
    return _cache[name]


def check(name, nprobe=None, rows=(0, -1)):
    import torch

    from paper_2501_17788_amd import Index

    data = workload(name)
    wl = data.workload
    nprobe = wl.nprobe if nprobe is None else nprobe
    nq = len(data.queries)
    rows = np.array(sorted({r % nq for r in rows}))
    say(f"[{name}] {data.n_embeddings} embeddings; whole batch of {nq} queries, nprobe={nprobe} "
        f"t'={wl.t_prime} k={wl.k}")
    t0 = time.time()
    with Index.from_synthetic(data) as ix:
        say(f"[{name}] index loaded in {time.time() - t0:.1f} s")
        q = torch.from_numpy(data.queries).cuda()
        t0 = time.time()
        ids, scores, counts, fixed = ix.search_async(q, nprobe, wl.t_prime, wl.k)
        ix.sync()
        say(f"[{name}] batch searched in {time.time() - t0:.2f} s")
        got = {"ids": ids.cpu().numpy(), "scores": scores.cpu().numpy(), "counts": counts.cpu().numpy(),
               "fixed": fixed.cpu().numpy()}
        say(f"[{name}] debug search of queries {rows.tolist()}")
        dbg = ix.search_debug(data.queries[rows], nprobe, wl.t_prime, wl.k)
    say(f"[{name}] oracle on queries {rows.tolist()} ({THREADS} threads)")
    t0 = time.time()
    want = oracle.search_index(data, queries=data.queries[rows], nprobe=nprobe, threads=THREADS)
    say(f"[{name}] oracle took {time.time() - t0:.1f} s; scored per query {want['n_scored'].tolist()}")
    for key in ("ids", "fixed", "counts", "scores"):
        np.testing.assert_array_equal(got[key][rows], want[key], err_msg=f"{name}: batch {key}")
    for key in ("ids", "fixed", "counts", "sel", "m_fixed", "cand_bitmap", "n_scored"):
        np.testing.assert_array_equal(dbg[key], want[key], err_msg=f"{name}: debug {key}")
    t0 = time.time()
    arrays = index_arrays(data)
    for qi in rows:
        gap = check_real_valued(got["scores"][qi], got["counts"][qi], got["ids"][qi], arrays, data.queries[qi],
                                nprobe, wl.t_prime)
        say(f"[{name}] query {qi}: {int(got['counts'][qi])} returned scores within {gap:.2e} relative of "
            f"the fp64 explicit-decompression scores")
    say(f"[{name}] real-valued check took {time.time() - t0:.1f} s")
    hit = float((got["ids"][:, 0] == data.query_targets).mean())
    say(f"[{name}] target document ranked first for {hit:.1%} of the batch")


@pytest.mark.timeout(600)
def test_mid_workload():
    check("mid", rows=(0, 511, -1))


@pytest.mark.timeout(600)
def test_long_workload():
    check("long", rows=(0, -1))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("nprobe", [16, 32, 64])
def test_full_workload(nprobe):
    check("full", nprobe=nprobe, rows=(0, -1))
