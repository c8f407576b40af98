"""Parity on the larger synthetic workloads, at full size (run on an MI355X).

The whole query batch goes through the engine in one call, as in the benchmark;
the oracle then checks sampled queries element by element: top-k ids, fixed-point
scores and counts from that batch, and probed centroids, missing-similarity
estimates, candidate sets and embeddings scored from a debug search of the same
queries. The long and full workloads take minutes to generate and check, so they
run only with WARP_LARGE_TESTS=1.
"""
from __future__ import annotations

import os
import time

import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu
LARGE = os.environ.get("WARP_LARGE_TESTS") == "1"
large = pytest.mark.skipif(not LARGE, reason="set WARP_LARGE_TESTS=1 (several minutes per workload)")


def say(*a):
    print(*a, flush=True)


_cache: dict = {}


def workload(name):
    if name not in _cache:
        _cache.clear()
        t0 = time.time()
        say(f"[{name}] generating")
        _cache[name] = synth.make_index(synth.WORKLOADS[name], workers=min(16, os.cpu_count() or 1),
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
    with Index.from_synthetic(data) as ix:
        q = torch.from_numpy(data.queries).cuda()
        t0 = time.time()
        ids, scores, counts, fixed = ix.search_async(q, nprobe, wl.t_prime, wl.k)
        ix.sync()
        say(f"[{name}] batch searched in {time.time() - t0:.2f} s")
        got = {"ids": ids.cpu().numpy(), "scores": scores.cpu().numpy(), "counts": counts.cpu().numpy(),
               "fixed": fixed.cpu().numpy()}
        say(f"[{name}] debug search of queries {rows.tolist()}")
        dbg = ix.search_debug(data.queries[rows], nprobe, wl.t_prime, wl.k)
    say(f"[{name}] oracle on queries {rows.tolist()}")
    t0 = time.time()
    want = oracle.search_index(data, queries=data.queries[rows], nprobe=nprobe, threads=len(rows))
    say(f"[{name}] oracle took {time.time() - t0:.1f} s; scored per query {want['n_scored'].tolist()}")
    for key in ("ids", "fixed", "counts", "scores"):
        np.testing.assert_array_equal(got[key][rows], want[key], err_msg=f"{name}: batch {key}")
    for key in ("ids", "fixed", "counts", "sel", "m_fixed", "cand_bitmap", "n_scored"):
        np.testing.assert_array_equal(dbg[key], want[key], err_msg=f"{name}: debug {key}")
    hit = float((got["ids"][:, 0] == data.query_targets).mean())
    say(f"[{name}] target document ranked first for {hit:.1%} of the batch")


def test_mid_workload():
    check("mid", rows=(0, 511, -1))


@large
def test_long_workload():
    check("long", rows=(0, -1))


@large
@pytest.mark.parametrize("nprobe", [16, 32, 64])
def test_full_workload(nprobe):
    check("full", nprobe=nprobe, rows=(0, -1))
