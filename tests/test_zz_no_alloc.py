"""warp_search_noalloc, the search entry point that allocates nothing, against
warp_search_async on the same index and queries (run on an MI355X).

Both are called through the C ABI with device pointers. The results must be
identical: top-k ids, float scores, counts and fixed-point scores. Each case makes
two calls in a row, the second with fewer queries, so the second finds what the
first left in the static scratch.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def _outs(nq, k, dev):
    import torch

    return (torch.full((nq, k), -7, dtype=torch.int32, device=dev),
            torch.full((nq, k), 7.0, dtype=torch.float32, device=dev),
            torch.full((nq,), -7, dtype=torch.int32, device=dev),
            torch.full((nq, k), 7, dtype=torch.int64, device=dev))


def _call(fn, ix, q, nprobe, t_prime, k):
    """One search through the C entry point `fn` (warp_search_async or warp_search_noalloc)."""
    import torch

    from paper_2501_17788_amd import warp

    nq, nt, _ = q.shape
    ids, scores, counts, fixed = _outs(nq, k, q.device)
    stream = torch.cuda.current_stream(q.device)
    P = ctypes.c_void_p
    rc = fn(ix.handle, P(q.data_ptr()), nq, nt, nprobe, int(t_prime), k, P(ids.data_ptr()), P(scores.data_ptr()),
            P(counts.data_ptr()), P(fixed.data_ptr()), P(stream.cuda_stream))
    if rc != 0:
        raise warp.WarpError(rc, warp.last_error())
    ix.sync()
    return {"ids": ids.cpu().numpy(), "scores": scores.cpu().numpy(), "counts": counts.cpu().numpy(),
            "fixed": fixed.cpu().numpy()}


def _both(ix, Q, nprobe, t_prime, k, label):
    import torch

    from paper_2501_17788_amd import lib

    q = torch.from_numpy(np.ascontiguousarray(Q, np.float32)).cuda()
    say(f"[{label}] {q.shape[0]} queries: warp_search_noalloc")
    got = _call(lib.warp_search_noalloc, ix, q, nprobe, t_prime, k)
    say(f"[{label}] {q.shape[0]} queries: warp_search_async")
    want = _call(lib.warp_search_async, ix, q, nprobe, t_prime, k)
    for key in ("ids", "scores", "counts", "fixed"):
        np.testing.assert_array_equal(got[key], want[key], err_msg=f"{label}: {key}")
    return got


def test_noalloc_matches_async_small_workload():
    """100k documents: about 17 MB of scratch per query, so the 256 MiB array takes waves
    of a dozen queries; 40 queries, then 5."""
    from paper_2501_17788_amd import Index

    data = synth.make_index(synth.WORKLOADS["small"], workers=min(16, len(os.sched_getaffinity(0))))
    wl = data.workload
    with Index.from_synthetic(data) as ix:
        _both(ix, data.queries[:40], wl.nprobe, wl.t_prime, wl.k, "small 40")
        _both(ix, data.queries[100:105], wl.nprobe, wl.t_prime, wl.k, "small 5")


@pytest.mark.parametrize("literal", [False, True], ids=["paper", "eq1_literal"])
def test_noalloc_matches_async_tiny(literal):
    from paper_2501_17788_amd import SCORING_EQ1_LITERAL, Index

    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=9, nprobe=32, k=50),
                            workers=1)
    wl = data.workload
    with Index.from_synthetic(data) as ix:
        if literal:
            ix.set_scoring(SCORING_EQ1_LITERAL)
        _both(ix, data.queries, wl.nprobe, wl.t_prime, wl.k, f"tiny 9 literal={literal}")
        _both(ix, data.queries[2:4, :17], wl.nprobe, wl.t_prime, wl.k, f"tiny 2x17 literal={literal}")


def test_noalloc_matches_async_large_nprobe_and_k():
    """n_probe above 256 and k above 4096 take the sort-based selection and top-k, whose
    sort buffers then also live in the static array."""
    from paper_2501_17788_amd import Index

    data = synth.make_index(synth.random_small_workload(21, n_centroids=1000, n_docs=20000, max_len=20, nbits=2,
                                                        n_queries=4, n_qtok=8, nprobe=300, t_prime=4000,
                                                        k=6000), workers=1)
    with Index.from_synthetic(data) as ix:
        _both(ix, data.queries, 300, 4000, 6000, "large 4")
        _both(ix, data.queries[1:3, :5], 600, 900, 5000, "large 2x5")


def test_noalloc_rejects_an_index_too_large_for_its_scratch():
    """With 3M documents one query's token-max table alone is 384 MiB: the call fails with
    WARP_ENOMEM and enqueues nothing; warp_search_async still serves the index."""
    from paper_2501_17788_amd import ENOMEM, Index, WarpError, lib

    import torch

    data = synth.make_index(synth.random_small_workload(9, n_centroids=40, n_docs=300, max_len=4, n_queries=2,
                                                        n_qtok=32, nprobe=5, t_prime=7, k=10), workers=1)
    with Index(data.centroids, data.offsets, data.doc_ids, data.codes, data.nbits, data.bucket_weights,
               3_000_000) as ix:
        q = torch.from_numpy(data.queries).cuda()
        with pytest.raises(WarpError) as e:
            _call(lib.warp_search_noalloc, ix, q, 5, 7, 10)
        assert e.value.code == ENOMEM and "static scratch" in e.value.msg
        say(f"[too large] {e.value.msg}")
        _call(lib.warp_search_async, ix, q, 5, 7, 10)
