"""Parity of the HIP engine with the CPU oracle (run on an MI355X).

Bit-exact: probed centroids and their order, the missing-similarity estimates,
candidate sets, embeddings scored, top-k ids and fixed-point document scores.
Float scores: the float of the same fixed-point value (identical), and within
1e-4 relative of the fp64 real-valued score from explicit decompression
(helpers.realvalued_doc_scores, which recomputes selection and m_i itself).
"""
from __future__ import annotations

import os

import numpy as np
import pytest

import oracle
import synth
from helpers import FRAC, check_real_valued, index_arrays, load_dyadic, unpack_msb_first

pytestmark = pytest.mark.gpu

EXACT = ("ids", "fixed", "counts", "sel", "m_fixed", "cand_bitmap", "n_scored")


def _engine():
    import paper_2501_17788_amd as w
    return w


def say(*a):
    print(*a, flush=True)


def compare(got: dict, want: dict, rows=None, label=""):
    for key in EXACT:
        g = got[key] if rows is None else got[key][rows]
        if not np.array_equal(g, want[key]):
            bad = np.argwhere(g != want[key]) if g.shape == want[key].shape else "shape"
            raise AssertionError(f"{label}: {key} differs at {bad[:5] if not isinstance(bad, str) else bad}")
    g = got["scores"] if rows is None else got["scores"][rows]
    np.testing.assert_array_equal(g, want["scores"])


def run_both(data, queries=None, nprobe=None, t_prime=None, k=None, label="", literal=False):
    w = _engine()
    wl = data.workload
    Q = data.queries if queries is None else queries
    nprobe = wl.nprobe if nprobe is None else nprobe
    t_prime = wl.t_prime if t_prime is None else t_prime
    k = wl.k if k is None else k
    say(f"[{label}] n_emb={data.n_embeddings} n_c={len(data.offsets) - 1} nbits={data.nbits} "
        f"queries={Q.shape} nprobe={nprobe} t'={t_prime} k={k} literal={literal}")
    with w.Index.from_synthetic(data) as ix:
        if literal:
            ix.set_scoring(w.SCORING_EQ1_LITERAL)
        got = ix.search_debug(Q, nprobe, t_prime, k)
    want = oracle.search_index(data, queries=Q, nprobe=nprobe, t_prime=t_prime, k=k,
                               flags=oracle.EQ1_LITERAL if literal else 0)
    compare(got, want, label=label)
    return got


# ----------------------------------------------------------------------------- hand-built

@pytest.mark.parametrize("case", range(8))
def test_dyadic_example(case):
    w = _engine()
    g, ix_arrays, Q = load_dyadic()
    c = g["cases"][case]
    say(f"[dyadic {c['name']}] nprobe={c['nprobe']} t'={c['t_prime']} k={c['k']}")
    with w.Index(**ix_arrays) as ix:
        got = ix.search_debug(Q, c["nprobe"], c["t_prime"], c["k"])
    assert got["ids"].tolist() == c["ids"]
    assert got["sel"].tolist() == c["sel"]
    assert (got["m_fixed"] / FRAC).tolist() == c["m"]
    assert got["n_scored"].tolist() == c["n_scored"]
    assert got["counts"].tolist() == c["counts"]
    want = oracle.search(queries=Q, nprobe=c["nprobe"], t_prime=c["t_prime"], k=c["k"], **ix_arrays)
    compare(got, want, label=f"dyadic {c['name']}")


# ----------------------------------------------------------------------------- random small

CASES = [
    # seed, n_centroids, n_docs, max_len, nbits, n_queries, n_qtok, nprobe, t_prime, k
    (0, 16, 40, 8, 4, 3, 4, 4, 10, 5),
    (1, 16, 40, 8, 2, 3, 4, 4, 10, 5),
    (2, 1, 10, 3, 4, 2, 32, 1, 0, 20),          # one centroid
    (3, 50, 300, 12, 4, 5, 32, 7, 0, 50),       # t' = 0
    (4, 50, 300, 12, 2, 5, 17, 7, 10 ** 9, 50),  # t' above N: lowest score
    (5, 64, 200, 10, 4, 4, 32, 64, 100, 300),   # nprobe = all clusters, k above candidates
    (6, 200, 1000, 20, 4, 7, 32, 32, 500, 100),
    (7, 200, 1000, 20, 2, 7, 1, 3, 50, 1),      # one query token, k = 1
    (8, 300, 5000, 30, 4, 3, 32, 256, 2000, 4096),  # largest nprobe and k
    (9, 40, 100000, 1, 4, 2, 8, 5, 7, 10),      # most documents have no embedding at all
    (10, 60, 400, 12, 1, 4, 32, 9, 100, 30),    # one bit per dimension
    (11, 60, 400, 12, 8, 4, 32, 9, 100, 30),    # eight bits per dimension
    (12, 300, 3000, 40, 8, 3, 32, 48, 800, 200),
    (13, 40, 303, 12, 4, 3, 32, 9, 100, 30),     # a document count that is not a multiple of 4
]

# n_probe above 256 (the selection sorts every (token, centroid) score) and k above 4096 (the
# top-k sorts every document key): the same results as the boundary-band selection and the
# LDS top-k give below those limits
LARGE_CASES = [
    # seed, n_centroids, n_docs, max_len, nbits, n_queries, n_qtok, nprobe, t_prime, k
    (20, 600, 3000, 20, 4, 3, 32, 600, 1500, 5000),    # all clusters, k above n_docs
    (21, 1000, 20000, 20, 2, 4, 8, 300, 4000, 6000),   # 300 of 1000 clusters
    (22, 400, 2000, 10, 4, 2, 16, 400, 10 ** 9, 50),   # t' above N: lowest score
    (23, 300, 2000, 10, 8, 2, 32, 257, 0, 4097),       # t' = 0, one past each limit
    (24, 700, 5000, 12, 1, 5, 32, 520, 700, 4096),     # large n_probe alone
    (25, 60, 9000, 12, 4, 3, 32, 9, 100, 8000),        # large k alone
    (26, 4000, 40000, 6, 4, 3, 1, 260, 100, 10000),    # fewer candidates than k, one token
]


@pytest.mark.parametrize("case", CASES, ids=[f"seed{c[0]}" for c in CASES])
def test_random_small(case):
    seed, n_c, n_docs, max_len, nbits, nq, nt, nprobe, tp, k = case
    if seed == 9:
        wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=300, max_len=max_len, nbits=nbits,
                                         n_queries=nq, n_qtok=nt, nprobe=nprobe, t_prime=tp, k=k)
        data = synth.make_index(wl, workers=1)
        data.workload = synth.with_overrides(wl, n_docs=n_docs)  # ids < 300 of 100000 docs
    else:
        wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=n_docs, max_len=max_len, nbits=nbits,
                                         n_queries=nq, n_qtok=nt, nprobe=nprobe, t_prime=tp, k=k)
        data = synth.make_index(wl, workers=1)
    run_both(data, label=f"random seed {seed}")


@pytest.mark.parametrize("case", LARGE_CASES, ids=[f"seed{c[0]}" for c in LARGE_CASES])
def test_large_nprobe_and_k(case):
    seed, n_c, n_docs, max_len, nbits, nq, nt, nprobe, tp, k = case
    wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=n_docs, max_len=max_len, nbits=nbits,
                                     n_queries=nq, n_qtok=nt, nprobe=nprobe, t_prime=tp, k=k)
    data = synth.make_index(wl, workers=1)
    run_both(data, label=f"large seed {seed}")
    if seed == 20:
        run_both(data, label=f"large seed {seed} literal", literal=True)


def test_selection_band_overflow_falls_back_to_sorting():
    """2,000 identical centroids and a query token equal to them: all 2,000 share the top
    selection bin, more than the 1,024 that the band rescoring holds. The blocking search runs
    again with the selection that sorts every score and must give the oracle's results; the
    asynchronous one reports WARP_ENOTSUP at sync, and the index keeps working."""
    import dataclasses

    import torch

    w = _engine()
    wl = synth.random_small_workload(30, n_centroids=3000, n_docs=2000, max_len=12, nbits=4, n_queries=3,
                                     n_qtok=8, nprobe=32, t_prime=500, k=20)
    data = synth.make_index(wl, workers=1)
    C = data.centroids.copy()
    C[1:2001] = C[0]
    Q = data.queries.copy()
    Q[0, 0] = C[0]
    data = dataclasses.replace(data, centroids=C, queries=Q)
    run_both(data, label="band overflow, blocking search")
    with w.Index.from_synthetic(data) as ix:
        say("[band overflow] asynchronous search")
        ix.search_async(torch.from_numpy(Q).cuda(), wl.nprobe, wl.t_prime, wl.k)
        with pytest.raises(w.WarpError) as e:
            ix.sync()
        assert e.value.code == w.ENOTSUP and "overflow" in e.value.msg
        compare(ix.search_debug(Q[1:], wl.nprobe, wl.t_prime, wl.k),
                oracle.search_index(data, queries=Q[1:]), label="band overflow, after the error")


@pytest.mark.parametrize("slices", ["3", "7"])
def test_split_selection(slices, monkeypatch):
    """Waves of few tokens split each token's selection over several workgroups (histogram and
    band lists in global memory). WARP_SELECT_SLICES forces the split on every wave: the
    probed centroids, m_i and the results must be the oracle's, at t' = 0, t' above N, nprobe
    = all clusters, nprobe 256 with k 4096, one query token, and in both scoring modes."""
    monkeypatch.setenv("WARP_SELECT_SLICES", slices)
    for case in (CASES[2], CASES[3], CASES[4], CASES[5], CASES[7], CASES[8], CASES[12]):
        seed, n_c, n_docs, max_len, nbits, nq, nt, nprobe, tp, k = case
        wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=n_docs, max_len=max_len, nbits=nbits,
                                         n_queries=nq, n_qtok=nt, nprobe=nprobe, t_prime=tp, k=k)
        run_both(synth.make_index(wl, workers=1), label=f"slices={slices} seed {seed}")
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=5, nprobe=24, k=40), workers=1)
    run_both(data, label=f"slices={slices} tiny")
    run_both(data, label=f"slices={slices} tiny literal", literal=True)


@pytest.mark.parametrize("narrow_max", ["0", "3", "4096"], ids=["all-wide", "narrow3", "all-narrow"])
def test_wide_and_narrow_scans_agree(narrow_max, monkeypatch):
    """Chunks probed by few tokens take the narrow scan (one wave per chunk, groups of three
    tokens per matrix-core tile), the others the wide one; WARP_NARROW_MAX moves the split.
    Every split gives the oracle's results: all chunks wide, a three-token split, and every
    chunk narrow (up to 32 tokens in eleven groups), in both scoring modes and at b = 1, 2, 4, 8."""
    monkeypatch.setenv("WARP_NARROW_MAX", narrow_max)
    for case in (CASES[3], CASES[6], CASES[10], CASES[11], CASES[12]):
        seed, n_c, n_docs, max_len, nbits, nq, nt, nprobe, tp, k = case
        wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=n_docs, max_len=max_len, nbits=nbits,
                                         n_queries=nq, n_qtok=nt, nprobe=nprobe, t_prime=tp, k=k)
        run_both(synth.make_index(wl, workers=1), label=f"narrow_max={narrow_max} seed {seed}")
    wl = synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=6, nbits=2, nprobe=24, k=40)
    data = synth.make_index(wl, workers=1)
    run_both(data, label=f"narrow_max={narrow_max} tiny b=2")
    run_both(data, label=f"narrow_max={narrow_max} tiny b=2 literal", literal=True)


def test_empty_clusters_and_ragged_tiles():
    # many centroids, few embeddings: most clusters are empty; tails of every tile are ragged
    wl = synth.random_small_workload(11, n_centroids=1024, n_docs=700, max_len=9, nbits=4, n_queries=6,
                                     n_qtok=32, nprobe=40, t_prime=30, k=25, zipf_s=0.3)
    data = synth.make_index(wl, workers=1)
    assert (np.diff(data.offsets) == 0).sum() > 20
    run_both(data, label="empty clusters")


def test_cluster_offsets_over_several_passes():
    # 70,001 clusters: the work plan's pair offsets (one workgroup, 32,768 clusters per pass)
    # carry a running total over three passes and end in a ragged tail; most clusters are empty
    wl = synth.random_small_workload(11, n_centroids=70001, n_docs=3000, max_len=24, nbits=2, n_queries=4,
                                     n_qtok=32, nprobe=64, t_prime=50, k=20)
    data = synth.make_index(wl, workers=1)
    assert len(data.offsets) - 1 == 70001 and (np.diff(data.offsets) == 0).sum() > 50000
    run_both(data, label="70001 clusters")


# ----------------------------------------------------------------------------- workloads

def test_tiny_workload_exact_and_real_valued():
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=4), workers=1)
    wl = data.workload
    got = run_both(data, label="tiny")
    for qi in range(len(data.queries)):
        gap = check_real_valued(got["scores"][qi], got["counts"][qi], got["ids"][qi], index_arrays(data),
                                data.queries[qi], wl.nprobe, wl.t_prime)
        say(f"[tiny] query {qi}: largest relative gap to the fp64 scores {gap:.2e}")
    assert got["ids"][0, 0] == data.query_targets[0]


@pytest.mark.parametrize("case", range(4))
@pytest.mark.parametrize("mode", ["paper", "eq1_literal"])
def test_eq1_literal_hand_worked(case, mode):
    """The hand-worked example that separates Section 4.5's imputation from Eq. 1 read
    literally (a fully retrieved document whose best score is below m_i, a partly
    retrieved one): the engine gives the hand-worked results in both modes."""
    w = _engine()
    g, ix_arrays, Q = load_dyadic("eq1_literal_example.json")
    c = g["cases"][case]
    say(f"[eq1 hand-worked {c['name']} {mode}] nprobe={c['nprobe']} t'={c['t_prime']} k={c['k']}")
    with w.Index(**ix_arrays) as ix:
        if mode == "eq1_literal":
            ix.set_scoring(w.SCORING_EQ1_LITERAL)
        got = ix.search_debug(Q, c["nprobe"], c["t_prime"], c["k"])
    want = c[mode]
    assert got["ids"].tolist() == want["ids"]
    assert got["counts"].tolist() == want["counts"]
    for qi in range(len(want["ids"])):
        for v, f in zip(want["scores"][qi], got["fixed"][qi].tolist()):
            assert f == (np.iinfo(np.int64).min if v is None else int(v * FRAC))
    assert got["sel"].tolist() == c["sel"]
    assert (got["m_fixed"] / FRAC).tolist() == c["m"]
    assert got["n_scored"].tolist() == c["n_scored"]
    flags = oracle.EQ1_LITERAL if mode == "eq1_literal" else 0
    compare(got, oracle.search(queries=Q, nprobe=c["nprobe"], t_prime=c["t_prime"], k=c["k"], flags=flags,
                               **ix_arrays), label=f"eq1 hand-worked {c['name']} {mode}")


@pytest.mark.parametrize("nbits", [1, 2, 4, 8])
def test_tiny_workload_code_widths(nbits):
    wl = synth.with_overrides(synth.WORKLOADS["tiny"], nbits=nbits, n_queries=3, nprobe=32, k=100)
    run_both(synth.make_index(wl, workers=1), label=f"tiny nbits={nbits}")


def test_many_waves_match_one_wave(monkeypatch):
    w = _engine()
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=9), workers=1)
    wl = data.workload
    say("[waves] one wave")
    with w.Index.from_synthetic(data) as ix:
        one = ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k)
        monkeypatch.setenv("WARP_SCRATCH_MB", "1")  # forces one query per wave
        say("[waves] one query per wave")
        many = ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k)
    for key in EXACT + ("scores",):
        np.testing.assert_array_equal(one[key], many[key])


def test_deterministic_and_async_matches_sync():
    import torch

    w = _engine()
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=5), workers=1)
    wl = data.workload
    with w.Index.from_synthetic(data) as ix:
        say("[async] sync twice")
        a = ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k)
        b = ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k)
        for key in EXACT + ("scores",):
            np.testing.assert_array_equal(a[key], b[key])
        say("[async] device tensors")
        q = torch.from_numpy(data.queries).cuda()
        ids, scores, counts, fixed = ix.search_async(q, wl.nprobe, wl.t_prime, wl.k)
        ix.sync()
        np.testing.assert_array_equal(ids.cpu().numpy(), a["ids"])
        np.testing.assert_array_equal(scores.cpu().numpy(), a["scores"])
        np.testing.assert_array_equal(counts.cpu().numpy(), a["counts"])
        np.testing.assert_array_equal(fixed.cpu().numpy(), a["fixed"])


@pytest.mark.parametrize("nbits", [1, 2, 4, 8])
def test_index_from_device_tensors(nbits):
    """warp_index_load_device copies the small arrays to the host for validation at every
    code width, then searches like a host-loaded index."""
    import torch

    w = _engine()
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=2, nbits=nbits), workers=1)
    wl = data.workload
    t = {k: torch.from_numpy(np.ascontiguousarray(getattr(data, k))).cuda()
         for k in ("centroids", "offsets", "doc_ids", "codes", "bucket_weights")}
    say(f"[device load] nbits={nbits}")
    with w.Index.from_device(t["centroids"], t["offsets"], t["doc_ids"], t["codes"], data.nbits,
                             t["bucket_weights"], data.n_docs) as ix:
        got = ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k)
    compare(got, oracle.search_index(data), label=f"device load nbits={nbits}")
    # validation still runs on device arrays: a non-unit centroid is rejected
    bad = t["centroids"].clone()
    bad[3] *= 1.01
    with pytest.raises(w.WarpError) as e:
        w.Index.from_device(bad, t["offsets"], t["doc_ids"], t["codes"], data.nbits, t["bucket_weights"],
                            data.n_docs)
    assert e.value.code == w.EINVAL and "unit norm" in e.value.msg


def test_scratch_cap_gives_enomem_then_recovers(monkeypatch):
    """WARP_MAX_SCRATCH_BYTES caps an index's search scratch: below what one query needs the
    search fails with WARP_ENOMEM; a cap that holds a few queries splits the batch into
    waves; without it the same index searches normally."""
    w = _engine()
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=6), workers=1)
    wl = data.workload
    want = oracle.search_index(data)
    with w.Index.from_synthetic(data) as ix:
        monkeypatch.setenv("WARP_MAX_SCRATCH_BYTES", "4096")
        say("[scratch cap] 4 KiB")
        with pytest.raises(w.WarpError) as e:
            ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k)
        assert e.value.code == w.ENOMEM and "WARP_MAX_SCRATCH_BYTES" in e.value.msg
        monkeypatch.setenv("WARP_MAX_SCRATCH_BYTES", str(3 << 20))
        say("[scratch cap] 3 MiB")
        compare(ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k), want, label="3 MiB cap")
        monkeypatch.delenv("WARP_MAX_SCRATCH_BYTES")
        say("[scratch cap] none")
        compare(ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k), want, label="no cap")


def test_freed_handle_is_rejected():
    """A freed handle is no longer live: a second free is a no-op and a search on it fails
    with WARP_EINVAL instead of touching freed memory."""
    import ctypes

    w = _engine()
    data = synth.make_index(synth.random_small_workload(4), workers=1)
    ix = w.Index.from_synthetic(data)
    h = ctypes.c_void_p(ix.handle.value)
    ix.close()
    w.lib.warp_index_free(h)  # second free: ignored
    assert "invalid" in w.last_error()
    Q = np.ascontiguousarray(data.queries, np.float32)
    ids = np.empty((len(Q), 3), np.int32)
    sc = np.empty((len(Q), 3), np.float32)
    rc = w.lib.warp_search(h, Q.ctypes.data_as(ctypes.c_void_p), len(Q), Q.shape[1], 2, 0, 3,
                           ids.ctypes.data_as(ctypes.c_void_p), sc.ctypes.data_as(ctypes.c_void_p), None)
    assert rc == w.EINVAL and "handle" in w.last_error()
    assert w.lib.warp_index_info(h, None, None, None, None) == w.EINVAL


def test_filter_scores_within_selection_margin():
    w = _engine()
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=8), workers=1)
    toks = data.queries.reshape(-1, 128)
    say("[filter] tiny, 256 tokens")
    with w.Index.from_synthetic(data) as ix:
        F = ix.filter_scores(toks)
    S = toks.astype(np.float64) @ data.centroids.astype(np.float64).T
    err = np.abs(F - S).max()
    say(f"[filter] max |f - S64| = {err:.3g}")
    assert err <= 2.0 ** -16  # the selection assumes 2^-13


def test_gpu_argument_errors():
    w = _engine()
    data = synth.make_index(synth.random_small_workload(1), workers=1)
    with w.Index.from_synthetic(data) as ix:
        Q = data.queries
        say("[errors]")
        for args, code in [((Q, 0, 1, 1), w.EINVAL), ((Q, 17, 1, 1), w.EINVAL), ((Q, 4, -1, 1), w.EINVAL),
                           ((Q, 4, 1, 0), w.EINVAL),
                           ((Q * 1.01, 4, 1, 3), w.EINVAL), ((np.zeros((1, 33, 128)), 4, 1, 3), w.EINVAL)]:
            with pytest.raises(w.WarpError) as e:
                ix.search(*args)
            assert e.value.code == code, (e.value, args[1:])
        # the index still works after rejected calls
        compare(ix.search_debug(Q, 4, 10, 5), oracle.search_index(data), label="after errors")
    bad = data.doc_ids.copy()
    bad[0] = data.n_docs
    with pytest.raises(w.WarpError) as e:
        w.Index(data.centroids, data.offsets, bad, data.codes, data.nbits, data.bucket_weights, data.n_docs)
    assert e.value.code == w.EINVAL and "document id" in e.value.msg


def test_async_query_norm_error_reported_by_sync():
    import torch

    w = _engine()
    data = synth.make_index(synth.random_small_workload(2), workers=1)
    with w.Index.from_synthetic(data) as ix:
        q = torch.from_numpy(data.queries * 1.1).cuda()
        ix.search_async(q, 4, 10, 5)
        with pytest.raises(w.WarpError) as e:
            ix.sync()
        assert e.value.code == w.EINVAL and "norm" in e.value.msg
        ix.search_async(torch.from_numpy(data.queries).cuda(), 4, 10, 5)
        ix.sync()  # cleared
        # the table written by the failed search is zeroed before it is used again
        got = ix.search_debug(data.queries, 4, 10, 5)
    compare(got, oracle.search_index(data, nprobe=4, t_prime=10, k=5), label="after a norm error")


# ----------------------------------------------------------------------------- the 256-query workload

@pytest.fixture(scope="module")
def small_data():
    return synth.make_index(synth.WORKLOADS["small"], workers=min(16, os.cpu_count() or 1))


def test_small_workload_sampled_queries(small_data):
    """All 256 queries in one launch (the benchmark's configuration); a sample of
    them checked against the oracle element by element."""
    w = _engine()
    data = small_data
    wl = data.workload
    say(f"[small] {data.n_embeddings} embeddings, 256 queries, nprobe={wl.nprobe} t'={wl.t_prime} k={wl.k}")
    rows = np.array([0, 1, 37, 100, 128, 200, 254, 255])
    with w.Index.from_synthetic(data) as ix:
        got = ix.search_debug(data.queries, wl.nprobe, wl.t_prime, wl.k)
        # the sampled queries on their own (256 tokens: the split selection) and one query
        got_few = ix.search_debug(data.queries[rows], wl.nprobe, wl.t_prime, wl.k)
        got_one = ix.search_debug(data.queries[rows[2:3]], wl.nprobe, wl.t_prime, wl.k)
    say(f"[small] oracle on queries {rows.tolist()}")
    want = oracle.search_index(data, queries=data.queries[rows])
    compare(got, want, rows=rows, label="small")
    compare(got_few, want, label="small, sampled queries alone")
    compare(got_one, {key: v[2:3] for key, v in want.items()}, label="small, one query")
    for qi in rows:
        gap = check_real_valued(got["scores"][qi], got["counts"][qi], got["ids"][qi], index_arrays(data),
                                data.queries[qi], wl.nprobe, wl.t_prime)
        say(f"[small] query {qi}: largest relative gap to the fp64 scores {gap:.2e}")
    hit = (got["ids"][:, 0] == data.query_targets).mean()
    say(f"[small] target doc ranked first for {hit:.1%} of queries; mean scored/query "
        f"{got['n_scored'].mean():.3g}")


# ----------------------------------------------------------------------------- Eq. 1 literal

LITERAL_CASES = [
    # seed, n_centroids, n_docs, max_len, nbits, nprobe, t_prime, k: short documents and many probes
    # make fully retrieved documents common, so both branches of the literal rule occur
    (20, 12, 200, 4, 4, 6, 50, 40),
    (21, 30, 500, 6, 2, 10, 200, 60),
    (22, 64, 1000, 12, 4, 32, 1000, 100),
    (23, 8, 100, 3, 1, 8, 0, 30),   # every cluster probed: every candidate fully retrieved
]


@pytest.mark.parametrize("case", LITERAL_CASES, ids=[f"seed{c[0]}" for c in LITERAL_CASES])
def test_eq1_literal_scoring(case):
    seed, n_c, n_docs, max_len, nbits, nprobe, tp, k = case
    wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=n_docs, max_len=max_len, nbits=nbits,
                                     n_queries=4, n_qtok=32, nprobe=nprobe, t_prime=tp, k=k)
    data = synth.make_index(wl, workers=1)
    lit = run_both(data, label=f"literal seed {seed}", literal=True)
    paper = run_both(data, label=f"paper seed {seed}")
    if seed != 23:  # with partial retrieval the two readings must differ somewhere
        assert not np.array_equal(lit["fixed"], paper["fixed"])


def test_eq1_literal_tiny_and_switch_back():
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=3, nprobe=64, k=50),
                            workers=1)
    w = _engine()
    with w.Index.from_synthetic(data) as ix:
        ix.set_scoring(w.SCORING_EQ1_LITERAL)
        compare(ix.search_debug(data.queries, 64, 10_000, 50),
                oracle.search_index(data, k=50, flags=oracle.EQ1_LITERAL), label="tiny literal")
        ix.set_scoring(w.SCORING_PAPER)
        compare(ix.search_debug(data.queries, 64, 10_000, 50), oracle.search_index(data, k=50),
                label="tiny paper after literal")
        with pytest.raises(w.WarpError):
            ix.set_scoring(7)


def test_exact_halves_in_the_residual_term():
    # query values on a 2^-13 grid and bucket weights on a 2^-14 grid make every residual
    # term V = 2^17 sum_d k_d m_d, so V 2^-18 is an exact half whenever the sum is odd:
    # the engine must round those halves upward like the oracle
    wl = synth.random_small_workload(31, n_centroids=60, n_docs=500, max_len=14, nbits=4, n_queries=5,
                                     n_qtok=32, nprobe=12, t_prime=200, k=40)
    data = synth.make_index(wl, workers=1)
    data.bucket_weights = (np.round(data.bucket_weights.astype(np.float64) * 2 ** 14) / 2 ** 14).astype(np.float32)
    Q = (np.round(data.queries.astype(np.float64) * 0.999 * 2 ** 13) / 2 ** 13).astype(np.float32)
    k = np.round(Q.astype(np.float64) * 2 ** 13).astype(np.int64).reshape(-1, 128)
    m = np.round(data.bucket_weights.astype(np.float64) * 2 ** 14).astype(np.int64)
    per_dim = m[unpack_msb_first(data.codes[:200], data.nbits)]  # [200, 128]
    odd = ((k @ per_dim.T) % 2 != 0).mean()
    say(f"[halves] fraction of exact halves among sampled residual terms: {odd:.2f}")
    assert odd > 0.2
    run_both(data, queries=Q, label="exact halves")


@pytest.mark.parametrize("weight_scale", [1.0, 11.0], ids=["epochs", "resets"])
def test_consecutive_searches_reuse_the_token_max_table(weight_scale, monkeypatch):
    # Waves tag the token-max rows of each query slot with the slot's epoch, so a cell of an
    # earlier wave reads as absent and a slot's rows are zeroed only when its epochs run out
    # (7 of them for the tiny workload's weights); with bucket weights too large for a spare
    # bit (scaled by 11), the fold resets every cell instead. Every search of a sequence with
    # changing query counts (slots run out of epochs at different times) must match the
    # oracle: across several zeroings, around Eq.-1-literal searches (which reset cells, so
    # the table is zeroed before them), a search with 17 tokens per query (another layout of
    # the slots) and one with one query per wave (a 1 MiB scratch budget: several waves)
    w = _engine()
    data = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_queries=9), workers=1)
    data.bucket_weights = (data.bucket_weights * weight_scale).astype(np.float32)
    assert np.abs(data.bucket_weights).max() <= 1.99
    wl = data.workload
    rng = np.random.default_rng(5)
    sizes = [5, 2, 9, 1, 7, 7, 3, 9, 4, 6, 9, 2, 8, 1, 5, 9]
    with w.Index.from_synthetic(data) as ix:
        for j, n in enumerate(sizes):
            Q = data.queries[rng.permutation(9)[:n]]
            if j == 6:
                Q = np.ascontiguousarray(Q[:, :17])
            literal = j in (3, 12)
            ix.set_scoring(w.SCORING_EQ1_LITERAL if literal else w.SCORING_PAPER)
            if j == 9:
                monkeypatch.setenv("WARP_SCRATCH_MB", "1")
            if j == 11:
                monkeypatch.delenv("WARP_SCRATCH_MB")
            say(f"[table x{weight_scale}] search {j}: {n} queries, literal={literal}")
            got = ix.search_debug(Q, wl.nprobe, wl.t_prime, wl.k)
            want = oracle.search_index(data, queries=Q, nprobe=wl.nprobe, t_prime=wl.t_prime, k=wl.k,
                                       flags=oracle.EQ1_LITERAL if literal else 0)
            compare(got, want, label=f"table x{weight_scale} search {j}")


# ----------------------------------------------------------------------------- top-k

def _tied_index(seed=21, n_tied=5000, n_other=1000, nbits=2):
    """n_tied documents with one identical embedding each (equal scores, so the k-th
    key sits in a tie far wider than the gather buffer) and n_other documents with
    random codes in two other clusters."""
    rng = np.random.default_rng(seed)
    C = rng.standard_normal((4, 128))
    C = (C / np.linalg.norm(C, axis=1, keepdims=True)).astype(np.float32)
    other = rng.integers(1, 3, n_other)
    order = np.argsort(other, kind="stable")
    clusters = np.concatenate([np.zeros(n_tied, np.int64), other[order]])
    doc_ids = np.concatenate([rng.permutation(n_tied), n_tied + order]).astype(np.int32)
    per_dim = np.zeros((n_tied + n_other, 128), np.int64)
    per_dim[n_tied:] = rng.integers(0, 1 << nbits, (n_other, 128))
    from helpers import pack_msb_first
    offsets = np.zeros(5, np.int64)
    np.cumsum(np.bincount(clusters, minlength=4), out=offsets[1:])
    w = np.array([-0.05, -0.01, 0.01, 0.05], np.float32)
    Q = rng.standard_normal((3, 8, 128))
    Q = (Q / np.linalg.norm(Q, axis=2, keepdims=True)).astype(np.float32)
    return dict(centroids=C, offsets=offsets, doc_ids=doc_ids, codes=pack_msb_first(per_dim, nbits),
                nbits=nbits, bucket_weights=w, n_docs=n_tied + n_other), Q


@pytest.mark.parametrize("cap", [None, "1", "0"], ids=["pruned", "cap1", "unpruned"])
def test_topk_ties_and_block_pruning(cap, monkeypatch):
    """The top-k's pruned passes (blocks whose best key can reach the k-th), its
    fallback to every block, and its exact radix select inside a wide tie."""
    w = _engine()
    if cap is not None:
        monkeypatch.setenv("WARP_TOPK_LIST_BLOCKS", cap)
    arrays, Q = _tied_index()
    for k in (4096, 100, 1):
        say(f"[topk ties cap={cap}] k={k}")
        with w.Index(**arrays) as ix:
            got = ix.search_debug(Q, 4, 0, k)
        want = oracle.search(queries=Q, nprobe=4, t_prime=0, k=k, **arrays)
        compare(got, want, label=f"ties cap={cap} k={k}")
    wl = synth.random_small_workload(8, n_centroids=300, n_docs=5000, max_len=30, nbits=4, n_queries=3,
                                     n_qtok=32, nprobe=256, t_prime=2000, k=4096)
    run_both(synth.make_index(wl, workers=1), label=f"seed 8 cap={cap}")
