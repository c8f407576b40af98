"""Pins of the CPU oracle against what the paper and the mathematics fix.

O1  explicit decompression followed by a dot product equals the implicit
    selective sum (Section 4.4, Eq. decompress and Eq. warp_selective_sum);
O2  nprobe = all clusters makes every (doc, token) pair retrieved, so the
    search equals exhaustive MaxSim over decompressed vectors (Eq. 1 with A = 1);
O3  WARP_SELECT's estimate (Section 4.3) equals the size-weighted order
    statistic max{s : sum of sizes scoring >= s exceeds t'} and its special cases;
O4  the recursive stride merge of Section 4.5 (Eq. merge_strides with
    Eq. doc_level_reduce, any split point) equals the oracle's document sums;
O5  the two readings of imputation coincide when m_i is the smallest retrieved
    score (XTR's estimate), and the literal Eq. 1 reading never scores lower; a
    hand-worked example (tests/golden/eq1_literal_example.json) fixes both
    readings exactly, including a fully retrieved document whose best score is
    below m_i and a partly retrieved one, and oracle copies with the literal
    reading's count test changed are caught by it;
O6  results do not depend on the order of embeddings inside a cluster nor on
    centroid labels;
O7  a hand-built dyadic example whose outputs were worked out by hand.
"""
from __future__ import annotations

import math
import random

import numpy as np
import pytest

import oracle
import synth
from helpers import (FRAC, bruteforce_maxsim, check_real_valued, cluster_of_embeddings, explicit_decompress,
                     load_dyadic, realvalued_doc_scores, topp_by_score, unpack_msb_first,
                     weighted_order_statistic)



def tok_tol(q, w):
    """Largest gap between a fixed-point token score and the real-valued one.

    Each product q_d * w uses q_d and w rounded to 2^-22 (error at most
    (|q_d| + |w|) 2^-23 + 2^-46 per dimension); the centroid term and the summed
    residual term are each rounded once to 2^-26.
    """
    q = np.asarray(q, np.float64)
    return ((np.abs(q).sum() + q.size * float(np.abs(w).max())) * 2.0 ** -23
            + q.size * 2.0 ** -46 + 2 * 2.0 ** -27)


def doc_tol(Q, w):
    """A document score sums one token score (or estimate) per query token."""
    return sum(tok_tol(q, w) for q in Q)


def _index(seed=0, **kw):
    return synth.make_index(synth.random_small_workload(seed, **kw), workers=1)


# ----------------------------------------------------------------------------- O7

@pytest.mark.parametrize("case", range(8))
def test_o7_dyadic_example(case):
    g, ix, Q = load_dyadic()
    c = g["cases"][case]
    r = oracle.search(queries=Q, nprobe=c["nprobe"], t_prime=c["t_prime"], k=c["k"], **ix)
    assert r["ids"].tolist() == c["ids"]
    assert r["counts"].tolist() == c["counts"]
    assert r["sel"].tolist() == c["sel"]
    assert (r["m_fixed"] / FRAC).tolist() == c["m"]
    assert r["n_scored"].tolist() == c["n_scored"]
    for qi in range(len(Q)):
        want = [None if v is None else v for v in c["scores"][qi]]
        got_fixed = r["fixed"][qi].tolist()
        got = r["scores"][qi].tolist()
        for w, f, s in zip(want, got_fixed, got):
            if w is None:
                assert f == np.iinfo(np.int64).min and s == -math.inf
            else:
                assert f == int(w * FRAC) and s == w
        bm = r["cand_bitmap"][qi]
        cands = [d for d in range(g["n_docs"]) if (bm[d >> 5] >> (d & 31)) & 1]
        assert cands == c["candidates"][qi]


# ----------------------------------------------------------------------------- O1

@pytest.mark.parametrize("nbits", [1, 2, 4, 8])
def test_o1_explicit_equals_implicit(nbits):
    idx = _index(1, nbits=nbits, n_centroids=8, n_docs=60)
    X = explicit_decompress(idx.centroids, idx.offsets, idx.codes, nbits, idx.bucket_weights)
    cl = cluster_of_embeddings(idx.offsets)
    for q in idx.queries.reshape(-1, 128)[:4]:
        S = oracle.centroid_scores(idx.centroids, q)
        # S64 against a library matrix product in fp64
        np.testing.assert_allclose(S, idx.centroids.astype(np.float64) @ q.astype(np.float64),
                                   rtol=0, atol=1e-12)
        direct = X @ q.astype(np.float64)
        per_dim = unpack_msb_first(idx.codes, nbits)
        selective = S[cl] + (idx.bucket_weights.astype(np.float64)[per_dim] * q).sum(axis=1)
        np.testing.assert_allclose(direct, selective, rtol=0, atol=1e-12)
        for c in range(len(idx.offsets) - 1):
            e0, e1 = int(idx.offsets[c]), int(idx.offsets[c + 1])
            t = oracle.token_scores(q, S[c], idx.codes, nbits, idx.bucket_weights, e0, e1)
            assert np.all(np.abs(t / FRAC - direct[e0:e1]) <= tok_tol(q, idx.bucket_weights))


def test_o1_planted_mistake_is_caught():
    """A wrong bit order in the unpacking (a plausible oracle bug) breaks O1."""
    idx = _index(2, nbits=4, n_centroids=4, n_docs=30)
    X = explicit_decompress(idx.centroids, idx.offsets, idx.codes, 4, idx.bucket_weights)
    q = idx.queries[0, 0]
    S = oracle.centroid_scores(idx.centroids, q)
    swapped = idx.codes.copy()
    swapped = ((swapped >> 4) | (swapped << 4)).astype(np.uint8)  # nibble order flipped
    e1 = int(idx.offsets[1])
    t = oracle.token_scores(q, S[0], swapped, 4, idx.bucket_weights, 0, e1)
    assert np.any(np.abs(t / FRAC - X[:e1] @ q.astype(np.float64)) > tok_tol(q, idx.bucket_weights))


# ----------------------------------------------------------------------------- O2

def _check_against_bruteforce(idx, r, k):
    X = explicit_decompress(idx.centroids, idx.offsets, idx.codes, idx.nbits, idx.bucket_weights)
    for qi, Q in enumerate(idx.queries):
        docs, bf = bruteforce_maxsim(X, idx.doc_ids, idx.n_docs, Q)
        bf_of = dict(zip(docs.tolist(), bf.tolist()))
        DOC_TOL = doc_tol(Q, idx.bucket_weights)
        n = int(r["counts"][qi])
        assert n == min(k, len(docs))
        ids = r["ids"][qi, :n]
        # every reported score is the exhaustive MaxSim score of that doc
        for d, f in zip(ids.tolist(), r["fixed"][qi, :n].tolist()):
            assert abs(f / FRAC - bf_of[d]) <= DOC_TOL
        # reported order agrees with the exhaustive scores up to rounding
        got = np.array([bf_of[d] for d in ids.tolist()])
        assert np.all(np.diff(got) <= 2 * DOC_TOL)
        # nothing left out scores clearly better than the last reported doc
        rest = np.array([bf_of[d] for d in docs.tolist() if d not in set(ids.tolist())])
        if n == k and len(rest):
            assert rest.max() <= got[-1] + 2 * DOC_TOL
        # and the candidate set is every doc with an embedding
        bm = r["cand_bitmap"][qi]
        cands = np.flatnonzero([(bm[d >> 5] >> (d & 31)) & 1 for d in range(idx.n_docs)])
        assert cands.tolist() == sorted(docs.tolist())


@pytest.mark.parametrize("seed,nbits", [(3, 4), (4, 2), (5, 4)])
def test_o2_all_clusters_equals_bruteforce_maxsim(seed, nbits):
    idx = _index(seed, nbits=nbits, n_centroids=12, n_docs=80, n_queries=3, n_qtok=6)
    k = 20
    r = oracle.search_index(idx, nprobe=12, t_prime=0, k=k)
    _check_against_bruteforce(idx, r, k)


def test_o2_tiny_workload_all_clusters():
    idx = synth.make_index(synth.with_overrides(synth.WORKLOADS["tiny"], n_docs=300,
                                                n_centroids=64), workers=1)
    r = oracle.search_index(idx, nprobe=64, t_prime=0, k=50)
    _check_against_bruteforce(idx, r, 50)


def test_o2_planted_mistake_is_caught():
    """Dropping the centroid term (a plausible oracle bug) fails the brute-force check."""
    idx = _index(6, nbits=4, n_centroids=6, n_docs=40, n_queries=1, n_qtok=4)
    shifted = idx.centroids.copy() * 0  # oracle fed zero centroids == centroid term dropped
    r = oracle.search(shifted, idx.offsets, idx.doc_ids, idx.codes, 4, idx.bucket_weights,
                      idx.n_docs, idx.queries, 6, 0, 10)
    with pytest.raises(AssertionError):
        _check_against_bruteforce(idx, r, 10)


def test_o2_realvalued_reference_agrees_with_oracle():
    """The fp64 explicit-decompression reference that the GPU tests apply to returned
    documents (helpers.realvalued_doc_scores, which recomputes selection and m_i in numpy)
    agrees with the oracle's fixed-point scores within the rounding bound, in both scoring
    readings, at nprobe below the number of clusters (so imputation takes part)."""
    for seed, literal in ((40, False), (41, True), (42, False)):
        idx = _index(seed, n_centroids=24, n_docs=120, n_queries=3, n_qtok=8, nprobe=5, t_prime=40, k=25)
        w = idx.workload
        r = oracle.search_index(idx, flags=oracle.EQ1_LITERAL if literal else 0)
        arrays = dict(centroids=idx.centroids, offsets=idx.offsets, doc_ids=idx.doc_ids, codes=idx.codes,
                      nbits=idx.nbits, bucket_weights=idx.bucket_weights, n_docs=idx.n_docs)
        for qi, Q in enumerate(idx.queries):
            n = int(r["counts"][qi])
            ref = realvalued_doc_scores(Q=Q, docs=r["ids"][qi, :n], nprobe=w.nprobe, t_prime=w.t_prime,
                                        literal=literal, **arrays)
            # the estimate m_i enters as R(m_i) in the oracle: one more 2^-27 per token
            bound = doc_tol(Q, idx.bucket_weights) + len(Q) * 2.0 ** -27
            assert np.all(np.abs(r["fixed"][qi, :n] / FRAC - ref) <= bound)
            assert check_real_valued(r["scores"][qi], n, r["ids"][qi], arrays, Q, w.nprobe, w.t_prime,
                                     literal=literal) <= 1e-4


# ----------------------------------------------------------------------------- O3

def _random_scores(rng, n, ties):
    s = rng.standard_normal(n) * 0.1
    if ties:
        s = np.round(s * 20) / 20  # many exact ties
    return s


@pytest.mark.parametrize("seed", range(12))
def test_o3_select_matches_definitions(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60))
    scores = _random_scores(rng, n, ties=seed % 2 == 0)
    sizes = rng.integers(0, 5, n) * (rng.random(n) < 0.8)
    offsets = np.r_[0, np.cumsum(sizes)].astype(np.int64)
    N = int(offsets[-1])
    nprobe = int(rng.integers(1, n + 1))
    for t_prime in sorted({0, max(N - 1, 0), N, N + 5, int(rng.integers(0, N + 1))}):
        sel, m = oracle.select(scores, offsets, nprobe, t_prime)
        assert sel.tolist() == topp_by_score(scores, nprobe).tolist()
        assert m == weighted_order_statistic(scores, sizes, t_prime)


def test_o3_special_cases():
    scores = np.array([0.5, 0.9, 0.1, 0.9, -0.3, 0.2])
    sizes = np.array([3, 0, 2, 4, 1, 0])
    offsets = np.r_[0, np.cumsum(sizes)].astype(np.int64)
    N = int(sizes.sum())
    order = topp_by_score(scores, len(scores))           # 1, 3, 0, 5, 2, 4
    nonempty = [c for c in order if sizes[c] > 0]
    _, m = oracle.select(scores, offsets, 1, 0)
    assert m == scores[nonempty[0]]                       # t' = 0: first non-empty centroid
    _, m = oracle.select(scores, offsets, 1, N - 1)
    assert m == scores[nonempty[-1]]                      # t' = N - 1: last non-empty
    _, m = oracle.select(scores, offsets, 1, N)
    assert m == scores.min()                              # never exceeded: lowest score
    # inclusive cumulative sizes in order 1, 3, 0, 5, 2, 4 are 0, 4, 7, 7, 9, 10
    assert oracle.select(scores, offsets, 1, 3)[1] == 0.9    # 4 > 3 at centroid 3
    assert oracle.select(scores, offsets, 1, 4)[1] == 0.5    # strict: 4 is not > 4; 7 > 4 at centroid 0
    assert oracle.select(scores, offsets, 1, 7)[1] == 0.1    # 7, 7 not > 7; 9 > 7 at centroid 2


def test_o3_planted_mistake_is_caught():
    """A non-strict comparison (>= t') would pick an earlier centroid: the pin sees it."""
    scores = np.array([0.9, 0.5, 0.1])
    sizes = np.array([2, 2, 2])
    # with '>=' the answer for t'=2 would be 0.9; the definition gives 0.5
    assert weighted_order_statistic(scores, sizes, 2) == 0.5
    offsets = np.r_[0, np.cumsum(sizes)].astype(np.int64)
    assert oracle.select(scores, offsets, 1, 2)[1] == 0.5


# ----------------------------------------------------------------------------- O4

def _merge_strides(strides, m, lo, hi, rnd):
    """Section 4.5: S_{lo,hi} = reduce(r_doc,(lo,k,hi), S_{lo,k}, S_{k+1,hi}) for a random k."""
    if lo == hi:
        return dict(strides[lo])
    k = rnd.randint(lo, hi - 1)
    a = _merge_strides(strides, m, lo, k, rnd)
    b = _merge_strides(strides, m, k + 1, hi, rnd)
    m_left = sum(m[lo:k + 1])
    m_right = sum(m[k + 1:hi + 1])
    out = {}
    for key in set(a) | set(b):
        if key in a and key in b:
            out[key] = a[key] + b[key]
        elif key in a:
            out[key] = a[key] + m_right
        else:
            out[key] = m_left + b[key]
    return out


@pytest.mark.parametrize("seed", range(4))
def test_o4_stride_merge_equals_doc_sums(seed):
    idx = _index(10 + seed, nbits=2 + 2 * (seed % 2), n_centroids=10, n_docs=50, n_queries=2,
                 n_qtok=7, nprobe=3, t_prime=15)
    w = idx.workload
    r = oracle.search_index(idx, doc_scores=True)
    rnd = random.Random(seed)
    for qi, Q in enumerate(idx.queries):
        m = r["m_fixed"][qi].tolist()
        strides = []
        for i, q in enumerate(Q):
            S = oracle.centroid_scores(idx.centroids, q)
            stride = {}
            for c in r["sel"][qi, i].tolist():   # r_tok over the nprobe strides
                e0, e1 = int(idx.offsets[c]), int(idx.offsets[c + 1])
                t = oracle.token_scores(q, S[c], idx.codes, idx.nbits, idx.bucket_weights, e0, e1)
                for d, v in zip(idx.doc_ids[e0:e1].tolist(), t.tolist()):
                    stride[d] = max(stride[d], v) if d in stride else v
            strides.append(stride)
        for _ in range(3):
            merged = _merge_strides(strides, m, 0, w.n_qtok - 1, rnd)
            doc_fixed = r["doc_fixed"][qi]
            present = np.flatnonzero(doc_fixed != np.iinfo(np.int64).min)
            assert sorted(merged) == present.tolist()
            for d, v in merged.items():
                assert doc_fixed[d] == v


# ----------------------------------------------------------------------------- O5

@pytest.mark.parametrize("seed", range(3))
def test_o5_readings_coincide_with_min_retrieved_estimate(seed):
    idx = _index(20 + seed, n_centroids=10, n_docs=60, n_qtok=6, nprobe=3, t_prime=10)
    a = oracle.search_index(idx, flags=oracle.M_MIN_RETRIEVED, doc_scores=True)
    b = oracle.search_index(idx, flags=oracle.M_MIN_RETRIEVED | oracle.EQ1_LITERAL, doc_scores=True)
    for key in ("ids", "fixed", "counts", "doc_fixed"):
        np.testing.assert_array_equal(a[key], b[key])
    # with WARP's t' estimate the literal reading can only raise a doc's score
    a = oracle.search_index(idx, doc_scores=True)
    b = oracle.search_index(idx, flags=oracle.EQ1_LITERAL, doc_scores=True)
    assert np.all(b["doc_fixed"] >= a["doc_fixed"])


EQ1_CASES = range(4)


def _eq1_expected_check(r, c, mode, n_docs):
    want = c[mode]
    assert r["ids"].tolist() == want["ids"], (c["name"], mode)
    assert r["counts"].tolist() == want["counts"]
    for qi in range(len(want["ids"])):
        for w, f, s in zip(want["scores"][qi], r["fixed"][qi].tolist(), r["scores"][qi].tolist()):
            if w is None:
                assert f == np.iinfo(np.int64).min and s == -math.inf
            else:
                assert f == int(w * FRAC) and s == w, (c["name"], mode, w, f)
    assert r["sel"].tolist() == c["sel"]
    assert (r["m_fixed"] / FRAC).tolist() == c["m"]
    assert r["n_scored"].tolist() == c["n_scored"]
    for qi, bm in enumerate(r["cand_bitmap"]):
        assert [d for d in range(n_docs) if (bm[d >> 5] >> (d & 31)) & 1] == c["candidates"][qi]


@pytest.mark.parametrize("case", EQ1_CASES)
@pytest.mark.parametrize("mode", ["paper", "eq1_literal"])
def test_o5_eq1_literal_hand_worked(case, mode):
    g, ix, Q = load_dyadic("eq1_literal_example.json")
    assert np.bincount(ix["doc_ids"], minlength=g["n_docs"]).tolist() == g["doc_lengths"]
    c = g["cases"][case]
    flags = oracle.EQ1_LITERAL if mode == "eq1_literal" else 0
    r = oracle.search(queries=Q, nprobe=c["nprobe"], t_prime=c["t_prime"], k=c["k"], flags=flags, **ix)
    _eq1_expected_check(r, c, mode, g["n_docs"])


# The literal reading's test "some embedding of the document was not retrieved for this
# token" (retrieved count below the document's embedding count), and two plausible slips.
_COUNT_TEST = "seen && seen[(int64_t)i * n_docs + doc] < a->doc_len[doc]"
_MUTANTS = {
    "unchanged (control)": _COUNT_TEST,
    "count test <=": _COUNT_TEST.replace(" < a->", " <= a->"),
    "count test dropped": "seen",
}


@pytest.mark.parametrize("mutant", sorted(_MUTANTS))
def test_o5_eq1_literal_mutants_are_caught(mutant, tmp_path):
    """A copy of the oracle with the count test changed fails the hand-worked literal cases;
    the unchanged copy, built the same way, passes them."""
    src = open(oracle.SRC).read()
    assert src.count(_COUNT_TEST) == 1, "the oracle's count test moved; update the mutants"
    lib = oracle.load_library(oracle.build_variant(src.replace(_COUNT_TEST, _MUTANTS[mutant]), str(tmp_path)))
    g, ix, Q = load_dyadic("eq1_literal_example.json")
    caught = False
    for c in g["cases"]:
        r = oracle.search(queries=Q, nprobe=c["nprobe"], t_prime=c["t_prime"], k=c["k"],
                          flags=oracle.EQ1_LITERAL, lib=lib, **ix)
        try:
            _eq1_expected_check(r, c, "eq1_literal", g["n_docs"])
        except AssertionError:
            caught = True
    if mutant.startswith("unchanged"):
        assert not caught
    else:
        assert caught, f"mutant '{mutant}' passes the hand-worked literal cases"


# ----------------------------------------------------------------------------- O6

def test_o6_invariances():
    idx = _index(30, n_centroids=12, n_docs=70, n_qtok=5, nprobe=4, t_prime=20, k=15)
    base = oracle.search_index(idx)
    rng = np.random.default_rng(0)
    # permute embeddings inside every cluster
    perm = np.concatenate([rng.permutation(np.arange(a, b))
                           for a, b in zip(idx.offsets[:-1], idx.offsets[1:])]).astype(np.int64)
    r = oracle.search(idx.centroids, idx.offsets, idx.doc_ids[perm], idx.codes[perm], idx.nbits,
                      idx.bucket_weights, idx.n_docs, idx.queries, 4, 20, 15)
    for key in ("ids", "fixed", "counts", "sel", "m_fixed", "n_scored", "cand_bitmap"):
        np.testing.assert_array_equal(base[key], r[key])
    # relabel centroids (new label of old centroid c is lab[c])
    n_c = len(idx.offsets) - 1
    lab = rng.permutation(n_c)
    inv = np.argsort(lab)
    sizes = np.diff(idx.offsets)
    new_off = np.r_[0, np.cumsum(sizes[inv])].astype(np.int64)
    blocks = [np.arange(idx.offsets[c], idx.offsets[c + 1]) for c in inv]
    e = np.concatenate(blocks).astype(np.int64)
    r = oracle.search(idx.centroids[inv], new_off, idx.doc_ids[e], idx.codes[e], idx.nbits,
                      idx.bucket_weights, idx.n_docs, idx.queries, 4, 20, 15)
    for key in ("ids", "fixed", "counts", "m_fixed", "n_scored", "cand_bitmap"):
        np.testing.assert_array_equal(base[key], r[key])
    np.testing.assert_array_equal(lab[base["sel"]], r["sel"])


# ----------------------------------------------------------------------------- O8

def test_o8_residual_rounding_of_exact_halves():
    """Token score = R(S64) + floor(V 2^-18 + 1/2), halves upward (reading 11).

    q_0 = 2^-13 and bucket weight m 2^-14 quantise exactly to 2^9 and m 2^8, so an
    embedding whose dimension 0 takes that bucket (every other q_d = 0) has
    V = m 2^17: V 2^-18 = m / 2. Worked by hand for m = 1, 3, -1, -3, 2, 0:
    0.5 -> 1, 1.5 -> 2, -0.5 -> 0, -1.5 -> -1, 1 -> 1, 0 -> 0 (half to even would
    give 0, 2, 0, -2, 1, 0).
    """
    m = [1, 3, -1, -3, 2, 0]
    w = np.zeros(16, np.float32)
    w[:len(m)] = np.asarray(m, np.float64) * 2.0 ** -14
    q = np.zeros(128, np.float32)
    q[0] = 2.0 ** -13
    codes = np.zeros((len(m), 64), np.uint8)
    codes[:, 0] = np.arange(len(m), dtype=np.uint8) << 4  # dimension 0 is the high nibble of byte 0
    t = oracle.token_scores(q, 0.0, codes, 4, w, 0, len(m))
    assert t.tolist() == [1, 2, 0, -1, 1, 0]
    # the centroid term R(2^-26) = 1 is added to the rounded residual term
    t = oracle.token_scores(q, 2.0 ** -26, codes, 4, w, 0, len(m))
    assert t.tolist() == [2, 3, 1, 0, 2, 1]
