"""Pins of the oracle's index construction (Section 4.1) against numpy and closed forms.

B0  the starting centroids are the starting vectors normalised (numpy fp64, sequential sum of
    squares), and a zero vector is rejected;
B1  assignment is the fp64 argmax over centroids (numpy matrix product);
B2  one k-means step gives the normalised mean direction of each centroid's tokens
    (numpy, float64), and keeps centroids without tokens;
B3  the spherical k-means objective never decreases over iterations;
B4  cutoffs and weights are numpy's inverted-CDF quantiles of the residual components;
B5  codes are numpy's searchsorted of the residuals in the cutoffs, packed MSB-first;
    the layout is a stable sort by cluster with matching offsets;
B6  well-separated clusters are recovered exactly.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import synth
from helpers import unpack_msb_first


def _inputs(seed=0, n_docs=120, max_len=20, n_c=24):
    wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=n_docs, max_len=max_len, nbits=4)
    data = synth.make_index(wl, with_queries=False, workers=1)
    lens = data.doc_lengths.astype(np.int64)
    X = synth.token_vectors(data.workload, np.arange(int(lens.sum())))
    docs = np.repeat(np.arange(len(lens)), lens).astype(np.int32)
    return X, docs, lens


def _init(X, sample, n_c, seed=1):
    rng = np.random.default_rng(seed)
    pick = np.sort(rng.choice(len(sample), size=n_c, replace=False))
    C = X[sample[pick]].astype(np.float64)
    return (C / np.linalg.norm(C, axis=1, keepdims=True)).astype(np.float32)


def _objective(X, C):
    return float((X.astype(np.float64) @ C.astype(np.float64).T).max(axis=1).sum())


def test_b0_starting_centroids_are_normalised_inputs():
    X, docs, _ = _inputs(3)
    sample = np.arange(0, len(X), 4)
    rng = np.random.default_rng(9)
    V = (rng.standard_normal((20, 128)) * rng.uniform(0.1, 3.0, (20, 1))).astype(np.float32)
    r = oracle.build_index(X, docs, V, sample, iterations=0, nbits=2, n_quant=100)
    V64 = V.astype(np.float64)
    norm = np.sqrt(np.cumsum(V64 * V64, axis=1)[:, -1])  # sum of squares in dimension order
    np.testing.assert_array_equal(r["centroids"], (V64 / norm[:, None]).astype(np.float32))
    assert np.all(np.abs(np.linalg.norm(r["centroids"].astype(np.float64), axis=1) - 1) < 1e-6)
    V[3] = 0
    with pytest.raises(ValueError):
        oracle.build_index(X, docs, V, sample, iterations=0, nbits=2, n_quant=100)


def test_b1_assignment_is_argmax():
    X, docs, _ = _inputs(0)
    sample = np.arange(0, len(X), 3)
    C0 = _init(X, sample, 24)
    r = oracle.build_index(X, docs, C0, sample, iterations=2, nbits=2, n_quant=200)
    S = X.astype(np.float64) @ r["centroids"].astype(np.float64).T
    best = S.max(axis=1)
    got = S[np.arange(len(X)), r["assign"]]
    assert np.all(got >= best - 1e-12)
    clear = (np.sort(S, axis=1)[:, -2] < best - 1e-9)  # no near tie
    assert np.array_equal(r["assign"][clear], S.argmax(axis=1)[clear])


def test_b2_one_kmeans_step_is_the_mean_direction():
    X, docs, _ = _inputs(1)
    sample = np.arange(0, len(X), 2)
    n_c = 40
    C0 = _init(X, sample, n_c)
    C0[5] = C0[4]  # a duplicate centroid: ties go to the lower id, so centroid 5 keeps no token
    r = oracle.build_index(X, docs, C0, sample, iterations=1, nbits=4, n_quant=100)
    Xs = X[sample].astype(np.float64)
    a = (Xs @ C0.astype(np.float64).T).argmax(axis=1)
    for c in range(n_c):
        members = Xs[a == c]
        if len(members) == 0:
            assert np.array_equal(r["centroids"][c], C0[c])
            continue
        m = members.sum(axis=0)
        np.testing.assert_allclose(r["centroids"][c], m / np.linalg.norm(m), rtol=0, atol=2e-7)
    assert np.array_equal(r["centroids"][5], C0[5])


def test_b3_objective_never_decreases():
    X, docs, _ = _inputs(2)
    sample = np.arange(0, len(X), 2)
    C0 = _init(X, sample, 32)
    prev = -np.inf
    for it in range(6):
        r = oracle.build_index(X, docs, C0, sample, iterations=it, nbits=2, n_quant=50)
        obj = _objective(X[sample], r["centroids"])
        assert obj >= prev - 1e-6
        prev = obj


@pytest.mark.parametrize("nbits", [1, 2, 4, 8])
def test_b4_b5_quantiles_codes_layout(nbits):
    X, docs, _ = _inputs(3)
    sample = np.arange(0, len(X), 2)
    C0 = _init(X, sample, 24)
    n_quant = 300
    r = oracle.build_index(X, docs, C0, sample, iterations=2, nbits=nbits, n_quant=n_quant)
    C, a = r["centroids"], r["assign"]
    R = X - C[a]  # float32 residuals, as in the definition
    comp = np.sort(R[:n_quant].ravel())
    nb = 1 << nbits
    want_cut = np.quantile(comp, np.arange(1, nb) / nb, method="inverted_cdf").astype(np.float32)
    want_w = np.quantile(comp, (2 * np.arange(nb) + 1) / (2 * nb), method="inverted_cdf").astype(np.float32)
    assert np.array_equal(r["cutoffs"], want_cut)
    assert np.array_equal(r["weights"], want_w)
    perm = np.argsort(a, kind="stable")
    assert np.array_equal(r["doc_ids"], docs[perm])
    assert np.array_equal(r["offsets"], np.concatenate([[0], np.cumsum(np.bincount(a, minlength=len(C)))]))
    codes = unpack_msb_first(r["codes"], nbits)
    want_codes = np.searchsorted(r["cutoffs"], R[perm], side="right")
    assert np.array_equal(codes, want_codes)


def test_b6_recovers_separated_clusters():
    rng = np.random.default_rng(7)
    K, per = 12, 60
    centers = rng.standard_normal((K, 128))
    centers /= np.linalg.norm(centers, axis=1, keepdims=True)
    truth = np.repeat(np.arange(K), per)
    X = centers[truth] + 0.03 * rng.standard_normal((K * per, 128))
    X = (X / np.linalg.norm(X, axis=1, keepdims=True)).astype(np.float32)
    order = rng.permutation(len(X))
    X, truth = X[order], truth[order]
    docs = np.arange(len(X), dtype=np.int32) // 6
    sample = np.arange(len(X))
    C0 = np.stack([X[np.nonzero(truth == k)[0][0]] for k in range(K)])  # one token of each cluster
    r = oracle.build_index(X, docs, C0, sample, iterations=3, nbits=2, n_quant=100)
    # the partition equals the true one (up to labels), and centroids approach the centers
    pairs = {(int(t), int(c)) for t, c in zip(truth, r["assign"])}
    assert len(pairs) == K and len({c for _, c in pairs}) == K
    for t, c in pairs:
        assert float(centers[t] @ r["centroids"][c]) > 0.995  # mean of 60 tokens with noise norm 0.34
