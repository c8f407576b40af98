"""The synthetic workload generator: determinism, layout and quantisation."""
import numpy as np
import pytest

import synth
from helpers import cluster_of_embeddings, pack_msb_first, unpack_msb_first


def _small(seed=0, **kw):
    return synth.make_index(synth.random_small_workload(seed, **kw), workers=1)


def test_deterministic_per_seed():
    a, b = _small(1), _small(1)
    for key in ("centroids", "offsets", "doc_ids", "codes", "bucket_weights", "queries"):
        np.testing.assert_array_equal(getattr(a, key), getattr(b, key))
    c = _small(2)
    assert not np.array_equal(a.centroids, c.centroids)


def test_parallel_generation_matches_serial():
    w = synth.with_overrides(synth.WORKLOADS["tiny"], n_docs=5000)
    a = synth.make_index(w, workers=1)
    b = synth.make_index(w, workers=3)
    for key in ("offsets", "doc_ids", "codes", "queries"):
        np.testing.assert_array_equal(getattr(a, key), getattr(b, key))


@pytest.mark.parametrize("nbits", [1, 2, 4, 8])
def test_packing_matches_independent_packer(nbits):
    rng = np.random.default_rng(nbits)
    per_dim = rng.integers(0, 1 << nbits, size=(7, 128))
    packed = synth.pack_codes(per_dim, nbits)
    np.testing.assert_array_equal(packed, pack_msb_first(per_dim, nbits))
    np.testing.assert_array_equal(unpack_msb_first(packed, nbits), per_dim)


def test_layout_and_quantisation():
    idx = synth.make_index(synth.WORKLOADS["tiny"], workers=1)
    w = idx.workload
    assert idx.offsets[0] == 0 and np.all(np.diff(idx.offsets) >= 0)
    assert idx.n_embeddings == idx.doc_lengths.sum() == len(idx.doc_ids) == len(idx.codes)
    assert idx.doc_lengths.min() >= 16 and idx.doc_lengths.max() <= 48
    assert np.allclose(np.linalg.norm(idx.centroids, axis=1), 1, atol=1e-6)
    assert np.allclose(np.linalg.norm(idx.queries, axis=-1), 1, atol=1e-6)
    # docs ascending inside every cluster
    cl = cluster_of_embeddings(idx.offsets)
    key = cl.astype(np.int64) * (1 << 32) + idx.doc_ids
    assert np.all(np.diff(key) >= 0)
    # every doc's embeddings are all present
    np.testing.assert_array_equal(np.bincount(idx.doc_ids, minlength=w.n_docs), idx.doc_lengths)
    # codes decode to the bucket that holds the residual: regenerate some tokens
    assert np.all(np.diff(idx.bucket_weights) > 0) and np.all(np.diff(idx.bucket_cutoffs) > 0)
    # Zipf skew: the largest cluster holds a large share
    assert np.diff(idx.offsets).max() > 0.05 * idx.n_embeddings
    # queries are noisy copies of tokens of their target document
    assert idx.queries.shape == (1, 32, 128)


def test_codes_quantise_the_residuals():
    w = synth.random_small_workload(5, n_docs=30, n_centroids=8)
    idx = synth.make_index(w, workers=1)
    # regenerate the fp32 tokens in generation order (docs in order) and map to sorted order
    n = idx.n_embeddings
    x = synth.token_vectors(w, np.arange(n))
    cl_gen = np.empty(n, np.int64)
    # generation order -> cluster-sorted order is a stable sort by cluster; rebuild it
    doc_gen = np.repeat(np.arange(w.n_docs), idx.doc_lengths)
    C = idx.centroids
    # the cluster of a generated token is the one whose residual codes match; recover it
    # through the stored layout: within a cluster, docs ascend and generation order is kept
    cl_sorted = cluster_of_embeddings(idx.offsets)
    order = np.lexsort((np.arange(n), doc_gen))  # generation order is already doc order
    assert np.all(order == np.arange(n))
    # rebuild the permutation: for each cluster, its embeddings in generation order
    dec = unpack_msb_first(idx.codes, w.nbits)
    lo = np.r_[-np.inf, idx.bucket_cutoffs]
    hi = np.r_[idx.bucket_cutoffs, np.inf]
    # match every stored embedding to a generated token of the same doc whose residual
    # falls in the decoded buckets for every dimension
    used = np.zeros(n, bool)
    for e in range(n):
        d = idx.doc_ids[e]
        cands = np.flatnonzero((doc_gen == d) & ~used)
        ok = False
        for g in cands:
            r = x[g] - C[cl_sorted[e]]
            if np.all((r >= lo[dec[e]]) & (r < hi[dec[e]])):
                used[g] = True
                cl_gen[g] = cl_sorted[e]
                ok = True
                break
        assert ok, f"embedding {e} matches no generated token"
