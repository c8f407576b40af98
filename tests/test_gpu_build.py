"""Index construction on the MI355X against the oracle (Section 4.1), bit for bit:
centroids after k-means, assignment, offsets, document ids, packed codes, bucket
cutoffs and weights; then a search over the device-built index."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def _inputs(seed, n_docs, max_len, n_c=64):
    wl = synth.random_small_workload(seed, n_centroids=n_c, n_docs=n_docs, max_len=max_len, nbits=4)
    data = synth.make_index(wl, with_queries=True, workers=1)
    lens = data.doc_lengths.astype(np.int64)
    X = synth.token_vectors(data.workload, np.arange(int(lens.sum())))
    docs = np.repeat(np.arange(len(lens)), lens).astype(np.int32)
    return data, X, docs, lens


def _build_both(X, docs, n_docs, C0, sample, iterations, nbits, n_quant, label):
    import torch

    import paper_2501_17788_amd as w

    say(f"[{label}] n={len(X)} n_c={len(C0)} sample={len(sample)} it={iterations} b={nbits} n_quant={n_quant}")
    got = w.build_index(torch.from_numpy(X).cuda(), torch.from_numpy(docs).cuda(), n_docs, C0, sample,
                        iterations, nbits, n_quant)
    got = {k: v.cpu().numpy() for k, v in got.items()}
    want = oracle.build_index(X, docs, C0, sample, iterations, nbits, n_quant)
    for key in ("assign", "centroids", "offsets", "doc_ids", "codes", "cutoffs", "weights"):
        assert np.array_equal(got[key], want[key]), f"{label}: {key} differs"
    return got, want


@pytest.mark.parametrize("nbits", [1, 2, 4, 8])
def test_build_matches_oracle(nbits):
    import paper_2501_17788_amd as w

    data, X, docs, lens = _inputs(30 + nbits, n_docs=600, max_len=40, n_c=128)
    sample = w.sample_passages(lens, c=12.0, seed=nbits)
    C0 = w.initial_centroids(X, sample, 128, seed=nbits)
    _build_both(X, docs, len(lens), C0, sample, 4, nbits, 1500, label=f"b={nbits}")


def test_build_many_tiles_and_radix_passes():
    """600 centroids (two 8-bit passes of the stable sort by cluster) over about 60k tokens
    (15 tiles of 4,096 keys), quantiles over 20,000 tokens (2.56M residual components: four
    passes over 625 tiles): the hand-written sorts and prefix sums at several tiles."""
    import paper_2501_17788_amd as w

    data, X, docs, lens = _inputs(44, n_docs=3000, max_len=40, n_c=600)
    sample = w.sample_passages(lens, c=20.0, seed=5)
    C0 = w.initial_centroids(X, sample, 600, seed=6)
    assert len(X) > 8 * 4096
    _build_both(X, docs, len(lens), C0, sample, 2, 2, 20000, label="600 centroids, 20k quantile tokens")


def test_build_edge_cases():
    import paper_2501_17788_amd as w

    data, X, docs, lens = _inputs(40, n_docs=200, max_len=12, n_c=48)
    sample = w.sample_passages(lens, c=5.0, seed=1)
    C0 = w.initial_centroids(X, sample, 48, seed=2)
    _build_both(X, docs, len(lens), C0, sample, 0, 4, len(X), label="no k-means step, all tokens for quantiles")
    _build_both(X, docs, len(lens), C0[:1], sample[:1], 3, 2, 1, label="one centroid, one sample token")
    C1 = C0.copy()
    C1[7] = C1[3]  # duplicate centroids: ties go to the lower id
    C1[20] = C1[3]
    got, _ = _build_both(X, docs, len(lens), C1, sample, 2, 4, 200, label="duplicate centroids")


def test_build_errors():
    import torch

    import paper_2501_17788_amd as w

    data, X, docs, lens = _inputs(41, n_docs=50, max_len=6, n_c=16)
    sample = w.sample_passages(lens, c=5.0, seed=1)
    C0 = w.initial_centroids(X, sample, 16, seed=2)
    Xt, Dt = torch.from_numpy(X).cuda(), torch.from_numpy(docs).cuda()
    Z = C0.copy()
    Z[2] = 0
    with pytest.raises(w.WarpError) as e:
        w.build_index(Xt, Dt, len(lens), Z, sample, 1, 4, 10)
    assert e.value.code == w.EINVAL and "zero" in e.value.msg
    bad = sample.copy()
    bad[0] = len(X)
    with pytest.raises(w.WarpError) as e:
        w.build_index(Xt, Dt, len(lens), C0, bad, 1, 4, 10)
    assert e.value.code == w.EINVAL and "sample id" in e.value.msg
    with pytest.raises(w.WarpError) as e:
        w.build_index(Xt * 1.5, Dt, len(lens), C0, sample, 1, 4, 10)
    assert e.value.code == w.EINVAL and "norm" in e.value.msg
    with pytest.raises(w.WarpError) as e:
        w.build_index(Xt, Dt, len(lens) - 1, C0, sample, 1, 4, 10)
    assert e.value.code == w.EINVAL and "document id" in e.value.msg
    with pytest.raises(w.WarpError):
        w.build_index(Xt, Dt, len(lens), C0, sample, 1, 3, 10)


def test_search_over_device_built_index():
    import torch

    import paper_2501_17788_amd as w

    data, X, docs, lens = _inputs(42, n_docs=800, max_len=40, n_c=128)
    sample = w.sample_passages(lens, c=12.0, seed=3)
    C0 = w.initial_centroids(X, sample, 128, seed=4)
    built = w.build_index(torch.from_numpy(X).cuda(), torch.from_numpy(docs).cuda(), len(lens), C0, sample, 4, 4,
                          3000)
    with w.Index.from_device(built["centroids"], built["offsets"], built["doc_ids"], built["codes"], 4,
                             built["weights"], len(lens)) as ix:
        got = ix.search_debug(data.queries, 16, 2000, 50)
    b = {k: v.cpu().numpy() for k, v in built.items()}
    want = oracle.search(b["centroids"], b["offsets"], b["doc_ids"], b["codes"], 4, b["weights"], len(lens),
                         data.queries, 16, 2000, 50)
    for key in ("ids", "fixed", "counts", "sel", "m_fixed", "cand_bitmap", "n_scored"):
        assert np.array_equal(got[key], want[key]), key
    hit = float(np.mean(got["ids"][:, 0] == data.query_targets))
    say(f"device-built index: target document first for {hit:.0%} of {len(data.queries)} queries")
    assert hit >= 0.5
