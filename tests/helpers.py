"""Shared test helpers: fixture loading and independent reference computations.

Nothing here imports the engine or the oracle; these are plain numpy
restatements used to pin the oracle and to build inputs.
"""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
FRAC = 2.0 ** 26


def load_dyadic():
    """The hand-built example of tests/golden/dyadic_example.json as arrays."""
    with open(os.path.join(GOLDEN, "dyadic_example.json")) as f:
        g = json.load(f)
    dim, nbits = g["dim"], g["nbits"]
    C = np.zeros((len(g["centroids_sparse"]), dim), np.float32)
    for c, entries in enumerate(g["centroids_sparse"]):
        for d, v in entries:
            C[c, d] = v
    emb = g["embeddings"]
    n_c = len(C)
    clusters = np.array([e[0] for e in emb])
    assert np.all(np.diff(clusters) >= 0)
    offsets = np.zeros(n_c + 1, np.int64)
    np.cumsum(np.bincount(clusters, minlength=n_c), out=offsets[1:])
    doc_ids = np.array([e[1] for e in emb], np.int32)
    per_dim = np.zeros((len(emb), dim), np.int64)
    per_dim[:, 0] = [e[2] for e in emb]
    per_dim[:, 1] = [e[3] for e in emb]
    codes = pack_msb_first(per_dim, nbits)
    Q = np.zeros((len(g["queries_sparse"]), len(g["queries_sparse"][0]), dim), np.float32)
    for qi, toks in enumerate(g["queries_sparse"]):
        for ti, entries in enumerate(toks):
            for d, v in entries:
                Q[qi, ti, d] = v
    w = np.array(g["bucket_weights"], np.float32)
    return g, dict(centroids=C, offsets=offsets, doc_ids=doc_ids, codes=codes, nbits=nbits,
                   bucket_weights=w, n_docs=g["n_docs"]), Q


def pack_msb_first(per_dim: np.ndarray, nbits: int) -> np.ndarray:
    """Pack codes with the first dimension of each byte in its most significant bits
    (written independently of the generator's packer: bit strings via np.packbits)."""
    n, dim = per_dim.shape
    bits = ((per_dim[:, :, None] >> np.arange(nbits - 1, -1, -1)) & 1).astype(np.uint8)
    return np.packbits(bits.reshape(n, dim * nbits), axis=1)


def unpack_msb_first(codes: np.ndarray, nbits: int, dim: int = 128) -> np.ndarray:
    """Inverse of pack_msb_first via np.unpackbits."""
    bits = np.unpackbits(codes, axis=1).reshape(codes.shape[0], dim, nbits).astype(np.int64)
    return (bits << np.arange(nbits - 1, -1, -1)).sum(axis=2)


def cluster_of_embeddings(offsets: np.ndarray) -> np.ndarray:
    return np.repeat(np.arange(len(offsets) - 1), np.diff(offsets))


def explicit_decompress(centroids, offsets, codes, nbits, bucket_weights) -> np.ndarray:
    """Eq. decompress: x_e = C[c_e] + sum_d e_d * w[code_{e,d}] in fp64."""
    per_dim = unpack_msb_first(codes, nbits, centroids.shape[1])
    cl = cluster_of_embeddings(offsets)
    return centroids[cl].astype(np.float64) + bucket_weights.astype(np.float64)[per_dim]


def bruteforce_maxsim(X: np.ndarray, doc_ids: np.ndarray, n_docs: int, Q: np.ndarray):
    """Exhaustive MaxSim over explicitly decompressed vectors: for every doc with at
    least one embedding, sum over query tokens of the max dot product (fp64).
    Returns (docs, scores) for the docs that have embeddings."""
    order = np.argsort(doc_ids, kind="stable")
    d_sorted = doc_ids[order]
    starts = np.flatnonzero(np.r_[True, d_sorted[1:] != d_sorted[:-1]])
    docs = d_sorted[starts]
    sims = Q.astype(np.float64) @ X[order].T            # [n_qtok, N]
    per_tok = np.maximum.reduceat(sims, starts, axis=1)  # [n_qtok, n_present_docs]
    return docs, per_tok.sum(axis=0)


def weighted_order_statistic(scores: np.ndarray, sizes: np.ndarray, t_prime: int) -> float:
    """max{ s : sum of sizes of centroids scoring >= s exceeds t' }, over the scores
    that occur; the lowest score when no s qualifies (brute force over distinct values)."""
    best = None
    for s in np.unique(scores):
        if sizes[scores >= s].sum() > t_prime:
            best = s if best is None else max(best, s)
    return float(scores.min()) if best is None else float(best)


def topp_by_score(scores: np.ndarray, nprobe: int) -> np.ndarray:
    """The nprobe best ids by (score desc, id asc) via lexsort."""
    order = np.lexsort((np.arange(len(scores)), -scores))
    return order[:nprobe]
