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


def load_dyadic(name: str = "dyadic_example.json"):
    """A hand-built example of tests/golden (by default dyadic_example.json) as arrays."""
    with open(os.path.join(GOLDEN, name)) as f:
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


def realvalued_doc_scores(centroids, offsets, doc_ids, codes, nbits, bucket_weights, n_docs, Q, docs,
                          nprobe, t_prime, literal=False):
    """fp64 scores of `docs` for one query Q [n_qtok, 128], from explicit decompression.

    Independent of the oracle and the engine: for every query token, the centroid
    scores are a numpy fp64 matrix product (Section 4.3), the probed centroids the
    nprobe best by (score desc, id asc), and m_i the score at the first position
    (same order) whose inclusive cumulative cluster size exceeds t' (the last one if
    none does). Only the documents' own embeddings are decompressed (Eq. decompress:
    x = C[c] + w[code]); a token's entry is the max of q_i . x over the document's
    embeddings in its probed clusters, else m_i (Section 4.5); with `literal`, a
    retrieved entry is raised to m_i when some embedding of the document was not
    retrieved for that token (Eq. 1 read literally). Cheap at any index size: one
    pass over doc_ids plus work proportional to len(docs).
    """
    docs = np.asarray(docs, np.int64)
    C64 = np.asarray(centroids, np.float64)
    w64 = np.asarray(bucket_weights, np.float64)
    sizes = np.diff(np.asarray(offsets, np.int64))
    n_c = len(sizes)
    want = np.zeros(n_docs, bool)
    want[docs] = True
    pos = np.flatnonzero(want[doc_ids])
    cl = np.searchsorted(offsets, pos, side="right") - 1
    X = C64[cl] + w64[unpack_msb_first(np.asarray(codes)[pos], nbits, C64.shape[1])]
    slot = np.full(n_docs, -1, np.int64)
    slot[docs] = np.arange(len(docs))
    e_slot = slot[np.asarray(doc_ids)[pos]]
    doc_len = np.bincount(e_slot, minlength=len(docs))
    out = np.zeros(len(docs))
    ids = np.arange(n_c)
    for q in np.asarray(Q, np.float64):
        S = C64 @ q
        order = np.lexsort((ids, -S))
        cum = np.cumsum(sizes[order])
        hit = np.flatnonzero(cum > t_prime)
        m = S[order[hit[0]]] if len(hit) else S[order[-1]]
        probed = np.isin(cl, order[:nprobe])
        s = X[probed] @ q
        best = np.full(len(docs), -np.inf)
        np.maximum.at(best, e_slot[probed], s)
        seen = np.bincount(e_slot[probed], minlength=len(docs))
        tok = np.where(np.isneginf(best), m, best)
        if literal:
            tok = np.where(~np.isneginf(best) & (seen < doc_len), np.maximum(tok, m), tok)
        out += tok
    return out


def check_real_valued(scores, counts, ids, data_arrays, Q, nprobe, t_prime, literal=False, rel_tol=1e-4):
    """Every returned float score within rel_tol * max(1, |ref|) of the fp64 explicit-
    decompression score of that document (realvalued_doc_scores); returns the largest
    relative gap. The returned order agrees with the reference up to the same tolerance."""
    n = int(counts)
    ref = realvalued_doc_scores(Q=Q, docs=ids[:n], nprobe=nprobe, t_prime=t_prime, literal=literal,
                                **data_arrays)
    got = np.asarray(scores[:n], np.float64)
    tol = rel_tol * np.maximum(1.0, np.abs(ref))
    gap = np.abs(got - ref)
    assert np.all(gap <= tol), f"real-valued score gap {gap.max():.3g} above {rel_tol} relative"
    assert np.all(np.diff(ref) <= tol[1:] + tol[:-1]), "returned order disagrees with the fp64 scores"
    return float((gap / np.maximum(1.0, np.abs(ref))).max()) if n else 0.0


def index_arrays(data) -> dict:
    """The index arrays of a synth.SyntheticIndex, as keyword arguments."""
    return dict(centroids=data.centroids, offsets=data.offsets, doc_ids=data.doc_ids, codes=data.codes,
                nbits=data.nbits, bucket_weights=data.bucket_weights, n_docs=data.n_docs)
