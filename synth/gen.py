"""Synthetic WARP workloads: index arrays and query token embeddings.

Recipe (stands in for the BEIR / LoTTE collections of the paper's evaluation,
whose passages, queries and trained encoder are not available):

* centroids ``C_c = g / ||g||`` with ``g ~ N(0, I_128)``, stored as fp32;
* cluster popularity: Zipf, ``p_r ~ r^-s`` over ranks ``r = 1..n_c``; rank ``r``
  is mapped to centroid ``perm[r]`` by a random permutation;
* document lengths: uniform integers, or ``round(LogNormal(mu, 0.6))`` with
  ``mu = ln(mean) - 0.6^2 / 2`` clamped to ``[1, cap]``;
* document tokens: draw a rank ``z ~ p``; the token is
  ``x = normalize(C[perm[z]] + 0.1 n)``, ``n ~ N(0, I)``, stored as fp32.  The
  token is assigned to cluster ``perm[z]`` by construction;
* residual ``r = x - C[cluster]`` quantised per dimension with quantile buckets
  (Section 4.1, index construction): the ``2^b - 1`` cutoffs are the quantiles
  ``j / 2^b`` of the pooled residual components of the first 65,536 tokens, the
  ``2^b`` bucket weights are the quantiles ``(j + 1/2) / 2^b``, and the code of a
  component is the number of cutoffs that are ``<=`` it;
* codes are packed ``8 / b`` per byte, most significant bits first (dimension
  ``2j`` of a 4-bit code sits in bits 7..4 of byte ``j``);
* embeddings are grouped by cluster and, inside a cluster, ordered by document
  id (then by position in the document);
* queries: a target document is drawn uniformly, then ``n_qtok`` of its tokens
  uniformly with replacement; each query token is ``normalize(x + 0.05 n)``.

Every random draw comes from a counter-based Philox stream keyed by
``(seed, stream, chunk)``, so any token can be regenerated from its embedding
id, and chunks can be generated in parallel.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ProcessPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

DIM = 128
CHUNK = 1 << 16          # embeddings per generation chunk
QUANTILE_SAMPLE = 1 << 16  # tokens pooled for the quantile cutoffs

# Philox stream identifiers.
S_CENTROIDS, S_PERM, S_LENGTHS, S_DRAWS, S_NOISE, S_QUERIES = 1, 2, 3, 4, 5, 7


@dataclass(frozen=True)
class Workload:
    name: str
    n_docs: int
    len_kind: str          # "uniform" (len_a..len_b inclusive) or "lognormal" (mean len_a, cap len_b)
    len_a: float
    len_b: float
    n_centroids: int
    zipf_s: float
    nbits: int
    n_queries: int
    nprobe: int
    t_prime: int
    k: int
    seed: int
    n_qtok: int = 32
    token_noise: float = 0.1
    query_noise: float = 0.05
    len_sigma: float = 0.6


_SEED0 = 20250129

WORKLOADS = {
    # 4,096 docs of 16-48 tokens, 1,024 centroids, Zipf 1.1, b = 4, one query.
    "tiny": Workload("tiny", 4096, "uniform", 16, 48, 1024, 1.1, 4, 1, 16, 10_000, 10, _SEED0 + 0),
    # 100k docs, lognormal mean 64 (cap 180), 2^15 centroids, b = 4, 256 queries.
    "small": Workload("small", 100_000, "lognormal", 64, 180, 1 << 15, 1.1, 4, 256, 32, 40_000, 100,
                      _SEED0 + 1),
    # 1M docs, lognormal mean 70, 2^17 centroids, b = 2, 1,024 queries (t' = 100,000: the
    # square-root rule that fits the other workloads, capped).
    "mid": Workload("mid", 1_000_000, "lognormal", 70, 512, 1 << 17, 1.1, 2, 1024, 32, 100_000, 100,
                    _SEED0 + 2),
    # 2M docs, lognormal mean 120 (cap 512), 2^18 centroids, Zipf 1.3, b = 4, 512 queries.
    "long": Workload("long", 2_000_000, "lognormal", 120, 512, 1 << 18, 1.3, 4, 512, 32, 100_000, 1000,
                     _SEED0 + 3),
    # 8.8M passages, lognormal mean 68, 2^18 centroids, b = 2, 4,096 queries.
    "full": Workload("full", 8_800_000, "lognormal", 68, 512, 1 << 18, 1.1, 2, 4096, 32, 100_000, 1000,
                     _SEED0 + 4),
}


@dataclass
class SyntheticIndex:
    workload: Workload
    centroids: np.ndarray      # [n_c, 128] float32, unit rows
    offsets: np.ndarray        # [n_c + 1] int64
    doc_ids: np.ndarray        # [N] int32, grouped by cluster, ascending inside a cluster
    codes: np.ndarray          # [N, 128 * b / 8] uint8
    bucket_weights: np.ndarray  # [2^b] float32
    bucket_cutoffs: np.ndarray  # [2^b - 1] float64 (index construction only)
    doc_lengths: np.ndarray    # [n_docs] int32
    queries: np.ndarray | None = None        # [n_queries, n_qtok, 128] float32
    query_targets: np.ndarray | None = None  # [n_queries] int32
    extra: dict = field(default_factory=dict)

    @property
    def nbits(self) -> int:
        return self.workload.nbits

    @property
    def n_docs(self) -> int:
        return self.workload.n_docs

    @property
    def n_embeddings(self) -> int:
        return int(self.offsets[-1])

    @property
    def cluster_sizes(self) -> np.ndarray:
        return np.diff(self.offsets)


def _rng(seed: int, stream: int, chunk: int = 0) -> np.random.Generator:
    key = np.array([seed & ((1 << 64) - 1), (stream << 40) | chunk], dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


def _normalize_rows(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def make_centroids(w: Workload) -> np.ndarray:
    g = _rng(w.seed, S_CENTROIDS).standard_normal((w.n_centroids, DIM))
    return _normalize_rows(g).astype(np.float32)


def zipf_cdf(n: int, s: float) -> np.ndarray:
    p = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(p)
    return c / c[-1]


def make_doc_lengths(w: Workload) -> np.ndarray:
    rng = _rng(w.seed, S_LENGTHS)
    if w.len_kind == "uniform":
        return rng.integers(int(w.len_a), int(w.len_b) + 1, size=w.n_docs).astype(np.int32)
    mu = math.log(w.len_a) - w.len_sigma ** 2 / 2
    lens = np.rint(rng.lognormal(mu, w.len_sigma, size=w.n_docs))
    return np.clip(lens, 1, w.len_b).astype(np.int32)


def pack_codes(codes: np.ndarray, nbits: int) -> np.ndarray:
    """Pack per-dimension codes [n, 128] into bytes, most significant bits first."""
    per = 8 // nbits
    c = codes.astype(np.uint8).reshape(codes.shape[0], DIM // per, per)
    out = np.zeros(c.shape[:2], dtype=np.uint8)
    for p in range(per):
        out |= (c[:, :, p] << (8 - nbits * (p + 1))).astype(np.uint8)
    return out


# ----------------------------------------------------------------------------
# chunked token generation (fork-based process pool; outputs in shared memory)

_G: dict = {}


def _draw_clusters(chunk: int, n: int) -> np.ndarray:
    """Cluster ids of the n tokens of chunk `chunk` (Zipf rank -> permuted centroid)."""
    w: Workload = _G["w"]
    u = _rng(w.seed, S_DRAWS, chunk).random(n)
    z = np.minimum(np.searchsorted(_G["cdf"], u, side="right"), w.n_centroids - 1)
    return _G["perm"][z].astype(np.int32)


def _tokens(chunk: int, e0: int, e1: int):
    """Tokens [e0, e1) of chunk `chunk`: (cluster ids, fp32 unit vectors)."""
    w: Workload = _G["w"]
    n = e1 - e0
    cl = _draw_clusters(chunk, n)
    noise = _rng(w.seed, S_NOISE, chunk).standard_normal((n, DIM), dtype=np.float32)
    x = _G["C"][cl]
    x += np.float32(w.token_noise) * noise
    x /= np.sqrt(np.einsum("ij,ij->i", x, x))[:, None]
    return cl, x


def _codes(r: np.ndarray, nbits: int) -> np.ndarray:
    """Per-dimension code = number of cutoffs <= r, packed MSB-first. The cutoffs are
    compared as the smallest float32 at or above each fp64 cutoff, which gives the same
    decision for float32 residuals as the fp64 comparison."""
    cut32 = _G["cut32"]
    code = np.zeros(r.shape, np.uint8)
    for c in cut32:
        code += r >= c
    return pack_codes(code, nbits)


def _chunk_range(s: int):
    """Chunks of super-range s (contiguous, so each worker walks docs in order)."""
    n_chunks, n_super = _G["n_chunks"], _G["n_super"]
    return range(s * n_chunks // n_super, (s + 1) * n_chunks // n_super)


def _count_job(s: int) -> np.ndarray:
    w: Workload = _G["w"]
    counts = np.zeros(w.n_centroids, np.int64)
    for chunk in _chunk_range(s):
        e0 = chunk * CHUNK
        e1 = min(_G["n_total"], e0 + CHUNK)
        counts += np.bincount(_draw_clusters(chunk, e1 - e0), minlength=w.n_centroids)
    return counts


def _write_job(s: int):
    """Generate the chunks of super-range s and write codes and doc ids into their
    final (cluster-grouped, doc-ascending) positions; return the query tokens."""
    w: Workload = _G["w"]
    cursor = _G["start"][s].copy()
    codes_out, docs_out, doc_of = _G["codes_out"], _G["docs_out"], _G["doc_of"]
    want = _G["want"]
    picked = []
    for chunk in _chunk_range(s):
        e0 = chunk * CHUNK
        e1 = min(_G["n_total"], e0 + CHUNK)
        cl, x = _tokens(chunk, e0, e1)
        packed = _codes(x - _G["C"][cl], w.nbits)
        order = np.argsort(cl, kind="stable")
        scl = cl[order]
        first = np.r_[True, scl[1:] != scl[:-1]]
        starts = np.flatnonzero(first)
        rank = np.arange(len(scl)) - np.repeat(starts, np.diff(np.r_[starts, len(scl)]))
        pos = cursor[scl] + rank
        codes_out[pos] = packed[order]
        docs_out[pos] = doc_of(e0 + order)
        u, cnt = scl[starts], np.diff(np.r_[starts, len(scl)])
        cursor[u] += cnt
        lo, hi = np.searchsorted(want, [e0, e1])
        if hi > lo:
            picked.append((want[lo:hi], x[want[lo:hi] - e0]))
    return picked


def _state(w: Workload, C, perm, cdf, n_total) -> dict:
    return {"w": w, "C": C, "perm": perm, "cdf": cdf, "n_total": n_total}


def _shared(shape, dtype) -> np.ndarray:
    """An array in anonymous shared memory, inherited by forked workers."""
    import mmap

    nbytes = int(np.prod(shape)) * np.dtype(dtype).itemsize
    buf = mmap.mmap(-1, max(nbytes, 1))
    return np.frombuffer(buf, dtype=dtype, count=int(np.prod(shape))).reshape(shape)


def _run(jobs, fn, workers):
    if workers > 1 and len(jobs) > 1:
        import multiprocessing as mp

        with ProcessPoolExecutor(min(workers, len(jobs)), mp_context=mp.get_context("fork")) as ex:
            return list(ex.map(fn, jobs))
    return [fn(j) for j in jobs]


def token_vectors(w: Workload, emb_ids: np.ndarray) -> np.ndarray:
    """Regenerate the fp32 token vectors of the given embedding ids (generation order)."""
    C = make_centroids(w)
    perm = _rng(w.seed, S_PERM).permutation(w.n_centroids)
    cdf = zipf_cdf(w.n_centroids, w.zipf_s)
    _G.clear()
    _G.update(_state(w, C, perm, cdf, None))
    out = np.zeros((len(emb_ids), DIM), np.float32)
    ids = np.asarray(emb_ids, dtype=np.int64)
    for chunk in np.unique(ids // CHUNK):
        sel = np.nonzero(ids // CHUNK == chunk)[0]
        e0 = int(chunk) * CHUNK
        _, x = _tokens(int(chunk), e0, int(ids[sel].max()) + 1)
        out[sel] = x[ids[sel] - e0]
    return out


def make_index(w: Workload, with_queries: bool = True, workers: int | None = None,
               progress=None) -> SyntheticIndex:
    """Generate the whole index (and, optionally, the query batch) of workload `w`.
    `progress(msg)` is called between the phases of a large generation."""
    if DIM % (8 // w.nbits) != 0 or w.nbits not in (1, 2, 4, 8):
        raise ValueError("nbits must be 1, 2, 4 or 8")
    say = progress or (lambda msg: None)
    C = make_centroids(w)
    perm = _rng(w.seed, S_PERM).permutation(w.n_centroids).astype(np.int64)
    cdf = zipf_cdf(w.n_centroids, w.zipf_s)
    lens = make_doc_lengths(w)
    doc_start = np.zeros(w.n_docs + 1, np.int64)
    np.cumsum(lens, out=doc_start[1:])
    n_total = int(doc_start[-1])
    _G.clear()
    _G.update(_state(w, C, perm, cdf, n_total))

    # quantile cutoffs and bucket weights from the residuals of the first tokens
    ns = min(n_total, QUANTILE_SAMPLE)
    cl_s, x_s = _tokens(0, 0, ns)
    sample = (x_s - C[cl_s]).astype(np.float64).ravel()
    nb = 1 << w.nbits
    cutoffs = np.quantile(sample, np.arange(1, nb) / nb)
    weights = np.quantile(sample, (np.arange(nb) + 0.5) / nb).astype(np.float32)
    cut32 = cutoffs.astype(np.float32)
    cut32 = np.where(cut32.astype(np.float64) < cutoffs, np.nextafter(cut32, np.float32(np.inf)), cut32)
    _G["cut32"] = cut32.astype(np.float32)

    # query targets: documents and token positions, drawn before the token pass so that
    # the pass keeps exactly the tokens the queries need
    want = np.zeros(0, np.int64)
    if with_queries:
        qr = _rng(w.seed, S_QUERIES)
        targets = qr.integers(0, w.n_docs, size=w.n_queries)
        pos = qr.integers(0, 1 << 62, size=(w.n_queries, w.n_qtok)) % lens[targets][:, None]
        q_emb = doc_start[targets][:, None] + pos
        q_noise = qr.standard_normal((w.n_queries, w.n_qtok, DIM))
        want = np.unique(q_emb.ravel())
    _G["want"] = want

    if workers is None:
        workers = min(16, os.cpu_count() or 1)
    n_chunks = (n_total + CHUNK - 1) // CHUNK
    n_super = max(1, min(n_chunks, 4 * workers))
    _G["n_chunks"], _G["n_super"] = n_chunks, n_super

    # pass 1: cluster sizes per super-range -> cluster offsets and write cursors
    counts = np.stack(_run(list(range(n_super)), _count_job, workers))
    sizes = counts.sum(axis=0)
    offsets = np.zeros(w.n_centroids + 1, np.int64)
    np.cumsum(sizes, out=offsets[1:])
    start = offsets[:-1][None, :] + np.cumsum(counts, axis=0) - counts
    _G["start"] = start
    say(f"cluster sizes done ({n_total} embeddings, {n_chunks} chunks)")

    # pass 2: tokens, codes, and their scatter into cluster order
    codes = _shared((n_total, DIM * w.nbits // 8), np.uint8)
    doc_ids = _shared((n_total,), np.int32)
    _G["codes_out"], _G["docs_out"] = codes, doc_ids
    _G["doc_of"] = lambda e: (np.searchsorted(doc_start, e, side="right") - 1).astype(np.int32)
    picked = [p for part in _run(list(range(n_super)), _write_job, workers) for p in part]
    say("codes done")

    idx = SyntheticIndex(
        workload=w, centroids=C, offsets=offsets, doc_ids=doc_ids, codes=codes,
        bucket_weights=weights, bucket_cutoffs=cutoffs, doc_lengths=lens)
    if with_queries:
        ids = np.concatenate([p[0] for p in picked]) if picked else np.zeros(0, np.int64)
        xs = np.concatenate([p[1] for p in picked]) if picked else np.zeros((0, DIM), np.float32)
        row = np.searchsorted(ids, q_emb)
        x = xs[row].astype(np.float64)
        idx.queries = _normalize_rows(x + w.query_noise * q_noise).astype(np.float32)
        idx.query_targets = targets.astype(np.int32)
    _G.clear()
    return idx


def make_queries(idx: SyntheticIndex) -> np.ndarray:
    if idx.queries is None:
        raise ValueError("index was generated without queries")
    return idx.queries


def random_small_workload(seed: int, *, n_centroids: int = 16, n_docs: int = 40, max_len: int = 8,
                          nbits: int = 4, n_queries: int = 2, n_qtok: int = 4, nprobe: int = 4,
                          t_prime: int = 10, k: int = 5, zipf_s: float = 1.1) -> Workload:
    """A tiny workload for exhaustive checks."""
    return Workload(f"rand{seed}", n_docs, "uniform", 1, max_len, n_centroids, zipf_s, nbits,
                    n_queries, nprobe, t_prime, k, 0x5EED0000 + seed, n_qtok=n_qtok)


def with_overrides(w: Workload, **kw) -> Workload:
    return replace(w, **kw)
