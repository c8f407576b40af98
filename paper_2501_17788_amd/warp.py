"""Python binding of libwarp.so: argument marshalling only.

Every step of a search runs in the HIP kernels behind the C ABI of
include/warp.h; this module converts arrays, checks shapes and raises
WarpError on a non-OK status. torch is used only for device tensors and
streams in the asynchronous entry point. There is no CPU fallback: if the
library is not built, importing the binding raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libwarp.so")

OK, EINVAL, ENOMEM, EDEVICE, ENOTSUP = 0, -1, -2, -3, -4
_NAMES = {EINVAL: "EINVAL", ENOMEM: "ENOMEM", EDEVICE: "EDEVICE", ENOTSUP: "ENOTSUP"}
STAGES = ("filter_gemm", "select", "plan", "scan", "fold", "topk")
SCORING_PAPER, SCORING_EQ1_LITERAL = 0, 1  # warp_set_scoring modes

EXPORTS = (
    "warp_fixed_point_bits", "warp_last_error", "warp_index_load", "warp_index_load_device",
    "warp_index_free", "warp_index_info", "warp_search", "warp_search_async", "warp_index_sync",
    "warp_search_debug", "warp_centroid_filter_scores", "warp_set_timing", "warp_stage_timings",
    "warp_t_prime_policy", "warp_set_scoring", "warp_build_index", "warp_search_noalloc",
    "warp_kmeans_sample_size",
)


class WarpError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_NAMES.get(code, code)}: {msg}")
        self.code = code
        self.msg = msg


def _load() -> ctypes.CDLL:
    # torch ships its own HIP runtime with the same soname as /opt/rocm's. Loading
    # torch first makes libwarp.so bind to that runtime, so there is one HIP
    # runtime in the process and torch's device pointers and streams are valid here.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "warp_fixed_point_bits": ([], ctypes.c_int),
        "warp_last_error": ([], ctypes.c_char_p),
        "warp_index_load": ([P, i32, i32, P, P, P, i32, P, i32, P], ctypes.c_int),
        "warp_index_load_device": ([P, i32, i32, P, P, P, i32, P, i32, P], ctypes.c_int),
        "warp_index_free": ([P], None),
        "warp_index_info": ([P, P, P, P, P], ctypes.c_int),
        "warp_search": ([P, P, i32, i32, i32, i64, i32, P, P, P], ctypes.c_int),
        "warp_search_async": ([P, P, i32, i32, i32, i64, i32, P, P, P, P, P], ctypes.c_int),
        "warp_search_noalloc": ([P, P, i32, i32, i32, i64, i32, P, P, P, P, P], ctypes.c_int),
        "warp_index_sync": ([P, P], ctypes.c_int),
        "warp_search_debug": ([P, P, i32, i32, i32, i64, i32, P, P, P, P, P, P, P, P], ctypes.c_int),
        "warp_centroid_filter_scores": ([P, P, i32, P], ctypes.c_int),
        "warp_set_timing": ([P, i32], ctypes.c_int),
        "warp_stage_timings": ([P, P, P, i32], ctypes.c_int),
        "warp_t_prime_policy": ([i64, ctypes.c_double, i64, P], ctypes.c_int),
        "warp_kmeans_sample_size": ([i64, ctypes.c_double, P], ctypes.c_int),
        "warp_set_scoring": ([P, i32], ctypes.c_int),
        "warp_build_index": ([P, P, i64, i32, P, i32, P, i64, i32, i32, i64, P, P, P, P, P, P, P], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


lib = _load()
FRAC_BITS = lib.warp_fixed_point_bits()


# Section 4.6 leaves the constants of its t' policy open; these defaults reproduce the
# t' of the synthetic workloads (40,000 for 6.3M embeddings, capped at 100,000 above).
T_PRIME_C = 15.8
T_PRIME_MAX = 100_000


def t_prime_policy(n_embeddings: int, c: float = T_PRIME_C, t_max: int = T_PRIME_MAX) -> int:
    """t' = min(t_max, floor(c * sqrt(n_embeddings))) (Section 4.6), computed by the library."""
    out = ctypes.c_int64()
    _check(lib.warp_t_prime_policy(int(n_embeddings), float(c), int(t_max), ctypes.byref(out)))
    return out.value


def last_error() -> str:
    return lib.warp_last_error().decode()


def _check(rc: int) -> None:
    if rc != OK:
        raise WarpError(rc, last_error())


def _ptr(a):
    if a is None:
        return None
    if isinstance(a, np.ndarray):
        return a.ctypes.data_as(ctypes.c_void_p)
    return ctypes.c_void_p(a.data_ptr())  # torch tensor


def _host(a, dtype, shape=None) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=dtype)
    if shape is not None and a.shape != shape:
        raise ValueError(f"expected shape {shape}, got {a.shape}")
    return a


class Index:
    """A device-resident WARP index (owns its device memory)."""

    def __init__(self, centroids, offsets, doc_ids, codes, nbits: int, bucket_weights, n_docs: int):
        C = _host(centroids, np.float32)
        n_c, dim = C.shape
        off = _host(offsets, np.int64, (n_c + 1,))
        ids = _host(doc_ids, np.int32)
        cd = _host(codes, np.uint8)
        w = _host(bucket_weights, np.float32)
        if cd.ndim != 2 or cd.shape[0] != len(ids) or cd.shape[0] != int(off[-1]):
            raise ValueError("codes / doc_ids / offsets disagree on the number of embeddings")
        if cd.shape[1] != dim * nbits // 8 or len(w) != 1 << nbits:
            raise ValueError("codes row width or bucket weight count does not match nbits")
        h = ctypes.c_void_p()
        _check(lib.warp_index_load(_ptr(C), n_c, dim, _ptr(off), _ptr(ids), _ptr(cd), nbits, _ptr(w),
                                   int(n_docs), ctypes.byref(h)))
        self._h = h
        self.n_centroids, self.n_docs, self.nbits = n_c, int(n_docs), nbits

    @classmethod
    def from_synthetic(cls, idx) -> "Index":
        return cls(idx.centroids, idx.offsets, idx.doc_ids, idx.codes, idx.nbits, idx.bucket_weights,
                   idx.n_docs)

    @classmethod
    def from_device(cls, centroids, offsets, doc_ids, codes, nbits: int, bucket_weights, n_docs: int):
        """Load from torch device tensors (copied; the tensors may be freed afterwards)."""
        self = cls.__new__(cls)
        for t in (centroids, offsets, doc_ids, codes, bucket_weights):
            if not t.is_cuda or not t.is_contiguous():
                raise ValueError("from_device needs contiguous device tensors")
        n_c, dim = centroids.shape
        if offsets.numel() != n_c + 1 or codes.shape[0] != doc_ids.numel():
            raise ValueError("offsets / codes / doc_ids disagree")
        if codes.shape[1] != dim * nbits // 8 or bucket_weights.numel() != 1 << nbits:
            raise ValueError("codes row width or bucket weight count does not match nbits")
        h = ctypes.c_void_p()
        _check(lib.warp_index_load_device(_ptr(centroids), n_c, dim, _ptr(offsets), _ptr(doc_ids),
                                          _ptr(codes), nbits, _ptr(bucket_weights), int(n_docs),
                                          ctypes.byref(h)))
        self._h = h
        self.n_centroids, self.n_docs, self.nbits = n_c, int(n_docs), nbits
        return self

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            lib.warp_index_free(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def handle(self):
        return self._h

    def info(self) -> dict:
        n_c, n_docs, nbits = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        n_emb = ctypes.c_int64()
        _check(lib.warp_index_info(self._h, ctypes.byref(n_c), ctypes.byref(n_emb), ctypes.byref(n_docs),
                                   ctypes.byref(nbits)))
        return {"n_centroids": n_c.value, "n_embeddings": n_emb.value, "n_docs": n_docs.value,
                "nbits": nbits.value}

    def _queries(self, queries) -> np.ndarray:
        Q = _host(queries, np.float32)
        if Q.ndim == 2:
            Q = Q[None]
        if Q.ndim != 3:
            raise ValueError("queries must be [n_queries, n_qtok, dim]")
        return Q

    def search(self, queries, nprobe: int, t_prime: int, k: int):
        """Blocking search of host queries [n_queries, n_qtok, 128] -> (ids, scores, counts)."""
        Q = self._queries(queries)
        nq, nt, _ = Q.shape
        ids = np.empty((nq, k), np.int32)
        scores = np.empty((nq, k), np.float32)
        counts = np.empty(nq, np.int32)
        _check(lib.warp_search(self._h, _ptr(Q), nq, nt, nprobe, int(t_prime), k, _ptr(ids), _ptr(scores),
                               _ptr(counts)))
        return ids, scores, counts

    def search_debug(self, queries, nprobe: int, t_prime: int, k: int, bitmap: bool = True) -> dict:
        """Blocking search returning every intermediate the C ABI exposes (the candidate
        bitmap, n_queries x n_docs / 8 bytes, only with `bitmap`)."""
        Q = self._queries(queries)
        nq, nt, _ = Q.shape
        words = (self.n_docs + 31) // 32
        r = {
            "ids": np.empty((nq, k), np.int32),
            "scores": np.empty((nq, k), np.float32),
            "counts": np.empty(nq, np.int32),
            "fixed": np.empty((nq, k), np.int64),
            "sel": np.empty((nq, nt, nprobe), np.int32),
            "m_fixed": np.empty((nq, nt), np.int64),
            "cand_bitmap": np.empty((nq, words), np.uint32) if bitmap else None,
            "n_scored": np.empty(nq, np.int64),
        }
        _check(lib.warp_search_debug(self._h, _ptr(Q), nq, nt, nprobe, int(t_prime), k, _ptr(r["ids"]),
                                     _ptr(r["scores"]), _ptr(r["counts"]), _ptr(r["fixed"]), _ptr(r["sel"]),
                                     _ptr(r["m_fixed"]), _ptr(r["cand_bitmap"]), _ptr(r["n_scored"])))
        return r

    def search_async(self, queries, nprobe: int, t_prime: int, k: int, out=None, stream=None):
        """Enqueue a search of device queries (torch [n_queries, n_qtok, 128] fp32) on a stream.

        `out` may hold preallocated (ids, scores, counts, fixed) device tensors. Returns them."""
        import torch

        if not queries.is_cuda or queries.dtype != torch.float32 or queries.dim() != 3:
            raise ValueError("queries must be a float32 device tensor [n_queries, n_qtok, 128]")
        queries = queries.contiguous()
        nq, nt, _ = queries.shape
        dev = queries.device
        if out is None:
            out = (torch.empty((nq, k), dtype=torch.int32, device=dev),
                   torch.empty((nq, k), dtype=torch.float32, device=dev),
                   torch.empty(nq, dtype=torch.int32, device=dev),
                   torch.empty((nq, k), dtype=torch.int64, device=dev))
        ids, scores, counts, fixed = out
        s = stream if stream is not None else torch.cuda.current_stream(dev)
        _check(lib.warp_search_async(self._h, _ptr(queries), nq, nt, nprobe, int(t_prime), k, _ptr(ids),
                                     _ptr(scores), _ptr(counts), _ptr(fixed), ctypes.c_void_p(s.cuda_stream)))
        return out

    def search_noalloc(self, queries, nprobe: int, t_prime: int, k: int, out=None, stream=None):
        """As search_async through warp_search_noalloc: the library allocates nothing (its
        scratch is a static 256 MiB device array per GPU). `out` as in search_async; the
        output tensors are allocated here by torch only when `out` is None."""
        import torch

        if not queries.is_cuda or queries.dtype != torch.float32 or queries.dim() != 3:
            raise ValueError("queries must be a float32 device tensor [n_queries, n_qtok, 128]")
        queries = queries.contiguous()
        nq, nt, _ = queries.shape
        dev = queries.device
        if out is None:
            out = (torch.empty((nq, k), dtype=torch.int32, device=dev),
                   torch.empty((nq, k), dtype=torch.float32, device=dev),
                   torch.empty(nq, dtype=torch.int32, device=dev),
                   torch.empty((nq, k), dtype=torch.int64, device=dev))
        ids, scores, counts, fixed = out
        s = stream if stream is not None else torch.cuda.current_stream(dev)
        _check(lib.warp_search_noalloc(self._h, _ptr(queries), nq, nt, nprobe, int(t_prime), k, _ptr(ids),
                                       _ptr(scores), _ptr(counts), _ptr(fixed), ctypes.c_void_p(s.cuda_stream)))
        return out

    def sync(self, stream=None) -> None:
        import torch

        s = stream if stream is not None else torch.cuda.current_stream()
        _check(lib.warp_index_sync(self._h, ctypes.c_void_p(s.cuda_stream)))

    def filter_scores(self, tokens) -> np.ndarray:
        """fp32 matrix-core centroid scores of host tokens [n_tok, 128] -> [n_tok, n_centroids]."""
        T = _host(tokens, np.float32)
        out = np.empty((T.shape[0], self.n_centroids), np.float32)
        _check(lib.warp_centroid_filter_scores(self._h, _ptr(T), T.shape[0], _ptr(out)))
        return out

    def set_scoring(self, mode: int) -> None:
        """SCORING_PAPER (Section 4.5, the default) or SCORING_EQ1_LITERAL (Eq. 1 read literally)."""
        _check(lib.warp_set_scoring(self._h, int(mode)))

    def set_timing(self, enable: bool) -> None:
        _check(lib.warp_set_timing(self._h, 1 if enable else 0))

    def stage_timings(self) -> dict:
        ms = np.zeros(len(STAGES), np.float64)
        n = np.zeros(len(STAGES), np.int64)
        _check(lib.warp_stage_timings(self._h, _ptr(ms), _ptr(n), len(STAGES)))
        return {s: (float(ms[i]), int(n[i])) for i, s in enumerate(STAGES)}


# ----------------------------------------------------------------------------- index construction

def sample_passages(doc_lengths, c: float = 16.0, seed: int = 0) -> np.ndarray:
    """Token ids (document-major order) of warp_kmeans_sample_size(n_docs, c) passages
    drawn without replacement (the draw is the caller's choice; the size is Section 4.1's)."""
    lens = np.asarray(doc_lengths, np.int64)
    n_docs = len(lens)
    size = ctypes.c_int64()
    _check(lib.warp_kmeans_sample_size(n_docs, float(c), ctypes.byref(size)))
    k = size.value
    docs = np.sort(np.random.default_rng(seed).choice(n_docs, size=k, replace=False))
    starts = np.zeros(n_docs + 1, np.int64)
    np.cumsum(lens, out=starts[1:])
    return np.concatenate([np.arange(starts[d], starts[d + 1]) for d in docs]).astype(np.int64)


def initial_centroids(tokens, sample_ids, n_centroids: int, seed: int = 0) -> np.ndarray:
    """n_centroids distinct sample tokens: the k-means starting vectors (warp_build_index
    normalises them). A choice of the caller, like the sample itself."""
    ids = np.asarray(sample_ids, np.int64)
    if n_centroids > len(ids):
        raise ValueError("more centroids than sampled tokens")
    pick = np.random.default_rng(seed).choice(len(ids), size=n_centroids, replace=False)
    X = tokens[ids[np.sort(pick)]]
    return np.ascontiguousarray(X.cpu() if hasattr(X, "cpu") else X, np.float32)


def build_index(tokens, token_docs, n_docs: int, init_centroids, sample_ids, iterations: int, nbits: int,
                n_quant: int) -> dict:
    """Index construction on the device (warp_build_index): torch tensors in, torch tensors out.

    tokens [n, 128] float32 and token_docs [n] int32 on the device; init_centroids
    [n_c, 128] and sample_ids [n_sample] int64 on the device or host. Returns the index
    arrays (centroids, offsets, doc_ids, codes, weights, cutoffs, assign) as device tensors.
    """
    import torch

    dev = tokens.device
    X = tokens.contiguous()
    docs = token_docs.to(torch.int32).contiguous()
    C0 = torch.as_tensor(init_centroids, dtype=torch.float32).to(dev).contiguous()
    S = torch.as_tensor(sample_ids, dtype=torch.int64).to(dev).contiguous()
    n, n_c = X.shape[0], C0.shape[0]
    out = {
        "centroids": torch.empty((n_c, 128), dtype=torch.float32, device=dev),
        "offsets": torch.empty(n_c + 1, dtype=torch.int64, device=dev),
        "doc_ids": torch.empty(n, dtype=torch.int32, device=dev),
        "codes": torch.empty((n, 16 * nbits), dtype=torch.uint8, device=dev),
        "weights": torch.empty(1 << nbits, dtype=torch.float32, device=dev),
        "cutoffs": torch.empty((1 << nbits) - 1, dtype=torch.float32, device=dev),
        "assign": torch.empty(n, dtype=torch.int32, device=dev),
    }
    torch.cuda.synchronize(dev)
    _check(lib.warp_build_index(
        _tptr(X), _tptr(docs), n, int(n_docs), _tptr(C0), n_c, _tptr(S), S.numel(), int(iterations), int(nbits),
        int(n_quant), _tptr(out["centroids"]), _tptr(out["offsets"]), _tptr(out["doc_ids"]), _tptr(out["codes"]),
        _tptr(out["weights"]), _tptr(out["cutoffs"]), _tptr(out["assign"])))
    return out


def _tptr(t):
    return ctypes.c_void_p(t.data_ptr())
