"""ctypes front end of the plain CPU oracle (``warp_oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg are its only users. The HIP engine never imports
it, and it imports nothing from the engine.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "warp_oracle.c")
LIB = os.path.join(_HERE, "liboracle.so")
FRAC_BITS = 26
EQ1_LITERAL = 1
M_MIN_RETRIEVED = 2

_lib = None


def build() -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math, OpenMP over queries)."""
    tmp = LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                           "-fno-fast-math", SRC, "-o", tmp, "-lm"])
    os.replace(tmp, LIB)
    return LIB


def build_variant(src_text: str, out_dir: str) -> str:
    """Compile oracle source text (for example a copy with a planted mistake) into
    out_dir/liboracle_variant.so with the same flags; returns its path."""
    c = os.path.join(out_dir, "warp_oracle.c")
    with open(c, "w") as f:
        f.write(src_text)
    so = os.path.join(out_dir, "liboracle_variant.so")
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
                           "-I", _HERE, c, "-o", so, "-lm"])
    return so


def load_library(path: str) -> ctypes.CDLL:
    """A compiled oracle library with its function signatures set."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_centroid_scores.argtypes = [P, i32, i32, P, P]
    lib.oracle_centroid_scores.restype = None
    lib.oracle_select.argtypes = [P, P, i32, i32, i64, P, P]
    lib.oracle_select.restype = None
    lib.oracle_token_scores.argtypes = [P, i32, f64, P, i32, P, i64, i64, P]
    lib.oracle_token_scores.restype = None
    lib.oracle_search.argtypes = [P, i32, i32, P, P, P, i32, P, i32, P, i32, i32, i32, i64, i32,
                                  i32, P, P, P, P, P, P, P, P, P, i32]
    lib.oracle_search.restype = ctypes.c_int
    lib.oracle_build_index.argtypes = [P, P, i64, P, i32, P, i64, i32, i32, i64, P, P, P, P, P, P, P, i32]
    lib.oracle_build_index.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _lib = load_library(LIB)
    return _lib


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def centroid_scores(centroids: np.ndarray, q: np.ndarray) -> np.ndarray:
    C = _c(centroids, np.float32)
    q = _c(q, np.float32)
    out = np.empty(C.shape[0], np.float64)
    _load().oracle_centroid_scores(_ptr(C), C.shape[0], C.shape[1], _ptr(q), _ptr(out))
    return out


def select(scores: np.ndarray, offsets: np.ndarray, nprobe: int, t_prime: int):
    s = _c(scores, np.float64)
    off = _c(offsets, np.int64)
    sel = np.empty(nprobe, np.int32)
    m = ctypes.c_double()
    _load().oracle_select(_ptr(s), _ptr(off), len(s), nprobe, int(t_prime), _ptr(sel), ctypes.byref(m))
    return sel, m.value


def token_scores(q, centroid_score: float, codes, nbits: int, bucket_weights, e0: int, e1: int):
    q = _c(q, np.float32)
    codes = _c(codes, np.uint8)
    w = _c(bucket_weights, np.float32)
    out = np.empty(max(0, e1 - e0), np.int32)
    _load().oracle_token_scores(_ptr(q), len(q), float(centroid_score), _ptr(codes), nbits, _ptr(w),
                                e0, e1, _ptr(out))
    return out


def search(centroids, offsets, doc_ids, codes, nbits, bucket_weights, n_docs, queries, nprobe,
           t_prime, k, flags: int = 0, debug: bool = True, doc_scores: bool = False,
           threads: int = 0, lib: ctypes.CDLL | None = None) -> dict:
    """Run the oracle on a batch of queries [n_queries, n_qtok, dim] (with `lib`, a
    library from load_library instead of the built oracle)."""
    C = _c(centroids, np.float32)
    off = _c(offsets, np.int64)
    ids = _c(doc_ids, np.int32)
    cd = _c(codes, np.uint8)
    w = _c(bucket_weights, np.float32)
    Q = _c(queries, np.float32)
    if Q.ndim == 2:
        Q = Q[None]
    nq, nt, dim = Q.shape
    n_c = C.shape[0]
    words = (n_docs + 31) // 32
    r = {
        "ids": np.empty((nq, k), np.int32),
        "fixed": np.empty((nq, k), np.int64),
        "scores": np.empty((nq, k), np.float32),
        "counts": np.empty(nq, np.int32),
    }
    if debug:
        r["sel"] = np.empty((nq, nt, nprobe), np.int32)
        r["m_fixed"] = np.empty((nq, nt), np.int64)
        r["cand_bitmap"] = np.empty((nq, words), np.uint32)
        r["n_scored"] = np.empty(nq, np.int64)
    if doc_scores:
        r["doc_fixed"] = np.empty((nq, n_docs), np.int64)
    rc = (lib or _load()).oracle_search(
        _ptr(C), n_c, dim, _ptr(off), _ptr(ids), _ptr(cd), nbits, _ptr(w), int(n_docs), _ptr(Q), nq, nt,
        nprobe, int(t_prime), k, flags, _ptr(r["ids"]), _ptr(r["fixed"]), _ptr(r["scores"]),
        _ptr(r["counts"]), _ptr(r.get("sel")), _ptr(r.get("m_fixed")), _ptr(r.get("cand_bitmap")),
        _ptr(r.get("n_scored")), _ptr(r.get("doc_fixed")), int(threads))
    if rc != 0:
        raise ValueError("oracle_search rejected its arguments")
    return r


def search_index(idx, queries=None, nprobe=None, t_prime=None, k=None, **kw) -> dict:
    """`search` on a synth.SyntheticIndex with its workload's parameters as defaults."""
    w = idx.workload
    return search(idx.centroids, idx.offsets, idx.doc_ids, idx.codes, idx.nbits, idx.bucket_weights,
                  idx.n_docs, idx.queries if queries is None else queries,
                  w.nprobe if nprobe is None else nprobe, w.t_prime if t_prime is None else t_prime,
                  w.k if k is None else k, **kw)


def build_index(tokens, token_docs, init_centroids, sample_ids, iterations: int, nbits: int, n_quant: int,
                threads: int = 0) -> dict:
    """Section 4.1's index construction (oracle_build_index) on host arrays."""
    X = _c(tokens, np.float32)
    docs = _c(token_docs, np.int32)
    C0 = _c(init_centroids, np.float32)
    S = _c(sample_ids, np.int64)
    n, n_c = X.shape[0], C0.shape[0]
    nb = 1 << nbits
    r = {
        "centroids": np.empty((n_c, 128), np.float32),
        "offsets": np.empty(n_c + 1, np.int64),
        "doc_ids": np.empty(n, np.int32),
        "codes": np.empty((n, 16 * nbits), np.uint8),
        "weights": np.empty(nb, np.float32),
        "cutoffs": np.empty(nb - 1, np.float32),
        "assign": np.empty(n, np.int32),
    }
    rc = _load().oracle_build_index(
        _ptr(X), _ptr(docs), n, _ptr(C0), n_c, _ptr(S), len(S), int(iterations), int(nbits), int(n_quant),
        _ptr(r["centroids"]), _ptr(r["offsets"]), _ptr(r["doc_ids"]), _ptr(r["codes"]), _ptr(r["weights"]),
        _ptr(r["cutoffs"]), _ptr(r["assign"]), int(threads))
    if rc != 0:
        raise ValueError("oracle_build_index rejected its arguments")
    return r
