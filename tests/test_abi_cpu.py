"""The C ABI without a GPU: the library loads, exports every declared entry point,
and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "warp.h")
HAS_GPU = os.path.exists("/dev/kfd")

w = pytest.importorskip("paper_2501_17788_amd")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(warp_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 12
    lib = ctypes.CDLL(w.warp.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), f"{name} declared in warp.h but not exported"
    assert sorted(w.EXPORTS) == names


def test_fixed_point_bits():
    assert w.FRAC_BITS == 26


def test_null_handles():
    lib = w.lib
    lib.warp_index_free(None)  # NULL-safe
    rc = lib.warp_search(None, None, 1, 32, 1, 0, 1, None, None, None)
    assert rc == w.EINVAL
    rc = lib.warp_index_info(None, None, None, None, None)
    assert rc == w.EINVAL and "handle" in w.last_error()
    assert lib.warp_index_sync(None, None) == w.EINVAL
    assert lib.warp_set_timing(None, 1) == w.EINVAL


def test_unknown_handle_is_rejected():
    """A pointer that no load returned is not a live handle: every call rejects it without
    reading through it, and freeing it is a no-op."""
    lib = w.lib
    junk = ctypes.create_string_buffer(4096)  # readable memory that is not an index
    h = ctypes.cast(junk, ctypes.c_void_p)
    lib.warp_index_free(h)
    assert "invalid" in w.last_error()
    assert lib.warp_index_info(h, None, None, None, None) == w.EINVAL
    assert lib.warp_index_sync(h, None) == w.EINVAL
    assert lib.warp_set_scoring(h, 0) == w.EINVAL
    assert lib.warp_set_timing(h, 1) == w.EINVAL
    Q = np.zeros((1, 4, 128), np.float32)
    ids = np.empty((1, 2), np.int32)
    sc = np.empty((1, 2), np.float32)
    P = ctypes.c_void_p
    rc = lib.warp_search(h, Q.ctypes.data_as(P), 1, 4, 1, 0, 2, ids.ctypes.data_as(P), sc.ctypes.data_as(P), None)
    assert rc == w.EINVAL and "handle" in w.last_error()


def _arrays(**over):
    idx = synth.make_index(synth.random_small_workload(3, n_centroids=6, n_docs=20), workers=1)
    a = dict(centroids=idx.centroids, offsets=idx.offsets, doc_ids=idx.doc_ids, codes=idx.codes,
             nbits=idx.nbits, bucket_weights=idx.bucket_weights, n_docs=idx.n_docs)
    a.update(over)
    return a


def _load_rc(a):
    try:
        w.Index(**a)
    except w.WarpError as e:
        return e.code, e.msg
    return 0, ""


@pytest.mark.parametrize("case,code,needle", [
    ("bad_offsets", w.EINVAL, "decrease"),
    ("first_offset", w.EINVAL, "offsets[0]"),
    ("big_weight", w.EINVAL, "bucket weight"),
    ("weight_above_1.99", w.EINVAL, "bucket weight"),
    ("nan_weight", w.EINVAL, "bucket weight"),
    ("non_unit", w.EINVAL, "unit norm"),
    ("n_docs_zero", w.EINVAL, "n_docs"),
    ("n_docs_huge", w.EINVAL, "n_docs"),
    ("nbits3", w.EINVAL, "nbits"),
])
def test_index_validation_before_device(case, code, needle):
    a = _arrays()
    if case == "bad_offsets":
        off = a["offsets"].copy()
        off[2], off[3] = off[3], off[2] - 1 if off[2] > 0 else -1
        a["offsets"] = off
    elif case == "first_offset":
        a["offsets"] = a["offsets"] + 1
        a["offsets"][-1] -= 1
    elif case == "big_weight":
        a["bucket_weights"] = a["bucket_weights"].copy()
        a["bucket_weights"][0] = -2.5
    elif case == "weight_above_1.99":
        a["bucket_weights"] = a["bucket_weights"].copy()
        a["bucket_weights"][-1] = 1.995
    elif case == "nan_weight":
        a["bucket_weights"] = a["bucket_weights"].copy()
        a["bucket_weights"][1] = np.nan
    elif case == "non_unit":
        a["centroids"] = a["centroids"] * 1.01
    elif case == "n_docs_zero":
        a["n_docs"] = 0
    elif case == "n_docs_huge":
        a["n_docs"] = (1 << 24) + 1
    elif case == "nbits3":
        # bypass the binding's shape checks: call the C entry point directly
        h = ctypes.c_void_p()
        C = np.ascontiguousarray(a["centroids"])
        rc = w.lib.warp_index_load(C.ctypes.data_as(ctypes.c_void_p), len(C), 128,
                                   a["offsets"].ctypes.data_as(ctypes.c_void_p),
                                   a["doc_ids"].ctypes.data_as(ctypes.c_void_p),
                                   a["codes"].ctypes.data_as(ctypes.c_void_p), 3,
                                   a["bucket_weights"].ctypes.data_as(ctypes.c_void_p), 20, ctypes.byref(h))
        assert rc == code and needle in w.last_error()
        assert h.value is None
        return
    rc, msg = _load_rc(a)
    assert rc == code and needle in msg, (rc, msg)


def test_unsupported_shapes():
    a = _arrays()
    h = ctypes.c_void_p()
    P = ctypes.c_void_p
    rc = w.lib.warp_index_load(a["centroids"].ctypes.data_as(P), 6, 64, a["offsets"].ctypes.data_as(P),
                               a["doc_ids"].ctypes.data_as(P), a["codes"].ctypes.data_as(P), 4,
                               a["bucket_weights"].ctypes.data_as(P), 20, ctypes.byref(h))
    assert rc == w.ENOTSUP and "dim" in w.last_error()


@pytest.mark.skipif(HAS_GPU, reason="checks the no-device error path")
def test_valid_index_without_device_reports_edevice():
    rc, msg = _load_rc(_arrays())
    assert rc == w.EDEVICE and "device" in msg


def test_t_prime_policy():
    """Section 4.6: t' proportional to sqrt(N), bounded by t'_max (computed on the host)."""
    import math

    from paper_2501_17788_amd import t_prime_policy

    for n in (0, 1, 99, 10_000, 6_305_539, 70_000_000, 10 ** 12):
        for c in (0.0, 1.0, 15.8, 100.0):
            for t_max in (0, 1000, 100_000, 10 ** 15):
                want = min(t_max, math.floor(c * math.sqrt(n)))
                assert t_prime_policy(n, c, t_max) == want, (n, c, t_max)
    # proportional to sqrt(N) below the cap, constant above it
    assert t_prime_policy(4 * 1_000_000, 10.0, 10 ** 9) == 2 * t_prime_policy(1_000_000, 10.0, 10 ** 9)
    assert t_prime_policy(10 ** 12, 15.8, 100_000) == 100_000
    # the defaults give the synthetic workloads' t': 40,000 for small (capped at 100,000 beyond)
    assert abs(t_prime_policy(6_305_539) - 40_000) < 1000
    for bad in ((-1, 1.0, 10), (10, -1.0, 10), (10, float("nan"), 10), (10, 1.0, -1)):
        with pytest.raises(w.WarpError) as e:
            t_prime_policy(*bad)
        assert e.value.code == w.EINVAL


def test_kmeans_sample_size():
    """Section 4.1: the k-means sample of passages grows with the square root of the collection
    (computed on the host), never more than the collection; sample_passages draws that many."""
    import ctypes
    import math

    from paper_2501_17788_amd import sample_passages

    def size(n, c):
        out = ctypes.c_int64()
        rc = w.lib.warp_kmeans_sample_size(n, c, ctypes.byref(out))
        assert rc == 0, w.last_error()
        return out.value

    for n in (0, 1, 15, 256, 257, 100_000, 8_800_000):
        for c in (0.0, 1.0, 16.0):
            assert size(n, c) == min(n, math.ceil(c * math.sqrt(n))), (n, c)
    assert size(100_000, 16.0) == 5060  # the small workload's sample (16 sqrt(100,000) = 5059.6)
    assert size(4 * 10 ** 6, 16.0) == 2 * size(10 ** 6, 16.0)
    for bad in ((-1, 1.0), (10, -1.0), (10, float("nan"))):
        assert w.lib.warp_kmeans_sample_size(bad[0], bad[1], ctypes.byref(ctypes.c_int64())) == w.EINVAL
    assert w.lib.warp_kmeans_sample_size(10, 1.0, None) == w.EINVAL
    lens = np.full(400, 3, np.int64)
    ids = sample_passages(lens, 4.0, seed=1)
    assert len(ids) == 3 * 80 and len(np.unique(ids // 3)) == 80  # 4 sqrt(400) passages of 3 tokens

