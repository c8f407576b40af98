"""WARP multi-vector search engine for AMD Instinct MI355X (gfx950).

The search path (WARP_SELECT, implicit decompression, two-stage reduction,
top-k) runs in hand-written HIP kernels behind the C ABI of include/warp.h;
`warp` is its Python binding.
"""
from .warp import (  # noqa: F401
    EINVAL, EDEVICE, ENOMEM, ENOTSUP, EXPORTS, FRAC_BITS, SCORING_EQ1_LITERAL, SCORING_PAPER, STAGES, T_PRIME_C,
    T_PRIME_MAX, Index, WarpError, build_index, initial_centroids, last_error, lib, sample_passages, t_prime_policy,
)
