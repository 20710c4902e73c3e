"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no CKKS arithmetic: it only draws random numbers.  Every
random quantity the scheme consumes (database rows, queries, the projection
matrix, the secret key, key and encryption randomness, noise) is drawn here and
handed, identically, to the GPU library and to the CPU oracle.

Generators are NumPy PCG64 streams ``default_rng([workload_id, stream, ...])``.
The workloads stand in for the paper's public corpora (CLIP-like 512-d
embeddings with near-duplicates, 96-d descriptors zero-padded to 128, a face
centroid level); none of those datasets is read.
"""
from __future__ import annotations

import numpy as np

# stream ids
STREAM_DB = 0
STREAM_QUERY = 1
STREAM_W = 2
STREAM_SECRET = 3
STREAM_KEY_A = 4
STREAM_KEY_E = 5
STREAM_ENC_A = 6
STREAM_ENC_E = 7


def rng(workload_id: int, stream: int, *extra: int) -> np.random.Generator:
    return np.random.default_rng([int(workload_id), int(stream), *[int(x) for x in extra]])


def normalize_rows(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    nrm = np.linalg.norm(x, axis=-1, keepdims=True)
    nrm[nrm == 0] = 1.0
    return x / nrm


def gaussian_unit_rows(g: np.random.Generator, n: int, dim: int) -> np.ndarray:
    """n rows of N(0, I_dim), each scaled to unit L2 norm (float64)."""
    return normalize_rows(g.standard_normal((n, dim)))


def mixture_rows(g: np.random.Generator, n: int, dim: int, n_comp: int, sigma: float = 0.3,
                 dup_frac: float = 0.0, jitter: float = 0.01, centers: np.ndarray | None = None,
                 chunk: int = 1 << 16) -> np.ndarray:
    """Gaussian-mixture rows, unit L2 norm, float32.

    centres ~ N(0, I); row = centre[uniform component] + N(0, sigma^2 I), normalised.
    A fraction ``dup_frac`` of rows is replaced by near-duplicates of random
    non-duplicate rows: normalise(src + N(0, jitter^2 I)).
    """
    if centers is None:
        centers = g.standard_normal((n_comp, dim))
    out = np.empty((n, dim), dtype=np.float32)
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        comp = g.integers(0, centers.shape[0], size=m)
        x = centers[comp] + sigma * g.standard_normal((m, dim))
        out[s:s + m] = normalize_rows(x)
    n_dup = int(round(dup_frac * n))
    if n_dup > 0:
        dup_idx = g.choice(n, size=n_dup, replace=False)
        is_dup = np.zeros(n, dtype=bool)
        is_dup[dup_idx] = True
        src_pool = np.nonzero(~is_dup)[0]
        src = src_pool[g.integers(0, src_pool.size, size=n_dup)]
        x = out[src].astype(np.float64) + jitter * g.standard_normal((n_dup, dim))
        out[dup_idx] = normalize_rows(x)
    return out


def mixture_queries(g: np.random.Generator, n: int, dim: int, centers: np.ndarray,
                    sigma: float = 0.3) -> np.ndarray:
    comp = g.integers(0, centers.shape[0], size=n)
    return normalize_rows(centers[comp] + sigma * g.standard_normal((n, dim)))


def projection_matrix(g: np.random.Generator, d_in: int, r: int, var: float = 1.0 / 128) -> np.ndarray:
    """d_in x r matrix with i.i.d. N(0, var) entries (float64)."""
    return g.standard_normal((d_in, r)) * np.sqrt(var)


def ternary_secret(g: np.random.Generator, n: int) -> np.ndarray:
    """n coefficients uniform on {-1, 0, 1} (int64)."""
    return g.integers(-1, 2, size=n).astype(np.int64)


def rounded_gaussian(g: np.random.Generator, shape, sigma: float = 3.2, bound: int = 19) -> np.ndarray:
    """Rounded N(0, sigma^2) integers, resampled while |e| > bound (int64)."""
    shape = tuple(np.atleast_1d(shape))
    x = np.rint(g.standard_normal(shape) * sigma)
    bad = np.abs(x) > bound
    while bad.any():
        x[bad] = np.rint(g.standard_normal(int(bad.sum())) * sigma)
        bad = np.abs(x) > bound
    return x.astype(np.int64)


def uniform_residues(g: np.random.Generator, moduli, lead: int, n: int) -> np.ndarray:
    """[lead][len(moduli)][n] uint64 with entry [.., t, ..] uniform on [0, moduli[t])."""
    moduli = [int(m) for m in moduli]
    out = np.empty((lead, len(moduli), n), dtype=np.uint64)
    for i in range(lead):
        for t, m in enumerate(moduli):
            out[i, t] = g.integers(0, m, size=n, dtype=np.uint64)
    return out
