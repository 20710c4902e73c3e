"""The benchmark workloads and their seeded synthetic inputs.

Each workload is one configuration of the scoring path: ring size, primes,
candidate set, vector dimension and slot layout.  Inputs are drawn by
``gen`` (random numbers only, no CKKS arithmetic); the same draw feeds the
GPU library and the CPU oracle.  The candidate sets stand in for the paper's
public corpora (CLIP-like 512-d embeddings with near-duplicates; 96-d
descriptors zero-padded to 128; a face-centroid level); no dataset is read.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import gen


@dataclass
class Workload:
    name: str
    log_n: int
    L: int
    K: int
    rows: int
    dim: int
    d: int
    B: int
    wid: int
    desc: str
    n_comp: int = 0          # 0: isotropic Gaussian rows, else a Gaussian mixture
    dup: float = 0.0         # near-duplicate fraction
    layout: str = "diag"     # "diag" or "row"
    d_in: int = 0            # projection input dimension (0: no projection)
    B_proj: int = 0          # baby step of the projection
    extra: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return 1 << self.log_n

    @property
    def slots(self) -> int:
        return self.n // 2

    @property
    def G(self) -> int:
        return self.d // self.B

    @property
    def n_blocks(self) -> int:
        return -(-self.rows // self.slots)


WORKLOADS = {
    "tiny": Workload(
        "tiny", 13, 3, 1, rows=1024, dim=128, d=128, B=16, wid=1, layout="row",
        desc="tiny scoring: 1,024 x 128-d N(0,1) unit rows, CKKS N=2^13, 3+1 primes, row layout, "
             "ct x pt then 7 rotate-and-sum steps"),
    "fine": Workload(
        "fine", 15, 8, 2, rows=65_536, dim=96, d=128, B=32, wid=2, n_comp=1024,
        desc="fine level: 65,536 x 96-d (zero-padded to 128) mixture rows, CKKS N=2^15, 8+2 primes, "
             "diagonal blocks"),
    "rank": Workload(
        "rank", 16, 12, 3, rows=16_384, dim=128, d=128, B=16, wid=3, d_in=512, B_proj=16,
        desc="rank reduction: encrypted 512-d query projected by a plaintext 512x128 Gaussian W, then "
             "scored against 16,384 x 128-d candidates with norm correction, CKKS N=2^16, 12+3 primes"),
    "rerank": Workload(
        "rerank", 16, 12, 3, rows=110_000, dim=512, d=512, B=64, wid=4, n_comp=4096, dup=0.05,
        desc="rerank level: 110,000 x 512-d mixture rows with 5% near-duplicates vs one encrypted query, "
             "CKKS N=2^16, 12+3 primes of 50 bits, scale 2^40, diagonal blocks"),
    "three_level": Workload(
        "three_level", 16, 12, 3, rows=110_000, dim=512, d=512, B=64, wid=5, n_comp=4096, dup=0.05,
        desc="three-level query: coarse 222,049 + fine 65,536 + rerank 110,000 x 512-d per query, "
             "32 encrypted queries back to back, CKKS N=2^16, 12+3 primes",
        extra=dict(coarse=222_049, fine_pool_blocks=4, fine_blocks=2, rerank_pool_blocks=8, rerank_blocks=4,
                   rerank_last=11_696, queries=32, top_coarse=16, top_fine=64)),
    "face": Workload(
        "face", 16, 12, 3, rows=222_049, dim=128, d=128, B=32, wid=7, d_in=512, B_proj=16,
        desc="face membership scan: 222,049 identity centroids (unit 512-d rows, projected to R=128 and "
             "re-normalised) against one encrypted 512-d query, cos >= tau decided under encryption; "
             "CKKS N=2^16, 12+3 primes of 50 bits, scale 2^50 with rescaling, levels 12 -> 2",
        extra=dict(log_scale=50, tau=0.5, y_lo=0.5, y_hi=2.5, degree=7, m=4, iters=2, query_noise=1.0)),
}


def candidate_rows(w: Workload, n_rows: int | None = None, stream_extra: int = 0, centers=None):
    """(rows float32 [n][dim], centres or None) of the workload's candidate set; given
    centres are reused (several candidate pools around the same clusters)."""
    n_rows = w.rows if n_rows is None else n_rows
    g = gen.rng(w.wid, gen.STREAM_DB, stream_extra)
    if w.n_comp:
        if centers is None:
            centers = g.standard_normal((w.n_comp, w.dim))
        X = gen.mixture_rows(g, n_rows, w.dim, w.n_comp, sigma=0.3, dup_frac=w.dup, centers=centers)
        return X, centers
    return gen.gaussian_unit_rows(g, n_rows, w.dim).astype(np.float32), None


def raw_rows(w: Workload) -> np.ndarray:
    """The d_in-dimensional unit N(0, I) rows behind a projected workload (float64)."""
    return gen.gaussian_unit_rows(gen.rng(w.wid, gen.STREAM_DB), w.rows, w.d_in)


def projected_rows(w: Workload, W: np.ndarray) -> np.ndarray:
    """Candidates of a projected workload: normalise(W^T x) for its raw rows x, re-normalised
    at enrollment as the paper's client does (float64)."""
    return gen.normalize_rows(raw_rows(w) @ W)


def face_queries(w: Workload, count: int = 1):
    """Queries of the membership workload: each a noisy view of one enrolled identity,
    q = normalise(c_j + rho z/|z|) with z ~ N(0, I) and rho = query_noise, so that
    cos(q, c_j) is about 1/sqrt(1 + rho^2).  Returns (queries [count][d_in], identities j)."""
    g = gen.rng(w.wid, gen.STREAM_QUERY)
    C = raw_rows(w)
    j = g.integers(0, w.rows, count)
    z = gen.normalize_rows(g.standard_normal((count, w.d_in)))
    return gen.normalize_rows(C[j] + w.extra["query_noise"] * z), j


def query_vectors(w: Workload, count: int = 1, centers=None) -> np.ndarray:
    g = gen.rng(w.wid, gen.STREAM_QUERY)
    dim = w.d_in or w.dim
    if centers is not None:
        return gen.mixture_queries(g, count, dim, centers)
    return gen.gaussian_unit_rows(g, count, dim)


def projection(w: Workload) -> np.ndarray:
    return gen.projection_matrix(gen.rng(w.wid, gen.STREAM_W), w.d_in, w.d, var=1.0 / w.d)


def rotation_steps(w: Workload) -> list[int]:
    """Every rotation key the workload's scoring needs."""
    if w.layout == "row":
        steps = [1 << k for k in range(int(np.log2(w.d)))]
    else:
        steps = list(range(1, w.B)) + [g * w.B for g in range(1, w.G)]
    if w.d_in:
        Bp = w.B_proj
        steps += list(range(1, Bp)) + [g * Bp for g in range(1, w.d // Bp)]
        steps += [w.d << k for k in range(int(np.log2(w.d_in // w.d)))]
    return sorted(set(steps))


def key_randomness(w: Workload, step: int, primes, dnum: int):
    a = gen.uniform_residues(gen.rng(w.wid, gen.STREAM_KEY_A, step), primes, dnum, w.n)
    e = gen.rounded_gaussian(gen.rng(w.wid, gen.STREAM_KEY_E, step), (dnum, w.n))
    return a, e


def secret(w: Workload) -> np.ndarray:
    return gen.ternary_secret(gen.rng(w.wid, gen.STREAM_SECRET), w.n)


def enc_randomness(w: Workload, primes_q, tag: int = 0):
    a = gen.uniform_residues(gen.rng(w.wid, gen.STREAM_ENC_A, tag), primes_q, 1, w.n)[0]
    e = gen.rounded_gaussian(gen.rng(w.wid, gen.STREAM_ENC_E, tag), w.n)
    return a, e


def relin_randomness(w: Workload, primes, dnum: int):
    """Randomness of the relinearisation key (key streams, tag 0: rotation steps start at 1)."""
    return key_randomness(w, 0, primes, dnum)


def db_enc_randomness(w: Workload, primes_q, first: int, count: int, block: int = 0):
    """Encryption randomness of `count` database plaintexts starting at index `first` of
    block `block` (one generator per ciphertext, so any slice is reproducible):
    a [count][L][N] uniform residues, e [count][N] noise."""
    a = np.empty((count, len(primes_q), w.n), dtype=np.uint64)
    e = np.empty((count, w.n), dtype=np.int64)
    for j in range(count):
        tag = 1_000_000 + block * 100_000 + first + j
        a[j] = gen.uniform_residues(gen.rng(w.wid, gen.STREAM_ENC_A, tag), primes_q, 1, w.n)[0]
        e[j] = gen.rounded_gaussian(gen.rng(w.wid, gen.STREAM_ENC_E, tag), w.n)
    return a, e
