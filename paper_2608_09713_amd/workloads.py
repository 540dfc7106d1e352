"""Seeded synthetic sparse matrices shaped like the paper's workloads.

This module only draws inputs. It holds none of the method's arithmetic
(no products, no transposes, no accumulation) and is shared by the oracle
tests, the GPU parity tests and the benchmark.

The paper evaluates on real matrices (Sec. V-A, Table 3) that are not
available here; these generators stand in for them:

* ``uniform``  -- every row holds exactly ``d`` distinct columns drawn
  uniformly without replacement (the tiny case and the off-diagonal blocks).
* ``kmer``     -- genomics k-mer overlap shape (Sec. I; the ELBA/BELLA overlap
  use): ``d`` distinct columns per row drawn from a bounded Zipf law of
  exponent ``s`` over the column ranks, ranks mapped to column ids through a
  seeded odd-multiplier bijection, then every column holding more than
  ``max_col`` entries is dropped (high-frequency k-mers are filtered).
* ``rmat``     -- Kronecker / power-law graph (stands in for
  ``kron_g500-logn21`` of Table 3): R-MAT edges, duplicates merged,
  self-loops dropped, a seeded symmetric vertex relabel (the random
  permutation of Sec. III-A), kept directed.

All matrices are canonical CSR: int64 ``row_ptr``, int32 ``col_idx``
strictly increasing within each row, 0-based.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import os
from typing import Optional

import numpy as np

GENERATOR_VERSION = 1


@dataclasses.dataclass
class CSR:
    nrows: int
    ncols: int
    row_ptr: np.ndarray            # int64 [nrows + 1]
    col_idx: np.ndarray            # int32 [nnz]
    values: Optional[np.ndarray]   # float64 / float32 [nnz] or None (pattern only)

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def with_values(self, values: Optional[np.ndarray]) -> "CSR":
        return CSR(self.nrows, self.ncols, self.row_ptr, self.col_idx, values)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def rng_for(seed: int, *stream: int) -> np.random.Generator:
    """Independent PCG64 stream per (seed, config, block)."""
    return np.random.default_rng(np.random.SeedSequence(entropy=seed, spawn_key=tuple(stream)))


# --------------------------------------------------------------------------
# helpers


def _rows_from_matrix(cols: np.ndarray, ncols: int) -> tuple[np.ndarray, np.ndarray]:
    """(m, d) array of per-row distinct columns -> canonical CSR arrays."""
    m, d = cols.shape
    cols = np.sort(cols, axis=1)
    row_ptr = np.arange(0, (m + 1) * d, d, dtype=np.int64)
    return row_ptr, np.ascontiguousarray(cols.reshape(-1)).astype(np.int32)


def _dedup_rows(draw, m: int, d: int) -> np.ndarray:
    """Draw an (m, d) matrix whose rows hold distinct values.

    ``draw(k)`` returns ``k`` fresh samples.  Duplicates inside a row are
    redrawn until none remain (sampling without replacement by rejection).
    """
    a = draw(m * d).reshape(m, d)
    while True:
        a.sort(axis=1)
        dup = np.zeros(a.shape, dtype=bool)
        dup[:, 1:] = a[:, 1:] == a[:, :-1]
        k = int(dup.sum())
        if k == 0:
            return a
        a[dup] = draw(k)


def _values(rng: np.random.Generator, nnz: int, dtype) -> np.ndarray:
    """Values in (0, 1]: 1 - U[0, 1)."""
    v = 1.0 - rng.random(nnz)
    if dtype == np.float32:
        v = v.astype(np.float32)
        v[v == 0] = np.float32(1.0)  # cannot happen for 1-U, kept as a guard
    return v


# --------------------------------------------------------------------------
# bounded Zipf by rejection-inversion (Hoermann & Derflinger, ACM TOMACS 1996)


class BoundedZipf:
    """Exact sampler of P(r) proportional to r^-s on r = 1..N, any s > 0.

    Rejection-inversion against the continuous hat h(x) = x^-s: invert the
    integral of the hat on [1.5, N + 0.5], round to the nearest integer and
    accept with the squeeze of the published method.  numpy's own ``zipf``
    needs s > 1 and is unbounded, so it cannot serve s = 0.9.
    """

    def __init__(self, n: int, s: float):
        self.n = int(n)
        self.s = float(s)
        self.hx1 = self._H(1.5) - 1.0
        self.hn = self._H(self.n + 0.5)
        self.squeeze = 2.0 - self._Hinv(self._H(2.5) - self._h(2.0))

    @staticmethod
    def _expm1_over(x):
        x = np.asarray(x, dtype=np.float64)
        small = np.abs(x) <= 1e-8
        safe = np.where(small, 1.0, x)
        return np.where(small, 1.0 + 0.5 * x * (1.0 + x / 3.0 * (1.0 + 0.25 * x)), np.expm1(safe) / safe)

    @staticmethod
    def _log1p_over(x):
        x = np.asarray(x, dtype=np.float64)
        small = np.abs(x) <= 1e-8
        safe = np.where(small, 1.0, x)
        return np.where(small, 1.0 - x * (0.5 - x * (1.0 / 3.0 - 0.25 * x)), np.log1p(safe) / safe)

    def _h(self, x):
        return np.exp(-self.s * np.log(x))

    def _H(self, x):
        q = 1.0 - self.s
        if abs(q) > 1e-6:
            return np.expm1(q * np.log(x)) / q
        lx = np.log(x)
        return self._expm1_over(q * lx) * lx

    def _Hinv(self, y):
        q = 1.0 - self.s
        t = np.maximum(y * q, -1.0)
        if abs(q) > 1e-6:
            # exp(log1p(t) / q), with t = q * y
            return np.exp(np.log1p(t) / q)
        return np.exp(self._log1p_over(t) * y)

    def sample(self, rng: np.random.Generator, k: int) -> np.ndarray:
        """``k`` draws.  Large requests are cut into fixed 2^22 chunks, each
        from its own stream spawned off ``rng`` and run on a thread pool, so
        the result depends only on ``rng``'s state, not on the thread count."""
        chunk = 1 << 22
        if k <= chunk:
            return self._sample_one(rng, k)
        nchunks = (k + chunk - 1) // chunk
        subs = rng.spawn(nchunks)
        out = np.empty(k, dtype=np.int64)

        def job(c):
            lo = c * chunk
            hi = min(k, lo + chunk)
            out[lo:hi] = self._sample_one(subs[c], hi - lo)

        with concurrent.futures.ThreadPoolExecutor(max_workers=_threads()) as ex:
            list(ex.map(job, range(nchunks)))
        return out

    def _sample_one(self, rng: np.random.Generator, k: int) -> np.ndarray:
        out = np.empty(k, dtype=np.int64)
        todo = None
        n_todo = k
        while n_todo:
            u = rng.random(n_todo)
            u *= self.hx1 - self.hn
            u += self.hn
            x = self._Hinv(u)
            r = np.floor(x + 0.5)
            np.clip(r, 1, self.n, out=r)
            ok = (r - x) <= self.squeeze
            rest = np.flatnonzero(~ok)
            if rest.size:
                rr = r[rest]
                ok[rest] = u[rest] >= self._H(rr + 0.5) - self._h(rr)
            if todo is None:
                out[ok] = r[ok]
                todo = np.flatnonzero(~ok)
            else:
                out[todo[ok]] = r[ok]
                todo = todo[~ok]
            n_todo = todo.size
        return out


def _rank_to_col(rng: np.random.Generator, ncols: int):
    """Seeded bijection of ranks 1..ncols onto column ids 0..ncols-1.

    ncols must be a power of two: c = (a * (r - 1) + b) mod ncols with odd a.
    """
    assert ncols & (ncols - 1) == 0, "k-mer column space must be a power of two"
    a = int(rng.integers(0, ncols // 2)) * 2 + 1
    b = int(rng.integers(0, ncols))
    mask = ncols - 1

    def f(r: np.ndarray) -> np.ndarray:
        return ((np.uint64(a) * (r.astype(np.uint64) - np.uint64(1)) + np.uint64(b)) & np.uint64(mask)).astype(np.int64)

    return f


# --------------------------------------------------------------------------
# generators


def uniform(nrows: int, ncols: int, d: int, rng: np.random.Generator, dtype=np.float64,
            values: bool = True) -> CSR:
    """Exactly ``d`` distinct uniform columns per row, values U(0,1]."""
    if d > ncols:
        raise ValueError("d > ncols")
    cols = _dedup_rows(lambda k: rng.integers(0, ncols, size=k, dtype=np.int64), nrows, d)
    row_ptr, col_idx = _rows_from_matrix(cols, ncols)
    vals = _values(rng, len(col_idx), dtype) if values else None
    return CSR(nrows, ncols, row_ptr, col_idx, vals)


def kmer(nrows: int, ncols: int, d: int, rng: np.random.Generator, s: float = 0.9,
         max_col: int = 50) -> CSR:
    """k-mer overlap shape: ``d`` distinct Zipf(s) columns per row, columns
    holding more than ``max_col`` entries removed, binary pattern."""
    z = BoundedZipf(ncols, s)
    to_col = _rank_to_col(rng, ncols)
    ranks = _dedup_rows(lambda k: z.sample(rng, k), nrows, d)
    cols = to_col(ranks.reshape(-1)).reshape(nrows, d)
    # column frequency (after per-row dedup); ranks are a bijection of columns
    counts = np.bincount(ranks.reshape(-1), minlength=ncols + 1)
    keep = counts[ranks] <= max_col
    del counts
    cols = np.sort(np.where(keep, cols, np.iinfo(np.int64).max), axis=1)
    lens = keep.sum(axis=1)
    row_ptr = np.zeros(nrows + 1, dtype=np.int64)
    np.cumsum(lens, out=row_ptr[1:])
    flat = cols.reshape(-1)
    col_idx = flat[flat != np.iinfo(np.int64).max].astype(np.int32)
    return CSR(nrows, ncols, row_ptr, col_idx, None)


def rmat(scale: int, edge_factor: int, rng: np.random.Generator,
         abcd=(0.57, 0.19, 0.19, 0.05), dtype=np.float32) -> CSR:
    """Directed R-MAT graph: 2^scale vertices, edge_factor * 2^scale draws,
    one quadrant choice per level, no noise; duplicates merged, self-loops
    dropped, symmetric random vertex relabel; weights U(0,1]."""
    nv = 1 << scale
    ne = edge_factor * nv
    a, b, c, _ = abcd
    src = np.zeros(ne, dtype=np.int64)
    dst = np.zeros(ne, dtype=np.int64)
    for _level in range(scale):
        u = rng.random(ne)
        sbit = u >= a + b                       # quadrants c, d: lower half
        dbit = ((u >= a) & (u < a + b)) | (u >= a + b + c)  # quadrants b, d: right half
        src = (src << 1) | sbit
        dst = (dst << 1) | dbit
    perm = rng.permutation(nv)
    src = perm[src]
    dst = perm[dst]
    keep = src != dst
    key = np.unique((src[keep] << scale) | dst[keep])
    src = key >> scale
    dst = key & (nv - 1)
    row_ptr = np.zeros(nv + 1, dtype=np.int64)
    np.cumsum(np.bincount(src, minlength=nv), out=row_ptr[1:])
    col_idx = dst.astype(np.int32)
    vals = _values(rng, len(col_idx), dtype)
    return CSR(nv, nv, row_ptr, col_idx, vals)


# --------------------------------------------------------------------------
# the five workloads (full size) and scaled-down parity variants

WORKLOADS = {
    "tiny_uniform_f64": "4096 x 16384, 8 uniform distinct columns per row, fp64 U(0,1]; lower",
    "kmer_i32": "2^20 x 2^26, 32 Zipf(0.9) distinct columns per row, columns > 50 dropped, binary; int32 counts, lower",
    "rmat20_f32": "R-MAT scale 20, edge factor 16, (.57,.19,.19,.05), dedup, no self-loops, fp32 U(0,1]; lower + mirror",
    "offdiag_f64": "two blocks 2^19 x 2^24, 24 uniform columns per row, fp64 U(0,1]; offdiag(Ai,Aj) and lower(Ai)",
    "jaccard_large": "2^23 x 2^28, 16 Zipf(0.9) distinct columns per row, columns > 50 dropped, binary; Jaccard fp32, lower",
}


def make(name: str, seed: int = 1, scale_shift: int = 0):
    """Build a named workload.

    ``scale_shift`` > 0 shrinks rows and columns by 2^scale_shift (R-MAT: the
    scale) while keeping the per-row structure, for parity tests the oracle
    finishes in seconds.  Returns a dict with the matrices and the semiring.
    """
    k = scale_shift
    if name == "tiny_uniform_f64":
        A = uniform(max(4096 >> k, 1), max(16384 >> k, 8), 8, rng_for(seed, 0, 0))
        return {"A": A, "semiring": "f64", "ops": ["lower"]}
    if name == "kmer_i32":
        A = kmer(max(1 << (20 - k), 1), 1 << (26 - k), 32, rng_for(seed, 1, 0))
        return {"A": A, "semiring": "count", "ops": ["lower"]}
    if name == "rmat20_f32":
        A = rmat(20 - k, 16, rng_for(seed, 2, 0))
        return {"A": A, "semiring": "f32", "ops": ["lower", "mirror"]}
    if name == "offdiag_f64":
        Ai = uniform(max(1 << (19 - k), 1), 1 << (24 - k), 24, rng_for(seed, 3, 0))
        Aj = uniform(max(1 << (19 - k), 1), 1 << (24 - k), 24, rng_for(seed, 3, 1))
        return {"A": Ai, "B": Aj, "semiring": "f64", "ops": ["offdiag", "lower"]}
    if name == "jaccard_large":
        A = kmer(max(1 << (23 - k), 1), 1 << (28 - k), 16, rng_for(seed, 4, 0))
        return {"A": A, "semiring": "jaccard", "ops": ["lower"]}
    raise KeyError(name)
