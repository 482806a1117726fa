"""Seeded generators for the similarity-join workloads.

Every workload is a pair of row-major point sets P (n_p x d) and Q (n_q x d)
stored in one of three element types, a metric ("ip": report (i, j) when
<P_i, Q_j> >= s; "l2": report (i, j) when ||P_i - Q_j||^2 <= r2) and a
threshold.  The problem statement is the similarity join of Section 4 of
Ahle & Silvestri, "Similarity Search with Tensor Core Units"; inner product
and cosine follow the ip-distance examples of the same section, and the
squared-L2 threshold applies to the squared distance.

Storage conventions (what both the oracle and the GPU library read):
  "f16"  -> numpy float16 array (IEEE binary16 bits)
  "bf16" -> numpy uint16 array holding bfloat16 bit patterns
  "i8"   -> numpy int8 array

Random numbers come from numpy's PCG64 (`default_rng(seed)`).  Planted pairs
are built so that they satisfy the predicate by construction wherever that is
possible without evaluating the predicate here (the tests check all of them
against the oracle).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

DTYPES = ("f16", "bf16", "i8")
ESIZE = {"f16": 2, "bf16": 2, "i8": 1}


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns.  NaNs map to a quiet NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    t = (u >> np.uint32(16)) & np.uint32(1)
    t += u
    t += np.uint32(0x7FFF)          # finite inputs cannot wrap around
    t >>= np.uint32(16)
    rounded = t.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded = rounded.copy()
        rounded[nan] = 0x7FC0
    return rounded


def encode(values: np.ndarray, dtype: str) -> np.ndarray:
    """Encode float64/int values into the storage array of `dtype`."""
    if dtype == "f16":
        return np.ascontiguousarray(np.asarray(values, dtype=np.float64).astype(np.float16))
    if dtype == "bf16":
        return bf16_bits_from_f32(np.asarray(values, dtype=np.float64).astype(np.float32))
    if dtype == "i8":
        v = np.asarray(values)
        if v.dtype.kind == "f":
            if not np.all(np.isfinite(v)) or np.any(v != np.round(v)):
                raise ValueError("int8 storage needs integer values")
        if v.size and (v.min() < -128 or v.max() > 127):
            raise ValueError("int8 storage needs values in [-128, 127]")
        return np.ascontiguousarray(v.astype(np.int8))
    raise ValueError(f"unknown dtype {dtype!r}")


@dataclass
class Workload:
    name: str
    metric: str            # "ip" or "l2"
    dtype: str             # "f16", "bf16" or "i8"
    P: np.ndarray          # storage array, shape (n_p, d)
    Q: np.ndarray          # storage array, shape (n_q, d); may be P itself
    threshold: float       # s for "ip", r2 for "l2"
    planted: np.ndarray    # (m, 2) int64 index pairs that must match
    decoys: np.ndarray = field(default_factory=lambda: np.zeros((0, 2), np.int64))
    real_valued: bool = False   # True when stored values are not integers
    self_join: bool = False     # True when Q is P (same array)
    description: str = ""

    @property
    def n_p(self) -> int:
        return int(self.P.shape[0])

    @property
    def n_q(self) -> int:
        return int(self.Q.shape[0])

    @property
    def d(self) -> int:
        return int(self.P.shape[1])

    @property
    def pair_evals(self) -> int:
        return self.n_p * self.n_q


# Full-size shapes of the five workloads, by name.  The default seed of a
# workload is 1000 + its position in this table.
CONFIGS = {
    "ip_f16_2048x64": dict(n=2048, d=64, dtype="f16", metric="ip", threshold=300.0,
                           planted=50),
    "ip_bf16_65536x128": dict(n=65536, d=128, dtype="bf16", metric="ip", threshold=308.0,
                              planted=10_000),
    "cos_f16_262144x256": dict(n=262144, d=256, dtype="f16", metric="ip", threshold=0.9,
                               planted=100_000),
    "l2_i8_1048576x64": dict(n=1048576, d=64, dtype="i8", metric="l2", threshold=2000.0,
                             planted=1_000_000),
    "ip_bf16_clustered_131072x1024": dict(n=131072, d=1024, dtype="bf16", metric="ip",
                                          threshold=125.0, planted=0),
}
NAMES = list(CONFIGS)


def _pick_pairs(rng, n_p, n_q, m):
    """m index pairs with distinct P rows and distinct Q rows."""
    m = min(m, n_p, n_q)
    ip = rng.permutation(n_p)[:m]
    iq = rng.permutation(n_q)[:m]
    return np.stack([ip, iq], axis=1).astype(np.int64)


def _scaled(count, n, n_full, minimum=1):
    if count == 0:
        return 0
    return max(minimum, int(round(count * n / n_full)))


def make_config(name: str, n: int | None = None, seed: int | None = None,
                self_join: bool = False) -> Workload:
    """Build the named workload.  `n` overrides |P| = |Q| (planted counts are
    scaled with n) so the same distribution can be checked at small sizes."""
    cfg = CONFIGS[name]
    pos = NAMES.index(name)
    n_full = cfg["n"]
    n = n_full if n is None else int(n)
    seed = 1000 + pos if seed is None else seed
    rng = np.random.default_rng(seed)
    d = cfg["d"]
    builder = (_ip_f16_small, _ip_bf16, _cos_f16, _l2_i8, _ip_bf16_clustered)[pos]
    w = builder(rng, n, d, _scaled(cfg["planted"], n, n_full), self_join)
    if self_join and not w.self_join:
        # the workload's P joined with itself (its planted pairs refer to Q)
        w.Q = w.P
        w.self_join = True
        w.planted = np.zeros((0, 2), np.int64)
        w.decoys = np.zeros((0, 2), np.int64)
        w.description += "; Q is P"
    w.name = name if n == n_full else f"{name}@n={n}"
    return w


def _ip_f16_small(rng, n, d, planted, self_join):
    """fp16 integers uniform in [-8, 8]; Q rows overwritten by copies of P rows."""
    Pv = rng.integers(-8, 9, size=(n, d))
    if self_join:
        P = encode(Pv, "f16")
        pl = np.stack([np.arange(n), np.arange(n)], 1)[:0]
        return Workload("", "ip", "f16", P, P, 300.0, pl, self_join=True,
                        description="fp16 integers U{-8..8}, Q is P")
    Qv = rng.integers(-8, 9, size=(n, d))
    pl = _pick_pairs(rng, n, n, planted)
    Qv[pl[:, 1]] = Pv[pl[:, 0]]
    return Workload("", "ip", "f16", encode(Pv, "f16"), encode(Qv, "f16"), 300.0, pl,
                    description="fp16 integers U{-8..8}; planted y = x")


def _ip_bf16(rng, n, d, planted, self_join):
    """bf16 integers uniform in [-4, 4]; planted y = x with 6 of 128 coordinates
    (5 %) redrawn from the same distribution."""
    Pv = rng.integers(-4, 5, size=(n, d))
    Qv = rng.integers(-4, 5, size=(n, d))
    pl = _pick_pairs(rng, n, n, planted)
    nres = int(round(0.05 * d))
    for t in range(pl.shape[0]):
        y = Pv[pl[t, 0]].copy()
        idx = rng.choice(d, size=nres, replace=False)
        y[idx] = rng.integers(-4, 5, size=nres)
        Qv[pl[t, 1]] = y
    return Workload("", "ip", "bf16", encode(Pv, "bf16"), encode(Qv, "bf16"), 308.0, pl,
                    description="bf16 integers U{-4..4}; planted y = x with 5% coords redrawn")


def _unit_rows(X):
    return X / np.linalg.norm(X, axis=1, keepdims=True)


def _cos_f16(rng, n, d, planted, self_join):
    """fp16 unit rows: Gaussian rows normalised in float64 then rounded to fp16;
    planted y = normalise(x + 0.3 g) with g ~ N(0, I/d)."""
    Px = _unit_rows(rng.standard_normal((n, d)))
    Qx = _unit_rows(rng.standard_normal((n, d)))
    pl = _pick_pairs(rng, n, n, planted)
    g = rng.standard_normal((pl.shape[0], d)) / np.sqrt(d)
    Qx[pl[:, 1]] = _unit_rows(Px[pl[:, 0]] + 0.3 * g)
    return Workload("", "ip", "f16", encode(Px, "f16"), encode(Qx, "f16"), 0.9, pl,
                    real_valued=True,
                    description="fp16 unit Gaussian rows (cosine); planted normalise(x+0.3g)")


def _l2_i8(rng, n, d, planted, self_join):
    """int8 integers uniform in [-15, 15]; squared radius 2000.

    Planted pairs: y = clamp(x + delta, -15, 15) with delta uniform in [-5, 5];
    clamping toward the interval that holds x only shrinks |y_k - x_k|, so
    ||x - y||^2 <= 64 * 25 = 1600 <= 2000 for every one of them.
    Ties (about 1 per 1000 planted): 16 coordinates moved 11 toward zero and 16
    moved 2 toward zero give ||x - y||^2 = 16*121 + 16*4 = 2000 exactly.
    Decoys (as many as ties, never matching): the same plus one more coordinate
    moved by 1 gives 2001."""
    assert d == 64
    Pv = rng.integers(-15, 16, size=(n, d), dtype=np.int8)
    Qv = rng.integers(-15, 16, size=(n, d), dtype=np.int8)
    n_ties = max(1, planted // 1000) if planted >= 2 else 0
    n_dec = n_ties
    allp = _pick_pairs(rng, n, n, planted + n_dec)
    pl, dec = allp[:planted], allp[planted:]
    n_rand = planted - n_ties
    xr = Pv[pl[:n_rand, 0]]
    xr += rng.integers(-5, 6, size=xr.shape, dtype=np.int8)   # |x + delta| <= 20: no wrap
    np.clip(xr, -15, 15, out=xr)
    Qv[pl[:n_rand, 1]] = xr

    def toward_zero(x, idx, step):
        # move x[idx] toward zero by `step`; x == 0 moves to +step
        s = np.where(x[idx] > 0, -1, np.where(x[idx] < 0, 1, 1))
        x[idx] = x[idx] + s * step

    for rows, extra in ((pl[n_rand:], 0), (dec, 1)):
        for t in range(rows.shape[0]):
            y = Pv[rows[t, 0]].astype(np.int64)
            idx = rng.permutation(d)
            toward_zero(y, idx[:16], 11)
            toward_zero(y, idx[16:32], 2)
            if extra:
                toward_zero(y, idx[32:33], 1)
            Qv[rows[t, 1]] = y
    return Workload("", "l2", "i8", encode(Pv, "i8"), encode(Qv, "i8"), 2000.0, pl, decoys=dec,
                    description="int8 integers U{-15..15}; planted within r; exact ties at 2000")


def _ip_bf16_clustered(rng, n, d, planted, self_join):
    """bf16 integers in [-2, 2] around 256 seeded cluster centres; each
    coordinate is independently redrawn from U{-2..2} with probability 0.1.
    Cluster labels are uniform and rows are not sorted by cluster."""
    n_cent = 256
    C = rng.integers(-2, 3, size=(n_cent, d)).astype(np.int8)

    def rows(m):
        lab = rng.integers(0, n_cent, size=m)
        X = C[lab]
        flip = rng.random((m, d), dtype=np.float32) < 0.1
        X[flip] = rng.integers(-2, 3, size=int(flip.sum()), dtype=np.int8)
        return X, lab

    Pv, lp = rows(n)
    Qv, lq = rows(n)
    w = Workload("", "ip", "bf16", bf16_bits_from_f32(Pv.astype(np.float32)),
                 bf16_bits_from_f32(Qv.astype(np.float32)), 125.0, np.zeros((0, 2), np.int64),
                 description="bf16 clustered integers, 256 centres, 10% coords redrawn")
    w.labels_p, w.labels_q = lp, lq
    return w


def random_case(seed: int, n_p: int, n_q: int, d: int, dtype: str, lo: int = -4, hi: int = 4,
                real: bool = False, metric: str = "ip", threshold: float = 0.0) -> Workload:
    """Uniform integer entries in [lo, hi] (or, with real=True, Gaussian entries
    scaled by 1/sqrt(d) for fp16/bf16)."""
    rng = np.random.default_rng(seed)
    if real:
        if dtype == "i8":
            raise ValueError("real-valued int8 makes no sense")
        Pv = rng.standard_normal((n_p, d)) / np.sqrt(max(d, 1))
        Qv = rng.standard_normal((n_q, d)) / np.sqrt(max(d, 1))
    else:
        Pv = rng.integers(lo, hi + 1, size=(n_p, d))
        Qv = rng.integers(lo, hi + 1, size=(n_q, d))
    return Workload(f"rand{seed}_{n_p}x{n_q}x{d}_{dtype}", metric, dtype, encode(Pv, dtype),
                    encode(Qv, dtype), threshold, np.zeros((0, 2), np.int64), real_valued=real)


def to_torch(X: np.ndarray, dtype: str, device="cuda"):
    """The storage array as a torch tensor of the matching element type
    (float16, bfloat16 or int8) on `device`."""
    import torch
    X = np.ascontiguousarray(X)
    if dtype == "f16":
        t = torch.from_numpy(X)
    elif dtype == "bf16":
        t = torch.from_numpy(X.view(np.int16)).view(torch.bfloat16)
    elif dtype == "i8":
        t = torch.from_numpy(X)
    else:
        raise ValueError(dtype)
    return t.to(device)


@dataclass
class LshParams:
    """The random draws of an LSH-bucketed join: L tables of k concatenated
    functions, projection rows A ((L*k, d) int8, function t*k + u of table t
    is row t*k + u), offsets B ((L*k,) int32) and bucket width w (0: sign
    hashes, > 0: quantised projections)."""
    L: int
    k: int
    A: np.ndarray
    B: np.ndarray
    w: int


def lsh_params(seed: int, L: int, k: int, d: int, w: int = 0, sigma: float = 32.0) -> LshParams:
    """Projection entries are N(0, sigma^2) draws rounded to integers and
    clipped to [-127, 127]; offsets are uniform integers in [0, w) (zero for
    sign hashes)."""
    rng = np.random.default_rng(seed)
    A = np.clip(np.rint(rng.standard_normal((L * k, d)) * sigma), -127, 127).astype(np.int8)
    B = (rng.integers(0, w, size=L * k) if w > 0 else np.zeros(L * k)).astype(np.int32)
    return LshParams(int(L), int(k), np.ascontiguousarray(A), B, int(w))
