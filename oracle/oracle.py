"""Python side of the oracle -- TEST INFRASTRUCTURE ONLY.

A ctypes wrapper around sj_oracle.c (plain C nested loops in double, see the
header of that file) that takes the storage arrays produced by `workloads`.
It follows the similarity-join definition of Ahle & Silvestri, Section 4:
report (i, j) when <P_i, Q_j> >= s ("ip"; cosine on unit rows) or when
||P_i - Q_j||^2 <= r2 ("l2"), both inclusive.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sj_oracle.c")
_LIB = os.path.join(_HERE, "libsj_oracle.so")
_DT = {"f16": 1, "bf16": 2, "i8": 3}
_MET = {"ip": 0, "l2": 1}
_lib = None


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile sj_oracle.c with gcc (-O2, OpenMP) into a shared library."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", "-o", tmp, src, "-lm"])
        os.replace(tmp, out)
    return out


def load(path: str | None = None):
    """Load (building first when missing or stale) the oracle library."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or build(force=False)
    lib = ctypes.CDLL(p)
    i64, dbl, vp, i32 = ctypes.c_int64, ctypes.c_double, ctypes.c_void_p, ctypes.c_int
    lib.or_decode.argtypes = [i32, vp, i64, vp]
    lib.or_decode.restype = None
    lib.or_score_ip.argtypes = [i32, vp, i64, vp, i64, i64]
    lib.or_score_ip.restype = dbl
    lib.or_score_l2.argtypes = [i32, vp, i64, vp, i64, i64]
    lib.or_score_l2.restype = dbl
    lib.or_join.argtypes = [i32, i32, vp, i64, vp, i64, i64, dbl, vp, i64, dbl, vp, i64, vp, vp,
                            i64, vp, i32]
    lib.or_join.restype = i64
    lib.or_count.argtypes = [i32, i32, vp, i64, vp, i64, i64, dbl, vp, i64, vp, i32]
    lib.or_count.restype = i64
    lib.or_scores.argtypes = [i32, i32, vp, vp, i64, vp, i64, vp]
    lib.or_scores.restype = None
    lib.or_lsh_keys.argtypes = [i32, vp, i64, i64, i64, i64, vp, vp, i32, vp]
    lib.or_lsh_keys.restype = i32
    lib.or_lsh_join.argtypes = [i32, i32, vp, i64, vp, i64, i64, dbl, i64, i64, vp, vp, i32, vp,
                                i64, i32]
    lib.or_lsh_join.restype = i64
    lib.or_max_threads.argtypes = []
    lib.or_max_threads.restype = i32
    lib.or_round_f16.argtypes = [dbl]
    lib.or_round_f16.restype = ctypes.c_uint16
    lib.or_round_bf16.argtypes = [dbl]
    lib.or_round_bf16.restype = ctypes.c_uint16
    lib.or_normalize.argtypes = [i32, vp, i64, i64, i32, vp]
    lib.or_normalize.restype = i32
    lib.or_hamming.argtypes = [vp, i64, vp, i64, i64]
    lib.or_hamming.restype = i64
    lib.or_join_hamming.argtypes = [vp, i64, vp, i64, i64, dbl, vp, i64, i32]
    lib.or_join_hamming.restype = i64
    if path is None:
        _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(P, Q, dtype):
    if dtype not in _DT:
        raise ValueError(f"unknown dtype {dtype}")
    want = {"f16": np.float16, "bf16": np.uint16, "i8": np.int8}[dtype]
    for X in (P, Q):
        if X.dtype != want or X.ndim != 2 or not X.flags.c_contiguous:
            raise ValueError(f"expected a C-contiguous 2-D {want.__name__} array for {dtype}")
    if P.shape[1] != Q.shape[1]:
        raise ValueError("P and Q must have the same dimension")


def decode(dtype: str, X: np.ndarray, lib=None) -> np.ndarray:
    """Exact float64 values of the stored elements."""
    lib = lib or load()
    X = np.ascontiguousarray(X)
    out = np.empty(X.shape, np.float64)
    lib.or_decode(_DT[dtype], _ptr(X), X.size, _ptr(out))
    return out


@dataclass
class JoinResult:
    pairs: np.ndarray        # (m, 2) uint32, lexicographic (i, j)
    total: int
    band_pairs: np.ndarray   # (b, 2) uint32: pairs whose score is within `band` of the threshold
    band_match: np.ndarray   # (b,) bool: whether each band pair matched


def join(metric: str, dtype: str, P: np.ndarray, Q: np.ndarray, thr: float, rows=None,
         band: float = 0.0, threads: int | None = None, cap: int | None = None,
         lib=None) -> JoinResult:
    """All (i, j) with i in `rows` (all of P when None) and j in Q that match."""
    lib = lib or load()
    _check(P, Q, dtype)
    n_p, d = P.shape
    n_q = Q.shape[0]
    r = None if rows is None else np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    nr = n_p if r is None else r.size
    cap = (1 << 20) if cap is None else int(cap)
    bcap = 1 << 20 if band > 0 else 0
    bp = np.zeros((max(bcap, 1), 2), np.uint32)
    bm = np.zeros(max(bcap, 1), np.uint8)
    nb = ctypes.c_int64(0)
    while True:
        out = np.zeros((max(cap, 1), 2), np.uint32)
        tot = lib.or_join(_MET[metric], _DT[dtype], _ptr(P), n_p, _ptr(Q), n_q, d, float(thr),
                          None if r is None else _ptr(r), nr, float(band), _ptr(out), cap,
                          _ptr(bp), _ptr(bm), bcap, ctypes.byref(nb), threads or 0)
        if tot < 0:
            raise RuntimeError(f"oracle join failed ({tot})")
        if tot <= cap:
            break
        cap = int(tot)          # buffer too small: run again with the exact size
    nb = min(nb.value, bcap)
    return JoinResult(out[:tot].copy(), int(tot), bp[:nb].copy(), bm[:nb].astype(bool))


def count(metric: str, dtype: str, P: np.ndarray, Q: np.ndarray, thr: float, rows=None,
          threads: int | None = None, per_row: bool = False, lib=None):
    """Number of matches (and optionally the per-row counts)."""
    lib = lib or load()
    _check(P, Q, dtype)
    n_p, d = P.shape
    r = None if rows is None else np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    nr = n_p if r is None else r.size
    pr = np.zeros(max(nr, 1), np.int64)
    tot = lib.or_count(_MET[metric], _DT[dtype], _ptr(P), n_p, _ptr(Q), Q.shape[0], d,
                       float(thr), None if r is None else _ptr(r), nr, _ptr(pr), threads or 0)
    if tot < 0:
        raise RuntimeError(f"oracle count failed ({tot})")
    return (int(tot), pr[:nr].copy()) if per_row else int(tot)


def scores(metric: str, dtype: str, P: np.ndarray, Q: np.ndarray, pairs, lib=None) -> np.ndarray:
    """The metric's score (inner product or squared distance) of each listed pair."""
    lib = lib or load()
    _check(P, Q, dtype)
    pr = np.ascontiguousarray(np.asarray(pairs, dtype=np.int64).reshape(-1, 2))
    out = np.zeros(max(pr.shape[0], 1), np.float64)
    lib.or_scores(_MET[metric], _DT[dtype], _ptr(P), _ptr(Q), P.shape[1], _ptr(pr), pr.shape[0],
                  _ptr(out))
    return out[:pr.shape[0]].copy()


def max_threads(lib=None) -> int:
    lib = lib or load()
    return int(lib.or_max_threads())


def _lsh_check(L: int, k: int, A: np.ndarray, B, w: int, d: int):
    if A.dtype != np.int8 or A.shape != (L * k, d) or not A.flags.c_contiguous:
        raise ValueError(f"A must be a C-contiguous ({L * k}, {d}) int8 array")
    B = np.zeros(L * k, np.int32) if B is None else np.ascontiguousarray(B, dtype=np.int32)
    if B.shape != (L * k,):
        raise ValueError(f"B must hold {L * k} int32 offsets")
    return B


def lsh_keys(dtype: str, X: np.ndarray, L: int, k: int, A: np.ndarray, B=None, w: int = 0,
             lib=None) -> np.ndarray:
    """(L, n) uint64 bucket keys of the rows of X (see or_lsh_keys in sj_oracle.c:
    L tables of k concatenated random-projection hashes, Section 4's LSH
    join; w == 0 sign hashes, w > 0 quantised projections with offsets B)."""
    lib = lib or load()
    _check(X, X, dtype)
    B = _lsh_check(L, k, A, B, w, X.shape[1])
    out = np.zeros((max(L, 1), max(X.shape[0], 1)), np.uint64)
    keys = np.zeros(L * X.shape[0] + 1, np.uint64)
    st = lib.or_lsh_keys(_DT[dtype], _ptr(X), X.shape[0], X.shape[1], L, k, _ptr(A), _ptr(B),
                         int(w), _ptr(keys))
    if st != 0:
        raise RuntimeError(f"oracle lsh_keys failed ({st})")
    out = keys[:L * X.shape[0]].reshape(L, X.shape[0]).copy()
    return out


def lsh_join(metric: str, dtype: str, P: np.ndarray, Q: np.ndarray, thr: float, L: int, k: int,
             A: np.ndarray, B=None, w: int = 0, threads: int | None = None,
             lib=None) -> np.ndarray:
    """The LSH-bucketed join (Section 4): all (i, j) sharing a bucket in some
    table that pass the exact test, as an (m, 2) uint32 array in (i, j) order."""
    lib = lib or load()
    _check(P, Q, dtype)
    B = _lsh_check(L, k, A, B, w, P.shape[1])
    cap = 1 << 16
    while True:
        out = np.zeros((cap, 2), np.uint32)
        tot = lib.or_lsh_join(_MET[metric], _DT[dtype], _ptr(P), P.shape[0], _ptr(Q),
                              Q.shape[0], P.shape[1], float(thr), L, k, _ptr(A), _ptr(B),
                              int(w), _ptr(out), cap, threads or 0)
        if tot < 0:
            raise RuntimeError(f"oracle lsh_join failed ({tot})")
        if tot <= cap:
            return out[:tot].copy()
        cap = int(tot)


# ------------------------------------------- Section 4's ip-distance front ends

def round_to(out_dtype: str, v: float, lib=None) -> int:
    """The nearest binary16 ("f16") or bfloat16 ("bf16") bit pattern of the
    double v, ties to even."""
    lib = lib or load()
    return int(lib.or_round_f16(float(v)) if out_dtype == "f16" else lib.or_round_bf16(float(v)))


def normalize(dtype: str, X: np.ndarray, lib=None) -> np.ndarray:
    """Every row divided by its Euclidean norm (double, ascending k) and
    rounded to the nearest value of the output type, ties to even: the
    storage array of f = g = x / ||x||, Section 4's cosine ip-distance.  The
    output type is the input's for fp16/bf16 and fp16 for int8; zero rows stay
    zero."""
    lib = lib or load()
    _check(X, X, dtype)
    out_dtype = "bf16" if dtype == "bf16" else "f16"
    out = np.zeros(X.shape, np.uint16)
    st = lib.or_normalize(_DT[dtype], _ptr(X), X.shape[0], X.shape[1], _DT[out_dtype], _ptr(out))
    if st != 0:
        raise RuntimeError(f"oracle normalize failed ({st})")
    return out.view(np.float16) if out_dtype == "f16" else out


def _check_bits(X: np.ndarray, d: int):
    if X.dtype != np.uint8 or X.ndim != 2 or not X.flags.c_contiguous or \
            X.shape[1] != (d + 7) // 8:
        raise ValueError(f"expected a C-contiguous (n, {(d + 7) // 8}) uint8 array of bit rows")


def hamming(P: np.ndarray, i: int, Q: np.ndarray, j: int, d: int, lib=None) -> int:
    """Number of the d coordinates in which bit rows P_i and Q_j differ
    (coordinate m is bit m % 8 of byte m / 8)."""
    lib = lib or load()
    _check_bits(P, d)
    _check_bits(Q, d)
    return int(lib.or_hamming(_ptr(P), i, _ptr(Q), j, d))


def hamming_join(P: np.ndarray, Q: np.ndarray, d: int, r: float, threads: int | None = None,
                 lib=None) -> np.ndarray:
    """All (i, j) with Hamming(P_i, Q_j) <= r, as an (m, 2) uint32 array in
    (i, j) order (rows of d bits, ceil(d / 8) bytes each)."""
    lib = lib or load()
    _check_bits(P, d)
    _check_bits(Q, d)
    cap = 1 << 16
    while True:
        out = np.zeros((cap, 2), np.uint32)
        tot = lib.or_join_hamming(_ptr(P), P.shape[0], _ptr(Q), Q.shape[0], d, float(r),
                                  _ptr(out), cap, threads or 0)
        if tot < 0:
            raise RuntimeError(f"oracle hamming_join failed ({tot})")
        if tot <= cap:
            return out[:tot].copy()
        cap = int(tot)
