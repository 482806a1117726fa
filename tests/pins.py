"""Pins for the oracle: checks that tie it to something other than itself.

Each pin takes the loaded oracle library (so that the mutation tests can run
the same pins against deliberately broken copies of the oracle) and raises
AssertionError when the oracle disagrees with

  * a library routine (numpy's integer matrix product, numpy/torch decoders),
  * a closed form (binomial counts on the hypercube, one-hot and cluster
    counts, identical rows),
  * exact rational arithmetic within the recursive-summation error bound,
  * the paper's own ip-distance transforms (Section 4: Hamming and squared L2
    as f(x).g(y)), or
  * an invariant of the join definition (Section 4: the set of pairs with
    D(x, y) <= r): symmetry, monotonicity, permutation equivariance,
    zero padding, translation, scaling, block decomposition, row subsets.

The pins decode the stored values themselves (numpy float16, torch bfloat16),
independently of the oracle's own decoder.
"""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np

import oracle
from workloads import encode

DT = ("f16", "bf16", "i8")


def values(dtype, X):
    """Exact float64 values of a storage array, decoded with numpy/torch."""
    if dtype == "f16":
        return X.astype(np.float64)
    if dtype == "i8":
        return X.astype(np.float64)
    import torch
    return torch.from_numpy(X.view(np.int16).copy()).view(torch.bfloat16).double().numpy()


def pairset(pairs):
    return set(map(tuple, np.asarray(pairs, dtype=np.int64).reshape(-1, 2).tolist()))


def mask_to_pairs(mask):
    i, j = np.nonzero(mask)
    return np.stack([i, j], 1)


def rand_int(rng, n, d, lo, hi, dtype):
    return encode(rng.integers(lo, hi + 1, size=(n, d)), dtype)


# ---------------------------------------------------------------- decoding

def pin_decode_f16_exhaustive(lib):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    X = bits.view(np.float16).reshape(1, -1)
    got = oracle.decode("f16", X, lib=lib).ravel()
    want = X.astype(np.float64).ravel()
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


def pin_decode_bf16_exhaustive(lib):
    X = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).reshape(1, -1)
    got = oracle.decode("bf16", X, lib=lib).ravel()
    want = values("bf16", X).ravel()
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


def pin_decode_i8_exhaustive(lib):
    X = np.arange(-128, 128, dtype=np.int64).astype(np.int8).reshape(1, -1)
    got = oracle.decode("i8", X, lib=lib).ravel()
    assert np.array_equal(got, np.arange(-128, 128, dtype=np.float64))


# ------------------------------------------------- library-routine pins

def pin_ip_equals_integer_matmul(lib):
    """Inner-product join == threshold of numpy's exact int64 product P.Q^T."""
    rng = np.random.default_rng(11)
    for dtype in DT:
        for (n_p, n_q, d, lo, hi) in ((37, 53, 1, -8, 8), (29, 41, 7, -8, 8), (40, 33, 33, -4, 4),
                                      (23, 31, 130, -3, 5)):
            P = rand_int(rng, n_p, d, lo, hi, dtype)
            Q = rand_int(rng, n_q, d, lo, hi, dtype)
            S = values(dtype, P).astype(np.int64) @ values(dtype, Q).astype(np.int64).T
            for s in np.unique(np.quantile(S, [0.0, 0.3, 0.9, 0.99, 1.0]).round()):
                got = oracle.join("ip", dtype, P, Q, float(s), lib=lib)
                want = mask_to_pairs(S >= s)
                assert got.total == want.shape[0], (dtype, n_p, n_q, d, s)
                assert np.array_equal(got.pairs.astype(np.int64), want), (dtype, d, s)


def pin_l2_equals_norm_expansion(lib):
    """Squared-L2 join == threshold of N_x + N_y - 2 P.Q^T (numpy int64)."""
    rng = np.random.default_rng(12)
    for dtype in DT:
        for (n_p, n_q, d, lo, hi) in ((31, 45, 1, -15, 15), (26, 38, 9, -15, 15),
                                      (33, 21, 64, -6, 6)):
            P = rand_int(rng, n_p, d, lo, hi, dtype)
            Q = rand_int(rng, n_q, d, lo, hi, dtype)
            Pv = values(dtype, P).astype(np.int64)
            Qv = values(dtype, Q).astype(np.int64)
            D = (Pv * Pv).sum(1)[:, None] + (Qv * Qv).sum(1)[None, :] - 2 * (Pv @ Qv.T)
            for r2 in np.unique(np.quantile(D, [0.0, 0.01, 0.2, 0.7, 1.0]).round()):
                got = oracle.join("l2", dtype, P, Q, float(r2), lib=lib)
                want = mask_to_pairs(D <= r2)
                assert np.array_equal(got.pairs.astype(np.int64), want), (dtype, d, r2)


def pin_l2_equals_paper_fg(lib):
    """Section 4's squared-L2 ip-distance: f(x) = (x_k^2, 1, -2 x_k)_k and
    g(y) = (1, y_k^2, y_k)_k (the last triple of g read as (1, y^2, y), see
    the readings in the design notes) give f(x).g(y) = ||x - y||^2 for every
    pair; checked exactly against the oracle's scores with numpy int64."""
    rng = np.random.default_rng(13)
    for dtype in DT:
        P = rand_int(rng, 17, 11, -15, 15, dtype)
        Q = rand_int(rng, 19, 11, -15, 15, dtype)
        x = values(dtype, P).astype(np.int64)
        y = values(dtype, Q).astype(np.int64)
        F = np.stack([x * x, np.ones_like(x), -2 * x], axis=2).reshape(x.shape[0], -1)
        G = np.stack([np.ones_like(y), y * y, y], axis=2).reshape(y.shape[0], -1)
        D = F @ G.T
        pr = np.array([(i, j) for i in range(17) for j in range(19)])
        got = oracle.scores("l2", dtype, P, Q, pr, lib=lib)
        assert np.array_equal(got, D.ravel().astype(np.float64)), dtype


def pin_hamming_closed_form(lib):
    """On {0,1}^d the squared distance is the Hamming distance, which Section
    4's Hamming ip-distance f(x) = (x_k, 1 - x_k)_k, g(y) = (1 - y_k, y_k)_k
    also computes; both checked against popcount(x xor y)."""
    rng = np.random.default_rng(14)
    d = 23
    bp = rng.integers(0, 2, size=(21, d))
    bq = rng.integers(0, 2, size=(18, d))
    pr = np.array([(i, j) for i in range(21) for j in range(18)])
    ham = np.array([bin(int("".join(map(str, bp[i])), 2) ^ int("".join(map(str, bq[j])), 2))
                    .count("1") for i, j in pr], dtype=np.float64)
    F = np.stack([bp, 1 - bp], 2).reshape(21, -1)
    G = np.stack([1 - bq, bq], 2).reshape(18, -1)
    assert np.array_equal((F @ G.T).ravel().astype(np.float64), ham)
    for dtype in DT:
        got = oracle.scores("l2", dtype, encode(bp, dtype), encode(bq, dtype), pr, lib=lib)
        assert np.array_equal(got, ham), dtype


# ------------------------------------------------------- closed forms

def pin_hypercube_ip_counts(lib):
    """P = Q = all of {-1,+1}^d: <x, y> = d - 2 Ham(x, y) and each x has
    C(d, h) partners at Hamming distance h, so the join has
    2^d * sum_{h : d - 2h >= s} C(d, h) pairs (ties included)."""
    for d in (1, 6, 9):
        cube = np.array([[1 if (v >> k) & 1 else -1 for k in range(d)] for v in range(1 << d)])
        for dtype in DT:
            X = encode(cube, dtype)
            for s in (-d - 1, -d, -1, 0, 1, 2, d - 2, d - 1, d, d + 1, 0.5, -0.5):
                want = (1 << d) * sum(math.comb(d, h) for h in range(d + 1) if d - 2 * h >= s)
                got = oracle.count("ip", dtype, X, X.copy(), float(s), lib=lib)
                assert got == want, (d, dtype, s, got, want)


def pin_binary_l2_counts(lib):
    """P = Q = all of {0,1}^d: ||x - y||^2 = Ham(x, y), so the join at radius
    r2 has 2^d * sum_{h <= r2} C(d, h) pairs."""
    for d in (1, 5, 8):
        cube = np.array([[(v >> k) & 1 for k in range(d)] for v in range(1 << d)])
        for dtype in DT:
            X = encode(cube, dtype)
            for r2 in (-1, 0, 0.5, 1, 2, d - 1, d, d + 3):
                want = (1 << d) * sum(math.comb(d, h) for h in range(d + 1) if h <= r2)
                got = oracle.count("l2", dtype, X, X.copy(), float(r2), lib=lib)
                assert got == want, (d, dtype, r2, got, want)


def pin_identical_rows(lib):
    """n_p copies of x joined with n_q copies of x: all n_p * n_q pairs when
    s <= ||x||^2, none above; for L2 all pairs at any r2 >= 0."""
    rng = np.random.default_rng(15)
    for dtype in DT:
        x = rng.integers(-7, 8, size=13)
        nx = int((x * x).sum())
        P = encode(np.tile(x, (9, 1)), dtype)
        Q = encode(np.tile(x, (14, 1)), dtype)
        assert oracle.count("ip", dtype, P, Q, float(nx), lib=lib) == 126
        assert oracle.count("ip", dtype, P, Q, nx + 0.5, lib=lib) == 0
        assert oracle.count("ip", dtype, P, Q, float(nx + 1), lib=lib) == 0
        assert oracle.count("l2", dtype, P, Q, 0.0, lib=lib) == 126
        assert oracle.count("l2", dtype, P, Q, -0.5, lib=lib) == 0


def pin_one_hot_counts(lib):
    """Rows c * e_k: <x, y> = c^2 when the hot coordinates agree and 0
    otherwise, so for 0 < s <= c^2 the join has sum_k |P_k| |Q_k| pairs and for
    s <= 0 all of them; squared distance is 0 or 2 c^2."""
    rng = np.random.default_rng(16)
    d, c = 10, 3
    kp = rng.integers(0, d, size=40)
    kq = rng.integers(0, d, size=35)
    Pv = np.zeros((40, d), np.int64)
    Qv = np.zeros((35, d), np.int64)
    Pv[np.arange(40), kp] = c
    Qv[np.arange(35), kq] = c
    same = sum(int((kp == k).sum()) * int((kq == k).sum()) for k in range(d))
    for dtype in DT:
        P, Q = encode(Pv, dtype), encode(Qv, dtype)
        assert oracle.count("ip", dtype, P, Q, float(c * c), lib=lib) == same
        assert oracle.count("ip", dtype, P, Q, 1.0, lib=lib) == same
        assert oracle.count("ip", dtype, P, Q, 0.0, lib=lib) == 40 * 35
        assert oracle.count("ip", dtype, P, Q, c * c + 1.0, lib=lib) == 0
        assert oracle.count("l2", dtype, P, Q, 0.0, lib=lib) == same
        assert oracle.count("l2", dtype, P, Q, 2.0 * c * c - 1, lib=lib) == same
        assert oracle.count("l2", dtype, P, Q, 2.0 * c * c, lib=lib) == 40 * 35
        got = oracle.join("ip", dtype, P, Q, 1.0, lib=lib).pairs.astype(np.int64)
        want = mask_to_pairs(kp[:, None] == kq[None, :])
        assert np.array_equal(got, want)


def pin_orthogonal_clusters(lib):
    """Rows with positive entries on disjoint coordinate blocks (one block per
    cluster): <x, y> > 0 exactly within a cluster, so at s = 1 the join is the
    union of the cluster products."""
    rng = np.random.default_rng(17)
    nc, bw = 5, 4
    lp = rng.integers(0, nc, size=30)
    lq = rng.integers(0, nc, size=27)
    Pv = np.zeros((30, nc * bw), np.int64)
    Qv = np.zeros((27, nc * bw), np.int64)
    for i, a in enumerate(lp):
        Pv[i, a * bw:(a + 1) * bw] = rng.integers(1, 4, size=bw)
    for j, a in enumerate(lq):
        Qv[j, a * bw:(a + 1) * bw] = rng.integers(1, 4, size=bw)
    want = mask_to_pairs(lp[:, None] == lq[None, :])
    for dtype in DT:
        got = oracle.join("ip", dtype, encode(Pv, dtype), encode(Qv, dtype), 1.0, lib=lib)
        assert np.array_equal(got.pairs.astype(np.int64), want), dtype


# --------------------------------------------- exact rational arithmetic

def pin_real_scores_within_summation_bound(lib):
    """Real-valued fp16/bf16 rows: every product of two decoded elements is
    exact in binary64 (at most 11 x 11 significand bits), so the oracle's only
    error is the recursive summation, bounded by gamma_{d} * sum_k |x_k y_k|
    with gamma_d = d u / (1 - d u), u = 2^-53.  Exact values come from Python
    Fractions."""
    rng = np.random.default_rng(18)
    u = 2.0 ** -53
    for dtype in ("f16", "bf16"):
        for d in (3, 64, 256):
            P = encode(rng.standard_normal((6, d)) / math.sqrt(d), dtype)
            Q = encode(rng.standard_normal((7, d)) / math.sqrt(d), dtype)
            x, y = values(dtype, P), values(dtype, Q)
            pr = np.array([(i, j) for i in range(6) for j in range(7)])
            for metric in ("ip", "l2"):
                got = oracle.scores(metric, dtype, P, Q, pr, lib=lib)
                g = d * u / (1 - d * u)
                for t, (i, j) in enumerate(pr):
                    if metric == "ip":
                        terms = [Fraction(a) * Fraction(b) for a, b in zip(x[i], y[j])]
                    else:
                        terms = [(Fraction(a) - Fraction(b)) ** 2 for a, b in zip(x[i], y[j])]
                    exact = sum(terms, Fraction(0))
                    mag = float(sum(abs(v) for v in terms))
                    # the l2 terms also round the difference and the square
                    bound = g * mag + (4 * u * mag if metric == "l2" else 0.0)
                    assert abs(Fraction(got[t]) - exact) <= Fraction(bound), (dtype, d, metric)


# ----------------------------------------------------------- invariants

def pin_self_join_symmetry(lib):
    """P joined with itself: (i, j) matches iff (j, i) does, for both metrics."""
    rng = np.random.default_rng(19)
    for dtype in DT:
        X = rand_int(rng, 60, 12, -6, 6, dtype)
        for metric, thr in (("ip", 20.0), ("l2", 200.0)):
            got = pairset(oracle.join(metric, dtype, X, X, thr, lib=lib).pairs)
            assert got, (dtype, metric)
            assert got == {(j, i) for (i, j) in got}, (dtype, metric)


def pin_monotone_in_threshold(lib):
    """Raising s shrinks the inner-product join; raising r2 grows the L2 join
    (as sets, not just counts)."""
    rng = np.random.default_rng(20)
    for dtype in DT:
        P = rand_int(rng, 40, 16, -5, 5, dtype)
        Q = rand_int(rng, 45, 16, -5, 5, dtype)
        prev = None
        for s in (-50.0, 0.0, 10.0, 25.0, 40.0, 80.0):
            cur = pairset(oracle.join("ip", dtype, P, Q, s, lib=lib).pairs)
            if prev is not None:
                assert cur <= prev
            prev = cur
        prev = None
        for r2 in (0.0, 200.0, 300.0, 400.0, 900.0):
            cur = pairset(oracle.join("l2", dtype, P, Q, r2, lib=lib).pairs)
            if prev is not None:
                assert prev <= cur
            prev = cur


def pin_permutation_equivariance(lib):
    """Permuting the rows of P and Q permutes the join's index pairs."""
    rng = np.random.default_rng(21)
    for dtype in DT:
        P = rand_int(rng, 33, 10, -6, 6, dtype)
        Q = rand_int(rng, 28, 10, -6, 6, dtype)
        pp, pq = rng.permutation(33), rng.permutation(28)
        for metric, thr in (("ip", 15.0), ("l2", 150.0)):
            base = pairset(oracle.join(metric, dtype, P, Q, thr, lib=lib).pairs)
            perm = pairset(oracle.join(metric, dtype, np.ascontiguousarray(P[pp]),
                                       np.ascontiguousarray(Q[pq]), thr, lib=lib).pairs)
            inv_p, inv_q = np.argsort(pp), np.argsort(pq)
            assert perm == {(int(inv_p[i]), int(inv_q[j])) for (i, j) in base}


def pin_zero_padding(lib):
    """Appending zero coordinates to every point changes neither metric."""
    rng = np.random.default_rng(22)
    for dtype in DT:
        Pv = rng.integers(-6, 7, size=(25, 9))
        Qv = rng.integers(-6, 7, size=(31, 9))
        pad = lambda X: np.concatenate([X, np.zeros((X.shape[0], 23), np.int64)], 1)  # noqa
        for metric, thr in (("ip", 12.0), ("l2", 120.0)):
            a = oracle.join(metric, dtype, encode(Pv, dtype), encode(Qv, dtype), thr, lib=lib)
            b = oracle.join(metric, dtype, encode(pad(Pv), dtype), encode(pad(Qv), dtype), thr,
                            lib=lib)
            assert np.array_equal(a.pairs, b.pairs)


def pin_translation_invariance_l2(lib):
    """Adding one vector t to every point leaves squared distances unchanged."""
    rng = np.random.default_rng(23)
    for dtype in DT:
        Pv = rng.integers(-9, 10, size=(27, 14))
        Qv = rng.integers(-9, 10, size=(26, 14))
        t = rng.integers(-9, 10, size=14)
        a = oracle.join("l2", dtype, encode(Pv, dtype), encode(Qv, dtype), 300.0, lib=lib)
        b = oracle.join("l2", dtype, encode(Pv + t, dtype), encode(Qv + t, dtype), 300.0, lib=lib)
        assert a.total > 0 and np.array_equal(a.pairs, b.pairs)


def pin_scaling(lib):
    """Doubling P doubles every inner product: join(2P, Q, 2s) = join(P, Q, s).
    Doubling both sets quadruples squared distances."""
    rng = np.random.default_rng(24)
    for dtype in DT:
        Pv = rng.integers(-7, 8, size=(30, 12))
        Qv = rng.integers(-7, 8, size=(29, 12))
        a = oracle.join("ip", dtype, encode(Pv, dtype), encode(Qv, dtype), 30.0, lib=lib)
        b = oracle.join("ip", dtype, encode(2 * Pv, dtype), encode(Qv, dtype), 60.0, lib=lib)
        assert a.total > 0 and np.array_equal(a.pairs, b.pairs)
        a = oracle.join("l2", dtype, encode(Pv, dtype), encode(Qv, dtype), 400.0, lib=lib)
        b = oracle.join("l2", dtype, encode(2 * Pv, dtype), encode(2 * Qv, dtype), 1600.0, lib=lib)
        assert a.total > 0 and np.array_equal(a.pairs, b.pairs)


def pin_block_decomposition(lib):
    """The join of P and Q is the union of the joins of their row blocks,
    with the blocks' index offsets added back."""
    rng = np.random.default_rng(25)
    for dtype in DT:
        P = rand_int(rng, 37, 8, -6, 6, dtype)
        Q = rand_int(rng, 41, 8, -6, 6, dtype)
        for metric, thr in (("ip", 10.0), ("l2", 100.0)):
            full = pairset(oracle.join(metric, dtype, P, Q, thr, lib=lib).pairs)
            parts = set()
            for a0, a1 in ((0, 15), (15, 37)):
                for b0, b1 in ((0, 20), (20, 41)):
                    r = oracle.join(metric, dtype, np.ascontiguousarray(P[a0:a1]),
                                    np.ascontiguousarray(Q[b0:b1]), thr, lib=lib)
                    parts |= {(i + a0, j + b0) for (i, j) in pairset(r.pairs)}
            assert full == parts


def pin_row_subset_and_order(lib):
    """Joining only some rows of P gives those rows' pairs; output pairs are in
    lexicographic (i, j) order and carry no duplicates."""
    rng = np.random.default_rng(26)
    for dtype in DT:
        P = rand_int(rng, 50, 6, -5, 5, dtype)
        Q = rand_int(rng, 47, 6, -5, 5, dtype)
        full = oracle.join("ip", dtype, P, Q, 8.0, lib=lib)
        pr = full.pairs.astype(np.int64)
        key = pr[:, 0] * (1 << 32) + pr[:, 1]
        assert np.all(np.diff(key) > 0)
        rows = np.array([3, 7, 20, 21, 49])
        sub = oracle.join("ip", dtype, P, Q, 8.0, rows=rows, lib=lib)
        assert pairset(sub.pairs) == {p for p in pairset(pr) if p[0] in set(rows.tolist())}
        cnt, per = oracle.count("ip", dtype, P, Q, 8.0, rows=rows, per_row=True, lib=lib)
        assert cnt == sub.total
        assert per.tolist() == [int((pr[:, 0] == r).sum()) for r in rows]


def pin_band_report(lib):
    """Boundary-band pairs are exactly the pairs whose score is within the
    band of the threshold, with the right match flag."""
    rng = np.random.default_rng(27)
    P = rand_int(rng, 30, 10, -5, 5, "i8")
    Q = rand_int(rng, 35, 10, -5, 5, "i8")
    x, y = P.astype(np.int64), Q.astype(np.int64)
    S = x @ y.T
    r = oracle.join("ip", "i8", P, Q, 12.0, band=2.0, lib=lib)
    want = mask_to_pairs(np.abs(S - 12) <= 2)
    assert np.array_equal(r.band_pairs.astype(np.int64), want)
    assert np.array_equal(r.band_match, S[want[:, 0], want[:, 1]] >= 12)




# ------------------------------------------------- LSH-bucketed join (Thm 3)

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden_lsh():
    rows = {}
    for line in open(os.path.join(GOLDEN, "lsh_keys_small.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            name, rest = line.split(None, 1)
            rows[name] = [[int(v) for v in part.split()] for part in rest.split(";")]
    return rows


def pin_lsh_keys_worked_example(lib):
    """Keys of a hand-worked example (tests/golden/lsh_keys_small.txt): the
    inclusive sign at z = 0, floor of negative quotients, two's-complement
    truncation, the bit position of each function and the table-major layout."""
    g = _golden_lsh()
    X = np.array(g["points"], np.int8)
    A = np.array(g["A"], np.int8)
    B = np.array(g["B"][0], np.int32)
    ks = oracle.lsh_keys("i8", X, 2, 2, A, B, 0, lib=lib)
    assert ks.tolist() == [[v for v in r] for r in g["sign"]], ks
    kq = oracle.lsh_keys("i8", X, 2, 2, A, B, 4, lib=lib)
    assert kq.tolist() == [[v for v in r] for r in g["quant4"]], kq
    # the same points stored as fp16 and bf16 give the same keys
    for dt in ("f16", "bf16"):
        Xf = encode(X.astype(np.float64), dt)
        assert np.array_equal(oracle.lsh_keys(dt, Xf, 2, 2, A, B, 0, lib=lib), ks)
        assert np.array_equal(oracle.lsh_keys(dt, Xf, 2, 2, A, B, 4, lib=lib), kq)


def pin_lsh_one_hot_keys(lib):
    """On scaled one-hot rows c e_m the projection is c A[f][m], so each key
    bit is the sign of a single known entry (pins the A index mapping)."""
    rng = np.random.default_rng(31)
    d, L, k = 9, 3, 5
    A = rng.integers(-20, 21, size=(L * k, d)).astype(np.int8)
    A[A == 0] = 1
    X = np.zeros((2 * d, d), np.int8)
    for m in range(d):
        X[m, m] = 3
        X[d + m, m] = -2
    keys = oracle.lsh_keys("i8", X, L, k, A, None, 0, lib=lib)
    for t in range(L):
        for r in range(2 * d):
            m, c = (r, 3) if r < d else (r - d, -2)
            want = sum(int(c * int(A[t * k + u, m]) >= 0) << (12 * u) for u in range(k))
            assert int(keys[t, r]) == want


def pin_lsh_one_bucket_is_exact_join(lib):
    """k = 0 (or all-zero projections) puts every point in one bucket: the
    LSH join is then the exact join."""
    rng = np.random.default_rng(32)
    for dtype, metric, thr in (("i8", "ip", 10.0), ("bf16", "ip", 6.0), ("f16", "l2", 60.0)):
        P = rand_int(rng, 37, 11, -4, 4, dtype)
        Q = rand_int(rng, 29, 11, -4, 4, dtype)
        x, y = values(dtype, P), values(dtype, Q)
        want = mask_to_pairs(x @ y.T >= thr) if metric == "ip" else \
            mask_to_pairs(((x[:, None, :] - y[None]) ** 2).sum(-1) <= thr)
        got0 = oracle.lsh_join(metric, dtype, P, Q, thr, 3, 0, np.zeros((0, 11), np.int8),
                               lib=lib)
        assert pairset(got0) == pairset(want)
        gotz = oracle.lsh_join(metric, dtype, P, Q, thr, 2, 4, np.zeros((8, 11), np.int8),
                               lib=lib)
        assert pairset(gotz) == pairset(want)


def pin_lsh_subset_union_and_planted(lib):
    """For any draws: the LSH join is the exact join restricted to pairs that
    share a bucket in some table, so it is a subset of the exact join, equals
    the union of its single-table joins, and contains every pair of identical
    rows that matches."""
    rng = np.random.default_rng(33)
    d, L, k = 16, 4, 3
    P = rand_int(rng, 60, d, -6, 6, "i8")
    Q = rand_int(rng, 50, d, -6, 6, "i8")
    Q[:10] = P[5:15]
    A = rng.integers(-30, 31, size=(L * k, d)).astype(np.int8)
    B = rng.integers(0, 40, size=L * k).astype(np.int32)
    for metric, thr, w in (("ip", 25.0, 0), ("l2", 500.0, 40)):
        exact = pairset(oracle.join(metric, "i8", P, Q, thr, lib=lib).pairs)
        got = pairset(oracle.lsh_join(metric, "i8", P, Q, thr, L, k, A, B, w, lib=lib))
        assert got <= exact and 0 < len(got) < len(exact)
        union = set()
        for t in range(L):
            union |= pairset(oracle.lsh_join(metric, "i8", P, Q, thr, 1, k,
                                             A[t * k:(t + 1) * k].copy(), B[t * k:(t + 1) * k],
                                             w, lib=lib))
        assert union == got
        for q in range(10):
            if (q + 5, q) in exact:
                assert (q + 5, q) in got
        # colliding pairs are exactly those with equal keys in some table
        kp = oracle.lsh_keys("i8", P, L, k, A, B, w, lib=lib)
        kq = oracle.lsh_keys("i8", Q, L, k, A, B, w, lib=lib)
        coll = (kp[:, :, None] == kq[:, None, :]).any(0)
        assert got == {p for p in exact if coll[p]}


def pin_lsh_sign_collision_probability(lib):
    """Random-hyperplane signs collide with probability 1 - theta / pi for
    points at angle theta (Charikar's SimHash, the classical LSH for angular
    distance).  Near-Gaussian integer projections (sd 32) on fp16 pairs at
    theta = pi / 3 and pi / 2: the empirical rate over 40 000 functions x 8
    pairs is within 0.012 of the law."""
    rng = np.random.default_rng(34)
    d, nf = 48, 40_000
    A = np.clip(np.rint(rng.standard_normal((nf, d)) * 32), -127, 127).astype(np.int8)
    for theta in (np.pi / 3, np.pi / 2):
        u = rng.standard_normal((8, d))
        u /= np.linalg.norm(u, axis=1, keepdims=True)
        v = rng.standard_normal((8, d))
        v -= (v * u).sum(1, keepdims=True) * u
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        y = np.cos(theta) * u + np.sin(theta) * v
        Xp, Xq = encode(u, "f16"), encode(y, "f16")
        kp = oracle.lsh_keys("f16", Xp, nf, 1, A, None, 0, lib=lib)
        kq = oracle.lsh_keys("f16", Xq, nf, 1, A, None, 0, lib=lib)
        up, yq = Xp.astype(np.float64), Xq.astype(np.float64)
        th = np.arccos((up * yq).sum(1) / np.linalg.norm(up, axis=1) / np.linalg.norm(yq, axis=1))
        rate = (kp == kq).mean()
        assert abs(rate - (1 - th / np.pi).mean()) < 0.012, (theta, rate)


def pin_lsh_quantised_collision_probability(lib):
    """Quantised Gaussian projections with uniform offsets (the p-stable LSH of
    Datar et al. for Euclidean distance) collide with probability
    p(c) = 1 - 2 Phi(-w / c) - 2 c / (sqrt(2 pi) w) (1 - exp(-w^2 / (2 c^2)))
    when the projected difference has standard deviation c.  Here c = 32 times
    the pair's distance; over 40 000 functions the rate is within 0.012."""
    rng = np.random.default_rng(35)
    d, nf = 32, 40_000
    A = np.clip(np.rint(rng.standard_normal((nf, d)) * 32), -127, 127).astype(np.int8)
    for w, delta_norm2 in ((256, 8), (512, 32)):
        x = rng.integers(-10, 11, size=(6, d))
        y = x.copy()
        for r in range(6):   # move delta_norm2 coordinates by one
            idx = rng.choice(d, size=delta_norm2, replace=False)
            y[r, idx] += 1
        B = rng.integers(0, w, size=nf).astype(np.int32)
        Xp, Xq = encode(x, "i8"), encode(y, "i8")
        kp = oracle.lsh_keys("i8", Xp, nf, 1, A, B, w, lib=lib)
        kq = oracle.lsh_keys("i8", Xq, nf, 1, A, B, w, lib=lib)
        c = 32.0 * math.sqrt(delta_norm2)
        phi = 0.5 * math.erfc((w / c) / math.sqrt(2))
        p = 1 - 2 * phi - 2 * c / (math.sqrt(2 * math.pi) * w) * (1 - math.exp(-w * w / (2 * c * c)))
        rate = (kp == kq).mean()
        assert abs(rate - p) < 0.012, (w, delta_norm2, rate, p)



# ------------------------------------- Section 4's ip-distance front ends

def _finite_table(dtype):
    """Every finite nonnegative binary16 / bfloat16 pattern in increasing order,
    with its exact value (decoded by the pins' own decoder)."""
    top = 0x7C00 if dtype == "f16" else 0x7F80
    bits = np.arange(top, dtype=np.uint16)
    vals = bits.view(np.float16).astype(np.float64) if dtype == "f16" else \
        values("bf16", bits.reshape(1, -1)).ravel()
    return bits, vals


def _nearest_by_search(dtype, v, bits, vals):
    """Round-to-nearest-even by its definition: the closest finite value (the
    two neighbours' distances are exact differences of nearby doubles), ties
    to the even pattern; beyond the midpoint above the largest finite value,
    infinity."""
    a = abs(v)
    sign = 0x8000 if math.copysign(1.0, v) < 0 else 0
    inf = 0x7C00 if dtype == "f16" else 0x7F80
    k = int(np.searchsorted(vals, a))
    if k < len(vals) and vals[k] == a:
        return sign | int(bits[k])
    if k == len(vals):
        ulp = vals[-1] - vals[-2]
        mid = vals[-1] + ulp / 2
        return sign | (inf if a >= mid else int(bits[-1]))
    lo, hi = k - 1, k
    dl, dh = a - vals[lo], vals[hi] - a
    if dl < dh:
        return sign | int(bits[lo])
    if dh < dl:
        return sign | int(bits[hi])
    return sign | int(bits[lo] if bits[lo] % 2 == 0 else bits[hi])


def pin_round_to_nearest_even(lib):
    """The oracle's double -> binary16 / bfloat16 rounding against a search of
    all finite patterns: random values in every binade (subnormals included),
    every kind of exact midpoint (ties), zeros, the overflow threshold;
    binary16 also against numpy's conversion."""
    rng = np.random.default_rng(31)
    for dtype in ("f16", "bf16"):
        bits, vals = _finite_table(dtype)
        ks = rng.choice(len(vals) - 1, 2500, replace=False)
        ks = np.concatenate([ks, np.arange(8), len(vals) - 2 - np.arange(4)])
        mids = (vals[ks] + vals[ks + 1]) / 2
        inside = vals[ks] + (vals[ks + 1] - vals[ks]) * rng.random(ks.size)
        ulp_top = vals[-1] - vals[-2]
        edge = [0.0, -0.0, vals[-1] + ulp_top / 2, vals[-1] + ulp_top / 2 * (1 - 2 ** -30),
                vals[-1] * 4, vals[1] / 2, vals[1] / 3]
        tests = np.concatenate([mids, inside, -mids[:300], -inside[:300], np.array(edge)])
        for v in tests:
            want = _nearest_by_search(dtype, float(v), bits, vals)
            got = oracle.round_to(dtype, float(v), lib=lib)
            assert got == want, (dtype, float(v), hex(got), hex(want))
            if dtype == "f16":
                with np.errstate(over="ignore"):
                    ref = int(np.float16(v).view(np.uint16))
                assert got == ref, (float(v), hex(got))


def _bits_of(dtype, v):
    return int(np.float16(v).view(np.uint16)) if dtype == "f16" else \
        _nearest_by_search("bf16", v, *_finite_table("bf16"))


def pin_normalize_exact_cases(lib):
    """Rows whose normalisation is known exactly: scaled one-hot rows give +-1
    at the hot coordinate and 0 elsewhere; (3, 4) gives the roundings of 3/5
    and 4/5, (1, 2, 2) those of 1/3 and 2/3, (2, 3, 6) those of 2/7, 3/7 and
    6/7 (Pythagorean quadruples: the norm is an integer); a zero row stays zero.
    Output type: fp16 for fp16 and int8 inputs, bf16 for bf16."""
    for dtype in DT:
        out_dt = "bf16" if dtype == "bf16" else "f16"
        X = np.array([[0, -5, 0, 0, 0, 0, 0], [3, 4, 0, 0, 0, 0, 0], [1, 2, 2, 0, 0, 0, 0],
                      [0, 0, 0, 0, 0, 0, 0], [-2, 3, -6, 0, 0, 0, 0], [0, 0, 0, 0, 0, 0, 7]])
        got = oracle.normalize(dtype, encode(X, dtype), lib=lib)
        got = got.view(np.uint16)
        want = np.zeros(X.shape, np.uint16)
        for i, norm in enumerate((5, 5, 3, 0, 7, 7)):
            for k in range(X.shape[1]):
                if X[i, k] != 0:
                    want[i, k] = _bits_of(out_dt, X[i, k] / norm)
        assert np.array_equal(got, want), (dtype, got, want)


def pin_normalize_within_half_ulp(lib):
    """Random rows of every input type: each normalised value lies within half
    an output ulp of the exact x_k / ||x|| (exact rational sum of squares,
    50-digit square root; slack 2^-50 relative for the double norm and
    quotient), the output is invariant under scaling the row by powers of two
    and equivariant under permuting its coordinates."""
    from decimal import Decimal, getcontext
    getcontext().prec = 50
    rng = np.random.default_rng(32)
    for dtype in DT:
        out_dt = "bf16" if dtype == "bf16" else "f16"
        if dtype == "i8":
            X = encode(rng.integers(-120, 121, size=(40, 37)), dtype)
        else:
            X = encode(rng.standard_normal((40, 37)) * np.exp(rng.uniform(-3, 3, (40, 1))), dtype)
        x = values(dtype, X)
        Y = oracle.normalize(dtype, X, lib=lib)
        y = values(out_dt, Y.view(np.uint16)) if out_dt == "bf16" else Y.astype(np.float64)
        for i in range(x.shape[0]):
            S = sum(Fraction(float(t)) ** 2 for t in x[i])
            norm = Decimal(S.numerator).sqrt() / Decimal(S.denominator).sqrt()
            for k in range(x.shape[1]):
                q = Decimal(float(x[i, k])) / norm
                yk = float(y[i, k])
                a = abs(yk) if yk != 0 else abs(float(q))
                e = math.frexp(a)[1] - 1 if a > 0 else -200
                p = 11 if out_dt == "f16" else 8
                emin = -14 if out_dt == "f16" else -126
                ulp = 2.0 ** (max(e, emin) - (p - 1))
                err = abs(Decimal(yk) - q)
                assert err <= Decimal(ulp / 2) + abs(q) * Decimal(2.0 ** -50), \
                    (dtype, i, k, yk, float(q))
        # scaling by 2 (fp16 / bf16 rows stay exact) and a permutation
        if dtype != "i8":
            X2 = encode(x * 2.0, dtype)
            assert np.array_equal(oracle.normalize(dtype, X2, lib=lib).view(np.uint16),
                                  Y.view(np.uint16))
        perm = rng.permutation(x.shape[1])
        Yp = oracle.normalize(dtype, np.ascontiguousarray(X[:, perm]), lib=lib)
        # the sum of squares runs in a different order: allow the rare
        # one-ulp change of the norm, compare within one output ulp
        a = Y.view(np.uint16)[:, perm].astype(np.int64)
        b = Yp.view(np.uint16).astype(np.int64)
        assert np.abs(a - b).max() <= 1


def _bitrows(B):
    """Pack (n, d) 0/1 rows: coordinate m in bit m % 8 of byte m / 8."""
    return np.packbits(np.asarray(B, dtype=np.uint8), axis=1, bitorder="little")


def pin_hamming_join_definition(lib):
    """The Hamming join: on all of {0,1}^d joined with itself the count within
    r is 2^d sum_{h <= r} C(d, h); on random rows (with random garbage in the
    padding bits past d) each distance equals numpy's unpackbits and xor
    count, and the join equals the squared-L2 join of the unpacked 0/1 rows."""
    for d in (5, 9):
        cube = np.array([[(v >> m) & 1 for m in range(d)] for v in range(1 << d)])
        Bc = _bitrows(cube)
        for r in (-1, 0, 1, 2.5, d):
            want = (1 << d) * sum(math.comb(d, h) for h in range(d + 1) if h <= r)
            assert len(oracle.hamming_join(Bc, Bc.copy(), d, r, lib=lib)) == want, (d, r)
    rng = np.random.default_rng(33)
    d = 45
    bp, bq = rng.integers(0, 2, size=(30, d)), rng.integers(0, 2, size=(26, d))
    Bp, Bq = _bitrows(bp), _bitrows(bq)
    Bp[:, -1] |= rng.integers(0, 256, size=30).astype(np.uint8) & 0xE0   # bits 45..47
    Bq[:, -1] |= rng.integers(0, 256, size=26).astype(np.uint8) & 0xE0
    up = np.unpackbits(Bp, axis=1, bitorder="little")[:, :d]
    uq = np.unpackbits(Bq, axis=1, bitorder="little")[:, :d]
    for i in range(0, 30, 7):
        for j in range(26):
            assert oracle.hamming(Bp, i, Bq, j, d, lib=lib) == int((up[i] ^ uq[j]).sum())
    for r in (5, 18, 22.7):
        got = oracle.hamming_join(Bp, Bq, d, r, lib=lib)
        l2 = oracle.join("l2", "i8", encode(bp, "i8"), encode(bq, "i8"), float(r), lib=lib)
        assert pairset(got) == pairset(l2.pairs) and len(got) == l2.total

PINS = {name[4:]: fn for name, fn in sorted(globals().items()) if name.startswith("pin_")}
