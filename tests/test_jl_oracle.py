"""The JL-transform oracle (oracle/jl.py) against its pins (CPU only): a
hand-worked example, the block form of Lemma 3's figure (each level reduces
r_i blocks of the vector by the same A_i), identity and single-factor
special cases, linearity, and the JL property the lemma states (norms kept
up to 1 +- eps with high probability; E ||Mx||^2 = ||x||^2 for factors with
entries N(0, 1 / k_i))."""
import os

import numpy as np
import pytest

from oracle import jl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden():
    rows = {}
    for line in open(os.path.join(GOLDEN, "jl_small.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            name, rest = line.split(None, 1)
            rows[name] = [[float(v) for v in part.split()] for part in rest.split(";")]
    return rows


def chain(d, k, zeta):
    """Lemma 3's sizes: k_i = i k (k_l = k), c_1 = zeta k, c_i = zeta k_{i-1},
    r_i = zeta^(l - i), with zeta^l = d / k."""
    l = int(round(np.log(d / k) / np.log(zeta)))
    assert zeta ** l * k == d
    shapes = []
    for i in range(1, l + 1):
        ki = k if i == l else i * k
        ci = zeta * k if i == 1 else zeta * shapes[-1][0]
        ri = zeta ** (l - i)
        shapes.append((ki, ci, ri))
    return shapes


def gaussian_factors(rng, shapes):
    return [rng.standard_normal((k, c)) / np.sqrt(k) for (k, c, r) in shapes]


def test_worked_example():
    g = _golden()
    shapes = [tuple(int(v) for v in s) for s in g["shapes"]]
    As = [np.array(g["A1"]), np.array(g["A2"])]
    Y = jl.transform(np.array(g["x"]), shapes, As)
    assert np.array_equal(Y, np.array(g["y"]))


@pytest.mark.parametrize("d,k,zeta", [(256, 32, 2), (1024, 16, 4), (96, 12, 2)])
def test_block_form_equals_dense(d, k, zeta):
    """Level by level: the vector as r_i blocks of c_i entries, each block
    times A_i^T (numpy matmul on the reshaped batch) -- the figure of Lemma 3's
    proof -- equals the dense product of Kronecker factors."""
    rng = np.random.default_rng(d + k)
    shapes = chain(d, k, zeta)
    assert jl.check_chain(d, shapes) == k
    As = gaussian_factors(rng, shapes)
    X = rng.standard_normal((7, d))
    Z = X.copy()
    for (ki, ci, ri), A in zip(shapes, As):
        Z = (Z.reshape(-1, ci) @ A.T).reshape(X.shape[0], ri * ki)
    Y = jl.transform(X, shapes, As)
    assert np.allclose(Y, Z, rtol=1e-12, atol=1e-12 * np.abs(Y).max())


def test_special_cases_and_linearity():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((5, 24))
    ident = [(6, 6, 4), (12, 12, 2), (24, 24, 1)]
    assert np.array_equal(jl.transform(X, ident, [np.eye(6), np.eye(12), np.eye(24)]), X)
    A = rng.standard_normal((5, 24))
    assert np.allclose(jl.transform(X, [(5, 24, 1)], [A]), X @ A.T, rtol=1e-13)
    shapes = [(3, 6, 4), (4, 12, 1)]
    As = [rng.standard_normal((3, 6)), rng.standard_normal((4, 12))]
    a, b = 2.5, -0.75
    lhs = jl.transform(a * X[:2] + b * X[2:4], shapes, As)
    rhs = a * jl.transform(X[:2], shapes, As) + b * jl.transform(X[2:4], shapes, As)
    assert np.allclose(lhs, rhs, rtol=1e-12, atol=1e-12)
    with pytest.raises(ValueError):
        jl.check_chain(24, [(3, 5, 4)])


def test_jl_norm_preservation():
    """Lemma 3's guarantee in distribution: with factors of i.i.d. N(0, 1/k_i)
    entries, ||Mx||^2 / ||x||^2 has mean 1 (over 400 draws of M, within 4
    standard errors), and with k = 64 at least 95% of the draws keep the norm
    within eps = 0.35 (a Gaussian JL matrix of that k keeps it within 0.35
    with probability > 0.99)."""
    rng = np.random.default_rng(11)
    d, k, zeta = 512, 64, 2
    shapes = chain(d, k, zeta)
    x = rng.standard_normal(d)
    ratios = []
    for _ in range(400):
        As = gaussian_factors(rng, shapes)
        y = jl.transform(x[None, :], shapes, As)[0]
        ratios.append((y @ y) / (x @ x))
    ratios = np.array(ratios)
    se = ratios.std() / np.sqrt(ratios.size)
    assert abs(ratios.mean() - 1) < 4 * se
    assert (np.abs(np.sqrt(ratios) - 1) <= 0.35).mean() >= 0.95


def test_abs_bound_worked_example():
    """|A_l| ... |A_1| |x| (the scale of the JL parity tolerance) on the
    hand-worked example, whose second factor and inputs have negative entries:
    a missing absolute value on x or on either factor changes a value."""
    g = _golden()
    shapes = [tuple(int(v) for v in s) for s in g["shapes"]]
    As = [np.array(g["A1"]), np.array(g["A2"])]
    B = jl.abs_bound(np.array(g["x"]), shapes, As)
    assert np.array_equal(B, np.array(g["absbound"]))


def _abs_bound_fractions(x, shapes, As):
    """Lemma 3's levels applied block by block to |x| with |A_i|, in exact
    rational arithmetic: level i splits its input into r_i blocks of c_i
    entries and maps each block b to |A_i| b."""
    from fractions import Fraction
    v = [abs(Fraction(float(t))) for t in x]
    for (k, c, r), A in zip(shapes, As):
        out = []
        for blk in range(r):
            seg = v[blk * c:(blk + 1) * c]
            for row in range(k):
                out.append(sum(abs(Fraction(float(A[row][col]))) * seg[col] for col in range(c)))
        v = out
    return v


@pytest.mark.parametrize("shapes", [[(3, 4, 3), (2, 9, 1)], [(4, 2, 4), (2, 4, 4), (3, 8, 1)]])
def test_abs_bound_exact_rationals(shapes):
    """abs_bound against an exact, level-by-level evaluation with Fractions on
    random real inputs and factors of both signs (within the relative
    rounding of the float64 evaluation, gamma(n) for sums of n nonnegative
    terms, n at most the dense row length)."""
    rng = np.random.default_rng(17 + len(shapes))
    d = shapes[0][1] * shapes[0][2]
    As = [rng.standard_normal((k, c)) for (k, c, r) in shapes]
    X = rng.standard_normal((3, d))
    B = jl.abs_bound(X, shapes, As)
    u = 2.0 ** -53
    tol = 4 * d * len(shapes) * u
    for row in range(X.shape[0]):
        exact = _abs_bound_fractions(X[row], shapes, As)
        assert len(exact) == B.shape[1]
        for got, want in zip(B[row], exact):
            assert want > 0 and abs(got - float(want)) <= tol * float(want)


def test_abs_bound_mutants_are_caught(monkeypatch):
    """Plausible slips in abs_bound (no absolute value on x, none on a later
    factor, |M| of the signed product instead of the product of |A_i|) each
    fail one of the two pins above."""
    orig_dense = jl.dense_matrix

    def no_abs_x(X, shapes, As):
        M = orig_dense(np.shape(X)[1], shapes, [np.abs(A) for A in As])
        return np.asarray(X, np.float64) @ M.T

    def no_abs_last(X, shapes, As):
        M = orig_dense(np.shape(X)[1], shapes, [np.abs(A) for A in As[:-1]] + [As[-1]])
        return np.abs(np.asarray(X, np.float64)) @ M.T

    def abs_of_product(X, shapes, As):
        M = np.abs(orig_dense(np.shape(X)[1], shapes, As))
        return np.abs(np.asarray(X, np.float64)) @ M.T

    for mutant in (no_abs_x, no_abs_last, abs_of_product):
        monkeypatch.setattr(jl, "abs_bound", mutant)
        failed = 0
        for pin, args in ((test_abs_bound_worked_example, ()),
                          (test_abs_bound_exact_rationals, ([(3, 4, 3), (2, 9, 1)],))):
            try:
                pin(*args)
            except AssertionError:
                failed += 1
        assert failed >= 1, mutant.__name__
