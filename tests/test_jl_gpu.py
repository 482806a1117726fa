"""GPU TCU JL transform (sj_jl) vs the oracle (dense Kronecker product in
float64), value by value.

Tolerance, from the arithmetic: every level is an fp32 product whose sums
have at most c_i terms, so (to first order, for any summation order) the
computed level differs from the exact one by at most gamma(c_i) |A_i| |input|
with gamma(n) = n u / (1 - n u), u = 2^-24; the levels' errors add up through
|M|, so |Y - Y_exact| <= 2 sum_i gamma(c_i) (|M| |x|) (factor 2 of margin for
the second-order terms).  The first level decodes its inputs exactly.  With
integer factors and integer inputs small enough that every partial sum stays
below 2^24 the result is exact, and the tests require equality there.
"""
import os
import sys

import numpy as np
import pytest

import workloads
from gpu_util import to_device
from oracle import jl

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2006_12608_amd  # noqa: F401
    yield
    torch.cuda.synchronize()


def chain(d, k, zeta):
    l = int(round(np.log(d / k) / np.log(zeta)))
    assert zeta ** l * k == d
    shapes = []
    for i in range(1, l + 1):
        ki = k if i == l else i * k
        ci = zeta * k if i == 1 else zeta * shapes[-1][0]
        shapes.append((ki, ci, zeta ** (l - i)))
    return shapes


def gamma(n):
    u = 2.0 ** -24
    return n * u / (1 - n * u)


def run(X, dtype, shapes, As):
    import torch
    import paper_2006_12608_amd as sj
    Xd = to_device(X, dtype)
    Ad = [torch.from_numpy(np.ascontiguousarray(A, dtype=np.float32)).cuda() for A in As]
    return sj.jl_transform(Xd, shapes, Ad).cpu().numpy().astype(np.float64)


def values(dtype, X):
    from pins import values as v
    return v(dtype, X)


@pytest.mark.parametrize("dtype,n,d,k,zeta", [("f16", 1000, 256, 32, 2), ("bf16", 333, 1024, 16, 4),
                                              ("i8", 777, 96, 12, 2), ("f16", 4099, 64, 8, 2)])
def test_jl_parity_real_factors(dtype, n, d, k, zeta):
    rng = np.random.default_rng(n + d)
    shapes = chain(d, k, zeta)
    As = [(rng.standard_normal((kk, c)) / np.sqrt(kk)).astype(np.float32).astype(np.float64)
          for (kk, c, r) in shapes]
    if dtype == "i8":
        X = workloads.encode(rng.integers(-20, 21, size=(n, d)), "i8")
    else:
        X = workloads.encode(rng.standard_normal((n, d)), dtype)
    say("jl", dtype, n, d, shapes)
    Y = run(X, dtype, shapes, As)
    x = values(dtype, X)
    ref = jl.transform(x, shapes, As)
    bound = 2 * sum(gamma(c) for (_, c, _) in shapes) * jl.abs_bound(x, shapes, As)
    err = np.abs(Y - ref)
    assert np.all(err <= bound), (err / np.maximum(bound, 1e-300)).max()


@pytest.mark.parametrize("dtype", ["i8", "bf16", "f16"])
def test_jl_exact_on_integers(dtype):
    """Integer factors and inputs: every partial sum is an integer below 2^24,
    so fp32 is exact and the GPU must equal the oracle."""
    rng = np.random.default_rng(7)
    shapes = [(8, 16, 6), (12, 24, 2), (5, 24, 1)]   # d = 96 -> 48 -> 24 -> 5
    As = [rng.integers(-3, 4, size=(kk, c)).astype(np.float64) for (kk, c, r) in shapes]
    X = workloads.encode(rng.integers(-4, 5, size=(517, 96)), dtype)
    Y = run(X, dtype, shapes, As)
    ref = jl.transform(values(dtype, X), shapes, As)
    assert np.array_equal(Y, ref)


def test_jl_worked_example():
    rows = {}
    for line in open(os.path.join(GOLDEN, "jl_small.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            name, rest = line.split(None, 1)
            rows[name] = [[float(v) for v in part.split()] for part in rest.split(";")]
    shapes = [tuple(int(v) for v in s) for s in rows["shapes"]]
    X = workloads.encode(np.array(rows["x"], dtype=np.int64), "i8")
    Y = run(X, "i8", shapes, [np.array(rows["A1"]), np.array(rows["A2"])])
    assert np.array_equal(Y, np.array(rows["y"]))


def test_jl_errors():
    import torch
    import paper_2006_12608_amd as sj
    X = torch.zeros((10, 24), dtype=torch.float16, device="cuda")
    A = torch.zeros(1000, dtype=torch.float32, device="cuda")
    Y = torch.zeros((10, 100), dtype=torch.float32, device="cuda")
    ctx = sj.context()
    bad = [[(3, 5, 4)], [(3, 6, 4), (2, 5, 2)], [(0, 6, 4)]]
    for shape in bad:
        st = sj.sj_jl(ctx, sj.SJ_F16, X.data_ptr(), 10, 24, len(shape), shape, A.data_ptr(),
                      Y.data_ptr())
        assert st == sj.SJ_E_INVAL, shape
    st = sj.sj_jl(ctx, sj.SJ_F16, X.data_ptr(), 10, 24, 0, [], A.data_ptr(), Y.data_ptr())
    assert st == sj.SJ_E_INVAL
    # buffers smaller than their shapes (checked against the allocation, which
    # the caching allocator rounds up: so ask for far more than it holds)
    st = sj.sj_jl(ctx, sj.SJ_F16, X.data_ptr(), 1 << 24, 24, 1, [(5, 24, 1)], A.data_ptr(),
                  Y.data_ptr())
    assert st == sj.SJ_E_INVAL      # X
    bigA = torch.zeros(65536 * 24, dtype=torch.float32, device="cuda")
    st = sj.sj_jl(ctx, sj.SJ_F16, X.data_ptr(), 10, 24, 1, [(65536, 24, 1)], bigA.data_ptr(),
                  Y.data_ptr())
    assert st == sj.SJ_E_INVAL      # Y holds far less than 10 x 65536 floats
    # a size chain whose last level would hold 10 x 2^47 values (more than
    # 2^48): rejected before any buffer is sized from it
    huge = [(65536, 24, 1), (65536, 1, 65536), (65536, 2, 1 << 31)]
    st = sj.sj_jl(ctx, sj.SJ_F16, X.data_ptr(), 10, 24, 3, huge, A.data_ptr(), Y.data_ptr())
    assert st == sj.SJ_E_UNSUPPORTED, sj.sj_last_error()
    st = sj.sj_jl(ctx, sj.SJ_F16, X.data_ptr(), 0, 24, 1, [(5, 24, 1)], A.data_ptr(),
                  Y.data_ptr())
    assert st == sj.SJ_OK


def test_jl_full_size_sampled_rows():
    """The cosine workload's 262144 x 256 fp16 rows reduced to k = 32 (three
    levels, zeta = 2) as bench.py runs it; the oracle checks sampled rows."""
    w = workloads.make_config("cos_f16_262144x256")
    rng = np.random.default_rng(1402)
    shapes = chain(256, 32, 2)
    As = [(rng.standard_normal((kk, c)) / np.sqrt(kk)).astype(np.float32).astype(np.float64)
          for (kk, c, r) in shapes]
    Y = run(w.P, "f16", shapes, As)
    rows = np.sort(rng.choice(w.n_p, size=64, replace=False))
    x = values("f16", w.P[rows])
    ref = jl.transform(x, shapes, As)
    bound = 2 * sum(gamma(c) for (_, c, _) in shapes) * jl.abs_bound(x, shapes, As)
    assert np.all(np.abs(Y[rows] - ref) <= bound)
    # the JL property on unit rows: norms within 1 +- 0.5 for nearly all rows
    nrm = np.linalg.norm(Y, axis=1)
    assert (np.abs(nrm - 1) <= 0.5).mean() > 0.99


def test_jl_most_levels():
    """32 levels, the most one call takes: row lengths 12 -> 8 -> 12 -> ...
    through (k, c, r) = (2, 3, 4) and (3, 2, 4), each factor a signed selection
    (one +-1 per row), so every value stays a small integer and the result
    must equal the oracle's exactly."""
    rng = np.random.default_rng(3232)
    shapes = [(2, 3, 4) if i % 2 == 0 else (3, 2, 4) for i in range(32)]
    As = []
    for (k, c, r) in shapes:
        A = np.zeros((k, c))
        A[np.arange(k), rng.integers(0, c, size=k)] = rng.choice([-1.0, 1.0], size=k)
        As.append(A)
    X = workloads.encode(rng.integers(-4, 5, size=(301, 12)), "f16")
    say("jl 32 levels")
    Y = run(X, "f16", shapes, As)
    assert Y.shape == (301, 12)
    assert np.array_equal(Y, jl.transform(values("f16", X), shapes, As))


@pytest.mark.parametrize("dtype,n,d,shapes", [
    ("f16", 1, 6, [(3, 6, 1)]),                      # one row, one level
    ("bf16", 129, 15, [(2, 5, 3), (7, 6, 1)]),       # odd sizes: no 4-entry loads
    ("i8", 65, 200, [(130, 200, 1)]),                 # more than 128 output columns
])
def test_jl_edge_shapes(dtype, n, d, shapes):
    rng = np.random.default_rng(n + d)
    As = [rng.integers(-3, 4, size=(k, c)).astype(np.float64) for (k, c, r) in shapes]
    X = workloads.encode(rng.integers(-4, 5, size=(n, d)), dtype)
    Y = run(X, dtype, shapes, As)
    assert np.array_equal(Y, jl.transform(values(dtype, X), shapes, As))
