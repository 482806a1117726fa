"""Section 4's ip-distance front ends on the GPU against the oracle.

Cosine (f = g = x / ||x||): sj_normalize's rows bit for bit against the
oracle's normalisation (both: double norm in ascending k, one double division,
rounding to the nearest binary16 / bfloat16, ties to even -- a decision both
sides take in the same precision); the cosine join (SJ_FLAG_COSINE) against
the oracle's inner-product join of the oracle's normalised rows, identical
outside the boundary band 1e-3 |s| (the normalised rows are real-valued).

Hamming (f(x) = (x, 1 - x), g(y) = (1 - y, y) on {0, 1}^d): sj_join_hamming's
pairs against the oracle's Hamming join on the same bit rows, exactly (integer
scores), across the resident and K-streamed kernels, both modes, ragged
shapes, garbage in the padding bits, the self-join, ties at r and the edges.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads
from gpu_util import compare, keys, sorted_pairs, to_device

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2006_12608_amd  # noqa: F401  (fails loudly when libsj.so is missing)
    yield
    torch.cuda.synchronize()


def _rows(rng, dtype, n, d, kind):
    if dtype == "i8":
        v = rng.integers(-128, 128, size=(n, d))
    elif kind == "wide":
        v = rng.standard_normal((n, d)) * np.exp(rng.uniform(-12, 8, size=(n, 1)))
    else:
        v = rng.standard_normal((n, d))
    X = workloads.encode(v if dtype != "f16" else np.clip(v, -6e4, 6e4), dtype)
    X[: max(1, n // 50)] = 0                 # zero rows stay zero
    return X


@pytest.mark.parametrize("dtype", ["f16", "bf16", "i8"])
@pytest.mark.parametrize("d,n,kind", [(1, 33, "unit"), (7, 300, "wide"), (64, 1000, "unit"),
                                      (256, 513, "wide"), (300, 129, "unit")])
def test_normalize_bit_exact(dtype, d, n, kind):
    import torch
    import paper_2006_12608_amd as sj
    rng = np.random.default_rng(500 + d + n)
    X = _rows(rng, dtype, n, d, kind)
    say("normalize", dtype, n, d, kind)
    Y = sj.normalize(to_device(X, dtype))
    want = oracle.normalize(dtype, X).view(np.uint16)
    got = Y.view(torch.int16).cpu().numpy().view(np.uint16)
    assert got.shape == want.shape
    bad = np.argwhere(got != want)
    assert bad.size == 0, f"{bad.shape[0]} values differ, first {bad[:3].tolist()}"


def _cos_case(dtype, n_p, n_q, d, seed, q=0.995):
    rng = np.random.default_rng(seed)
    P = _rows(rng, dtype, n_p, d, "unit")
    Q = _rows(rng, dtype, n_q, d, "unit")
    Q[5:25] = P[40:60]                      # identical rows: cosine 1
    Pn, Qn = oracle.normalize(dtype, P), oracle.normalize(dtype, Q)
    out_dt = "bf16" if dtype == "bf16" else "f16"
    from pins import values
    S = values(out_dt, Pn.view(np.uint16) if out_dt == "bf16" else Pn) @ \
        values(out_dt, Qn.view(np.uint16) if out_dt == "bf16" else Qn).T
    s = float(np.quantile(S, q))
    return P, Q, Pn, Qn, out_dt, s


@pytest.mark.parametrize("dtype,d,two_pass", [("f16", 64, False), ("bf16", 96, True),
                                              ("i8", 40, False), ("f16", 300, True),
                                              ("bf16", 17, False)])
def test_cosine_join(dtype, d, two_pass):
    import paper_2006_12608_amd as sj
    P, Q, Pn, Qn, out_dt, s = _cos_case(dtype, 700, 610, d, 600 + d)
    say("cosine join", dtype, d, s, "two_pass" if two_pass else "single")
    g = sorted_pairs(sj.join_ip(to_device(P, dtype), to_device(Q, dtype), s, cosine=True,
                                two_pass=two_pass, cap=None if two_pass else 700 * 610))
    Pd = Pn if out_dt == "f16" else Pn.view(np.uint16)
    Qd = Qn if out_dt == "f16" else Qn.view(np.uint16)
    ref = oracle.join("ip", out_dt, Pd, Qd, s, band=1e-3 * abs(s))
    info = compare(g, ref, True)
    assert ref.total > 20
    say("band", info)


def test_cosine_self_join_and_default_sizing():
    """P == Q (one normalisation, the upper triangle mirrored); the Python
    default (no capacity) sizes the output with a counting call."""
    import paper_2006_12608_amd as sj
    P, _, Pn, _, _, s = _cos_case("f16", 900, 30, 48, 611, q=0.99)
    Pd = to_device(P, "f16")
    say("cosine self-join", s)
    g = sorted_pairs(sj.join_ip(Pd, Pd, s, cosine=True, cap=900 * 900, two_pass=False))
    ref = oracle.join("ip", "f16", Pn, Pn.copy(), s, band=1e-3 * abs(s))
    compare(g, ref, True)
    assert all((i, i) in set(map(tuple, g.tolist())) for i in range(18, 900))   # nonzero rows
    h = sorted_pairs(sj.join_ip(Pd, Pd, s, cosine=True))
    assert np.array_equal(g, h)


def test_cosine_on_the_cosine_workload():
    """The cosine workload's distribution (rows already normalised in float64
    and rounded to fp16) normalised again on the GPU: its planted neighbours
    are found and the pairs equal the oracle's outside the band."""
    import paper_2006_12608_amd as sj
    w = workloads.make_config("cos_f16_262144x256", n=3000)
    say("cosine workload", w.name)
    g = sorted_pairs(sj.join_ip(to_device(w.P, "f16"), to_device(w.Q, "f16"), w.threshold,
                                cosine=True))
    Pn, Qn = oracle.normalize("f16", w.P), oracle.normalize("f16", w.Q)
    ref = oracle.join("ip", "f16", Pn, Qn, w.threshold, band=1e-3 * w.threshold)
    compare(g, ref, True)
    assert set(map(tuple, w.planted.tolist())) <= set(map(tuple, g.astype(np.int64).tolist()))


def _bits(rng, n, d, garbage=True):
    B = rng.integers(0, 2, size=(n, d)).astype(np.uint8)
    X = np.packbits(B, axis=1, bitorder="little")
    if garbage and d % 8:
        X[:, -1] |= rng.integers(0, 256, size=n).astype(np.uint8) & np.uint8((0xFF << (d % 8)) & 0xFF)
    return np.ascontiguousarray(X), B


def _bits_device(X):
    import torch
    return torch.from_numpy(X).cuda()


@pytest.mark.parametrize("d,n_p,n_q,two_pass", [(1, 40, 33, False), (8, 300, 517, True),
                                                (45, 513, 129, False), (64, 700, 600, True),
                                                (100, 257, 300, False), (256, 300, 301, True),
                                                (300, 270, 333, False), (1000, 130, 140, True),
                                                (16384, 33, 70, False), (16384, 33, 70, True)])
def test_hamming_join(d, n_p, n_q, two_pass):
    import paper_2006_12608_amd as sj
    rng = np.random.default_rng(700 + d)
    P, bp = _bits(rng, n_p, d)
    Q, bq = _bits(rng, n_q, d)
    Q[3:13] = P[20:30]                        # distance 0
    flip = rng.integers(0, d, size=10)
    for t in range(10):                       # distance 1
        Q[20 + t, flip[t] // 8] ^= np.uint8(1 << (flip[t] % 8))
    for r in (0, d // 3, d / 2 - 0.5, d / 2):
        say("hamming", d, n_p, n_q, r, "two_pass" if two_pass else "single")
        g = sorted_pairs(sj.join_hamming(_bits_device(P), _bits_device(Q), d, r,
                                         two_pass=two_pass,
                                         cap=None if two_pass else n_p * n_q))
        want = oracle.hamming_join(P, Q, d, r)
        assert np.array_equal(keys(g), keys(want)), (d, r, g.shape[0], len(want))


def test_hamming_self_join_and_larger():
    """The same pointer (upper triangle, mirrored: symmetric, diagonal
    present) and a 12000-row, 128-bit join with planted near-duplicates."""
    import paper_2006_12608_amd as sj
    rng = np.random.default_rng(710)
    P, _ = _bits(rng, 1100, 64)
    P[500:520] = P[0:20]
    Pd = _bits_device(P)
    say("hamming self-join")
    g = sorted_pairs(sj.join_hamming(Pd, Pd, 64, 22, two_pass=False, cap=1100 * 1100))
    want = oracle.hamming_join(P, P.copy(), 64, 22)
    assert np.array_equal(keys(g), keys(want))
    s = set(map(tuple, g.tolist()))
    assert all((i, i) in s for i in range(1100)) and all((j, i) in s for (i, j) in s)
    P, _ = _bits(rng, 12000, 128, garbage=False)
    Q, _ = _bits(rng, 12000, 128, garbage=False)
    Q[:300] = P[1000:1300]
    for t in range(300):
        Q[t, rng.integers(0, 16)] ^= np.uint8(1 << rng.integers(0, 8))
    say("hamming 12000 x 128 bits")
    g = sorted_pairs(sj.join_hamming(_bits_device(P), _bits_device(Q), 128, 40))
    want = oracle.hamming_join(P, Q, 128, 40)
    assert np.array_equal(keys(g), keys(want)) and len(want) >= 300


def test_frontend_edges_and_errors():
    import torch
    import paper_2006_12608_amd as sj
    ctx = sj.context()
    say("front-end edges")
    Z = torch.zeros((0, 2), dtype=torch.uint8, device="cuda")
    P = torch.zeros((5, 2), dtype=torch.uint8, device="cuda")
    assert sj.join_hamming(Z, P, 16, 3).shape[0] == 0
    E = torch.zeros((6, 0), dtype=torch.uint8, device="cuda")
    F = torch.zeros((7, 0), dtype=torch.uint8, device="cuda")
    assert sj.join_hamming(E, F, 0, 0).shape[0] == 42          # d = 0: every distance 0
    assert sj.join_hamming(E, F, 0, -0.5).shape[0] == 0
    X, _ = _bits(np.random.default_rng(3), 64, 20)
    Xd = _bits_device(X)
    total = len(oracle.hamming_join(X, X.copy(), 20, 6))
    out = torch.empty((total, 2), dtype=torch.int32, device="cuda")
    for flags in (0, sj.SJ_FLAG_TWO_PASS):
        st, n = sj.sj_join_hamming(ctx, Xd.data_ptr(), 64, Xd.data_ptr(), 64, 20, 6,
                                   out.data_ptr(), total - 1, flags)
        assert st == sj.SJ_E_OVERFLOW and n == total
    assert sj.sj_join_hamming(ctx, Xd.data_ptr(), 64, Xd.data_ptr(), 64, 20, float("nan"),
                              out.data_ptr(), total)[0] == sj.SJ_E_INVAL
    assert sj.sj_join_hamming(ctx, Xd.data_ptr(), 1, Xd.data_ptr(), 1, 16385, 1.0,
                              out.data_ptr(), total)[0] in (sj.SJ_E_UNSUPPORTED, sj.SJ_E_INVAL)
    # cosine of empty and zero-dimensional inputs; a zero row normalises to zeros
    H = torch.zeros((0, 8), dtype=torch.float16, device="cuda")
    assert sj.join_ip(H, H, 0.0, cosine=True).shape[0] == 0
    H0 = torch.zeros((3, 0), dtype=torch.float16, device="cuda")
    assert sj.join_ip(H0, H0, 0.0, cosine=True).shape[0] == 9
    Zr = torch.zeros((4, 8), dtype=torch.bfloat16, device="cuda")
    assert torch.count_nonzero(sj.normalize(Zr).float()) == 0
    assert sj.join_ip(Zr, Zr, 0.0, cosine=True).shape[0] == 16  # <0, 0> = 0 >= 0
