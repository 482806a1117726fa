"""GPU LSH-bucketed join (sj_join_lsh) vs the oracle's LSH join, pair set by
pair set, on seeded inputs and seeded LSH draws.

The bucket keys are integers computed exactly (or in double precision in the
same order) on both sides -- the GPU's matrix-core hash keeps only the
decisions its fp32 sums make certain and recomputes the rest that way -- so
the candidate sets agree exactly; the exact test then follows the all-pairs
join's rules: identical sets for integer-valued inputs, identical outside the
boundary band for real-valued ones.  Cases cover both hash families, every
dtype, both metrics, ragged sizes against the 128-row tiles, buckets
spanning several tiles, unaligned rows, the self-join, k = 0 (the exact
join), the first-table rule (no duplicates), decisions the fp32 hash cannot
take, the candidate count, overflow and argument errors.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads
from gpu_util import compare, sorted_pairs, to_device, keys

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


def lsh_device(h):
    import torch
    A = torch.from_numpy(h.A).cuda()
    B = torch.from_numpy(h.B).cuda() if h.w > 0 else None
    return A, B


def expected_candidates(w, h, rows=False):
    """Sum over tables and keys of (#P rows with the key) x (#Q rows with it),
    from the oracle's keys; with rows=True also the sum of (#P rows + #Q rows)
    over the keys both have."""
    kp = oracle.lsh_keys(w.dtype, w.P, h.L, h.k, h.A, h.B, h.w)
    kq = oracle.lsh_keys(w.dtype, w.Q, h.L, h.k, h.A, h.B, h.w)
    tot = nrows = 0
    for t in range(h.L):
        up, cp = np.unique(kp[t], return_counts=True)
        uq, cq = np.unique(kq[t], return_counts=True)
        _, ip, iq = np.intersect1d(up, uq, return_indices=True)
        tot += int((cp[ip].astype(np.int64) * cq[iq]).sum())
        nrows += int(cp[ip].sum() + cq[iq].sum())
    return (tot, nrows) if rows else tot


def run_lsh(w, h, thr=None, self_join=False, check_cand=True):
    import paper_2006_12608_amd as sj
    thr = w.threshold if thr is None else thr
    Pd = to_device(w.P, w.dtype)
    Qd = Pd if self_join else to_device(w.Q, w.dtype)
    A, B = lsh_device(h)
    say(w.name, w.metric, w.dtype, w.n_p, w.n_q, w.d, thr, f"L={h.L} k={h.k} w={h.w}")
    got, cand = sj.join_lsh(Pd, Qd, thr, w.metric, L=h.L, k=h.k, A=A, B=B, w=h.w)
    g = sorted_pairs(got)
    ref_pairs = oracle.lsh_join(w.metric, w.dtype, w.P, w.Q, thr, h.L, h.k, h.A, h.B, h.w)
    band = 1e-3 * abs(thr) if w.real_valued else 0.0
    exact = oracle.join(w.metric, w.dtype, w.P, w.Q, thr, band=band)
    ref = oracle.JoinResult(ref_pairs, len(ref_pairs), exact.band_pairs, exact.band_match)
    info = compare(g, ref, w.real_valued)
    if check_cand:
        e_cand, e_rows = expected_candidates(w, h, rows=True)
        assert cand == e_cand
        assert sj.sj_get_stats(sj.context(Pd.device.index)).lsh_rows == e_rows
    return g, ref_pairs, exact, cand, info


def case(seed, n_p, n_q, d, dtype, metric, thr, lo=-4, hi=4, real=False):
    w = workloads.random_case(seed, n_p, n_q, d, dtype, lo, hi, real=real, metric=metric,
                              threshold=thr)
    return w


@pytest.mark.parametrize("dtype,metric,thr,d,wid", [
    ("i8", "ip", 20.0, 64, 0),
    ("bf16", "ip", 18.0, 128, 0),
    ("f16", "ip", 30.0, 72, 0),
    ("i8", "l2", 400.0, 48, 300),
    ("bf16", "l2", 420.0, 96, 400),
    ("f16", "l2", 500.0, 40, 350),
    ("i8", "l2", 600.0, 96, 400),     # 96-byte rows: the longest that travel as records
    ("f16", "l2", 500.0, 48, 350),
    ("i8", "l2", 600.0, 97, 400),     # 112-byte padded rows: gathered without records
])
def test_lsh_parity_integer(dtype, metric, thr, d, wid):
    w = case(700 + d, 333, 290, d, dtype, metric, thr)
    # planted near-duplicates so the buckets share close pairs
    w.Q[:40] = w.P[100:140]
    h = workloads.lsh_params(900 + d, L=6, k=3, d=d, w=wid)
    g, ref, exact, cand, _ = run_lsh(w, h)
    assert 0 < len(ref) <= exact.total
    assert cand < w.n_p * w.n_q * h.L


@pytest.mark.parametrize("dtype,d,L,k,wid,metric,thr", [
    # 1200-byte rows: the keys from 512-byte segments of the rows in LDS, the
    # functions in passes of 16; the bucket join gathers 10 chunks per row
    ("f16", 600, 5, 20, 0, "ip", 150.0),
    ("i8", 1100, 3, 6, 900, "l2", 4000.0),    # 1104-byte rows, quantised hashes
    # 70 tables of 8 signs (560 functions): more than the matrix-core hash takes
    ("bf16", 64, 70, 8, 0, "ip", 20.0),
])
def test_lsh_general_hash_long_rows_many_functions(dtype, d, L, k, wid, metric, thr):
    w = case(800 + d + L, 300, 280, d, dtype, metric, thr)
    w.Q[:40] = w.P[100:140]
    h = workloads.lsh_params(950 + d + L, L=L, k=k, d=d, w=wid)
    g, ref, exact, cand, _ = run_lsh(w, h)
    assert 40 <= len(ref) <= exact.total


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_lsh_parity_real_cosine(dtype):
    """Unit rows (real-valued), sign hashes: identical outside the band."""
    wl = workloads.make_config("cos_f16_262144x256", n=1500)
    if dtype == "bf16":
        P = workloads.bf16_bits_from_f32(wl.P.astype(np.float32))
        Q = workloads.bf16_bits_from_f32(wl.Q.astype(np.float32))
        wl = workloads.Workload(wl.name + "-bf16", "ip", "bf16", P, Q, wl.threshold,
                                wl.planted, real_valued=True)
    h = workloads.lsh_params(77, L=8, k=6, d=wl.d)
    g, ref, exact, cand, info = run_lsh(wl, h)
    assert len(ref) > 0
    say("band", info)


def test_lsh_buckets_span_tiles_and_ragged():
    """k = 1: two big buckets per table, each hundreds of rows (several 128-row
    tiles plus ragged tails on both sides)."""
    w = case(41, 517, 389, 33, "i8", "ip", 15.0, -6, 6)   # 33-byte rows: repacked
    h = workloads.lsh_params(42, L=3, k=1, d=33)
    run_lsh(w, h)


def test_lsh_quantised_wide_keys_many_rows():
    """Seven quantised values of 9 bits and 8 tables (63-bit keys: sorted by
    the top half of their mix, then the rare runs whose halves collide by the
    whole mix) on 6000 int8 rows of the squared-L2 workload: the sorts span
    many radix blocks."""
    wl = workloads.make_config("l2_i8_1048576x64", n=6000)
    h = workloads.lsh_params(1303, L=8, k=7, d=wl.d, w=2000)
    g, ref, exact, cand, _ = run_lsh(wl, h)
    assert 0 < len(ref) <= exact.total


def test_lsh_k0_is_exact_join():
    import paper_2006_12608_amd as sj
    w = case(43, 200, 150, 64, "bf16", "ip", 12.0)
    h = workloads.lsh_params(44, L=2, k=0, d=64)
    g, ref, exact, cand, _ = run_lsh(w, h)
    assert np.array_equal(keys(g), keys(exact.pairs))
    assert cand == w.n_p * w.n_q * h.L
    full = sorted_pairs(sj.join_ip(to_device(w.P, "bf16"), to_device(w.Q, "bf16"), 12.0))
    assert np.array_equal(full, g)


@pytest.mark.parametrize("metric,thr,k,wid", [("l2", 200.0, 0, 0), ("l2", 180.0, 1, 120),
                                             ("ip", 2.0, 2, 0)])
def test_lsh_dense_matches(metric, thr, k, wid):
    """Short int8 rows (joined as row records) with thresholds that most pairs
    pass: waves find from a few to thousands of pairs per tile, so the pairs
    go both through the per-wave staging (many flushes) and straight out."""
    w = case(51 + k, 700, 650, 16, "i8", metric, thr, -3, 3)
    h = workloads.lsh_params(52 + k, L=3, k=k, d=16, w=wid)
    g, ref, exact, *_ = run_lsh(w, h)
    assert len(ref) > w.n_p * w.n_q // 10


def test_lsh_self_join_same_pointer():
    w = case(45, 300, 300, 32, "i8", "l2", 300.0, -5, 5)
    w.Q = w.P
    w.P[50:60] = w.P[0:10]
    h = workloads.lsh_params(46, L=5, k=2, d=32, w=250)
    g, ref, *_ = run_lsh(w, h, self_join=True)
    s = set(map(tuple, g.tolist()))
    assert all((i, i) in s for i in range(300))      # every point collides with itself
    assert all((j, i) in s for (i, j) in s)          # symmetric


@pytest.mark.parametrize("d,L,thr", [(16, 24, 6.0), (64, 56, 64.0), (80, 20, 72.0),
                                     (96, 24, 78.0), (128, 24, 90.0), (32, 256, 20.0)])
def test_lsh_many_tables_first_table_rule(d, L, thr):
    """Many tables and few functions: most pairs collide in several tables;
    each must still be reported once.  Short rows carry fingerprints of the
    first 112 - (row bytes rounded up to 32) tables in their records (80, 48
    and 16 tables here, later tables by their keys); 128-byte rows carry 16.
    256 tables is the most one call takes (its hash on the general kernel)."""
    w = case(47 + d, 260, 240, d, "i8", "ip", thr, -3, 3)
    h = workloads.lsh_params(48 + d, L=L, k=2, d=d)
    g, ref, *_ = run_lsh(w, h)
    assert len(g) == len(ref) > 0


def test_lsh_overflow_and_errors():
    import torch
    import paper_2006_12608_amd as sj
    w = case(49, 128, 128, 32, "i8", "ip", 4.0)
    h = workloads.lsh_params(50, L=4, k=2, d=32)
    Pd, Qd = to_device(w.P, "i8"), to_device(w.Q, "i8")
    A, B = lsh_device(h)
    n_ref = len(oracle.lsh_join("ip", "i8", w.P, w.Q, 4.0, h.L, h.k, h.A, h.B, h.w))
    assert n_ref > 10
    out = torch.empty((5, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(sj.SjError) as e:
        sj.join_lsh(Pd, Qd, 4.0, "ip", L=4, k=2, A=A, w=0, cap=5, out=out)
    assert e.value.status == sj.SJ_E_OVERFLOW and e.value.n_out == n_ref
    ctx = sj.context()
    args = (ctx, sj.SJ_IP, sj.SJ_I8, Pd.data_ptr(), 128, Qd.data_ptr(), 128, 32, 4.0)
    assert sj.sj_join_lsh(*args, 0, 2, A.data_ptr(), None, 0, None, 0)[0] == sj.SJ_E_INVAL
    assert sj.sj_join_lsh(*args, 4, 65, A.data_ptr(), None, 0, None, 0)[0] == sj.SJ_E_INVAL
    assert sj.sj_join_lsh(*args, 4, 2, None, None, 0, None, 0)[0] == sj.SJ_E_INVAL
    assert sj.sj_join_lsh(*args, 4, 2, A.data_ptr(), None, 5, None, 0)[0] == sj.SJ_E_INVAL
    assert sj.sj_join_lsh(*args, 4, 2, A.data_ptr(), None, -1, None, 0)[0] == sj.SJ_E_INVAL
    st, n, nc = sj.sj_join_lsh(ctx, sj.SJ_IP, sj.SJ_I8, Pd.data_ptr(), 0, Qd.data_ptr(), 128,
                               32, 4.0, 4, 2, A.data_ptr(), None, 0, None, 0)
    assert (st, n, nc) == (sj.SJ_OK, 0, 0)


def test_lsh_cosine_workload_recall():
    """The cosine workload's distribution at 16384 rows with the LSH
    parameters the benchmark uses at full size (16 tables of 10 signs):
    parity with the oracle's LSH join, and every planted neighbour that
    matches is found unless no table makes it collide."""
    wl = workloads.make_config("cos_f16_262144x256", n=16384)
    h = workloads.lsh_params(1302, L=16, k=10, d=wl.d)
    g, ref, exact, cand, info = run_lsh(wl, h, check_cand=False)
    say("pairs", len(g), "exact", exact.total, "candidates", cand, "band", info)
    assert cand < wl.n_p * wl.n_q // 8
    assert len(ref) >= 0.9 * exact.total


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("wid", [0, 5])
def test_lsh_uncertain_decisions_are_exact(dtype, wid):
    """Rows built so that many projections are exactly zero (sign hashes) or
    land exactly on a bucket boundary (width 5): the matrix-core hash cannot
    decide those from its fp32 sums and recomputes them exactly; the pairs must
    still be the oracle's, and the same integer points stored as int8 (which
    take the exact int32 hash throughout) must give the same pairs."""
    import paper_2006_12608_amd as sj
    import torch
    rng = np.random.default_rng(91 + wid)
    d, L, k = 32, 6, 4
    h = workloads.lsh_params(92, L=L, k=k, d=d, w=wid)
    h.A[:, 16:] = 0                       # projections see only the first 16 coordinates
    x = rng.integers(-3, 4, size=(400, d))
    x[:150, :16] = 0                      # ... which are zero for 150 rows: z = 0 exactly
    y = rng.integers(-3, 4, size=(380, d))
    y[:120, :16] = 0
    y[200:260] = x[200:260]
    w = workloads.Workload("zeros", "ip", dtype, workloads.encode(x, dtype),
                           workloads.encode(y, dtype), 10.0, np.zeros((0, 2), np.int64))
    g, ref, exact, cand, _ = run_lsh(w, h)
    wi = workloads.Workload("zeros-i8", "ip", "i8", workloads.encode(x, "i8"),
                            workloads.encode(y, "i8"), 10.0, np.zeros((0, 2), np.int64))
    gi, *_ = run_lsh(wi, h)
    assert np.array_equal(keys(g), keys(gi))


def test_lsh_many_functions_matrix_core_hash():
    """24 tables of 12 signs (288 functions: the matrix-core hash's function
    masks span several 64-bit words, and tables straddle them) on real-valued
    unit rows: parity with the oracle outside the band."""
    wl = workloads.make_config("cos_f16_262144x256", n=1200)
    h = workloads.lsh_params(78, L=24, k=12, d=wl.d)
    g, ref, exact, cand, info = run_lsh(wl, h)
    assert len(ref) > 0


@pytest.mark.parametrize("dtype,n_p,n_q,d,L,k,wid,metric,thr", [
    ("f16", 1, 1, 7, 2, 3, 0, "ip", -1000.0),    # one point each, odd d (repacked rows)
    ("bf16", 1, 300, 9, 3, 64, 0, "ip", 5.0),    # 64 sign bits per table (one bit each)
    ("i8", 257, 1, 5, 4, 2, 3, "l2", 40.0),      # quantised with a tiny bucket width
    ("f16", 130, 129, 1, 2, 5, 0, "ip", 2.0),    # d = 1: every projection is a multiple of x
])
def test_lsh_edge_shapes(dtype, n_p, n_q, d, L, k, wid, metric, thr):
    w = case(60 + d + n_p, n_p, n_q, d, dtype, metric, thr, -3, 3)
    h = workloads.lsh_params(61 + k, L=L, k=k, d=d, w=wid)
    run_lsh(w, h)


def test_lsh_full_size_sampled_rows():
    """The full cosine workload (262144 x 256 fp16) with the benchmark's LSH
    parameters (16 tables of 10 signs, its seed): the oracle computes every
    row's keys and, for sampled rows of P, the exact matches; the LSH join's
    pairs of those rows must be exactly the matches that share a key with them
    in some table (outside the boundary band)."""
    import paper_2006_12608_amd as sj
    wl = workloads.make_config("cos_f16_262144x256")
    h = workloads.lsh_params(1300 + workloads.NAMES.index("cos_f16_262144x256"), L=16, k=10,
                             d=wl.d)
    Pd, Qd = to_device(wl.P, wl.dtype), to_device(wl.Q, wl.dtype)
    A, _ = lsh_device(h)
    say("lsh full", wl.name)
    got, cand = sj.join_lsh(Pd, Qd, wl.threshold, "ip", L=h.L, k=h.k, A=A)
    g = sorted_pairs(got)
    rng = np.random.default_rng(4321)
    rows = np.sort(np.concatenate([rng.choice(wl.n_p, size=16, replace=False),
                                   wl.planted[:16, 0]]))
    rows = np.unique(rows)
    kq = oracle.lsh_keys(wl.dtype, wl.Q, h.L, h.k, h.A)
    kp = oracle.lsh_keys(wl.dtype, np.ascontiguousarray(wl.P[rows]), h.L, h.k, h.A)
    ex = oracle.join("ip", wl.dtype, wl.P, wl.Q, wl.threshold, rows=rows,
                     band=1e-3 * wl.threshold)
    pos = {int(r): t for t, r in enumerate(rows)}
    keep = np.array([bool((kp[:, pos[int(i)]] == kq[:, int(j)]).any()) for i, j in ex.pairs],
                    dtype=bool) if ex.total else np.zeros(0, bool)
    ref = oracle.JoinResult(ex.pairs[keep], int(keep.sum()), ex.band_pairs, ex.band_match)
    info = compare(g[np.isin(g[:, 0], rows)], ref, True)
    say("rows", rows.size, "pairs", ref.total, "band", info)
    assert ref.total >= 16


def test_lsh_quantised_benchmark_parameters():
    """Six quantised values of 10 bits and 16 tables (60-bit keys: sorted by
    the top half of their mix; the benchmark's configuration on the int8
    squared-L2 workload) on 6000 rows of that workload: parity with the
    oracle's LSH join, its candidate count and its bucket rows."""
    wl = workloads.make_config("l2_i8_1048576x64", n=6000)
    h = workloads.lsh_params(1303, L=16, k=6, d=wl.d, w=2000)
    g, ref, exact, cand, _ = run_lsh(wl, h)
    assert 0 < len(ref) <= exact.total


def test_lsh_full_size_quantised_sampled_rows():
    """The full int8 squared-L2 workload (1048576 x 64) with the benchmark's
    LSH parameters (16 tables of 6 quantised projections, width 2000, its
    seed): the oracle computes every row's keys and, for sampled rows of P
    (random ones and planted ones), the exact matches; the LSH join's pairs
    of those rows must be exactly the matches that share a key with them in
    some table.  Every reported pair must pass the exact test, and none may
    repeat."""
    import paper_2006_12608_amd as sj
    name = "l2_i8_1048576x64"
    wl = workloads.make_config(name)
    h = workloads.lsh_params(1300 + workloads.NAMES.index(name), L=16, k=6, d=wl.d, w=2000)
    Pd, Qd = to_device(wl.P, wl.dtype), to_device(wl.Q, wl.dtype)
    A, B = lsh_device(h)
    say("lsh full", wl.name, f"L={h.L} k={h.k} w={h.w}")
    got, cand = sj.join_lsh(Pd, Qd, wl.threshold, "l2", L=h.L, k=h.k, A=A, B=B, w=h.w)
    g = sorted_pairs(got)
    assert np.unique(keys(g)).size == g.shape[0]
    sc = oracle.scores("l2", wl.dtype, wl.P, wl.Q, g.astype(np.int64))
    assert np.all(sc <= wl.threshold)
    rng = np.random.default_rng(4322)
    rows = np.unique(np.concatenate([rng.choice(wl.n_p, size=24, replace=False),
                                     wl.planted[:40, 0], wl.planted[-8:, 0]]))
    kq = oracle.lsh_keys(wl.dtype, wl.Q, h.L, h.k, h.A, h.B, h.w)
    kp = oracle.lsh_keys(wl.dtype, np.ascontiguousarray(wl.P[rows]), h.L, h.k, h.A, h.B, h.w)
    ex = oracle.join("l2", wl.dtype, wl.P, wl.Q, wl.threshold, rows=rows)
    pos = {int(r): t for t, r in enumerate(rows)}
    keep = np.array([bool((kp[:, pos[int(i)]] == kq[:, int(j)]).any()) for i, j in ex.pairs],
                    dtype=bool)
    ref = oracle.JoinResult(ex.pairs[keep], int(keep.sum()), ex.band_pairs, ex.band_match)
    compare(g[np.isin(g[:, 0], rows)], ref, False)
    say("rows", rows.size, "exact", ex.total, "found", ref.total, "candidates", cand,
        "pairs", g.shape[0])
    assert ref.total >= 30


@pytest.mark.parametrize("name,wid,dist_far", [("cos_f16_262144x256", 0, None),
                                               ("l2_i8_1048576x64", 2000, 101.2)])
def test_lsh_merged_instances_from_the_plan(name, wid, dist_far):
    """Section 4's parameters from sj_lsh_plan (recall target 0.9), and its
    high-probability scheme: the planned number of instances, each with its
    own draws, run as one call with all their tables (the first-table rule
    merges them).  The result equals the union of the oracle's LSH joins of
    the instances taken one by one, with no pair twice, and every planted
    pair the union holds."""
    import math
    import paper_2006_12608_amd as sj
    wl = workloads.make_config(name, n=2500)
    if wid == 0:
        p1 = sj.sj_lsh_collision(0, 1.0, math.acos(wl.threshold))
        p2 = sj.sj_lsh_collision(0, 1.0, math.pi / 2)
    else:
        p1 = sj.sj_lsh_collision(wid, 32.0, math.sqrt(wl.threshold))
        p2 = sj.sj_lsh_collision(wid, 32.0, dist_far)
    st, k, L_inst, reps = sj.sj_lsh_plan(p1, p2, wl.n_p, 128, 0.9)
    assert st == sj.SJ_OK
    k = max(k, 1)
    L_inst = min(L_inst, 256 // reps)
    insts = [workloads.lsh_params(2000 + 7 * r, L=L_inst, k=k, d=wl.d, w=wid) for r in range(reps)]
    h = workloads.LshParams(L_inst * reps, k, np.concatenate([x.A for x in insts]),
                            np.concatenate([x.B for x in insts]), wid)
    say("plan", name, "p1", p1, "p2", p2, "k", k, "L_inst", L_inst, "reps", reps)
    g, ref, exact, cand, _ = run_lsh(wl, h, check_cand=False)
    assert np.unique(keys(g)).size == g.shape[0]
    union = set()
    for x in insts:
        union |= set(map(tuple, oracle.lsh_join(wl.metric, wl.dtype, wl.P, wl.Q, wl.threshold,
                                                x.L, x.k, x.A, x.B, x.w).tolist()))
    assert set(map(tuple, np.asarray(ref).tolist())) == union
    say("found", len(union), "of", exact.total)
