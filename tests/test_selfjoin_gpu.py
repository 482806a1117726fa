"""Self-joins (P and Q the same pointer): the single pass computes only the
upper triangle of P.P^T and writes every off-diagonal match twice.

The pair set must equal the oracle's full join of P with itself, (i, i)
included and every (i, j) with its mirror (j, i), for every resident variant
(d picks the k-step variant), both metrics, sizes that span several
workgroups and Q tiles with ragged tails (so tiles straddle the diagonal in
every position), and at the size the benchmark's workloads use, on sampled
rows.  The two-pass mode (which computes the whole square) must give the
same set.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads
from gpu_util import compare, gpu_join, keys, sorted_pairs, to_device
from pins import values

pytestmark = pytest.mark.gpu


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


def self_case(seed, n, d, dtype, metric, quantile):
    w = workloads.random_case(seed, n, n, d, dtype, lo=-3, hi=3, metric=metric)
    w.P[n // 3: n // 3 + 20] = w.P[:20]      # duplicate rows: equal points
    w.Q = w.P
    w.self_join = True
    x = values(dtype, w.P).astype(np.int64)
    if metric == "ip":
        S = x @ x.T
        w.threshold = float(np.quantile(S, quantile, method="nearest"))
    else:
        N = (x * x).sum(1)
        D = N[:, None] + N[None, :] - 2 * (x @ x.T)
        w.threshold = float(np.quantile(D, 1 - quantile, method="nearest"))
    return w


@pytest.mark.parametrize("dtype,d", [("f16", 16), ("bf16", 64), ("f16", 128), ("bf16", 256),
                                     ("i8", 32), ("i8", 64), ("i8", 128), ("i8", 250)])
@pytest.mark.parametrize("metric", ["ip", "l2"])
def test_self_join_triangle_parity(dtype, d, metric):
    n = 1500 if d <= 128 else 1100
    w = self_case(31 + d, n, d, dtype, metric, 0.995)
    P = to_device(w.P, dtype)
    say("self", dtype, d, metric, n, w.threshold)
    g = sorted_pairs(gpu_join(metric, P, P, w.threshold))
    ref = oracle.join(metric, dtype, w.P, w.P, w.threshold)
    compare(g, ref, False)
    s = set(map(tuple, g.tolist()))
    assert all((i, i) in s for i in range(n)) or metric == "ip"
    assert all((j, i) in s for (i, j) in s)
    g2 = sorted_pairs(gpu_join(metric, P, P, w.threshold, two_pass=True))
    assert np.array_equal(keys(g2), keys(g))


def test_self_join_triangle_full_size_sampled_rows():
    """The 65536-row bf16 workload joined with itself in the benchmark's
    launch configuration; the oracle recomputes sampled rows."""
    w = workloads.make_config("ip_bf16_65536x128")
    P = to_device(w.P, w.dtype)
    say("self full", w.name)
    g = sorted_pairs(gpu_join("ip", P, P, w.threshold))
    rng = np.random.default_rng(77)
    rows = np.sort(rng.choice(w.n_p, size=24, replace=False))
    ref = oracle.join("ip", w.dtype, w.P, w.P, w.threshold, rows=rows)
    compare(g[np.isin(g[:, 0], rows)], ref, False)
    s = keys(g)
    mirrored = keys(g[:, ::-1].copy())
    assert np.array_equal(np.sort(mirrored), s)


@pytest.mark.parametrize("dtype,d,metric,n", [("bf16", 300, "ip", 700), ("f16", 600, "l2", 530),
                                              ("bf16", 1024, "ip", 600), ("i8", 600, "ip", 777),
                                              ("i8", 1024, "l2", 513)])
def test_self_join_triangle_streamed(dtype, d, metric, n):
    """Rows of more than 512 bytes take the K-streamed kernel: its single pass
    skips the 256 x 256 tiles below the diagonal and mirrors the pairs of the
    others; the set equals the oracle's and the two-pass mode's (ragged last
    tiles on both sides)."""
    w = self_case(51 + d, n, d, dtype, metric, 0.99)
    P = to_device(w.P, dtype)
    say("self streamed", dtype, d, metric, n, w.threshold)
    g = sorted_pairs(gpu_join(metric, P, P, w.threshold))
    ref = oracle.join(metric, dtype, w.P, w.P, w.threshold)
    compare(g, ref, False)
    s = set(map(tuple, g.tolist()))
    assert all((j, i) in s for (i, j) in s)
    g2 = sorted_pairs(gpu_join(metric, P, P, w.threshold, two_pass=True))
    assert np.array_equal(keys(g2), keys(g))


@pytest.mark.parametrize("dtype,d,n", [("i8", 64, 5000), ("bf16", 128, 4100), ("f16", 40, 2600)])
def test_self_join_triangle_block_pairing(dtype, d, n):
    """Several blocks of P rows (odd and even counts): the triangle's
    workgroups pair block pb with block n_pb - 1 - pb, and every pair is
    still found once per orientation."""
    w = self_case(61 + d, n, d, dtype, "ip", 0.998)
    P = to_device(w.P, dtype)
    say("self pairing", dtype, d, n, w.threshold)
    g = sorted_pairs(gpu_join("ip", P, P, w.threshold))
    ref = oracle.join("ip", dtype, w.P, w.P, w.threshold)
    compare(g, ref, False)
