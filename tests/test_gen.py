"""The seeded workload generators (CPU only)."""
import numpy as np
import pytest

import oracle
import workloads
from pins import values


def test_deterministic_per_seed():
    a = workloads.make_config("ip_f16_2048x64")
    b = workloads.make_config("ip_f16_2048x64")
    c = workloads.make_config("ip_f16_2048x64", seed=7)
    assert np.array_equal(a.P, b.P) and np.array_equal(a.Q, b.Q)
    assert np.array_equal(a.planted, b.planted)
    assert not np.array_equal(a.P, c.P)
    r1 = workloads.random_case(5, 10, 11, 7, "bf16")
    r2 = workloads.random_case(5, 10, 11, 7, "bf16")
    assert np.array_equal(r1.P, r2.P) and np.array_equal(r1.Q, r2.Q)


@pytest.mark.parametrize("k,n,lo,hi", [("ip_f16_2048x64", None, -8, 8),
                                       ("ip_bf16_65536x128", 2048, -4, 4),
                                       ("l2_i8_1048576x64", 4096, -15, 15),
                                       ("ip_bf16_clustered_131072x1024", 1024, -2, 2)])
def test_value_ranges_integer(k, n, lo, hi):
    w = workloads.make_config(k, n=n)
    for X in (w.P, w.Q):
        v = values(w.dtype, X)
        assert v.min() >= lo and v.max() <= hi
        assert np.all(v == np.round(v))
    assert not w.real_valued


def test_shapes_full_size_small_configs():
    for k in ("ip_f16_2048x64", "ip_bf16_65536x128"):
        w = workloads.make_config(k)
        cfg = workloads.CONFIGS[k]
        assert w.P.shape == (cfg["n"], cfg["d"]) and w.Q.shape == (cfg["n"], cfg["d"])
        assert w.planted.shape == (cfg["planted"], 2)
        assert len(set(w.planted[:, 0].tolist())) == cfg["planted"]
        assert len(set(w.planted[:, 1].tolist())) == cfg["planted"]


def test_cosine_rows_are_unit():
    w = workloads.make_config("cos_f16_262144x256", n=2048)
    for X in (w.P, w.Q):
        nrm = (X.astype(np.float64) ** 2).sum(1)
        # fp16 rounding of each coordinate moves ||x||^2 by at most ~2 * 2^-11 relative
        assert np.all(np.abs(nrm - 1.0) < 4e-3)
    assert w.real_valued


@pytest.mark.parametrize("k,n", [("ip_f16_2048x64", None), ("ip_bf16_65536x128", 4096),
                                 ("cos_f16_262144x256", 4096), ("l2_i8_1048576x64", 16384)])
def test_planted_pairs_match(k, n):
    w = workloads.make_config(k, n=n)
    sc = oracle.scores(w.metric, w.dtype, w.P, w.Q, w.planted)
    assert w.planted.shape[0] > 0
    if w.metric == "ip":
        assert np.all(sc >= w.threshold), sc.min()
        if w.real_valued:   # keep clear of the 1e-3 boundary band
            assert np.all(sc >= w.threshold * 1.001)
    else:
        assert np.all(sc <= w.threshold), sc.max()


def test_l2_ties_and_decoys():
    w = workloads.make_config("l2_i8_1048576x64", n=65536)
    sc = oracle.scores("l2", "i8", w.P, w.Q, w.planted)
    n_ties = int((sc == 2000).sum())
    assert n_ties == w.decoys.shape[0] > 0
    dec = oracle.scores("l2", "i8", w.P, w.Q, w.decoys)
    assert np.all(dec == 2001)


def _ip_pmf(a, d):
    """Exact distribution of <x, y> for independent x, y uniform on
    {-a..a}^d: the d-fold convolution of the product distribution."""
    vals = np.arange(-a, a + 1)
    prod = np.zeros(2 * a * a + 1)
    for u in vals:
        for v in vals:
            prod[u * v + a * a] += 1.0 / (2 * a + 1) ** 2
    pmf = np.array([1.0])
    for _ in range(d):
        pmf = np.convolve(pmf, prod)
    return pmf, -d * a * a      # pmf[t] = P(<x, y> = t + offset)


@pytest.mark.parametrize("k,n,a", [("ip_f16_2048x64", None, 8), ("ip_bf16_65536x128", 2048, 4)])
def test_background_count_matches_exact_pmf(k, n, a):
    """Background matches agree with n^2 * P(<x,y> >= s) from the exact PMF."""
    w = workloads.make_config(k, n=n)
    pmf, off = _ip_pmf(a, w.d)
    t = np.arange(pmf.size) + off
    p = pmf[t >= w.threshold].sum()
    expect = w.n_p * w.n_q * p
    S = values(w.dtype, w.P) @ values(w.dtype, w.Q).T
    got = int((S >= w.threshold).sum()) - w.planted.shape[0]
    # pairs sharing a row are correlated; allow 5 "independent" sigmas doubled
    tol = 10 * np.sqrt(expect) + 0.01 * expect
    assert abs(got - expect) <= tol, (got, expect)


def test_clustered_structure():
    w = workloads.make_config("ip_bf16_clustered_131072x1024", n=1024)
    S = values("bf16", w.P) @ values("bf16", w.Q).T
    same = w.labels_p[:, None] == w.labels_q[None, :]
    assert S[same].min() > 1000          # same-cluster pairs always match s = 125
    dens = (S >= w.threshold).mean()
    assert 0.02 < dens < 0.04            # about 3 % of pairs match (about 5e8 at full size)


def test_bf16_encoding_is_round_to_nearest_even():
    import torch
    x = np.random.default_rng(3).standard_normal(1 << 16).astype(np.float32)
    x[:4] = [np.inf, -np.inf, 0.0, -0.0]
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(workloads.bf16_bits_from_f32(x), ref)
