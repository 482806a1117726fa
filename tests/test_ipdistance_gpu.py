"""Section 4's ip-distances through the GPU's inner-product join.

Section 4 reduces every ip-distance D(x, y) to an inner product f(x).g(y) of
transformed points and then joins F_P against G_Q with one matrix product.
The library evaluates the squared L2 distance with the norm expansion
N_x + N_y - 2<x, y> (d' = d) and offers no separate Hamming entry (on {0,1}^d
Hamming is the squared L2 distance).  These tests run the paper's own
transforms through sj_join_ip instead -- D(x, y) <= r  <=>  f(x).(-g(y)) >= -r
-- and check that the pair sets agree exactly with sj_join_l2 and with the
oracle: the squared-L2 transform f = (x_k^2, 1, -2 x_k), g = (1, y_k^2, y_k)
(d' = 3 d, a cross-check of the norm epilogue) and the Hamming transform
f = (x_k, 1 - x_k), g = (1 - y_k, y_k) (d' = 2 d, on the int8 matrix cores).
The transforms are applied here, on the host, to integer inputs, so every
transformed value and every score is an exact integer.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads
from gpu_util import keys, sorted_pairs, to_device

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


def l2_fg(x, y):
    F = np.stack([x * x, np.ones_like(x), -2 * x], axis=2).reshape(x.shape[0], -1)
    G = np.stack([np.ones_like(y), y * y, y], axis=2).reshape(y.shape[0], -1)
    return F, G


def hamming_fg(x, y):
    F = np.stack([x, 1 - x], axis=2).reshape(x.shape[0], -1)
    G = np.stack([1 - y, y], axis=2).reshape(y.shape[0], -1)
    return F, G


@pytest.mark.parametrize("n_p,n_q,d,r2", [(300, 257, 24, 600.0), (129, 520, 40, 1100.0)])
def test_paper_l2_transform_through_ip_join(n_p, n_q, d, r2):
    """F_P (d' = 3d) against -G_Q with threshold -r2 on the bf16 inner-product
    kernel (every value is an integer below 2^8 in magnitude, so bf16 holds
    it and the fp32 sums are exact) gives the same pairs as the L2 join."""
    import paper_2006_12608_amd as sj
    rng = np.random.default_rng(5000 + d)
    x = rng.integers(-7, 8, size=(n_p, d))
    y = rng.integers(-7, 8, size=(n_q, d))
    y[:30] = x[:30] + rng.integers(-2, 3, size=(30, d))
    P, Q = workloads.encode(x, "i8"), workloads.encode(y, "i8")
    F, G = l2_fg(x, y)
    say("l2 via f.g", n_p, n_q, d, r2)
    got_fg = sorted_pairs(sj.join_ip(to_device(workloads.encode(F, "bf16"), "bf16"),
                                     to_device(workloads.encode(-G, "bf16"), "bf16"), -r2))
    got_l2 = sorted_pairs(sj.join_l2(to_device(P, "i8"), to_device(Q, "i8"), r2))
    ref = oracle.join("l2", "i8", P, Q, r2)
    assert ref.total > 30
    assert np.array_equal(keys(got_fg), keys(ref.pairs))
    assert np.array_equal(keys(got_l2), keys(ref.pairs))


@pytest.mark.parametrize("n_p,n_q,d,r", [(400, 333, 48, 14.0), (97, 1030, 100, 38.0)])
def test_paper_hamming_transform_through_ip_join(n_p, n_q, d, r):
    """Hamming distance on {0,1}^d: F_P (d' = 2d) against -G_Q with threshold
    -r on the int8 inner-product kernel, the same set from sj_join_l2 on the
    bit vectors themselves (squared L2 = Hamming on {0,1}), and the oracle."""
    import paper_2006_12608_amd as sj
    rng = np.random.default_rng(6000 + d)
    x = rng.integers(0, 2, size=(n_p, d))
    y = rng.integers(0, 2, size=(n_q, d))
    flip = rng.random((40, d)) < 0.1
    y[:40] = np.where(flip, 1 - x[:40], x[:40])
    F, G = hamming_fg(x, y)
    P, Q = workloads.encode(x, "i8"), workloads.encode(y, "i8")
    say("hamming via f.g", n_p, n_q, d, r)
    got_fg = sorted_pairs(sj.join_ip(to_device(workloads.encode(F, "i8"), "i8"),
                                     to_device(workloads.encode(-G, "i8"), "i8"), -r))
    got_l2 = sorted_pairs(sj.join_l2(to_device(P, "i8"), to_device(Q, "i8"), r))
    ref = oracle.join("l2", "i8", P, Q, r)
    assert ref.total > 40
    ham = (x[:, None, :] != y[None, :, :]).sum(-1)
    want = np.argwhere(ham <= r)
    assert np.array_equal(keys(ref.pairs), keys(want))
    assert np.array_equal(keys(got_fg), keys(ref.pairs))
    assert np.array_equal(keys(got_l2), keys(ref.pairs))
