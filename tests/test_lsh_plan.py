"""Section 4's LSH parameter choice (sj_lsh_plan) and the families' collision
probabilities (sj_lsh_collision), host-only functions of the library, on the
CPU.  The collision probability of the quantised family is checked against a
numerical integration of its definition (scipy), the sign family against the
angle law at its fixed points; the plan against the inequalities that define
k, L and the number of instances, and against the exact miss probability of
the resulting scheme."""
import math

import numpy as np
import pytest


@pytest.fixture(scope="module")
def sj():
    import paper_2006_12608_amd as sj
    return sj


def test_sign_collision(sj):
    assert sj.sj_lsh_collision(0, 1.0, 0.0) == 1.0
    assert sj.sj_lsh_collision(0, 1.0, math.pi) == 0.0
    assert abs(sj.sj_lsh_collision(0, 1.0, math.pi / 2) - 0.5) < 1e-15
    theta = math.acos(0.9)
    assert abs(sj.sj_lsh_collision(0, 1.0, theta) - (1 - theta / math.pi)) < 1e-15
    assert math.isnan(sj.sj_lsh_collision(0, 1.0, 4.0))
    assert math.isnan(sj.sj_lsh_collision(-1, 1.0, 1.0))


@pytest.mark.parametrize("w,sigma,dist", [(2000, 32.0, math.sqrt(2000)), (2000, 32.0, 101.2),
                                          (5, 1.0, 0.3), (300, 7.0, 80.0), (1, 2.0, 40.0)])
def test_quantised_collision_against_integration(sj, w, sigma, dist):
    """floor((<a,x> + b) / w): the projections of the two points differ by
    u Z (u = sigma dist, Z standard normal) and, for an offset b uniform in
    [0, w), land in one bucket with probability max(0, 1 - u |Z| / w):
    integrated numerically over Z."""
    from scipy import integrate
    u = sigma * dist
    dens = lambda z: 2.0 * math.exp(-z * z / 2) / math.sqrt(2 * math.pi)   # |Z|
    want, _ = integrate.quad(lambda z: dens(z) * max(0.0, 1.0 - u * z / w), 0.0, w / u,
                             epsabs=1e-13, epsrel=1e-12)
    got = sj.sj_lsh_collision(w, sigma, dist)
    assert abs(got - want) < 1e-10, (got, want)
    assert sj.sj_lsh_collision(w, sigma, 0.0) == 1.0
    # monotone: farther points collide less often
    assert sj.sj_lsh_collision(w, sigma, dist * 1.5) < got


@pytest.mark.parametrize("p1,p2,n,tile,recall", [(0.8564, 0.5, 262144, 128, 0.99),
                                                 (0.48, 0.24, 1 << 20, 128, 0.9),
                                                 (0.9, 0.3, 100, 128, 0.5),
                                                 (0.7, 0.65, 50000, 64, 0.999)])
def test_plan_defining_inequalities(sj, p1, p2, n, tile, recall):
    st, k, L, R = sj.sj_lsh_plan(p1, p2, n, tile, recall)
    assert st == sj.SJ_OK, sj.sj_last_error()
    # k: the least integer with p2^k <= tile / n
    assert p2 ** k <= tile / n * (1 + 1e-12)
    assert k == 0 or p2 ** (k - 1) > tile / n
    # L: the least number of tables with L p1^k >= 1
    q = p1 ** k
    assert L * q >= 1 - 1e-9 and (L - 1) * q < 1
    # R: the least number of instances with e^-R <= 1 - recall
    assert math.exp(-R) <= 1 - recall + 1e-12
    assert R == 1 or math.exp(-(R - 1)) > 1 - recall
    # the merged scheme misses a pair at the threshold with probability
    # (1 - p1^k)^(L R) <= 1 - recall
    assert (1 - q) ** (L * R) <= 1 - recall + 1e-12


def test_plan_errors(sj):
    assert sj.sj_lsh_plan(0.5, 0.6, 1000, 128, 0.9)[0] == sj.SJ_E_INVAL   # p2 >= p1
    assert sj.sj_lsh_plan(1.0, 0.5, 1000, 128, 0.9)[0] == sj.SJ_E_INVAL
    assert sj.sj_lsh_plan(0.9, 0.5, 1000, 128, 1.0)[0] == sj.SJ_E_INVAL
    assert sj.sj_lsh_plan(0.9, 0.5, 0, 128, 0.9)[0] == sj.SJ_E_INVAL
    assert sj.sj_lsh_plan(0.9, 0.999, 1 << 40, 1, 0.9)[0] in (sj.SJ_E_INVAL, sj.SJ_E_UNSUPPORTED)
