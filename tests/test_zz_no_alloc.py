"""sj_join_noalloc (the join that allocates nothing: its device scratch is a
fixed region of the library) against the allocating entry points sj_join_l2 /
sj_join_ip, through the C-ABI: the same pair sets (integer inputs: exact), the
same arrays in count-then-emit order, two calls in a row with the second on a
smaller input (the region keeps the last call's contents, so its counters must
be cleared by each call), overflow, and a request too large for the region."""
import sys

import numpy as np
import pytest

import workloads
from gpu_util import sorted_pairs, to_device

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2006_12608_amd as sj
    ctx = sj.sj_create(0, int(torch.cuda.current_stream().cuda_stream))
    yield sj, ctx, torch
    torch.cuda.synchronize()
    sj.sj_destroy(ctx)


def _both(sj, ctx, torch, metric, dtype, Pd, n_p, Qd, n_q, d, thr, flags):
    """(allocating result, no-allocation result) as (n, 2) int32 tensors."""
    m = sj.SJ_IP if metric == "ip" else sj.SJ_L2
    dt = {"f16": sj.SJ_F16, "bf16": sj.SJ_BF16, "i8": sj.SJ_I8}[dtype]
    fn = sj.sj_join_ip if metric == "ip" else sj.sj_join_l2
    st, total = sj.sj_count(ctx, m, dt, Pd.data_ptr(), n_p, Qd.data_ptr(), n_q, d, thr)
    assert st == sj.SJ_OK, sj.sj_last_error()
    cap = max(total, 1)
    a = torch.full((cap, 2), -1, dtype=torch.int32, device="cuda")
    b = torch.full((cap, 2), -1, dtype=torch.int32, device="cuda")
    st, na = fn(ctx, dt, Pd.data_ptr(), n_p, Qd.data_ptr(), n_q, d, thr, a.data_ptr(), cap, flags)
    assert st == sj.SJ_OK, sj.sj_last_error()
    st, nb = sj.sj_join_noalloc(ctx, m, dt, Pd.data_ptr(), n_p, Qd.data_ptr(), n_q, d, thr,
                                b.data_ptr(), cap, flags)
    assert st == sj.SJ_OK, sj.sj_last_error()
    assert na == nb == total
    return a[:na], b[:nb]


@pytest.mark.parametrize("metric,dtype,d,big,small", [
    ("l2", "i8", 64, (3000, 2500), (700, 300)),      # row norms in the fixed region
    ("ip", "bf16", 100, (2100, 1900), (500, 70)),    # 200-byte rows: repacked there
    ("ip", "f16", 600, (900, 1100), (257, 130)),     # the K-streamed kernel
])
def test_noalloc_equals_allocating(env, metric, dtype, d, big, small):
    sj, ctx, torch = env
    from pins import values
    for (n_p, n_q), seed in ((big, 1), (small, 2)):
        w = workloads.random_case(300 + seed + d, n_p, n_q, d, dtype, lo=-3, hi=3)
        x = values(dtype, w.P).astype(np.int64)
        y = values(dtype, w.Q).astype(np.int64)
        if metric == "ip":
            thr = float(np.quantile(x @ y.T, 0.97, method="nearest"))
        else:
            d2 = (x * x).sum(1)[:, None] + (y * y).sum(1)[None, :] - 2 * (x @ y.T)
            thr = float(np.quantile(d2, 0.03, method="nearest"))
        Pd, Qd = to_device(w.P, dtype), to_device(w.Q, dtype)
        say("noalloc", metric, dtype, d, n_p, n_q, thr)
        a, b = _both(sj, ctx, torch, metric, dtype, Pd, n_p, Qd, n_q, d, thr, 0)
        assert a.shape[0] > 0
        assert np.array_equal(sorted_pairs(a), sorted_pairs(b))
        # count-then-emit: the same array, element by element (deterministic order)
        a2, b2 = _both(sj, ctx, torch, metric, dtype, Pd, n_p, Qd, n_q, d, thr,
                       sj.SJ_FLAG_TWO_PASS | sj.SJ_FLAG_RECOMPUTE)
        assert torch.equal(a2, b2)
        assert np.array_equal(sorted_pairs(a2), sorted_pairs(a))


def test_noalloc_self_join_and_overflow(env):
    sj, ctx, torch = env
    w = workloads.random_case(311, 1500, 1500, 64, "i8", lo=-4, hi=4)
    Pd = to_device(w.P, "i8")
    say("noalloc self-join / overflow")
    a, b = _both(sj, ctx, torch, "l2", "i8", Pd, 1500, Pd, 1500, 64, 500.0, 0)
    assert np.array_equal(sorted_pairs(a), sorted_pairs(b))
    total = a.shape[0]
    out = torch.empty((total, 2), dtype=torch.int32, device="cuda")
    st, n = sj.sj_join_noalloc(ctx, sj.SJ_L2, sj.SJ_I8, Pd.data_ptr(), 1500, Pd.data_ptr(), 1500,
                               64, 500.0, out.data_ptr(), total - 1, 0)
    assert st == sj.SJ_E_OVERFLOW and n == total


def test_noalloc_rejects_what_does_not_fit(env):
    """Row norms of 5 Mi rows need 20 MiB, more than the fixed region holds: an
    error before any launch, and the next call works."""
    sj, ctx, torch = env
    say("noalloc too large")
    n = 5 << 20
    P = torch.zeros((n // 2, 16), dtype=torch.int8, device="cuda")
    Q = torch.zeros((n - n // 2, 16), dtype=torch.int8, device="cuda")
    out = torch.empty((16, 2), dtype=torch.int32, device="cuda")
    st, _ = sj.sj_join_noalloc(ctx, sj.SJ_L2, sj.SJ_I8, P.data_ptr(), P.shape[0], Q.data_ptr(),
                               Q.shape[0], 16, 0.0, out.data_ptr(), 16, 0)
    assert st == sj.SJ_E_UNSUPPORTED
    assert "fixed scratch" in sj.sj_last_error()
    st, _ = sj.sj_join_noalloc(ctx, sj.SJ_L2, sj.SJ_I8, P.data_ptr(), 4, Q.data_ptr(), 4, 16,
                               0.0, out.data_ptr(), 16, sj.SJ_FLAG_TWO_PASS)
    assert st == sj.SJ_OK
    assert sj.sj_join_noalloc(None, 0, 1, None, 0, None, 0, 0, 0.0, None, 0)[0] == sj.SJ_E_INVAL
