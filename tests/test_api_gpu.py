"""Error handling of the C-ABI on a GPU: bad arguments are rejected with a
status, never a fault (the library checks pointers and buffer sizes against
their allocations before any launch)."""
import ctypes
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


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


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def test_host_pointer_is_rejected(env):
    sj, ctx, torch = env
    say("host pointer")
    host = np.zeros((64, 16), np.float16)
    Q = torch.zeros((64, 16), dtype=torch.float16, device="cuda")
    out = torch.empty((10, 2), dtype=torch.int32, device="cuda")
    st, n = sj.sj_join_ip(ctx, sj.SJ_F16, host.ctypes.data, 64, Q.data_ptr(), 64, 16, 0.0,
                          out.data_ptr(), 10)
    assert st == sj.SJ_E_INVAL, sj.sj_last_error()


def _range_query_works(ptr) -> bool:
    """The library bounds-checks buffers with hipMemGetAddressRange; only ask it
    to reject an oversized request when that query works for this allocation
    (otherwise the request would reach a kernel and read out of bounds)."""
    try:
        hip = ctypes.CDLL("libamdhip64.so")
    except OSError:
        return False
    base, size = ctypes.c_void_p(), ctypes.c_size_t()
    ok = hip.hipMemGetAddressRange(ctypes.byref(base), ctypes.byref(size), ctypes.c_void_p(ptr))
    return ok == 0 and base.value is not None and size.value > 0


def test_undersized_buffers_are_rejected(env):
    sj, ctx, torch = env
    say("undersized")
    P = torch.zeros((64, 16), dtype=torch.float16, device="cuda")
    out = torch.empty((10, 2), dtype=torch.int32, device="cuda")
    if not (_range_query_works(P.data_ptr()) and _range_query_works(out.data_ptr())):
        pytest.skip("hipMemGetAddressRange does not describe torch's allocations here")
    # claims more rows than P holds (the allocation is rounded up, so ask for far more)
    st, _ = sj.sj_join_ip(ctx, sj.SJ_F16, P.data_ptr(), 1 << 26, P.data_ptr(), 64, 16, 0.0,
                          out.data_ptr(), 10)
    assert st == sj.SJ_E_INVAL, sj.sj_last_error()
    st, _ = sj.sj_join_ip(ctx, sj.SJ_F16, P.data_ptr(), 64, P.data_ptr(), 64, 16, 0.0,
                          out.data_ptr(), 1 << 30)
    assert st == sj.SJ_E_INVAL, sj.sj_last_error()


def test_bad_values_are_rejected(env):
    sj, ctx, torch = env
    say("bad values")
    P = torch.zeros((8, 16), dtype=torch.int8, device="cuda")
    out = torch.empty((64, 2), dtype=torch.int32, device="cuda")
    st, _ = sj.sj_join_ip(ctx, sj.SJ_I8, P.data_ptr(), 8, P.data_ptr(), 8, 16, float("nan"),
                          out.data_ptr(), 64)
    assert st == sj.SJ_E_INVAL
    st, _ = sj.sj_join_ip(ctx, 9, P.data_ptr(), 8, P.data_ptr(), 8, 16, 0.0, out.data_ptr(), 64)
    assert st == sj.SJ_E_INVAL
    st, _ = sj.sj_count(ctx, 7, sj.SJ_I8, P.data_ptr(), 8, P.data_ptr(), 8, 16, 0.0)
    assert st == sj.SJ_E_INVAL
    big = torch.zeros((1, 40000), dtype=torch.int8, device="cuda")
    st, _ = sj.sj_join_ip(ctx, sj.SJ_I8, big.data_ptr(), 1, big.data_ptr(), 1, 40000, 0.0,
                          out.data_ptr(), 64)
    assert st == sj.SJ_E_UNSUPPORTED
    # flags a function does not take: unknown bits, and the cosine front end on L2
    st, _ = sj.sj_join_ip(ctx, sj.SJ_I8, P.data_ptr(), 8, P.data_ptr(), 8, 16, 0.0,
                          out.data_ptr(), 64, 16)
    assert st == sj.SJ_E_INVAL, sj.sj_last_error()
    st, _ = sj.sj_join_l2(ctx, sj.SJ_I8, P.data_ptr(), 8, P.data_ptr(), 8, 16, 0.0,
                          out.data_ptr(), 64, sj.SJ_FLAG_COSINE)
    assert st == sj.SJ_E_INVAL, sj.sj_last_error()
    n = ctypes.c_uint64(0)
    assert sj.lib.sj_join_ip(ctx, sj.SJ_I8, P.data_ptr(), 8, P.data_ptr(), 8, 16, 0.0,
                             out.data_ptr(), 64, None, 0) == sj.SJ_E_INVAL
    assert n.value == 0
    # the context still works after the failures
    st, n = sj.sj_join_ip(ctx, sj.SJ_I8, P.data_ptr(), 8, P.data_ptr(), 8, 16, 0.0,
                          out.data_ptr(), 64)
    assert st == sj.SJ_OK and n == 64


def test_stats_and_timing(env):
    sj, ctx, torch = env
    say("stats")
    P = torch.randint(-3, 4, (600, 64), dtype=torch.int8, device="cuda")
    out = torch.empty((600 * 600, 2), dtype=torch.int32, device="cuda")
    st, n = sj.sj_join_l2(ctx, sj.SJ_I8, P.data_ptr(), 600, P.data_ptr(), 600, 64, 300.0,
                          out.data_ptr(), 600 * 600, sj.SJ_FLAG_TIMING)
    assert st == sj.SJ_OK
    s = sj.sj_get_stats(ctx)
    assert s.total == n and s.timed == 1 and s.kernel == 1
    assert s.ms_join > 0 and s.ms_norms > 0
    st, n2 = sj.sj_join_l2(ctx, sj.SJ_I8, P.data_ptr(), 600, P.data_ptr(), 600, 64, 300.0,
                           out.data_ptr(), 600 * 600, sj.SJ_FLAG_TIMING | sj.SJ_FLAG_TWO_PASS)
    s = sj.sj_get_stats(ctx)
    assert n2 == n and s.ms_count > 0 and s.ms_emit > 0


def test_two_contexts_two_streams(env):
    sj, _, torch = env
    say("two streams")
    s1 = torch.cuda.Stream()
    P = torch.randint(-4, 5, (500, 32), dtype=torch.int8, device="cuda")
    ref = sj.count(P, P, 20.0)
    with torch.cuda.stream(s1):
        c = sj.count(P, P, 20.0)
    assert c == ref


def test_python_default_is_count_then_emit(env):
    """join_ip / join_l2 without a capacity size the output with sj_count and
    fill it by count-then-emit: the order is deterministic and equals an
    explicit two-pass call's; with two_pass=False the same set comes from the
    single pass."""
    sj, ctx, torch = env
    say("python default")
    P = torch.randint(-4, 5, (700, 64), dtype=torch.int8, device="cuda")
    Q = torch.randint(-4, 5, (650, 64), dtype=torch.int8, device="cuda")
    for f, thr in ((sj.join_ip, 40.0), (sj.join_l2, 700.0)):
        a = f(P, Q, thr, ctx=ctx)
        b = f(P, Q, thr, ctx=ctx)
        assert a.shape[0] > 0 and torch.equal(a, b)
        c = f(P, Q, thr, cap=a.shape[0], two_pass=True, ctx=ctx)
        assert torch.equal(a, c)
        d = f(P, Q, thr, two_pass=False, ctx=ctx)
        ka = (a[:, 0].long() << 32 | a[:, 1].long()).sort().values
        kd = (d[:, 0].long() << 32 | d[:, 1].long()).sort().values
        assert torch.equal(ka, kd)


def test_zero_dimension_reading(env):
    """d = 0: points of R^0 all coincide (every score is 0): every pair for
    s <= 0 or r2 >= 0, none otherwise, in both modes and through sj_count."""
    sj, ctx, torch = env
    say("d = 0")
    P0 = torch.zeros((7, 0), dtype=torch.bfloat16, device="cuda")
    Q0 = torch.zeros((9, 0), dtype=torch.bfloat16, device="cuda")
    for two_pass in (False, True):
        assert sj.join_ip(P0, Q0, 0.0, two_pass=two_pass, ctx=ctx).shape[0] == 63
        assert sj.join_ip(P0, Q0, 1e-30, two_pass=two_pass, ctx=ctx).shape[0] == 0
        assert sj.join_l2(P0, Q0, 0.0, two_pass=two_pass, ctx=ctx).shape[0] == 63
        assert sj.join_l2(P0, Q0, -1e-30, two_pass=two_pass, ctx=ctx).shape[0] == 0
    assert sj.count(P0, Q0, -5.0, "ip", ctx=ctx) == 63
    assert sj.count(P0, Q0, 3.0, "l2", ctx=ctx) == 63


def test_unknown_metric_is_rejected(env):
    sj, ctx, torch = env
    say("unknown metric")
    P = torch.zeros((8, 16), dtype=torch.int8, device="cuda")
    with pytest.raises(ValueError, match="metric"):
        sj.count(P, P, 0.0, "cos", ctx)
    A = torch.zeros((2, 16), dtype=torch.int8, device="cuda")
    with pytest.raises(ValueError, match="metric"):
        sj.join_lsh(P, P, 0.0, "L2", L=1, k=2, A=A, ctx=ctx)
