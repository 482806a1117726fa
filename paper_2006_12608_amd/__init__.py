"""MI355X-native similarity join (Ahle & Silvestri, "Similarity Search with
Tensor Core Units", Section 4, brute-force method): Python binding of libsj.so.

The raw C-ABI entry points are exposed under their C names (sj_create,
sj_join_ip, sj_join_l2, sj_count, sj_join_noalloc, sj_normalize,
sj_join_hamming, sj_join_lsh, sj_lsh_sort, sj_lsh_collision, sj_lsh_plan, sj_jl, sj_destroy,
sj_get_stats, sj_last_error) with plain integer pointers; `join_ip`, `join_l2`, `count` and
`join_lsh` (the LSH-bucketed join of Theorem 3) are conveniences over PyTorch
device tensors.  This module only marshals
arguments: every step of the join runs in the library's HIP kernels.  Import
fails when libsj.so has not been built (python paper_2006_12608_amd/build.py).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsj.so")

SJ_F16, SJ_BF16, SJ_I8 = 1, 2, 3
SJ_IP, SJ_L2 = 0, 1
SJ_OK, SJ_E_INVAL, SJ_E_OVERFLOW, SJ_E_NOMEM, SJ_E_HIP, SJ_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
SJ_FLAG_TWO_PASS, SJ_FLAG_TIMING, SJ_FLAG_RECOMPUTE, SJ_FLAG_COSINE = 1, 2, 4, 8

STATUS_NAMES = {0: "SJ_OK", -1: "SJ_E_INVAL", -2: "SJ_E_OVERFLOW", -3: "SJ_E_NOMEM",
                -4: "SJ_E_HIP", -5: "SJ_E_UNSUPPORTED"}


class SjError(RuntimeError):
    def __init__(self, status: int, message: str, n_out: int | None = None):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.n_out = n_out


class sj_stats(ctypes.Structure):
    _fields_ = [("total", ctypes.c_uint64), ("ms_norms", ctypes.c_double),
                ("ms_join", ctypes.c_double), ("ms_count", ctypes.c_double),
                ("ms_scan", ctypes.c_double), ("ms_emit", ctypes.c_double),
                ("kernel", ctypes.c_uint32), ("timed", ctypes.c_uint32),
                ("emit_from_bits", ctypes.c_uint32), ("lsh_rows", ctypes.c_uint64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python paper_2006_12608_amd/build.py` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, u32, u64, dbl, i32 = (ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_double,
                              ctypes.c_int)
    lib.sj_create.argtypes = [ctypes.POINTER(vp), i32, vp]
    lib.sj_create.restype = i32
    join_args = [vp, i32, vp, u32, vp, u32, u32, dbl, vp, u64, ctypes.POINTER(u64), ctypes.c_uint]
    lib.sj_join_ip.argtypes = join_args
    lib.sj_join_ip.restype = i32
    lib.sj_join_l2.argtypes = join_args
    lib.sj_join_l2.restype = i32
    lib.sj_count.argtypes = [vp, i32, i32, vp, u32, vp, u32, u32, dbl, ctypes.POINTER(u64)]
    lib.sj_count.restype = i32
    lib.sj_join_noalloc.argtypes = [vp, i32, i32, vp, u32, vp, u32, u32, dbl, vp, u64,
                                    ctypes.POINTER(u64), ctypes.c_uint]
    lib.sj_join_noalloc.restype = i32
    lib.sj_normalize.argtypes = [vp, i32, vp, u32, u32, vp]
    lib.sj_normalize.restype = i32
    lib.sj_join_hamming.argtypes = [vp, vp, u32, vp, u32, u32, dbl, vp, u64,
                                    ctypes.POINTER(u64), ctypes.c_uint]
    lib.sj_join_hamming.restype = i32
    lib.sj_join_lsh.argtypes = [vp, i32, i32, vp, u32, vp, u32, u32, dbl, u32, u32, vp, vp,
                                ctypes.c_int32, vp, u64, ctypes.POINTER(u64),
                                ctypes.POINTER(u64)]
    lib.sj_join_lsh.restype = i32
    lib.sj_lsh_sort.argtypes = [vp, vp, u32, u32, u32, vp]
    lib.sj_lsh_sort.restype = i32
    lib.sj_lsh_collision.argtypes = [ctypes.c_int32, dbl, dbl]
    lib.sj_lsh_collision.restype = dbl
    lib.sj_lsh_plan.argtypes = [dbl, dbl, u64, u32, dbl, ctypes.POINTER(u32), ctypes.POINTER(u32),
                                ctypes.POINTER(u32)]
    lib.sj_lsh_plan.restype = i32
    lib.sj_jl.argtypes = [vp, i32, vp, u32, u32, u32, vp, vp, vp]
    lib.sj_jl.restype = i32
    lib.sj_destroy.argtypes = [vp]
    lib.sj_destroy.restype = None
    lib.sj_get_stats.argtypes = [vp, ctypes.POINTER(sj_stats)]
    lib.sj_get_stats.restype = i32
    lib.sj_last_error.argtypes = []
    lib.sj_last_error.restype = ctypes.c_char_p
    return lib


lib = _load()


# ------------------------------------------------------------ raw C-ABI names

def sj_last_error() -> str:
    return lib.sj_last_error().decode()


def sj_create(device: int = 0, stream: int | None = None) -> int:
    """Returns an opaque context handle (int)."""
    h = ctypes.c_void_p()
    st = lib.sj_create(ctypes.byref(h), device, stream or None)
    if st != SJ_OK:
        raise SjError(st, sj_last_error())
    return h.value


def sj_destroy(ctx: int | None) -> None:
    lib.sj_destroy(ctx)


def _join_raw(fn, ctx, dtype, P, n_p, Q, n_q, d, thr, pairs, cap, flags):
    n = ctypes.c_uint64(0)
    st = fn(ctx, dtype, P, n_p, Q, n_q, d, float(thr), pairs, cap, ctypes.byref(n), flags)
    return st, n.value


def sj_join_ip(ctx, dtype, P, n_p, Q, n_q, d, s, pairs, cap, flags=0):
    """Returns (status, n_out); pointers are integers (device addresses)."""
    return _join_raw(lib.sj_join_ip, ctx, dtype, P, n_p, Q, n_q, d, s, pairs, cap, flags)


def sj_join_l2(ctx, dtype, P, n_p, Q, n_q, d, r2, pairs, cap, flags=0):
    """Returns (status, n_out); pointers are integers (device addresses)."""
    return _join_raw(lib.sj_join_l2, ctx, dtype, P, n_p, Q, n_q, d, r2, pairs, cap, flags)


def sj_join_noalloc(ctx, metric, dtype, P, n_p, Q, n_q, d, thr, pairs, cap, flags=0):
    """The join without device allocation (fixed library scratch); returns
    (status, n_out); pointers are integers (device addresses)."""
    n = ctypes.c_uint64(0)
    st = lib.sj_join_noalloc(ctx, metric, dtype, P, n_p, Q, n_q, d, float(thr), pairs, cap,
                             ctypes.byref(n), flags)
    return st, n.value


def sj_normalize(ctx, dtype, X, n, d, Y):
    """Returns the status; pointers are integers (device addresses)."""
    return lib.sj_normalize(ctx, dtype, X, n, d, Y)


def sj_join_hamming(ctx, P, n_p, Q, n_q, d, r, pairs, cap, flags=0):
    """Returns (status, n_out); P and Q are device bit rows (ceil(d / 8) bytes)."""
    n = ctypes.c_uint64(0)
    st = lib.sj_join_hamming(ctx, P, n_p, Q, n_q, d, float(r), pairs, cap, ctypes.byref(n),
                             flags)
    return st, n.value


def sj_count(ctx, metric, dtype, P, n_p, Q, n_q, d, threshold):
    """Returns (status, count)."""
    n = ctypes.c_uint64(0)
    st = lib.sj_count(ctx, metric, dtype, P, n_p, Q, n_q, d, float(threshold), ctypes.byref(n))
    return st, n.value


def sj_join_lsh(ctx, metric, dtype, P, n_p, Q, n_q, d, thr, L, k, A, B, w, pairs, cap):
    """Returns (status, n_out, n_cand); pointers are integers (device addresses)."""
    n = ctypes.c_uint64(0)
    nc = ctypes.c_uint64(0)
    st = lib.sj_join_lsh(ctx, metric, dtype, P, n_p, Q, n_q, d, float(thr), L, k, A, B, int(w),
                         pairs, cap, ctypes.byref(n), ctypes.byref(nc))
    return st, n.value, nc.value


def sj_lsh_sort(ctx, keys, n, L, bits, perm) -> int:
    return lib.sj_lsh_sort(ctx, keys, n, L, bits, perm)


def sj_lsh_collision(w: int, sigma: float, dist: float) -> float:
    return lib.sj_lsh_collision(int(w), float(sigma), float(dist))


def sj_lsh_plan(p1: float, p2: float, n: int, tile: int, recall: float):
    """Returns (status, k, L_inst, reps)."""
    k, L, r = ctypes.c_uint32(), ctypes.c_uint32(), ctypes.c_uint32()
    st = lib.sj_lsh_plan(float(p1), float(p2), int(n), int(tile), float(recall), ctypes.byref(k),
                         ctypes.byref(L), ctypes.byref(r))
    return st, k.value, L.value, r.value


def sj_jl(ctx, dtype, X, n, d, levels, shape, A, Y):
    """Returns the status; shape is a sequence of (k_i, c_i, r_i), pointers
    are integers (device addresses)."""
    flat = [int(v) for s in shape for v in s]
    arr = (ctypes.c_uint32 * max(len(flat), 1))(*flat)
    return lib.sj_jl(ctx, dtype, X, n, d, levels, arr, A, Y)


def sj_get_stats(ctx) -> sj_stats:
    out = sj_stats()
    st = lib.sj_get_stats(ctx, ctypes.byref(out))
    if st != SJ_OK:
        raise SjError(st, sj_last_error())
    return out


# ------------------------------------------------------ torch conveniences

_contexts: dict = {}


def context(device: int | None = None, stream=None) -> int:
    """A cached context bound to (device, stream); defaults to torch's
    current device and stream."""
    import torch
    dev = torch.cuda.current_device() if device is None else int(device)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    handle = int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream or 0)
    key = (dev, handle)
    if key not in _contexts:
        _contexts[key] = sj_create(dev, handle)
    return _contexts[key]


def dtype_code(t) -> int:
    import torch
    codes = {torch.float16: SJ_F16, torch.bfloat16: SJ_BF16, torch.int8: SJ_I8}
    if t.dtype not in codes:
        raise TypeError(f"unsupported dtype {t.dtype}; use float16, bfloat16 or int8")
    return codes[t.dtype]


def _metric_code(metric: str) -> int:
    if metric not in ("ip", "l2"):
        raise ValueError(f"metric must be 'ip' or 'l2', not {metric!r}")
    return SJ_IP if metric == "ip" else SJ_L2


def _check_pair(P, Q):
    if P.dim() != 2 or Q.dim() != 2 or P.shape[1] != Q.shape[1]:
        raise ValueError("P and Q must be 2-D with the same number of columns")
    if P.dtype != Q.dtype:
        raise ValueError("P and Q must have the same dtype")
    if not (P.is_cuda and Q.is_cuda):
        raise ValueError("P and Q must be device tensors")
    if not (P.is_contiguous() and Q.is_contiguous()):
        raise ValueError("P and Q must be contiguous")


def count(P, Q, threshold: float, metric: str = "ip", ctx=None) -> int:
    """Number of matching pairs (sj_count)."""
    _check_pair(P, Q)
    m = _metric_code(metric)
    ctx = ctx or context(P.device.index)
    st, n = sj_count(ctx, m, dtype_code(P), P.data_ptr(), P.shape[0], Q.data_ptr(), Q.shape[0],
                     P.shape[1], threshold)
    if st != SJ_OK:
        raise SjError(st, sj_last_error())
    return n


def _sized_call(call, flags, cap, out, device):
    """Runs call(pairs_ptr, cap, flags) -> (status, n); with neither a
    capacity nor an output buffer, a first count-then-emit call with no room
    sizes the output (it stops after the count) and a second one fills it."""
    import torch
    if cap is None and out is None:
        st, n = call(None, 0, flags | SJ_FLAG_TWO_PASS)
        if st not in (SJ_OK, SJ_E_OVERFLOW):
            raise SjError(st, sj_last_error(), n)
        cap = n
    if out is None:
        out = torch.empty((max(int(cap), 1), 2), dtype=torch.int32, device=device)
        cap = int(cap)
    else:
        cap = out.shape[0] if cap is None else int(cap)
    st, n = call(out.data_ptr() if cap else None, cap, flags)
    if st != SJ_OK:
        raise SjError(st, sj_last_error(), n)
    return out[:n]


def _join(metric, P, Q, thr, cap, two_pass, timing, ctx, out, recompute=False, cosine=False):
    import torch
    _check_pair(P, Q)
    ctx = ctx or context(P.device.index)
    if two_pass is None:
        # no capacity given: count-then-emit sizes the output exactly
        two_pass = cap is None and out is None
    flags = ((SJ_FLAG_TWO_PASS if two_pass else 0) | (SJ_FLAG_TIMING if timing else 0)
             | (SJ_FLAG_RECOMPUTE if recompute else 0) | (SJ_FLAG_COSINE if cosine else 0))
    if cosine:
        def call(ptr, c, f):
            return sj_join_ip(ctx, dtype_code(P), P.data_ptr(), P.shape[0], Q.data_ptr(),
                              Q.shape[0], P.shape[1], thr, ptr, c, f)
        return _sized_call(call, flags, cap, out, P.device)
    if cap is None and out is None:
        cap = count(P, Q, thr, metric, ctx)
    if out is None:
        out = torch.empty((max(int(cap), 1), 2), dtype=torch.int32, device=P.device)
        cap = int(cap)
    else:
        cap = out.shape[0] if cap is None else int(cap)
    fn = sj_join_ip if metric == "ip" else sj_join_l2
    st, n = fn(ctx, dtype_code(P), P.data_ptr(), P.shape[0], Q.data_ptr(), Q.shape[0], P.shape[1],
               thr, out.data_ptr() if cap else None, cap, flags)
    if st != SJ_OK:
        raise SjError(st, sj_last_error(), n)
    return out[:n]


def join_ip(P, Q, s: float, cap: int | None = None, two_pass: bool | None = None,
            timing: bool = False, ctx=None, out=None, recompute: bool = False,
            cosine: bool = False):
    """All (i, j) with <P_i, Q_j> >= s as an (n, 2) int32 tensor of uint32
    indices.  With cap=None (and no `out`) the output is sized by sj_count and
    filled by count-then-emit (deterministic order) unless two_pass=False asks
    for the single pass; with a capacity the single pass runs unless
    two_pass=True.  recompute makes the second pass of count-then-emit repeat
    the product even where the first pass's match bits would be kept.
    cosine=True normalises the rows in the library first (SJ_FLAG_COSINE)."""
    return _join("ip", P, Q, s, cap, two_pass, timing, ctx, out, recompute, cosine)


def join_l2(P, Q, r2: float, cap: int | None = None, two_pass: bool | None = None,
            timing: bool = False, ctx=None, out=None, recompute: bool = False):
    """All (i, j) with ||P_i - Q_j||^2 <= r2 (see join_ip)."""
    return _join("l2", P, Q, r2, cap, two_pass, timing, ctx, out, recompute)


def normalize(X, ctx=None):
    """Section 4's cosine front end (sj_normalize): the rows of X (float16,
    bfloat16 or int8 device tensor) divided by their norms, rounded to
    float16 (bfloat16 for bfloat16 input)."""
    import torch
    if X.dim() != 2 or not X.is_cuda or not X.is_contiguous():
        raise ValueError("X must be a contiguous 2-D device tensor")
    ctx = ctx or context(X.device.index)
    Y = torch.empty(X.shape, dtype=torch.bfloat16 if X.dtype == torch.bfloat16 else torch.float16,
                    device=X.device)
    st = sj_normalize(ctx, dtype_code(X), X.data_ptr(), X.shape[0], X.shape[1], Y.data_ptr())
    if st != SJ_OK:
        raise SjError(st, sj_last_error())
    return Y


def join_hamming(P, Q, d: int, r: float, cap: int | None = None, two_pass: bool | None = None,
                 timing: bool = False, ctx=None, out=None):
    """Section 4's Hamming join (sj_join_hamming): all (i, j) whose d-bit rows
    differ in at most r coordinates.  P and Q are (n, ceil(d / 8)) uint8
    device tensors of bit rows (coordinate m in bit m % 8 of byte m / 8).
    Sizing and modes as join_ip."""
    import torch
    for X in (P, Q):
        if X.dtype != torch.uint8 or X.dim() != 2 or X.shape[1] != (d + 7) // 8 or \
                not X.is_cuda or not X.is_contiguous():
            raise ValueError(f"bit rows must be contiguous (n, {(d + 7) // 8}) uint8 device "
                             "tensors")
    ctx = ctx or context(P.device.index)
    if two_pass is None:
        two_pass = cap is None and out is None
    flags = (SJ_FLAG_TWO_PASS if two_pass else 0) | (SJ_FLAG_TIMING if timing else 0)

    def call(ptr, c, f):
        return sj_join_hamming(ctx, P.data_ptr(), P.shape[0], Q.data_ptr(), Q.shape[0], d, r,
                               ptr, c, f)
    return _sized_call(call, flags, cap, out, P.device)


def join_lsh(P, Q, thr: float, metric: str = "ip", *, L: int, k: int, A, B=None, w: int = 0,
             cap: int | None = None, ctx=None, out=None):
    """LSH-bucketed join (sj_join_lsh): the pairs that share a bucket in one
    of L tables (k concatenated random projections each: signs when w == 0,
    quantised with offsets B when w > 0) and pass the exact test of `metric`.
    A is an (L*k, d) int8 device tensor, B an (L*k,) int32 device tensor (or
    None for sign hashes).  With cap=None a first call sizes the output.
    Returns (pairs as an (n, 2) int32 tensor of uint32 indices, number of pair
    evaluations made)."""
    import torch
    _check_pair(P, Q)
    if A.dtype != torch.int8 or not A.is_cuda or not A.is_contiguous() or \
            tuple(A.shape) != (L * k, P.shape[1]):
        raise ValueError(f"A must be a contiguous ({L * k}, {P.shape[1]}) int8 device tensor")
    if B is not None and (B.dtype != torch.int32 or not B.is_cuda or not B.is_contiguous()
                          or B.numel() != L * k):
        raise ValueError(f"B must be a contiguous ({L * k},) int32 device tensor")
    m = _metric_code(metric)
    ctx = ctx or context(P.device.index)
    args = (ctx, m, dtype_code(P), P.data_ptr(), P.shape[0], Q.data_ptr(), Q.shape[0],
            P.shape[1], thr, L, k, A.data_ptr() if A.numel() else None,
            None if B is None else B.data_ptr(), w)
    if out is None:
        if cap is None:
            st, n, _ = sj_join_lsh(*args, None, 0)
            if st not in (SJ_OK, SJ_E_OVERFLOW):
                raise SjError(st, sj_last_error(), n)
            cap = n
        out = torch.empty((max(int(cap), 1), 2), dtype=torch.int32, device=P.device)
        cap = int(cap)
    else:
        cap = out.shape[0] if cap is None else int(cap)
    st, n, nc = sj_join_lsh(*args, out.data_ptr() if cap else None, cap)
    if st != SJ_OK:
        raise SjError(st, sj_last_error(), n)
    return out[:n], nc


def lsh_sort(keys, bits: int, ctx=None):
    """The LSH join's grouping step (sj_lsh_sort): keys is an (L, n) int64
    device tensor of bucket keys (read as uint64, each below 2**bits).  Returns
    an (L, n) int32 tensor: per table the rows with equal keys contiguous and
    in increasing order, the groups in an order fixed by the key values."""
    import torch
    if keys.dim() != 2 or keys.dtype != torch.int64 or not keys.is_cuda or \
            not keys.is_contiguous():
        raise ValueError("keys must be a contiguous (L, n) int64 device tensor")
    L, n = keys.shape
    perm = torch.empty((L, n), dtype=torch.int32, device=keys.device)
    ctx = ctx or context(keys.device.index)
    st = sj_lsh_sort(ctx, keys.data_ptr() if keys.numel() else None, n, L, int(bits),
                     perm.data_ptr() if perm.numel() else None)
    if st != SJ_OK:
        raise SjError(st, sj_last_error())
    return perm


def jl_transform(X, shapes, As, ctx=None):
    """TCU Johnson-Lindenstrauss transform (sj_jl): the rows of X (n x d device
    tensor: float16, bfloat16 or int8) reduced by M = (I_{r_l} (x) A_l) ...
    (I_{r_1} (x) A_1); shapes is the list of (k_i, c_i, r_i), As the list of
    k_i x c_i float32 device tensors.  Returns an (n, r_l k_l) float32 tensor."""
    import torch
    if X.dim() != 2 or not X.is_cuda or not X.is_contiguous():
        raise ValueError("X must be a contiguous 2-D device tensor")
    shapes = [tuple(int(v) for v in s) for s in shapes]
    if len(As) != len(shapes):
        raise ValueError("one factor per level")
    for (k, c, r), A in zip(shapes, As):
        if tuple(A.shape) != (k, c) or A.dtype != torch.float32 or not A.is_cuda:
            raise ValueError(f"factor of shape {(k, c)} float32 on the device expected")
    Acat = torch.cat([A.reshape(-1) for A in As]).contiguous()
    out_dim = shapes[-1][0] * shapes[-1][2]
    Y = torch.empty((X.shape[0], out_dim), dtype=torch.float32, device=X.device)
    ctx = ctx or context(X.device.index)
    st = sj_jl(ctx, dtype_code(X), X.data_ptr(), X.shape[0], X.shape[1], len(shapes), shapes,
               Acat.data_ptr(), Y.data_ptr())
    if st != SJ_OK:
        raise SjError(st, sj_last_error())
    return Y
