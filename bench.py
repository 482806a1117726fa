#!/usr/bin/env python3
"""Benchmark of the MI355X similarity join (one GPU).

A step is one whole join call -- sj_join_ip / sj_join_l2 on one batch of
synthetic input already resident in HBM: (row norms for L2), the fused MFMA
product + threshold + compaction kernel, and the hand-back of the match count
(two passes plus the scan for workloads that need count-then-emit).  The
default workload is the largest one that fits one GPU: the 1048576 x 1048576,
d = 64, int8 squared-L2 join (1.1e12 pair evaluations).  After the timed
region the line also reports the join kernel's fraction of the dense MFMA
peak on the 65536 x 128 bf16 and 262144 x 256 fp16 inner-product workloads
(`other_workloads`); the others (--workload NAME, see workloads.NAMES) are
available for measurements but are not the headline line.

Prints ONE JSON line on stdout:
  metric/value/unit: pair-evaluations per second of the whole step
  roofline: the join kernel's algorithmic FLOP (2 d per pair) / its average
            duration measured with HIP events on the stream it runs on, against
            the MI355X dense MFMA peak for its dtype
  cpu_baseline: the oracle (plain C loops) on a bounded sample of the same
            workload on this host's cores
  other_workloads: kernel time and fraction of peak of the join on the other
            two workloads with a 60%-of-peak target (measured untimed, after
            the timed region)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# dense MFMA peaks of MI355X (TFLOP/s or TOP/s)
PEAK = {"f16": 2500.0, "bf16": 2500.0, "i8": 5000.0}
DEFAULT_WORKLOAD = "l2_i8_1048576x64"
# workloads whose join kernel fraction is reported beside the headline
OTHER_WORKLOADS = ("ip_bf16_65536x128", "cos_f16_262144x256")
TWO_PASS = {"ip_bf16_clustered_131072x1024"}   # high-output workload: count-then-emit


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _code_only(src: str) -> str:
    """C++ source without comments and blank space (string literals kept)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c == '"' or c == "'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            i = src.find("\n", i)
            i = n if i < 0 else i
        elif src.startswith("/*", i):
            i = src.find("*/", i + 2)
            i = n if i < 0 else i + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


# Sources of the all-pairs join, its count/emit passes and their launches
# (the kernels whose counters are recorded); the LSH front end is not among them.
JOIN_SOURCES = ("sj_api", "sj_aux", "sj_internal", "sj_join")


# Sources of the TCU JL transform (its own counter record).
JL_SOURCES = ("sj_jl", "sj_host")

# Sources of the LSH-bucketed join (it uses the join's MMA helpers too).
LSH_SOURCES = ("sj_lsh", "sj_sort", "sj_aux", "sj_internal", "sj_host", "sj_join")


def kernel_source_hash(prefixes=JOIN_SOURCES) -> str:
    """Hash of the code of the source files whose names start with one of
    `prefixes` (comments and layout ignored; default: the join's), to tell
    whether a stored counter record was taken on the current kernels."""
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2006_12608_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".h", ".hip", ".cpp")) and f.startswith(prefixes):
            h.update(f.encode())
            h.update(_code_only(open(os.path.join(d, f)).read()).encode())
    return h.hexdigest()[:16]


def _counter_record(key: str, prefixes=JOIN_SOURCES):
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        rec = json.load(open(p)).get(key)
    except (ValueError, OSError):
        return None
    if not rec or rec.get("kernel_sha") != kernel_source_hash(prefixes):
        return None
    return rec


def traffic_for(key: str, prefixes=JOIN_SOURCES):
    """HBM bytes per launch from the committed rocprofv3 counter summary (key:
    the workload name for its join or first-pass kernel, "<workload>:emit" for
    its emit-from-bits kernel), if it was taken on the current kernel sources;
    otherwise None."""
    rec = _counter_record(key, prefixes)
    return rec.get("hbm_bytes_per_launch") if rec else None


def busy_for(key: str):
    """The join kernel's matrix-core busy fraction and clock (GHz) from the
    committed rocprofv3 counters (SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE)
    of this workload, if taken on the current kernel sources; otherwise
    None.  Their product over 2.4 GHz is the fraction of the spec peak."""
    rec = _counter_record(key)
    if not rec or "mfma_busy" not in rec:
        return None
    return {"mfma_busy": rec["mfma_busy"], "clock_ghz": rec["clock_ghz"],
            "source": "profiles/join_resident_mfma_busy_and_clock_counters.md"}


def measured_mfma_peak(dtype: str, duration_ms: float, operands=None, waves_per_simd: int = 2):
    """The throughput of a loop of MFMAs alone on this GPU (libsj_peak.so:
    four accumulator chains per wave, `waves_per_simd` waves per SIMD, no
    memory traffic) over a run of `duration_ms`, with MFMA operands taken
    from `operands` (a device tensor, e.g. the workload's rows; random values
    if None), or None when the probe library is not built.  At full
    matrix-core duty the chip's power limit lowers the clock below what the
    join runs at, so this is context for the clock counters, not a ceiling."""
    import ctypes
    path = os.path.join(ROOT, "paper_2006_12608_amd", "libsj_peak.so")
    if not os.path.exists(path):
        return None
    lib = ctypes.CDLL(path)
    lib.sj_peak_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_void_p,
                                 ctypes.c_uint64, ctypes.POINTER(ctypes.c_double),
                                 ctypes.POINTER(ctypes.c_double)]
    lib.sj_peak_mfma.restype = ctypes.c_int
    tops, ms = ctypes.c_double(), ctypes.c_double()
    code = {"f16": 1, "bf16": 2, "i8": 3}[dtype]
    ptr = operands.data_ptr() if operands is not None else None
    nbytes = operands.numel() * operands.element_size() if operands is not None else 0
    if lib.sj_peak_mfma(code, waves_per_simd, max(duration_ms, 1.0), ptr, nbytes, ctypes.byref(tops),
                        ctypes.byref(ms)) != 0:
        return None
    return {"value": tops.value, "unit": "TOP/s" if dtype == "i8" else "TFLOP/s",
            "run_ms": ms.value,
            "operands": "the workload's P rows" if operands is not None else "random"}


def cpu_model() -> str:
    try:
        for l in open("/proc/cpuinfo"):
            if l.startswith("model name"):
                return l.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, target_s: float = 12.0):
    import numpy as np
    import oracle
    threads = oracle.max_threads()
    rng = np.random.default_rng(4242)
    per_row_work = w.n_q * max(w.d, 1)
    # the probe takes at least one row per thread (the oracle's threads split
    # the rows), so its rate is the rate of the timed sample
    r0 = max(threads, min(w.n_p, int(2e8 // per_row_work) or 1))
    r0 = min(r0, w.n_p)
    rows = np.sort(rng.choice(w.n_p, size=r0, replace=False))
    t = time.perf_counter()
    oracle.join(w.metric, w.dtype, w.P, w.Q, w.threshold, rows=rows, threads=threads)
    t0 = time.perf_counter() - t
    n_rows = int(max(1, min(w.n_p, round(r0 * target_s / max(t0, 1e-3)))))
    rows = np.sort(rng.choice(w.n_p, size=n_rows, replace=False))
    t = time.perf_counter()
    r = oracle.join(w.metric, w.dtype, w.P, w.Q, w.threshold, rows=rows, threads=threads)
    el = time.perf_counter() - t
    return {"value": n_rows * w.n_q / el, "unit": "pair-evaluations/s", "cores": threads,
            "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{n_rows} random rows of P against all {w.n_q} rows of Q "
                      f"({n_rows * w.n_q:.3g} pair evaluations, {el:.1f} s, {r.total} matches)"}


def copy_calibration():
    """A plain device copy of known size: 256 MiB read and 256 MiB written per
    launch.  Its counter readings give the factors that turn the join kernel's
    FETCH_SIZE and WRITE_SIZE into bytes."""
    import torch
    a = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_per_launch": 256 << 20, "launches": 3}))


def jl_chain(d, k, zeta):
    """Lemma 3's level sizes (k_i, c_i, r_i): k_i = i k (k_l = k), c_1 = zeta k,
    c_i = zeta k_{i-1}, r_i = zeta^(l - i), zeta^l = d / k."""
    import math
    l = int(round(math.log(d / k) / math.log(zeta)))
    if zeta ** l * k != d:
        raise SystemExit(f"--jl: d = {d} is not k zeta^l")
    shapes = []
    for i in range(1, l + 1):
        ki = k if i == l else i * k
        ci = zeta * k if i == 1 else zeta * shapes[-1][0]
        shapes.append((ki, ci, zeta ** (l - i)))
    return shapes


def bench_jl(args, w, Pd, ctx):
    """The TCU JL transform of P: one JSON line with its throughput and its
    HBM roofline (each level reads its input and writes its output once)."""
    import numpy as np
    import torch
    import paper_2006_12608_amd as sj
    k, zeta = (int(v) for v in args.jl.split(","))
    shapes = jl_chain(w.d, k, zeta)
    rng = np.random.default_rng(1400 + __import__("workloads").NAMES.index(args.workload))
    As = [torch.from_numpy((rng.standard_normal((kk, c)) / np.sqrt(kk)).astype(np.float32)).cuda()
          for (kk, c, r) in shapes]
    for _ in range(args.warmup):
        sj.jl_transform(Pd, shapes, As, ctx=ctx)
    torch.cuda.synchronize()
    ms = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        sj.jl_transform(Pd, shapes, As, ctx=ctx)
        ms.append(sj.sj_get_stats(ctx).ms_join)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) / args.steps * 1e3
    kms = float(np.mean(ms))
    esz = 1 if w.dtype == "i8" else 2
    nbytes = w.n_p * w.d * esz
    for i, (kk, c, r) in enumerate(shapes):
        nbytes += w.n_p * r * kk * 4 * (2 if i + 1 < len(shapes) else 1)
    flop = sum(2.0 * w.n_p * r * kk * c for (kk, c, r) in shapes)
    print(json.dumps({
        "metric": "rows reduced/sec (TCU JL transform)",
        "value": w.n_p / (ms_step / 1e3), "unit": "rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32 (inputs " + w.dtype + ")",
        "data": "synthetic (the workload's P; factors N(0, 1/k_i), seeded)",
        "config": {"workload": w.name, "n": w.n_p, "d": w.d, "k": k, "zeta": zeta,
                   "levels": [list(s) for s in shapes], "parallelism": "single GPU"},
        "phases_ms": {"transform": kms},
        "flop": flop,
        "roofline": {"bound": "hbm", "kernel": "jl_level (all levels)", "kernel_ms": kms,
                     "achieved": nbytes / (kms / 1e3) / 1e9, "peak": 8000.0, "unit": "GB/s",
                     "frac": nbytes / (kms / 1e3) / 1e9 / 8000.0,
                     "traffic": traffic_for(f"jl:{args.workload}:{args.jl}", JL_SOURCES),
                     "algorithmic_bytes": nbytes},
    }), flush=True)


def lsh_plan(args, w):
    """Section 4's parameters (sj_lsh_plan) for the workload at the recall
    target of --lsh-plan RECALL[,w]: one function's collision probability p1
    at the join's threshold and p2 at the workload's typical distance between
    unrelated points (cosine: orthogonal; squared L2: the median distance of
    2000 random pairs), the 128-row tile for sqrt(m).  Returns (L, k, w, plan
    record); L = L_inst * reps, capped at the library's 256 tables."""
    import math
    import numpy as np
    import paper_2006_12608_amd as sj
    parts = args.lsh_plan.split(",")
    recall = float(parts[0])
    wid = int(parts[1]) if len(parts) > 1 else (0 if w.metric == "ip" else 2000)
    sigma = 32.0   # workloads.lsh_params' projection scale
    if wid == 0:
        d1, d2 = math.acos(min(1.0, w.threshold)), math.pi / 2
    else:
        rng = np.random.default_rng(5)
        i, j = rng.integers(0, w.n_p, 2000), rng.integers(0, w.n_q, 2000)
        x = w.P[i].astype(np.float64)
        y = w.Q[j].astype(np.float64)
        d1, d2 = math.sqrt(w.threshold), float(np.median(np.sqrt(((x - y) ** 2).sum(1))))
    p1, p2 = sj.sj_lsh_collision(wid, sigma, d1), sj.sj_lsh_collision(wid, sigma, d2)
    st, k, L_inst, reps = sj.sj_lsh_plan(p1, p2, max(w.n_p, w.n_q), 128, recall)
    if st != sj.SJ_OK:
        raise SystemExit(f"sj_lsh_plan: {sj.sj_last_error()}")
    L = min(L_inst * reps, 256)
    return L, k, wid, {"recall_target": recall, "p1": p1, "p2": p2, "dist_near": d1,
                       "dist_far": d2, "k": k, "L_inst": L_inst, "reps": reps,
                       "tables_planned": L_inst * reps, "tables_run": L,
                       "guaranteed_recall_at_threshold":
                           1 - (1 - p1 ** k) ** L}


def bench_lsh(args, w, Pd, Qd, ctx, exact_total):
    """The LSH-bucketed join of Theorem 3 on the workload: one JSON line with
    its whole-call throughput, the share of the exact join it finds, its
    candidate pair evaluations, the bucket-join kernel's MFMA fraction on
    those candidates, and the all-pairs join's time on the same workload."""
    import numpy as np
    import torch
    import paper_2006_12608_amd as sj
    import workloads
    plan = None
    if args.lsh_plan:
        L, k, wid, plan = lsh_plan(args, w)
    else:
        parts = [int(v) for v in args.lsh.split(",")]
        L, k, wid = parts[0], parts[1], parts[2] if len(parts) > 2 else 0
    h = workloads.lsh_params(1300 + workloads.NAMES.index(args.workload), L, k, w.d, wid)
    A = torch.from_numpy(h.A).cuda()
    B = torch.from_numpy(h.B).cuda() if wid > 0 else None
    m = sj.SJ_IP if w.metric == "ip" else sj.SJ_L2
    dt = {"f16": sj.SJ_F16, "bf16": sj.SJ_BF16, "i8": sj.SJ_I8}[w.dtype]
    cap = max(exact_total, 1)
    out = torch.empty((cap, 2), dtype=torch.int32, device="cuda")

    def step():
        st, n, nc = sj.sj_join_lsh(ctx, m, dt, Pd.data_ptr(), w.n_p, Qd.data_ptr(), w.n_q, w.d,
                                   w.threshold, L, k, A.data_ptr(), None if B is None
                                   else B.data_ptr(), wid, out.data_ptr(), cap)
        if st != sj.SJ_OK:
            raise sj.SjError(st, sj.sj_last_error(), n)
        return n, nc

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    hash_ms, sort_ms, join_ms, rows = [], [], [], 0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        n_out, n_cand = step()
        s = sj.sj_get_stats(ctx)
        hash_ms.append(s.ms_norms)
        sort_ms.append(s.ms_scan)
        join_ms.append(s.ms_join)
        rows = s.lsh_rows
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) / args.steps * 1e3
    jms = float(np.mean(join_ms))
    flop = 2.0 * n_cand * max(w.d, 1)
    peak = PEAK[w.dtype]
    # the bucket join's algorithmic bytes: every row of every shared bucket
    # read once per table (with its norm for L2), the pairs written
    esz = 1 if w.dtype == "i8" else 2
    alg_bytes = rows * (w.d * esz + (4 if w.metric == "l2" else 0)) + 8 * n_out
    lsh_key = f"lsh:{w.name}:{L},{k},{wid}"
    # the all-pairs join of the same workload, for the speed-up at this recall
    fn = sj.sj_join_ip if w.metric == "ip" else sj.sj_join_l2
    out2 = torch.empty((max(exact_total, 1), 2), dtype=torch.int32, device="cuda")
    for _ in range(2):
        fn(ctx, dt, Pd.data_ptr(), w.n_p, Qd.data_ptr(), w.n_q, w.d, w.threshold,
           out2.data_ptr(), exact_total, 0)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    reps_ap = 3
    for _ in range(reps_ap):
        fn(ctx, dt, Pd.data_ptr(), w.n_p, Qd.data_ptr(), w.n_q, w.d, w.threshold,
           out2.data_ptr(), exact_total, 0)
    torch.cuda.synchronize()
    ap_ms = (time.perf_counter() - t1) / reps_ap * 1e3
    print(json.dumps({
        "metric": "pair-evaluations/sec (all-pairs equivalent, LSH-bucketed join)",
        "value": w.n_p * w.n_q / (ms_step / 1e3),
        "unit": "pair-evaluations/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded generator and seeded LSH draws, inputs resident in HBM)",
        "config": {"workload": w.name, "metric": w.metric, "n_p": w.n_p, "n_q": w.n_q,
                   "d": w.d, "threshold": w.threshold, "mode": "lsh", "L": L, "k": k, "w": wid,
                   "parallelism": "single GPU"},
        "n_out": int(n_out), "exact_total": int(exact_total),
        "recall": n_out / exact_total if exact_total else None,
        "all_pairs_ms_per_step": ap_ms,
        "speedup_vs_all_pairs": ap_ms / ms_step,
        "plan": plan,
        "candidate_pair_evals": int(n_cand),
        "candidate_fraction": n_cand / (w.n_p * w.n_q),
        "candidate_pair_evals_per_s": n_cand / (ms_step / 1e3),
        "phases_ms": {"hash": float(np.mean(hash_ms)), "sort_and_pairs": float(np.mean(sort_ms)),
                      "bucket_join": jms},
        "roofline": {"bound": "hbm", "kernel": "lsh join_kernel", "kernel_ms": jms,
                     "achieved": alg_bytes / (jms / 1e3) / 1e9, "peak": 8000.0, "unit": "GB/s",
                     "frac": alg_bytes / (jms / 1e3) / 1e9 / 8000.0,
                     "algorithmic_bytes": int(alg_bytes), "bucket_rows": int(rows),
                     "traffic": traffic_for(lsh_key, LSH_SOURCES),
                     "mfma_achieved": flop / (jms / 1e3) / 1e12, "mfma_peak": peak,
                     "mfma_unit": "TOP/s" if w.dtype == "i8" else "TFLOP/s",
                     "mfma_frac": flop / (jms / 1e3) / 1e12 / peak},
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    import workloads
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=workloads.NAMES)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the join kernel measurements on the other workloads")
    ap.add_argument("--mfma-loop", action="store_true",
                    help="only run the MFMA-only loop on the workload's rows (for counters)")
    ap.add_argument("--loop-ms", type=float, default=200.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy a 256 MiB buffer three times (the reference kernel for "
                         "scaling rocprofv3's FETCH_SIZE / WRITE_SIZE counters to HBM bytes)")
    ap.add_argument("--self-join", action="store_true",
                    help="join the workload's P with itself (same pointer: the single pass "
                         "computes the upper triangle and mirrors its pairs)")
    ap.add_argument("--jl", default=None, metavar="k,zeta",
                    help="time the TCU JL transform (sj_jl) of the workload's P to dimension k "
                         "with Lemma 3's levels for zeta; prints its own JSON line")
    ap.add_argument("--lsh-plan", default=None, metavar="RECALL[,w]",
                    help="time the LSH-bucketed join with Section 4's parameters for a recall "
                         "target (sj_lsh_plan); prints its own JSON line")
    ap.add_argument("--lsh", default=None, metavar="L,k[,w]",
                    help="time the LSH-bucketed join (sj_join_lsh) on the workload instead: "
                         "L tables of k concatenated projections (w = 0: signs; w > 0: "
                         "quantised with bucket width w); prints its own JSON line")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.mfma_loop:
        mfma_loop(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the join shards "
              "by rows of P across GPUs, which is not implemented", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2006_12608_amd as sj
    import workloads
    to_device = workloads.to_torch

    k = args.workload
    log(f"generating workload {k} ...")
    w = workloads.make_config(k, self_join=args.self_join)
    torch.cuda.set_device(0)
    Pd = to_device(w.P, w.dtype)
    Qd = Pd if w.self_join else to_device(w.Q, w.dtype)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ctx = sj.context(0, stream)
    dt = {"f16": sj.SJ_F16, "bf16": sj.SJ_BF16, "i8": sj.SJ_I8}[w.dtype]
    two_pass = k in TWO_PASS
    flags = sj.SJ_FLAG_TIMING | (sj.SJ_FLAG_TWO_PASS if two_pass else 0)
    fn = sj.sj_join_ip if w.metric == "ip" else sj.sj_join_l2

    if args.jl:
        bench_jl(args, w, Pd, ctx)
        return
    total = sj.count(Pd, Qd, w.threshold, w.metric, ctx=ctx)
    if args.lsh or args.lsh_plan:
        bench_lsh(args, w, Pd, Qd, ctx, total)
        return
    out = torch.empty((max(total, 1), 2), dtype=torch.int32, device="cuda")
    log(f"{w.name}: {total} matches; warmup {args.warmup}, steps {args.steps}")

    def step():
        st, n = fn(ctx, dt, Pd.data_ptr(), w.n_p, Qd.data_ptr(), w.n_q, w.d, w.threshold,
                   out.data_ptr(), total, flags)
        if st != sj.SJ_OK:
            raise sj.SjError(st, sj.sj_last_error(), n)
        return n

    # Setup, untimed: bring the GPU clocks to their sustained state with about
    # 0.3 s of counting passes before the warmup steps proper.
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < 0.3:
        sj.count(Pd, Qd, w.threshold, w.metric, ctx=ctx)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    kern_ms, emit_ms, count_ms, scan_ms, norm_ms = [], [], [], [], []
    from_bits = False
    t0 = time.perf_counter()
    n_out = 0
    for _ in range(args.steps):
        n_out = step()
        s = sj.sj_get_stats(ctx)
        kern_ms.append(s.ms_join if not two_pass else s.ms_count)
        emit_ms.append(s.ms_emit)
        count_ms.append(s.ms_count)
        scan_ms.append(s.ms_scan)
        norm_ms.append(s.ms_norms)
        from_bits = bool(s.emit_from_bits)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    ms_step = el / args.steps * 1e3
    pair_evals = w.n_p * w.n_q
    value = pair_evals / (ms_step / 1e3)
    kms = float(np.mean(kern_ms))
    flop = 2.0 * pair_evals * max(w.d, 1)
    # a self-join's distinct pairs: the upper triangle, diagonal included
    # (the kernel computes those and mirrors the rest)
    kflop = 2.0 * (w.n_p * (w.n_p + 1) // 2) * max(w.d, 1) if w.self_join and not two_pass \
        else flop
    achieved_k = kflop / (kms / 1e3) / 1e12
    achieved = achieved_k
    peak = PEAK[w.dtype]
    traffic = None if w.self_join else traffic_for(args.workload)
    line = {
        "metric": "pair-evaluations/sec",
        "value": value,
        "unit": "pair-evaluations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded generator, inputs resident in HBM)",
        "config": {"workload": w.name + ("+self-join" if w.self_join else ""),
                   "metric": w.metric, "n_p": w.n_p, "n_q": w.n_q, "d": w.d,
                   "threshold": w.threshold, "mode": "two-pass" if two_pass else "single-pass",
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak,
                     "unit": "TOP/s" if w.dtype == "i8" else "TFLOP/s", "frac": achieved / peak,
                     "traffic": traffic,
                     "kernel": "join_resident" if w.d * (1 if w.dtype == "i8" else 2) <= 512
                     else "join_streamed",
                     "kernel_ms": kms,
                     "counters": None if w.self_join or two_pass else busy_for(args.workload)},
        "effective_tflops_step": flop / (ms_step / 1e3) / 1e12,
        "pct_peak_step": flop / (ms_step / 1e3) / 1e12 / peak,
        "n_out": int(n_out),
        "pairs_emitted_per_s": n_out / (float(np.mean(emit_ms)) / 1e3) if two_pass
        else n_out / (ms_step / 1e3),
        "phases_ms": {"norms": float(np.mean(norm_ms)), "join_or_count": kms,
                      "scan": float(np.mean(scan_ms)), "emit": float(np.mean(emit_ms))},
        "kernel_sha": kernel_source_hash(),
    }
    if two_pass:
        # the second pass's algorithmic HBM bytes: 8 per pair written, plus the
        # first pass's match bits read (one bit per result of every 256 x 256
        # tile) when it reads them instead of recomputing the product
        tiles = -(-w.n_p // 256) * -(-w.n_q // 256)
        emit_bytes = n_out * 8 + (tiles * 256 * 256 // 8 if from_bits else 0)
        line["emit"] = {"from_match_bits": from_bits, "hbm_bytes_algorithmic": emit_bytes,
                        "hbm_gbps_algorithmic": emit_bytes / (float(np.mean(emit_ms)) / 1e3) / 1e9,
                        "traffic": traffic_for(args.workload + ":emit") if from_bits else None}
    if not args.no_other_workloads:
        line["other_workloads"] = {name: kernel_fraction(name, stream, ctx)
                                   for name in OTHER_WORKLOADS if name != w.name}
    if not args.no_cpu_baseline:
        log("timing the oracle on a sample ...")
        line["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(line), flush=True)


def kernel_fraction(name: str, stream, ctx, steps: int = 10):
    """The join kernel's average time over `steps` single-pass calls on the
    named workload (after the clock-settling count passes) and its fraction
    of the dense MFMA peak: 2 d FLOP per pair evaluation over the kernel time
    recorded with HIP events on the call's stream."""
    import numpy as np
    import torch
    import paper_2006_12608_amd as sj
    import workloads
    log(f"measuring the join kernel on {name} ...")
    w = workloads.make_config(name)
    Pd = workloads.to_torch(w.P, w.dtype)
    Qd = workloads.to_torch(w.Q, w.dtype)
    torch.cuda.synchronize()
    dt = {"f16": sj.SJ_F16, "bf16": sj.SJ_BF16, "i8": sj.SJ_I8}[w.dtype]
    fn = sj.sj_join_ip if w.metric == "ip" else sj.sj_join_l2
    total = sj.count(Pd, Qd, w.threshold, w.metric, ctx=ctx)
    out = torch.empty((max(total, 1), 2), dtype=torch.int32, device="cuda")
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < 0.3:
        sj.count(Pd, Qd, w.threshold, w.metric, ctx=ctx)
    ms = []
    for _ in range(steps + 2):
        st, n = fn(ctx, dt, Pd.data_ptr(), w.n_p, Qd.data_ptr(), w.n_q, w.d, w.threshold,
                   out.data_ptr(), total, sj.SJ_FLAG_TIMING)
        if st != sj.SJ_OK:
            raise sj.SjError(st, sj.sj_last_error(), n)
        ms.append(sj.sj_get_stats(ctx).ms_join)
    kms = float(np.mean(ms[2:]))
    achieved = 2.0 * w.n_p * w.n_q * w.d / (kms / 1e3) / 1e12
    return {"kernel_ms": kms, "achieved": achieved, "peak": PEAK[w.dtype],
            "unit": "TOP/s" if w.dtype == "i8" else "TFLOP/s",
            "frac": achieved / PEAK[w.dtype], "n_out": int(n), "dtype": w.dtype,
            "steps": steps, "counters": busy_for(name)}


def mfma_loop(args):
    """The MFMA-only loop (libsj_peak.so) on the workload's P rows for about
    --loop-ms milliseconds at 1, 2 and 4 waves per SIMD: one JSON line.  A
    command to take clock and matrix-core busy counters of the loop with."""
    import torch
    import workloads
    w = workloads.make_config(args.workload)
    Pd = workloads.to_torch(w.P, w.dtype)
    torch.cuda.synchronize()
    res = {}
    for wps in (1, 2, 4):
        res[f"{wps}_waves_per_simd"] = measured_mfma_peak(w.dtype, args.loop_ms, Pd, wps)
    print(json.dumps({"mfma_loop": res, "workload": w.name, "dtype": w.dtype,
                      "peak": PEAK[w.dtype]}), flush=True)


if __name__ == "__main__":
    main()
