"""Helpers shared by the GPU tests: move workloads to the device, run the
library, and compare its pair sets with the oracle's."""
from __future__ import annotations

import numpy as np

import oracle
import workloads


def to_device(X: np.ndarray, dtype: str, device="cuda"):
    return workloads.to_torch(X, dtype, device)


def keys(pairs: np.ndarray) -> np.ndarray:
    p = np.asarray(pairs).astype(np.uint64).reshape(-1, 2)
    return (p[:, 0] << np.uint64(32)) | p[:, 1]


def sorted_pairs(pairs) -> np.ndarray:
    """(m, 2) uint32 pairs sorted lexicographically by (i, j)."""
    if hasattr(pairs, "cpu"):
        pairs = pairs.cpu().numpy()
    pairs = np.ascontiguousarray(pairs)
    if pairs.dtype == np.int32:
        pairs = pairs.view(np.uint32)
    k = np.sort(keys(pairs))
    out = np.empty((k.size, 2), np.uint32)
    out[:, 0] = (k >> np.uint64(32)).astype(np.uint32)
    out[:, 1] = (k & np.uint64(0xFFFFFFFF)).astype(np.uint32)
    return out


def gpu_join(metric, Pd, Qd, thr, cap=None, two_pass=False, timing=False):
    """The library's join; two_pass=False is the single pass (sized by sj_count)."""
    import paper_2006_12608_amd as sj
    f = sj.join_ip if metric == "ip" else sj.join_l2
    return f(Pd, Qd, thr, cap=cap, two_pass=two_pass, timing=timing)


def compare(gpu_sorted: np.ndarray, ref: "oracle.JoinResult", real_valued: bool):
    """Integer-valued inputs: the sets must be identical.  Real-valued inputs:
    identical outside the boundary band (pairs whose fp64 score lies within the
    band of the threshold), whose size is returned with the agreement inside it."""
    g = keys(gpu_sorted)
    assert np.unique(g).size == g.size, "duplicate pairs in the GPU output"
    m = keys(ref.pairs)
    if not real_valued:
        if not np.array_equal(g, m):
            extra = np.setdiff1d(g, m)[:5]
            missing = np.setdiff1d(m, g)[:5]
            raise AssertionError(f"GPU {g.size} pairs vs oracle {m.size}; extra {extra} "
                                 f"missing {missing}")
        return {"band": 0, "gpu_in_band": 0, "oracle_in_band": 0}
    b = keys(ref.band_pairs)
    g_out = np.setdiff1d(g, b)
    m_out = np.setdiff1d(m, b)
    if not np.array_equal(g_out, m_out):
        raise AssertionError(f"outside the band: GPU {g_out.size} vs oracle {m_out.size}; "
                             f"extra {np.setdiff1d(g_out, m_out)[:5]} "
                             f"missing {np.setdiff1d(m_out, g_out)[:5]}")
    return {"band": int(b.size), "gpu_in_band": int(np.intersect1d(g, b).size),
            "oracle_in_band": int(np.intersect1d(m, b).size)}
