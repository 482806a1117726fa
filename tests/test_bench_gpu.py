"""bench.py's measurement helpers on the GPU."""
import pytest

pytestmark = pytest.mark.gpu


def test_mfma_only_peak_probe():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import bench
    ops = torch.randint(-4, 5, (4096, 128), device="cuda").to(torch.bfloat16)
    for dt, lo, hi, x in (("bf16", 300.0, 2600.0, None), ("i8", 600.0, 5200.0, None),
                          ("bf16", 300.0, 2600.0, ops)):
        m = bench.measured_mfma_peak(dt, 20.0, x)
        assert m is not None, "libsj_peak.so is not built"
        print("[case] mfma-only", dt, m, flush=True)
        assert lo < m["value"] < hi and m["run_ms"] > 0
