"""Host-side checks of bench.py: the per-configuration case list and the one-GPU guard.
No GPU is used."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_config_cases_cover_every_workload_and_sweep():
    from paper_2512_08061_amd import workloads as wl

    cases = bench.config_cases()
    labels = [c[0] for c in cases]
    assert len(labels) == len(set(labels))
    assert set(wl.WORKLOADS) <= set(labels)
    for causal in ("noncausal", "causal"):
        ns = sorted(w.n for label, w in cases if label.startswith(f"sweep_{causal}_"))
        assert ns == [1024, 2048, 4096, 8192, 16384]
    for label, w in cases:
        assert min(w.B, w.H, w.n, w.d, w.M, w.L) >= 1
        assert bench.bytes_per_token_head(w) == 4 * w.d * (2 if w.dtype == "bf16" else 4)
        assert bench.flops_per_token_head(w, w.causal) > bench.flops_per_token_head(w, False) or not w.causal


def test_flops_per_token_head_long_causal():
    # 4dM + 4Dd + 4D + 2C(D + d + 1) with d = 128, M = 32, D = 256, C = 64
    from paper_2512_08061_amd import workloads as wl

    w = wl.WORKLOADS["long_causal"]
    assert bench.flops_per_token_head(w, True) == 4 * 128 * 32 + 4 * 256 * 128 + 4 * 256 + 2 * 64 * (256 + 128 + 1)


def test_more_than_one_gpu_is_refused():
    for extra in ([], ["--configs"], ["--decode", "1"]):
        p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", *extra],
                           capture_output=True, text=True, timeout=120)
        assert p.returncode == 2, (extra, p.stderr)
        assert "one GPU" in p.stderr
