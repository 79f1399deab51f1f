"""The benchmark's host-side contract, without a GPU: it refuses more than
one GPU with a message, and its algorithmic byte counts are the per-step
figures the measurements are quoted in (70B-shaped verify step at K = 4,
B = 1, ctx 2048: 129.37 GB of weights + 5.37 GB of KV reads + the new K/V
and the logits = 134.77 GB; 7B-shaped: 14.30 GB)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_verify_bytes_at_the_quoted_shapes():
    import bench
    from paper_2302_01318_amd import configs
    s70 = configs.SEVENTY_B
    b70 = bench.verify_bytes(s70, 1, 4, 2048)
    assert abs(b70 - 134.77e9) < 0.01e9, b70
    # The pieces: every weight matrix once, the prior and new KV once each way.
    HD = s70.n_heads * s70.head_dim
    weights = s70.n_layers * (4 * s70.d_model * HD + 2 * s70.d_model * s70.d_ff) * 2 + s70.vocab * s70.d_model * 2
    assert abs(weights - 129.37e9) < 0.01e9
    kv_read = s70.n_layers * 2 * HD * (2048 + 5) * 2
    assert abs(kv_read - 5.38e9) < 0.01e9
    assert b70 > weights + kv_read
    b7 = bench.verify_bytes(configs.SEVEN_B, 1, 4, 2048)
    assert abs(b7 - 14.30e9) < 0.01e9, b7
    # FP8 projections: one byte per weight plus a scale per output row.
    b70_8 = bench.verify_bytes(s70.with_(dtype="fp8"), 1, 4, 2048)
    assert 69e9 < b70_8 < 71e9, b70_8


def test_profile_figures_only_for_the_profiled_workload():
    # profiles/ holds counters and traces of the 70B verify step at K = 4,
    # B = 1, ctx 2048; another shape or workload must not report them.
    import bench
    for args in (("7b", "bf16", 1, 4, 2048), ("70b", "bf16", 16, 8, 2048), ("70b", "bf16", 1, 4, 8192),
                 ("70b", "fp8", 4, 4, 2048)):
        assert bench.profiled_figures(*args) == {"traffic": None, "mfma": None, "trace": None}, args
    got = bench.profiled_figures("70b", "bf16", 1, 4, 2048)
    assert got["traffic"] == bench.measured_traffic("bf16")
    assert got["trace"] == bench.measured_trace("bf16")
