"""Host-side logic of bench.py (no GPU): the one-GPU guard and the rule that
counter-measured traffic is reported only for the kernel source and the
gradient-buffer mode the counters were taken with."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    msg = json.loads(p.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_traffic_follows_source_hash_and_grad_mode(tmp_path, monkeypatch):
    t = dict(bench.TRAFFIC["gemm_bwd_dw_tn"])
    src = tmp_path / "k.hip"
    src.write_bytes(b"kernel source")
    import hashlib
    t["source"] = str(src)
    t["sha256_16"] = hashlib.sha256(b"kernel source").hexdigest()[:16]
    monkeypatch.setitem(bench.TRAFFIC, "gemm_bwd_dw_tn", t)
    wl, mode = t["workload"], t["grad_buffers"]
    other = "accumulate" if mode == "overwrite" else "overwrite"
    assert bench.measured_traffic("gemm_bwd_dw_tn", wl, mode) == t["bytes_per_launch"]
    assert bench.measured_traffic("gemm_bwd_dw_tn", wl, other) is None
    assert bench.measured_traffic("gemm_bwd_dw_tn", "gpt3-13b-stage", mode) is None
    assert bench.measured_traffic("attn_fwd", wl, mode) is None
    src.write_bytes(b"kernel source, edited")
    assert bench.measured_traffic("gemm_bwd_dw_tn", wl, mode) is None


def test_recorded_traffic_is_not_below_algorithmic_bytes():
    """The recorded per-launch bytes of the dW GEMM cover at least its fp32
    output writes and operand reads on the 175B stage (2 layers, H = 12288,
    L = 2048: 8 launches per sequence, 12 H^2 weights per layer)."""
    H, L = 12288, 2048
    per_layer_out = 12 * H * H * 4
    operands = 2 * L * 2 * (H + 4 * H + H + H + 3 * H + H + 4 * H + H) / 4
    assert bench.TRAFFIC["gemm_bwd_dw_tn"]["bytes_per_launch"] >= per_layer_out / 4 + operands
