"""Host-side logic of bench.py (no GPU): the one-GPU contract and the
algorithmic work it divides by kernel durations for the rooflines."""
import os
import subprocess
import sys

import bench
from paper_2608_13524_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120, cwd=ROOT)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_projection_work_per_launch():
    """Per vocabulary row: U row (2h bytes), the bias row once per request
    (4b), one fp32 logit per parent row (4R); plus the R feature rows (2hR).
    flops 2 R h V (Sec. 3.2, one product per parent row and token)."""
    cfg = W.CONFIGS["qwen3-4b"]
    h, V = cfg.hidden, cfg.vocab
    for d, R in ((1, 1), (2, 8), (16, 8)):
        b_, f_ = bench.kernel_work(cfg, "logits", d)
        assert b_ == V * (2 * h + 4 * 1 + 4 * R) + 2 * h * R
        assert f_ == 2.0 * R * h * V
    # the steady-state figure the benchmark reports at 8 rows
    assert bench.kernel_work(cfg, "logits", 2)[0] == 783422976


def test_softmax_pass_work_is_one_read_of_z():
    cfg = W.CONFIGS["stress-x16"]
    R = cfg.batch * cfg.width                  # 1024 parent rows from depth 3 on
    assert bench.kernel_work(cfg, "lse_topk", 3) == (4 * R * cfg.vocab, 0.0)
    assert bench.kernel_work(cfg, "lse_topk", 3)[0] == 622329856


def test_traffic_is_reported_only_for_a_summarised_kernel():
    assert bench.measured_traffic("qwen3-4b", "lse_topk") is None
    assert bench.measured_traffic("no-such-workload", "logits") is None


def test_target_shape_is_the_stress_workload():
    """The per-kernel targets are measured at the stress workload's steady
    shape: 16 requests x 64 nodes = 1024 parent rows, V = 151936, h = 5120."""
    cfg = W.CONFIGS["stress-x16"]
    s = bench.TARGET_SHAPE
    assert s["rows"] == cfg.batch * cfg.width and s["vocab"] == cfg.vocab and s["hidden"] == cfg.hidden
    assert s["k"] == cfg.branch and s["rows"] // s["rows_per_group"] == cfg.batch
