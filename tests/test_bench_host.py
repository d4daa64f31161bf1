"""Host logic of bench.py, without a GPU: the one-GPU refusal, the algorithmic FLOP / byte formulas, and the rule
that the committed traffic figure is reported only for the kernel sources it was measured on."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env=None):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          env=e, cwd=ROOT, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run(["--gpus", "2"])
    assert r.returncode != 0 and "one GPU" in r.stderr
    r = _run([], env={"WORLD_SIZE": "4"})
    assert r.returncode != 0 and "one GPU" in r.stderr


def test_linear_flops_and_bytes():
    # one 2048 x 4096 -> 4096 linear at rank 16: base product, LoRA down and up
    M, K, N, r = 2048, 4096, 4096, 16
    assert bench.lin_flops(M, K, N, r) == 2 * M * K * N + 2 * M * K * r + 2 * M * r * N
    # bf16 x, W, A, B read once; fp32 y_off and y_on written once
    assert bench.lin_bytes(M, K, N, r) == 2 * (M * K + N * K + r * K + N * r) + 2 * 4 * M * N


def test_traffic_figure_only_for_the_measured_sources(monkeypatch):
    path = os.path.join(ROOT, "profiles", "traffic_prefill.txt")
    recorded = [ln.split("=", 1)[1].strip() for ln in open(path) if ln.startswith("kernel_source_sha256=")]
    fig = bench.committed_traffic("prefill")
    if recorded and recorded[0] == bench.kernel_source_digest():
        assert fig is not None
        assert abs(fig["bytes_per_launch"] - fig["read_bytes_per_launch"] - fig["write_bytes_per_launch"]) <= 2
        assert fig["bytes_per_launch"] >= fig["algorithmic_bytes_per_launch"] > 0
    else:
        assert fig is None  # measured on other sources: not reported
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 64)
    assert bench.committed_traffic("prefill") is None
    assert bench.committed_traffic("no_such_part") is None


def test_unknown_aux_entry_is_refused():
    r = _run(["--aux", "score_logits,no_such_entry"])
    assert r.returncode == 2 and "no_such_entry" in r.stderr
