"""Host logic of bench.py, without a GPU: the one-GPU refusal, the algorithmic FLOP / byte formulas, the rule that
the committed traffic figure is reported only for the kernel sources it was measured on, and the CPU baseline's
error report."""
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


def test_rel_err_is_relative_to_the_output_scale():
    import numpy as np
    ref = np.array([1.0, -2.0, 0.0, 4.0])
    assert bench.rel_err(ref, ref) == 0.0
    # an error at a zero entry is measured against the rms of the reference (sqrt(21 / 4))
    got = ref.copy()
    got[2] = 0.5
    assert abs(bench.rel_err(got, ref) - 0.5 / np.sqrt(21 / 4)) < 1e-15
    # at a large entry, against that entry
    got = ref.copy()
    got[3] = 4.4
    assert abs(bench.rel_err(got, ref) - 0.1) < 1e-12
    assert bench.rel_err(np.zeros(0), np.zeros(0)) == 0.0


def test_cpu_baseline_error_report():
    """The CPU baseline's comparison with the step's outputs, on small stand-in shapes: the oracle's own outputs (in
    fp32, as the GPU returns them) read as rounding-level errors, and a deviation planted in one output shows up with
    its size under that output's key only."""
    import numpy as np
    import workloads as WL
    from oracle import lora_linear_ref, score_head_ref, reward_ref

    dec = [WL.gen_linear(1 + i, 4, 64, 32, 8, name=n) for i, n in enumerate("qkvo")]
    pre = [WL.gen_linear(10 + i, 80, 64, 48, 8, name=n) for i, n in enumerate(("q", "down"))]
    sc = WL.gen_score_head(20, 2, 40, 64, 300, 8)

    def f32(a):
        return np.asarray(a, np.float32)

    res = score_head_ref(sc.h, sc.W_lm, sc.A, sc.B, sc.s, sc.ids)
    g = dict(decode=[tuple(f32(y) for y in lora_linear_ref(c.x, c.W, c.A, c.B, c.s)) for c in dec],
             prefill={c.name: tuple(f32(y) for y in lora_linear_ref(c.x, c.W, c.A, c.B, c.s)) for c in pre},
             score=dict(lp_on=f32(res["lp_on"]), lp_off=f32(res["lp_off"]), kl=f32(res["kl"]),
                        reward=f32(reward_ref(sc.h, sc.w_rm, sc.n_seq, sc.seq_len))))
    err = bench.cpu_baseline(0.05, (dec, pre, sc), g)["max_error_vs_oracle"]
    assert err["rows"] == 80
    for k, v in err.items():
        if k != "rows":
            assert v < 1e-5, (k, v)

    y_on = g["prefill"]["down"][1]
    y_on[7, 5] += 0.01 * max(abs(float(y_on[7, 5])), float(np.sqrt(np.mean(y_on.astype(np.float64) ** 2))))
    g["score"]["lp_on"][3] += 0.002
    err = bench.cpu_baseline(0.05, (dec, pre, sc), g)["max_error_vs_oracle"]
    assert 0.009 < err["prefill_y_rel"] < 0.011
    assert 0.0019 < err["score_lp_on_abs"] < 0.0021
    assert err["decode_y_rel"] < 1e-5 and err["score_kl_abs"] < 1e-5 and err["score_reward_rel"] < 1e-5
