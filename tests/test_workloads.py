"""The seeded input generators: bf16 rounding, determinism, shapes (CPU only)."""
import numpy as np
import pytest

import workloads as WL


def test_bf16_round_nearest_even_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.normal(0, 1, 100000), rng.normal(0, 1e-30, 1000), rng.normal(0, 1e30, 1000),
                        [0.0, -0.0, np.inf, -np.inf, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8]]).astype(np.float32)
    ours = WL.f32_to_bf16(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_widen_roundtrip():
    u = np.arange(0, 65536, dtype=np.uint32).astype(np.uint16)
    f = WL.bf16_bits_to_f32(u)
    finite = np.isfinite(f)
    assert np.array_equal(WL.f32_to_bf16(f[finite]), u[finite])


def test_generators_are_deterministic_and_shaped():
    a = WL.gen_linear(0, 16, 512, 512, 8)
    b = WL.gen_linear(0, 16, 512, 512, 8)
    for k in ("x", "W", "A", "B"):
        assert np.array_equal(getattr(a, k), getattr(b, k))
    assert a.x.shape == (16, 512) and a.W.shape == (512, 512) and a.A.shape == (8, 512) and a.B.shape == (512, 8)
    on, off, ids = WL.gen_logits(1, 8, 1000)
    assert on.dtype == np.float32 and ids.dtype == np.int32 and ids.min() >= 0 and ids.max() < 1000
    c = WL.gen_score_head(4, 2, 8, 64, 300, 4)
    assert c.h.shape == (16, 64) and c.W_lm.shape == (300, 64) and c.w_rm.shape == (64,)


def test_distribution_scales():
    c = WL.gen_linear(3, 64, 1024, 512, 16)
    W = WL.bf16_bits_to_f32(c.W).astype(np.float64)
    B = WL.bf16_bits_to_f32(c.B).astype(np.float64)
    assert abs(W.std() * np.sqrt(1024) - 1.0) < 0.02
    assert abs(B.std() * np.sqrt(16) - 1.0) < 0.03
    on, off, _ = WL.gen_logits(1, 16, 32000)
    assert abs(on.std() - 2.0) < 0.02
    assert abs((off - on).std() - 0.1) < 0.002


def test_shared_activation_per_width():
    cases = WL.gen_linears(3, 8, WL.PREFILL_PROJ[:2] + WL.PREFILL_PROJ[-1:], 4)
    assert cases[0].x is cases[1].x and cases[2].x.shape == (8, 11008)


def test_advantage_generator():
    a = WL.gen_advantages(5, 2, 16, 64, start=3)
    b = WL.gen_advantages(5, 2, 16, 64, start=3)
    assert a.h.shape == (32, 64) and a.w_v.shape == (64,) and a.kl.shape == (32,) and a.reward.shape == (2,)
    assert a.kl.dtype == np.float32 and a.reward.dtype == np.float32 and a.M == 32 and a.K == 64
    for k in ("kl", "reward", "h", "w_v"):
        assert np.array_equal(getattr(a, k), getattr(b, k))
    big = WL.gen_advantages(5, 4, 512, 256)
    assert abs(big.kl.std() - 0.1) < 0.005
    assert WL.WORKLOADS["ppo_advantages"]["seed"] == 5
