"""Pins of the float64 oracle against what the mathematics fixes (CPU only).

The paper prints no worked example for any quantity on this path, so each
oracle function is pinned by exact brute force on tiny inputs, closed forms,
invariants and independent library routines.  The mutation tests at the end
plant plausible mistakes in copies of the oracle and check that these pins
catch them.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import hydra_oracle as O
from workloads import f32_to_bf16, gen_linear, gen_logits, gen_score_head


# ---------------------------------------------------------------- helpers

def _int_bf16(rng, shape, lo=-8, hi=8):
    """Small integers: exactly representable in bf16 and in every partial sum."""
    v = rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    return f32_to_bf16(v), v.astype(np.int64)


def _frac_lora(xi, Wi, Ai, Bi, s):
    """Exact LoRA linear with Fractions and plain loops: y_off[m][n], y_on[m][n]."""
    M, K = xi.shape
    N, r = Bi.shape
    s = Fraction(s)
    y_off = [[Fraction(0)] * N for _ in range(M)]
    y_on = [[Fraction(0)] * N for _ in range(M)]
    for m in range(M):
        T = [sum(Fraction(int(xi[m, k])) * int(Ai[j, k]) for k in range(K)) for j in range(r)]
        for n in range(N):
            base = sum(Fraction(int(xi[m, k])) * int(Wi[n, k]) for k in range(K))
            y_off[m][n] = base
            y_on[m][n] = base + s * sum(T[j] * int(Bi[n, j]) for j in range(r))
    return y_off, y_on


# ---------------------------------------------------------------- LoRA linear

@pytest.mark.parametrize("M,K,N,r,s", [(3, 8, 5, 2, 2.0), (1, 16, 3, 1, -0.5), (4, 8, 7, 3, 0.25), (2, 8, 4, 0, 2.0)])
def test_lora_linear_exact_bruteforce(M, K, N, r, s):
    rng = np.random.default_rng(100 + M * 7 + K + N + r)
    x, xi = _int_bf16(rng, (M, K))
    W, Wi = _int_bf16(rng, (N, K))
    A, Ai = _int_bf16(rng, (r, K))
    B, Bi = _int_bf16(rng, (N, r))
    y_off, y_on = O.lora_linear_ref(x, W, A, B, s)
    e_off, e_on = _frac_lora(xi, Wi, Ai, Bi, s)
    for m in range(M):
        for n in range(N):
            assert Fraction(y_off[m, n]) == e_off[m][n]
            assert Fraction(y_on[m, n]) == e_on[m][n]


def test_lora_linear_float_bruteforce_loops():
    """Non-integer bf16 inputs: float64 triple loop (math.fsum, exact sums) vs the oracle."""
    c = gen_linear(7, M=5, K=24, N=6, r=3, s=2.0)
    X, W, A, B = (O.bf16_to_f64(t) for t in (c.x, c.W, c.A, c.B))
    y_off, y_on = O.lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    for m in range(5):
        T = [math.fsum(X[m, k] * A[j, k] for k in range(24)) for j in range(3)]
        for n in range(6):
            base = math.fsum(X[m, k] * W[n, k] for k in range(24))
            on = base + c.s * math.fsum(T[j] * B[n, j] for j in range(3))
            assert abs(y_off[m, n] - base) <= 1e-13 * max(1.0, abs(base))
            assert abs(y_on[m, n] - on) <= 1e-12 * max(1.0, abs(on))


def test_lora_linear_merged_weight_invariant():
    """y_on equals x (W + s B A)^T computed from the explicitly merged weight."""
    c = gen_linear(11, M=33, K=128, N=96, r=8, s=2.0)
    X, W, A, B = (O.bf16_to_f64(t) for t in (c.x, c.W, c.A, c.B))
    W_merged = W + c.s * (B @ A)            # [N x K]
    expect = X @ W_merged.T
    _, y_on = O.lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert np.max(np.abs(y_on - expect)) <= 1e-12 * np.max(np.abs(expect))


def test_lora_linear_b_zero_and_s_zero_are_lora_off():
    c = gen_linear(12, M=9, K=64, N=40, r=8, s=2.0)
    y_off, y_on = O.lora_linear_ref(c.x, c.W, c.A, np.zeros_like(c.B), c.s)
    assert np.array_equal(y_on, y_off)
    y_off2, y_on2 = O.lora_linear_ref(c.x, c.W, c.A, c.B, 0.0)
    assert np.array_equal(y_on2, y_off2)
    assert np.array_equal(y_off, y_off2)


def test_lora_linear_linear_in_scale_and_row_permutation():
    c = gen_linear(13, M=12, K=64, N=32, r=4, s=1.0)
    off1, on1 = O.lora_linear_ref(c.x, c.W, c.A, c.B, 1.0)
    _, on3 = O.lora_linear_ref(c.x, c.W, c.A, c.B, 3.0)
    d1 = on1 - off1
    assert np.allclose(on3 - off1, 3.0 * d1, rtol=1e-12, atol=1e-12)
    perm = np.random.default_rng(0).permutation(12)
    offp, onp = O.lora_linear_ref(c.x[perm], c.W, c.A, c.B, 1.0)
    assert np.array_equal(offp, off1[perm]) and np.array_equal(onp, on1[perm])


def test_lora_linear_adapter_selection():
    """Two adapter sets over one base (Hydra-PPO): each on-output uses only its own pair."""
    a = gen_linear(14, M=6, K=32, N=16, r=4)
    b = gen_linear(15, M=6, K=32, N=16, r=4)
    off_a, on_a = O.lora_linear_ref(a.x, a.W, a.A, a.B, 2.0)
    off_b, on_b = O.lora_linear_ref(a.x, a.W, b.A, b.B, 2.0)
    assert np.array_equal(off_a, off_b)
    assert not np.allclose(on_a, on_b)


def _multi_case(seed, M=3, K=8, N=5, r=2, n_on=2):
    rng = np.random.default_rng(seed)
    x_off = _int_bf16(rng, (M, K))
    W = _int_bf16(rng, (N, K))
    xs = [_int_bf16(rng, (M, K)) for _ in range(n_on)]
    As = [_int_bf16(rng, (r, K)) for _ in range(n_on)]
    Bs = [_int_bf16(rng, (N, r)) for _ in range(n_on)]
    ss = [2.0, -0.5, 0.25, 1.0][:n_on]
    return x_off, W, xs, As, Bs, ss


def _multi_pins_hold(fn):
    """True when fn reproduces the exact per-pass brute force (used to show the pin catches mistakes)."""
    for seed in (31, 32):
        x_off, W, xs, As, Bs, ss = _multi_case(seed)
        y_off, y_ons = fn(x_off[0], W[0], [x[0] for x in xs], [a[0] for a in As], [b[0] for b in Bs], ss)
        e_off, _ = _frac_lora(x_off[1], W[1], As[0][1], Bs[0][1], 0.0)
        if not np.array_equal(y_off, np.array([[float(v) for v in row] for row in e_off])):
            return False
        for a in range(len(xs)):
            _, e_on = _frac_lora(xs[a][1], W[1], As[a][1], Bs[a][1], ss[a])
            if not np.array_equal(y_ons[a], np.array([[float(v) for v in row] for row in e_on])):
                return False
    return True


def test_lora_linear_multi_exact_per_pass_bruteforce():
    """Several passes over one W (Alg. 2): each output is its own input's exact product with its own adapter."""
    assert _multi_pins_hold(O.lora_linear_multi_ref)


def test_lora_linear_multi_merged_weight_per_adapter():
    c = [gen_linear(40 + i, M=7, K=64, N=24, r=4, s=[2.0, 0.5][i]) for i in range(2)]
    off = gen_linear(42, M=7, K=64, N=24, r=4)
    y_off, y_ons = O.lora_linear_multi_ref(off.x, c[0].W, [c[0].x, c[1].x], [c[0].A, c[1].A], [c[0].B, c[1].B],
                                           [c[0].s, c[1].s])
    Wd = O.bf16_to_f64(c[0].W)
    assert np.max(np.abs(y_off - O.bf16_to_f64(off.x) @ Wd.T)) == 0.0
    for i in range(2):
        merged = Wd + c[i].s * (O.bf16_to_f64(c[i].B) @ O.bf16_to_f64(c[i].A))
        expect = O.bf16_to_f64(c[i].x) @ merged.T
        assert np.max(np.abs(y_ons[i] - expect)) <= 1e-12 * np.max(np.abs(expect))
    none_off, only_off = O.lora_linear_multi_ref(None, c[0].W, [], [], [], [])
    assert none_off is None and only_off == []


def _mut_multi_swapped_adapters(x_off, W, xs, As, Bs, ss):
    return O.lora_linear_multi_ref(x_off, W, xs, As[::-1], Bs[::-1], ss)


def _mut_multi_off_from_first_on_input(x_off, W, xs, As, Bs, ss):
    _, y_ons = O.lora_linear_multi_ref(x_off, W, xs, As, Bs, ss)
    y_off, _ = O.lora_linear_multi_ref(xs[0], W, [], [], [], [])
    return y_off, y_ons


def _mut_multi_shared_input(x_off, W, xs, As, Bs, ss):
    return O.lora_linear_multi_ref(x_off, W, [xs[0]] * len(xs), As, Bs, ss)


@pytest.mark.parametrize("mut", [_mut_multi_swapped_adapters, _mut_multi_off_from_first_on_input,
                                 _mut_multi_shared_input])
def test_pins_catch_multi_mutations(mut):
    assert not _multi_pins_hold(mut)


# ---------------------------------------------------------------- LoRA linear backward (update stage)
def _frac_loss(xi, Wi, Ai, Bi, s, dyi):
    """L = sum dY * y_on, exactly (Fractions): linear in each of x, A, B separately."""
    _, y_on = _frac_lora(xi, Wi, Ai, Bi, s)
    M, N = dyi.shape
    return sum(Fraction(int(dyi[m, n])) * y_on[m][n] for m in range(M) for n in range(N))


@pytest.mark.parametrize("M,K,N,r,s", [(2, 8, 3, 2, 2.0), (3, 8, 2, 1, -0.5), (1, 16, 4, 3, 0.25)])
def test_lora_backward_exact_difference_quotients(M, K, N, r, s):
    """L = <dY, y_on> is linear in x, in A and in B, so a unit step's difference quotient IS the derivative:
    every entry of dX, dA, dB equals L(theta + e) - L(theta), computed exactly from the forward definition."""
    rng = np.random.default_rng(M * 31 + K + r)
    xb, xi = _int_bf16(rng, (M, K), -4, 4)
    Wb, Wi = _int_bf16(rng, (N, K), -4, 4)
    Ab, Ai = _int_bf16(rng, (r, K), -4, 4)
    Bb, Bi = _int_bf16(rng, (N, r), -4, 4)
    dyb, dyi = _int_bf16(rng, (M, N), -4, 4)
    dX, dA, dB = O.lora_linear_backward_ref(xb, Wb, Ab, Bb, s, dyb)
    L0 = _frac_loss(xi, Wi, Ai, Bi, s, dyi)
    for m in range(M):
        for k in range(K):
            x2 = xi.copy()
            x2[m, k] += 1
            assert dX[m, k] == float(_frac_loss(x2, Wi, Ai, Bi, s, dyi) - L0)
    for j in range(r):
        for k in range(K):
            a2 = Ai.copy()
            a2[j, k] += 1
            assert dA[j, k] == float(_frac_loss(xi, Wi, a2, Bi, s, dyi) - L0)
    for n in range(N):
        for j in range(r):
            b2 = Bi.copy()
            b2[n, j] += 1
            assert dB[n, j] == float(_frac_loss(xi, Wi, Ai, b2, s, dyi) - L0)


def test_lora_backward_b_zero_and_shapes():
    """B = 0 (LoRA's zero init): dX is the base gradient dY W and dA vanishes, while dB does not."""
    c = gen_linear(60, M=9, K=64, N=40, r=8, s=2.0)
    rng = np.random.default_rng(1)
    dy = rng.standard_normal((9, 40))
    dX, dA, dB = O.lora_linear_backward_ref(c.x, c.W, c.A, np.zeros_like(c.B), c.s, dy)
    np.testing.assert_allclose(dX, dy @ O.bf16_to_f64(c.W), rtol=1e-13, atol=1e-13)
    assert np.all(dA == 0.0) and np.abs(dB).max() > 0
    assert dX.shape == (9, 64) and dA.shape == (8, 64) and dB.shape == (40, 8)


def _mut_bwd_db_from_swapped_factors(x, W, A, B, s, dy):
    # dB from the LoRA-down product of dY instead of X: s dY^T (dY B) is the wrong chain
    dX, dA, _ = O.lora_linear_backward_ref(x, W, A, B, s, dy)
    dYd = O.bf16_to_f64(dy)
    return dX, dA, s * dYd.T @ (dYd @ O.bf16_to_f64(B))


def _mut_bwd_missing_scale(x, W, A, B, s, dy):
    return O.lora_linear_backward_ref(x, W, A, B, 1.0, dy)


def _mut_bwd_lora_dx_dropped(x, W, A, B, s, dy):
    dX, dA, dB = O.lora_linear_backward_ref(x, W, A, B, s, dy)
    base, _, _ = O.lora_linear_backward_ref(x, W, A, np.zeros_like(B), s, dy)
    return base, dA, dB


@pytest.mark.parametrize("mut", [_mut_bwd_db_from_swapped_factors, _mut_bwd_missing_scale, _mut_bwd_lora_dx_dropped])
def test_pins_catch_backward_mutations(mut):
    rng = np.random.default_rng(77)
    M, K, N, r, s = 2, 8, 3, 2, 2.0
    xb, xi = _int_bf16(rng, (M, K), -4, 4)
    Wb, Wi = _int_bf16(rng, (N, K), -4, 4)
    Ab, Ai = _int_bf16(rng, (r, K), -4, 4)
    Bb, Bi = _int_bf16(rng, (N, r), -4, 4)
    dyb, dyi = _int_bf16(rng, (M, N), -4, 4)
    L0 = _frac_loss(xi, Wi, Ai, Bi, s, dyi)
    dX, dA, dB = mut(xb, Wb, Ab, Bb, s, dyb)
    ok = True
    for (m, k) in [(0, 0), (1, 5)]:
        x2 = xi.copy()
        x2[m, k] += 1
        ok &= dX[m, k] == float(_frac_loss(x2, Wi, Ai, Bi, s, dyi) - L0)
    for (j, k) in [(0, 1), (1, 7)]:
        a2 = Ai.copy()
        a2[j, k] += 1
        ok &= dA[j, k] == float(_frac_loss(xi, Wi, a2, Bi, s, dyi) - L0)
    for (n, j) in [(0, 0), (2, 1)]:
        b2 = Bi.copy()
        b2[n, j] += 1
        ok &= dB[n, j] == float(_frac_loss(xi, Wi, Ai, b2, s, dyi) - L0)
    assert not ok


# ---------------------------------------------------------------- log-softmax / gather

def test_log_softmax_rows_normalise():
    z = np.random.default_rng(1).normal(0, 2, (7, 1000))
    ids = np.arange(7, dtype=np.int32)
    _, lse = O.log_softmax_gather_ref(z, ids)
    for i in range(7):
        assert abs(np.exp(z[i] - lse[i]).sum() - 1.0) < 1e-12


def test_log_softmax_uniform_row_closed_form():
    V = 32000
    z = np.zeros((2, V))
    z[1] += 3.5
    lp, lse = O.log_softmax_gather_ref(z, np.array([5, V - 1], dtype=np.int32))
    assert lp[0] == -math.log(V)
    assert abs(lp[1] + 10.373491181781864) < 1e-12
    assert abs(lse[1] - (3.5 + math.log(V))) < 1e-12


def test_log_softmax_two_class_closed_form():
    rng = np.random.default_rng(2)
    z = rng.normal(0, 3, (50, 2))
    lp0, _ = O.log_softmax_gather_ref(z, np.zeros(50, np.int32))
    lp1, _ = O.log_softmax_gather_ref(z, np.ones(50, np.int32))
    assert np.allclose(lp0, -np.log1p(np.exp(z[:, 1] - z[:, 0])), rtol=0, atol=1e-13)
    assert np.allclose(lp1, -np.log1p(np.exp(z[:, 0] - z[:, 1])), rtol=0, atol=1e-13)


def test_log_softmax_shift_invariance_and_overflow():
    rng = np.random.default_rng(3)
    z = rng.normal(0, 2, (4, 500))
    ids = rng.integers(0, 500, 4).astype(np.int32)
    lp, _ = O.log_softmax_gather_ref(z, ids)
    lp2, _ = O.log_softmax_gather_ref(z + 1234.5, ids)
    assert np.allclose(lp, lp2, rtol=0, atol=1e-9)
    big = np.zeros((2, 100))
    big[:, 7] = 1e4
    lpb, _ = O.log_softmax_gather_ref(big, np.array([7, 8], np.int32))
    assert lpb[0] == 0.0 and lpb[1] == -1e4


def test_log_softmax_matches_torch_float64():
    torch = pytest.importorskip("torch")
    z = np.random.default_rng(4).normal(0, 2, (16, 32000))
    ids = np.random.default_rng(5).integers(0, 32000, 16).astype(np.int32)
    lp, _ = O.log_softmax_gather_ref(z, ids)
    ref = torch.log_softmax(torch.from_numpy(z), dim=1)[torch.arange(16), torch.from_numpy(ids).long()].numpy()
    assert np.max(np.abs(lp - ref)) < 1e-12


def test_log_softmax_matches_scipy_logsumexp():
    scipy_special = pytest.importorskip("scipy.special")
    z = np.random.default_rng(6).normal(0, 2, (8, 4000))
    _, lse = O.log_softmax_gather_ref(z, np.zeros(8, np.int32))
    assert np.max(np.abs(lse - scipy_special.logsumexp(z, axis=1))) < 1e-12


def test_log_softmax_out_of_range_token_is_nan():
    z = np.zeros((3, 10))
    lp, _ = O.log_softmax_gather_ref(z, np.array([-1, 10, 3], np.int32))
    assert math.isnan(lp[0]) and math.isnan(lp[1]) and not math.isnan(lp[2])


# ---------------------------------------------------------------- KL

def test_kl_zero_when_lora_off_for_both():
    on, off, ids = gen_logits(20, M=6, V=3000)
    r = O.score_logits_ref(off, off, ids)
    assert np.all(r["kl"] == 0.0)
    c = gen_score_head(21, 2, 4, 64, 300, 4)
    rr = O.score_head_ref(c.h, c.W_lm, c.A, np.zeros_like(c.B), c.s, c.ids)
    assert np.all(rr["kl"] == 0.0)


def test_kl_antisymmetric_and_shift_free():
    on, off, ids = gen_logits(22, M=6, V=3000)
    a = O.score_logits_ref(on, off, ids)
    b = O.score_logits_ref(off, on, ids)
    assert np.array_equal(a["kl"], -b["kl"])
    shift = np.arange(6, dtype=np.float64)[:, None] * 3.25
    c = O.score_logits_ref(on.astype(np.float64) + shift, on, ids)
    assert np.max(np.abs(c["kl"])) < 1e-12


def test_kl_sign_follows_sampled_token_logit():
    """Raising only the sampled token's logit raises lp_on, so KL = lp_on - lp_off > 0."""
    V = 50
    off = np.zeros((3, V))
    ids = np.array([1, 2, 3], np.int32)
    on = off.copy()
    on[np.arange(3), ids] += 1.0
    r = O.score_logits_ref(on, off, ids)
    expect = 1.0 - math.log((V - 1 + math.e) / V)
    assert np.allclose(r["kl"], expect, rtol=0, atol=1e-13)


# ---------------------------------------------------------------- reward head and composition

def test_reward_exact_bruteforce():
    rng = np.random.default_rng(30)
    n_seq, seq_len, K = 3, 4, 16
    h, hi = _int_bf16(rng, (n_seq * seq_len, K))
    w, wi = _int_bf16(rng, (K,))
    got = O.reward_ref(h, w, n_seq, seq_len)
    for b in range(n_seq):
        row = b * seq_len + seq_len - 1
        assert Fraction(got[b]) == sum(Fraction(int(hi[row, k])) * int(wi[k]) for k in range(K))


def test_reward_equals_lora_off_linear_with_one_output():
    c = gen_score_head(31, 3, 5, 64, 100, 4)
    rew = O.reward_ref(c.h, c.w_rm, 3, 5)
    last = np.array([b * 5 + 4 for b in range(3)])
    y_off, _ = O.lora_linear_ref(c.h[last], c.w_rm[None, :], np.zeros((0, 64), np.uint16),
                                 np.zeros((1, 0), np.uint16), 0.0)
    assert np.allclose(rew, y_off[:, 0], rtol=1e-14, atol=0)


def test_score_head_is_linear_then_log_softmax():
    c = gen_score_head(32, 2, 8, 64, 500, 8)
    r = O.score_head_ref(c.h, c.W_lm, c.A, c.B, c.s, c.ids, c.w_rm, 2, 8)
    z_off, z_on = O.lora_linear_ref(c.h, c.W_lm, c.A, c.B, c.s)
    r2 = O.score_logits_ref(z_on, z_off, c.ids)
    for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off"):
        assert np.array_equal(r[k], r2[k])
    assert r["reward"].shape == (2,)
    sub = np.array([3, 7, 15])
    rs = O.score_head_ref(c.h[sub], c.W_lm, c.A, c.B, c.s, c.ids[sub], c.w_rm, 2, 8, rows=sub)
    assert np.allclose(rs["lp_on"], r["lp_on"][sub], rtol=0, atol=1e-12)
    assert np.allclose(rs["reward"], r["reward"], rtol=0, atol=0)


# ---------------------------------------------------------------- two-input scoring head

def _two_input_case(seed, n_seq=2, seq_len=3, K=8, V=6, r=2):
    rng = np.random.default_rng(seed)
    M = n_seq * seq_len
    h_act = _int_bf16(rng, (M, K), -3, 3)
    h_off = _int_bf16(rng, (M, K), -3, 3)
    W = _int_bf16(rng, (V, K), -2, 2)
    A = _int_bf16(rng, (r, K), -2, 2)
    B = _int_bf16(rng, (V, r), -2, 2)
    w = _int_bf16(rng, (K,))
    ids = rng.integers(0, V, size=M)
    return h_act, h_off, W, A, B, w, ids, n_seq, seq_len


def _two_input_pins_hold(fn):
    """True when fn matches the brute force: exact Fraction logits of each pass from its own input (LoRA on the
    actor pass only), the log-softmax of each row from math.fsum over those exact logits, the exact reward from
    the LoRA-off input's last rows."""
    s = 0.5
    for seed in (51, 52):
        h_act, h_off, W, A, B, w, ids, n_seq, seq_len = _two_input_case(seed)
        res = fn(h_act[0], h_off[0], W[0], A[0], B[0], s, ids, w[0], n_seq, seq_len)
        _, z_on = _frac_lora(h_act[1], W[1], A[1], B[1], s)
        z_off, _ = _frac_lora(h_off[1], W[1], A[1], B[1], s)
        for i in range(len(ids)):
            for z, key in ((z_on, "on"), (z_off, "off")):
                row = [float(v) for v in z[i]]
                m = max(row)
                lse = m + math.log(math.fsum(math.exp(v - m) for v in row))
                if abs(res["lse_" + key][i] - lse) > 1e-12 or abs(res["lp_" + key][i] - (row[ids[i]] - lse)) > 1e-12:
                    return False
            if abs(res["kl"][i] - (res["lp_on"][i] - res["lp_off"][i])) > 0:
                return False
        for b in range(n_seq):
            last = b * seq_len + seq_len - 1
            if Fraction(res["reward"][b]) != sum(Fraction(int(h_off[1][last, k])) * int(w[1][k]) for k in range(8)):
                return False
    return True


def test_score_two_input_bruteforce():
    """The actor pass's logits come from h_act with the head's LoRA, the reference logits and the reward from h_off
    without it (App. A, Alg. 2): exact per-pass brute force."""
    assert _two_input_pins_hold(O.score_head_two_input_ref)


def test_score_two_input_equal_inputs_is_the_one_input_head():
    """With h_act == h_off the two-input head is the one-input head of score_head_ref."""
    c = gen_score_head(53, 2, 8, 64, 500, 8)
    a = O.score_head_two_input_ref(c.h, c.h, c.W_lm, c.A, c.B, c.s, c.ids, c.w_rm, 2, 8)
    b = O.score_head_ref(c.h, c.W_lm, c.A, c.B, c.s, c.ids, c.w_rm, 2, 8)
    for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off", "reward"):
        assert np.array_equal(a[k], b[k]), k


def _mut_two_lora_on_off_pass(h_act, h_off, W, A, B, s, ids, w, n_seq, seq_len):
    _, z_on = O.lora_linear_ref(h_act, W, A, B, s)
    _, z_off = O.lora_linear_ref(h_off, W, A, B, s)
    res = O.score_logits_ref(z_on, z_off, ids)
    res["reward"] = O.reward_ref(h_off, w, n_seq, seq_len)
    return res


def _mut_two_swapped_inputs(h_act, h_off, W, A, B, s, ids, w, n_seq, seq_len):
    return O.score_head_two_input_ref(h_off, h_act, W, A, B, s, ids, w, n_seq, seq_len)


def _mut_two_reward_from_actor(h_act, h_off, W, A, B, s, ids, w, n_seq, seq_len):
    res = O.score_head_two_input_ref(h_act, h_off, W, A, B, s, ids, w, n_seq, seq_len)
    res["reward"] = O.reward_ref(h_act, w, n_seq, seq_len)
    return res


def _mut_two_one_input(h_act, h_off, W, A, B, s, ids, w, n_seq, seq_len):
    return O.score_head_ref(h_act, W, A, B, s, ids, w, n_seq, seq_len)


@pytest.mark.parametrize("mut", [_mut_two_lora_on_off_pass, _mut_two_swapped_inputs, _mut_two_reward_from_actor,
                                 _mut_two_one_input])
def test_pins_catch_two_input_mutations(mut):
    assert not _two_input_pins_hold(mut)


# ---------------------------------------------------------------- mutation checks

def _pins_for_linear(fn):
    """Run the linear pins against ``fn``; return True iff all pass."""
    try:
        rng = np.random.default_rng(5)
        x, xi = _int_bf16(rng, (3, 8))
        W, Wi = _int_bf16(rng, (5, 8))
        A, Ai = _int_bf16(rng, (2, 8))
        B, Bi = _int_bf16(rng, (5, 2))
        y_off, y_on = fn(x, W, A, B, 2.0)
        e_off, e_on = _frac_lora(xi, Wi, Ai, Bi, 2.0)
        ok = all(Fraction(y_off[m, n]) == e_off[m][n] and Fraction(y_on[m, n]) == e_on[m][n]
                 for m in range(3) for n in range(5))
        c = gen_linear(11, M=9, K=32, N=12, r=4, s=2.0)
        X, Wd, Ad, Bd = (O.bf16_to_f64(t) for t in (c.x, c.W, c.A, c.B))
        _, on = fn(c.x, c.W, c.A, c.B, c.s)
        ok = ok and np.allclose(on, X @ (Wd + c.s * Bd @ Ad).T, rtol=1e-12, atol=1e-12)
        return bool(ok)
    except Exception:
        return False


def _pins_for_logsoftmax(fn):
    try:
        V = 32000
        lp, _ = fn(np.zeros((1, V)), np.array([0], np.int32))
        ok = abs(lp[0] + math.log(V)) < 1e-12
        z = np.random.default_rng(2).normal(0, 3, (20, 2))
        lp0, _ = fn(z, np.zeros(20, np.int32))
        ok = ok and np.allclose(lp0, -np.log1p(np.exp(z[:, 1] - z[:, 0])), atol=1e-12, rtol=0)
        big = np.zeros((1, 10))
        big[0, 3] = 1e4
        lpb, _ = fn(big, np.array([3], np.int32))
        ok = ok and lpb[0] == 0.0
        return bool(ok)
    except Exception:
        return False


def test_pins_accept_the_oracle():
    assert _pins_for_linear(O.lora_linear_ref)
    assert _pins_for_logsoftmax(O.log_softmax_gather_ref)


def _mut_no_scale(x, W, A, B, s):
    X, Wd, Ad, Bd = (O.bf16_to_f64(t) for t in (x, W, A, B))
    return X @ Wd.T, X @ Wd.T + (X @ Ad.T) @ Bd.T


def _mut_transposed_b(x, W, A, B, s):
    X, Wd, Ad, Bd = (O.bf16_to_f64(t) for t in (x, W, A, B))
    Bt = Bd.reshape(Bd.shape[1], Bd.shape[0]).T          # wrong memory order for B
    return X @ Wd.T, X @ Wd.T + s * (X @ Ad.T) @ Bt.T


def _mut_dropped_base(x, W, A, B, s):
    X, Wd, Ad, Bd = (O.bf16_to_f64(t) for t in (x, W, A, B))
    return X @ Wd.T, s * (X @ Ad.T) @ Bd.T


def _mut_w_reshaped(x, W, A, B, s):
    X, Wd, Ad, Bd = (O.bf16_to_f64(t) for t in (x, W, A, B))
    Wt = Wd.reshape(Wd.shape[1], Wd.shape[0]).T          # W read as [K x N]
    return X @ Wt.T if Wt.shape[1] == X.shape[1] else X @ Wd.T * 0, None


@pytest.mark.parametrize("mut", [_mut_no_scale, _mut_transposed_b, _mut_dropped_base, _mut_w_reshaped])
def test_pins_catch_linear_mutations(mut):
    assert not _pins_for_linear(mut)


def _mut_lse_without_max(z, ids):
    z = np.asarray(z, np.float64)
    with np.errstate(over="ignore"):
        lse = np.log(np.exp(z).sum(1))
    return z[np.arange(len(ids)), ids] - lse, lse


def _mut_lse_missing_max_term(z, ids):
    z = np.asarray(z, np.float64)
    m = z.max(1, keepdims=True)
    lse = np.log(np.exp(z - m).sum(1))                   # forgot "+ m"
    return z[np.arange(len(ids)), ids] - lse, lse


def _mut_wrong_sign(z, ids):
    lp, lse = O.log_softmax_gather_ref(z, ids)
    return -lp, lse


def _mut_off_by_one_token(z, ids):
    return O.log_softmax_gather_ref(z, (np.asarray(ids) + 1) % np.asarray(z).shape[1])


@pytest.mark.parametrize("mut", [_mut_lse_without_max, _mut_lse_missing_max_term, _mut_wrong_sign, _mut_off_by_one_token])
def test_pins_catch_log_softmax_mutations(mut):
    assert not _pins_for_logsoftmax(mut)
