"""Pins of the PPO advantage-step oracle (value head, per-token reward, GAE)
against things other than itself: exact rational brute force through the
one-step recursion (the oracle sums the series instead), closed forms for
lambda = 1 and lambda = 0, a geometric series, and planted mistakes."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import ppo_oracle as P
from workloads import f32_to_bf16


def _int_bf16(rng, shape, lo=-6, hi=6):
    v = rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    return f32_to_bf16(v), v.astype(np.int64)


# ---------------------------------------------------------------- value head
@pytest.mark.parametrize("M,K", [(1, 8), (3, 16), (5, 24)])
def test_value_head_exact_bruteforce(M, K):
    rng = np.random.default_rng(M * 100 + K)
    hb, hi = _int_bf16(rng, (M, K))
    wb, wi = _int_bf16(rng, (K,))
    got = P.value_head_ref(hb, wb)
    for m in range(M):
        want = sum(Fraction(int(hi[m, k])) * Fraction(int(wi[k])) for k in range(K))
        assert got[m] == float(want)


# ---------------------------------------------------------------- rewards
def _frac_rewards(kl, reward, n_seq, T, start, beta):
    out = []
    for b in range(n_seq):
        for t in range(T):
            v = Fraction(0)
            if t >= start:
                v -= Fraction(beta) * Fraction(kl[b * T + t])
            if t == T - 1:
                v += Fraction(reward[b])
            out.append(v)
    return out


@pytest.mark.parametrize("start", [0, 2, 4])
def test_rewards_exact(start):
    rng = np.random.default_rng(7 + start)
    n_seq, T = 3, 5
    kl = (rng.integers(-8, 9, n_seq * T) / 8.0).astype(np.float64)
    reward = (rng.integers(-8, 9, n_seq) / 4.0).astype(np.float64)
    beta = 0.25
    got = P.ppo_rewards_ref(kl, reward, n_seq, T, start, beta)
    want = _frac_rewards(kl, reward, n_seq, T, start, beta)
    assert [Fraction(g) for g in got] == want


# ---------------------------------------------------------------- GAE
def _frac_gae(r, V, n_seq, T, start, gamma, lam):
    """Exact rational GAE through the one-step recursion A_t = delta_t + gamma lam A_{t+1}."""
    A = [Fraction(0)] * (n_seq * T)
    R = [Fraction(0)] * (n_seq * T)
    g, c = Fraction(gamma), Fraction(gamma) * Fraction(lam)
    for b in range(n_seq):
        nxt = Fraction(0)
        for t in range(T - 1, -1, -1):
            v = Fraction(V[b * T + t])
            v1 = Fraction(V[b * T + t + 1]) if t + 1 < T else Fraction(0)
            delta = Fraction(r[b * T + t]) + g * v1 - v
            nxt = delta + c * nxt
            if t >= start:
                A[b * T + t] = nxt
                R[b * T + t] = nxt + v
    return A, R


def _small_case(seed, n_seq, T):
    rng = np.random.default_rng(seed)
    r = rng.integers(-16, 17, n_seq * T) / 8.0
    V = rng.integers(-16, 17, n_seq * T) / 4.0
    return r.astype(np.float64), V.astype(np.float64)


@pytest.mark.parametrize("T,start,gamma,lam", [(1, 0, 1.0, 0.95), (5, 0, 1.0, 0.95), (6, 2, 0.75, 0.5),
                                               (4, 3, 1.0, 0.0), (6, 0, 0.5, 1.0)])
def test_gae_matches_exact_recursion(T, start, gamma, lam):
    n_seq = 3
    r, V = _small_case(T * 10 + start, n_seq, T)
    A, R = P.gae_ref(r, V, n_seq, T, start, gamma, lam)
    eA, eR = _frac_gae(r, V, n_seq, T, start, gamma, lam)
    np.testing.assert_allclose(A, [float(x) for x in eA], rtol=0, atol=1e-12)
    np.testing.assert_allclose(R, [float(x) for x in eR], rtol=0, atol=1e-12)


def test_gae_lambda_one_is_return_minus_value():
    rng = np.random.default_rng(11)
    n_seq, T = 2, 40
    r = rng.standard_normal(n_seq * T)
    V = rng.standard_normal(n_seq * T)
    A, R = P.gae_ref(r, V, n_seq, T, 0, 1.0, 1.0)
    rr, VV = r.reshape(n_seq, T), V.reshape(n_seq, T)
    mc = np.cumsum(rr[:, ::-1], axis=1)[:, ::-1]   # sum_{k >= t} r_k
    np.testing.assert_allclose(A.reshape(n_seq, T), mc - VV, rtol=0, atol=1e-11)
    np.testing.assert_allclose(R.reshape(n_seq, T), mc, rtol=0, atol=1e-11)


def test_gae_lambda_zero_is_td_residual():
    rng = np.random.default_rng(12)
    n_seq, T, gamma = 3, 17, 0.9
    r = rng.standard_normal(n_seq * T)
    V = rng.standard_normal(n_seq * T)
    A, _ = P.gae_ref(r, V, n_seq, T, 0, gamma, 0.0)
    rr, VV = r.reshape(n_seq, T), V.reshape(n_seq, T)
    nxt = np.concatenate([VV[:, 1:], np.zeros((n_seq, 1))], axis=1)
    np.testing.assert_allclose(A.reshape(n_seq, T), rr + gamma * nxt - VV, rtol=0, atol=1e-12)


def test_gae_constant_residual_is_geometric():
    n_seq, T, gamma, lam, r0 = 1, 30, 1.0, 0.95, 0.3
    r = np.full(T, r0)
    V = np.zeros(T)
    A, _ = P.gae_ref(r, V, n_seq, T, 0, gamma, lam)
    c = gamma * lam
    t = np.arange(T)
    np.testing.assert_allclose(A, r0 * (1 - c ** (T - t)) / (1 - c), rtol=1e-13, atol=0)


def test_gae_one_step_recursion_holds_and_prompt_is_zero():
    rng = np.random.default_rng(13)
    n_seq, T, start, gamma, lam = 2, 64, 20, 1.0, 0.95
    r = rng.standard_normal(n_seq * T)
    V = rng.standard_normal(n_seq * T)
    A, R = P.gae_ref(r, V, n_seq, T, start, gamma, lam)
    A2, R2, V2, r2 = A.reshape(n_seq, T), R.reshape(n_seq, T), V.reshape(n_seq, T), r.reshape(n_seq, T)
    for t in range(start, T):
        nxt_v = V2[:, t + 1] if t + 1 < T else 0.0
        nxt_a = A2[:, t + 1] if t + 1 < T else 0.0
        np.testing.assert_allclose(A2[:, t] - gamma * lam * nxt_a, r2[:, t] + gamma * nxt_v - V2[:, t], atol=1e-12)
    assert np.all(A2[:, :start] == 0) and np.all(R2[:, :start] == 0)
    np.testing.assert_allclose(R2[:, start:], A2[:, start:] + V2[:, start:], atol=0)


# ---------------------------------------------------------------- planted mistakes
def _pins_for_gae(fn):
    """True when fn passes the pins above (used to show they catch mistakes)."""
    try:
        for T, start, gamma, lam in [(5, 0, 1.0, 0.95), (6, 2, 0.75, 0.5), (6, 0, 0.5, 1.0)]:
            r, V = _small_case(T * 10 + start, 3, T)
            A, R = fn(r, V, 3, T, start, gamma, lam)
            eA, eR = _frac_gae(r, V, 3, T, start, gamma, lam)
            if not np.allclose(A, [float(x) for x in eA], atol=1e-12):
                return False
            if not np.allclose(R, [float(x) for x in eR], atol=1e-12):
                return False
        return True
    except Exception:
        return False


def _mut_lambda_only(r, V, n, T, s, g, lam):
    return P.gae_ref(r, V, n, T, s, g, lam / g if g else lam)   # decay lambda instead of gamma*lambda


def _mut_no_bootstrap(r, V, n, T, s, g, lam):
    return P.gae_ref(r, V, n, T, s, 0.0 * g, lam)                 # drops gamma V_{t+1}


def _mut_sign(r, V, n, T, s, g, lam):
    A, R = P.gae_ref(r, V, n, T, s, g, lam)
    return -A, R


def _mut_returns_without_value(r, V, n, T, s, g, lam):
    A, R = P.gae_ref(r, V, n, T, s, g, lam)
    return A, A


@pytest.mark.parametrize("mut", [_mut_lambda_only, _mut_no_bootstrap, _mut_sign, _mut_returns_without_value])
def test_pins_catch_gae_mutations(mut):
    assert _pins_for_gae(P.gae_ref)
    assert not _pins_for_gae(mut)


# ---------------------------------------------------------------- PPO losses (update stage)
def _loss_case(seed, n_seq=3, T=20, start=5):
    rng = np.random.default_rng(seed)
    M = n_seq * T
    lp_old = -rng.uniform(0.5, 6.0, M)
    lp_new = lp_old + rng.normal(0, 0.3, M)
    A = rng.normal(0, 1, M)
    V = rng.normal(0, 1, M)
    R = V + rng.normal(0, 0.5, M)
    return lp_new, lp_old, A, V, R, n_seq, T, start


def test_ppo_loss_zero_advantage_and_equal_policies():
    lp_new, lp_old, A, V, R, n, T, st = _loss_case(21)
    z = P.ppo_loss_ref(lp_new, lp_old, np.zeros_like(A), V, R, n, T, st, 0.2)
    assert z["pg_loss"] == 0.0 and np.all(z["d_lp"] == 0.0)
    e = P.ppo_loss_ref(lp_old, lp_old, A, V, R, n, T, st, 0.2)   # rho = 1: no clipping, objective = mean A
    mask = (np.arange(n * T) % T) >= st
    cnt = n * (T - st)
    assert abs(e["pg_loss"] + A[mask].sum() / cnt) < 1e-12
    np.testing.assert_allclose(e["d_lp"], np.where(mask, -A / cnt, 0.0), rtol=0, atol=1e-15)
    assert e["clip_frac"] == 0.0


@pytest.mark.parametrize("rho,A,obj,active", [(1.5, 1.0, 1.2, False), (0.5, 1.0, 0.5, True),
                                              (0.5, -1.0, -0.8, False), (1.5, -1.0, -1.5, True),
                                              (1.1, 2.0, 2.2, True), (0.9, -3.0, -2.7, True)])
def test_ppo_loss_clip_cases_closed_form(rho, A, obj, active):
    """One response token: the objective is the textbook min of the plain and clipped terms (eps = 0.2)."""
    out = P.ppo_loss_ref([np.log(rho)], [0.0], [A], [0.0], [0.0], 1, 1, 0, 0.2)
    assert abs(out["pg_loss"] + obj) < 1e-12
    assert abs(out["d_lp"][0] - (-rho * A if active else 0.0)) < 1e-12
    assert out["clip_frac"] == (0.0 if active else 1.0)


def test_ppo_loss_gradients_match_finite_differences():
    lp_new, lp_old, A, V, R, n, T, st = _loss_case(22)
    base = P.ppo_loss_ref(lp_new, lp_old, A, V, R, n, T, st, 0.2)
    h = 1e-6
    rng = np.random.default_rng(0)
    for t in rng.choice(n * T, 25, replace=False):
        rho = np.exp(lp_new[t] - lp_old[t])
        if abs(rho - 0.8) < 1e-4 or abs(rho - 1.2) < 1e-4:
            continue   # a kink of the clip
        up, dn = lp_new.copy(), lp_new.copy()
        up[t] += h
        dn[t] -= h
        fd = (P.ppo_loss_ref(up, lp_old, A, V, R, n, T, st, 0.2)["pg_loss"] -
              P.ppo_loss_ref(dn, lp_old, A, V, R, n, T, st, 0.2)["pg_loss"]) / (2 * h)
        assert abs(fd - base["d_lp"][t]) < 1e-7
        vu, vd = V.copy(), V.copy()
        vu[t] += h
        vd[t] -= h
        fdv = (P.ppo_loss_ref(lp_new, lp_old, A, vu, R, n, T, st, 0.2)["v_loss"] -
               P.ppo_loss_ref(lp_new, lp_old, A, vd, R, n, T, st, 0.2)["v_loss"]) / (2 * h)
        assert abs(fdv - base["d_v"][t]) < 1e-7


def test_ppo_value_loss_closed_form_and_prompt_mask():
    lp_new, lp_old, A, V, R, n, T, st = _loss_case(23)
    out = P.ppo_loss_ref(lp_new, lp_old, A, V, R, n, T, st, 0.2)
    resp = np.concatenate([np.arange(b * T + st, (b + 1) * T) for b in range(n)])
    assert abs(out["v_loss"] - 0.5 * np.mean((V[resp] - R[resp]) ** 2)) < 1e-13
    prompt = np.setdiff1d(np.arange(n * T), resp)
    assert np.all(out["d_lp"][prompt] == 0.0) and np.all(out["d_v"][prompt] == 0.0)


def _loss_pins_hold(fn):
    try:
        for rho, A, obj, active in [(1.5, 1.0, 1.2, False), (0.5, 1.0, 0.5, True), (0.5, -1.0, -0.8, False),
                                    (1.5, -1.0, -1.5, True)]:
            out = fn([np.log(rho)], [0.0], [A], [0.0], [0.0], 1, 1, 0, 0.2)
            if abs(out["pg_loss"] + obj) > 1e-12 or abs(out["d_lp"][0] - (-rho * A if active else 0.0)) > 1e-12:
                return False
        lp_new, lp_old, A, V, R, n, T, st = _loss_case(24)
        out = fn(lp_new, lp_old, A, V, R, n, T, st, 0.2)
        ref = P.ppo_loss_ref(lp_new, lp_old, A, V, R, n, T, st, 0.2)
        resp = np.concatenate([np.arange(b * T + st, (b + 1) * T) for b in range(n)])
        return abs(out["v_loss"] - 0.5 * np.mean((V[resp] - R[resp]) ** 2)) < 1e-13 and \
            abs(out["pg_loss"] - ref["pg_loss"]) < 1e-13
    except Exception:
        return False


def _mut_max_instead_of_min(ln, lo, A, V, R, n, T, st, eps):
    out = P.ppo_loss_ref(ln, lo, A, V, R, n, T, st, eps)
    rho = np.exp(np.asarray(ln, float) - np.asarray(lo, float))
    A = np.asarray(A, float)
    obj = np.maximum(rho * A, np.clip(rho, 1 - eps, 1 + eps) * A)
    mask = (np.arange(len(A)) % T) >= st
    out["pg_loss"] = -obj[mask].sum() / (n * (T - st))
    return out


def _mut_swapped_clip_bounds(ln, lo, A, V, R, n, T, st, eps):
    return P.ppo_loss_ref(ln, lo, A, V, R, n, T, st, -eps)


def _mut_mean_over_all_tokens(ln, lo, A, V, R, n, T, st, eps):
    return P.ppo_loss_ref(ln, lo, A, V, R, n, T, 0, eps)


def _mut_inverse_ratio(ln, lo, A, V, R, n, T, st, eps):
    return P.ppo_loss_ref(lo, ln, A, V, R, n, T, st, eps)


@pytest.mark.parametrize("mut", [_mut_max_instead_of_min, _mut_swapped_clip_bounds, _mut_mean_over_all_tokens,
                                 _mut_inverse_ratio])
def test_pins_catch_ppo_loss_mutations(mut):
    assert _loss_pins_hold(P.ppo_loss_ref)
    assert not _loss_pins_hold(mut)
