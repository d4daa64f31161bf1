"""GPU parity of hydra_value_head, hydra_ppo_advantages and hydra_ppo_loss against the float64 oracle."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import gae_ref, ppo_loss_ref, ppo_rewards_ref, value_head_ref
from gpu_helpers import assert_rel, dev_bf16, host, say

pytestmark = pytest.mark.gpu


def _vals(h, w, device):
    import torch
    M = h.shape[0]
    out = torch.full((M,), float("nan"), device=device)
    H.hydra_value_head(dev_bf16(h, device), dev_bf16(w, device), out)
    torch.cuda.synchronize()
    return host(out)


@pytest.mark.parametrize("M,K", [(1, 8), (5, 520), (300, 4104), (33, 12288)])
def test_value_head_matches_oracle(M, K, dev):
    say("value_head", M, K)
    c = WL.gen_advantages(4000 + M + K, 1, M, K)
    got = _vals(c.h, c.w_v, dev)
    assert_rel(got, value_head_ref(c.h, c.w_v), "values")


def _adv(kl, reward, values, n_seq, T, start, beta, gamma, lam, device, with_rewards=True):
    import torch
    M = n_seq * T
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    adv = torch.full((M,), float("nan"), device=device)
    ret = torch.full((M,), float("nan"), device=device)
    rew = torch.full((M,), float("nan"), device=device) if with_rewards else None
    H.hydra_ppo_advantages(t(kl), t(reward), t(values), n_seq, T, adv, ret, rewards=rew, start=start,
                           beta=beta, gamma=gamma, lam=lam)
    torch.cuda.synchronize()
    return host(adv), host(ret), (host(rew) if with_rewards else None)


CASES = [
    # (n_seq, seq_len, start, gamma, lam): one token, lanes left empty (T < 64), ragged chunks,
    # long sequences, the prompt mask, lambda = 0 and 1, a discount below 1.
    (1, 1, 0, 1.0, 0.95), (3, 7, 0, 1.0, 0.95), (2, 100, 37, 1.0, 0.95), (4, 512, 0, 1.0, 0.95),
    (4, 512, 256, 1.0, 0.95), (1, 5000, 17, 0.99, 0.95), (33, 65, 64, 0.9, 0.0), (5, 130, 3, 1.0, 1.0),
]


@pytest.mark.parametrize("n_seq,T,start,gamma,lam", CASES)
def test_advantages_match_oracle(n_seq, T, start, gamma, lam, dev):
    say("ppo_advantages", dict(n_seq=n_seq, T=T, start=start, gamma=gamma, lam=lam))
    rng = np.random.default_rng(5000 + n_seq * T + start)
    kl = (rng.standard_normal(n_seq * T) * 0.1).astype(np.float32)
    reward = rng.standard_normal(n_seq).astype(np.float32)
    values = rng.standard_normal(n_seq * T).astype(np.float32)
    beta = 0.02
    adv, ret, rew = _adv(kl, reward, values, n_seq, T, start, beta, gamma, lam, dev)
    e_rew = ppo_rewards_ref(kl, reward, n_seq, T, start, beta)
    e_adv, e_ret = gae_ref(e_rew, values, n_seq, T, start, gamma, lam)
    assert_rel(rew, e_rew, "rewards")
    assert_rel(adv, e_adv, "advantages")
    assert_rel(ret, e_ret, "returns")
    prompt = (np.arange(n_seq * T) % T) < start
    assert np.all(adv[prompt] == 0) and np.all(ret[prompt] == 0) and np.all(rew[prompt] == 0)


def test_advantages_optional_rewards_and_determinism(dev):
    say("ppo_advantages determinism")
    rng = np.random.default_rng(77)
    kl = (rng.standard_normal(3 * 300) * 0.1).astype(np.float32)
    reward = rng.standard_normal(3).astype(np.float32)
    values = rng.standard_normal(3 * 300).astype(np.float32)
    a1, r1, _ = _adv(kl, reward, values, 3, 300, 10, 0.02, 1.0, 0.95, dev)
    a2, r2, _ = _adv(kl, reward, values, 3, 300, 10, 0.02, 1.0, 0.95, dev, with_rewards=False)
    assert np.array_equal(a1, a2) and np.array_equal(r1, r2)


def test_advantage_step_full_workload(dev):
    """4 sequences x 512 tokens, K = 4096: the critic value head on every row, then the rewards, advantages
    and returns, each checked on every token."""
    import torch
    c = WL.make("ppo_advantages")
    say("ppo_advantages full", c.n_seq, c.seq_len, c.K)
    vals = _vals(c.h, c.w_v, dev)
    e_vals = value_head_ref(c.h, c.w_v)
    assert_rel(vals, e_vals, "values")
    adv, ret, rew = _adv(c.kl, c.reward, vals, c.n_seq, c.seq_len, c.start, c.beta, c.gamma, c.lam, dev)
    e_rew = ppo_rewards_ref(c.kl, c.reward, c.n_seq, c.seq_len, c.start, c.beta)
    e_adv, e_ret = gae_ref(e_rew, e_vals, c.n_seq, c.seq_len, c.start, c.gamma, c.lam)
    assert_rel(rew, e_rew, "rewards")
    assert_rel(adv, e_adv, "advantages")
    assert_rel(ret, e_ret, "returns")


# ---------------------------------------------------------------- PPO losses
def _loss_inputs(seed, n_seq, T):
    rng = np.random.default_rng(seed)
    M = n_seq * T
    lp_old = -rng.uniform(0.5, 6.0, M).astype(np.float32)
    lp_new = (lp_old + rng.normal(0, 0.3, M)).astype(np.float32)
    A = rng.normal(0, 1, M).astype(np.float32)
    V = rng.normal(0, 1, M).astype(np.float32)
    R = (V + rng.normal(0, 0.5, M)).astype(np.float32)
    return lp_new, lp_old, A, V, R


def _run_loss(device, lp_new, lp_old, A, V, R, n_seq, T, start, eps):
    import torch
    t = [torch.from_numpy(np.ascontiguousarray(v)).to(device) for v in (lp_new, lp_old, A, V, R)]
    losses = torch.full((3,), float("nan"), device=device)
    d_lp = torch.full((n_seq * T,), float("nan"), device=device)
    d_v = torch.full((n_seq * T,), float("nan"), device=device)
    H.hydra_ppo_loss(*t, n_seq, T, losses, d_lp, d_v, start=start, eps=eps)
    torch.cuda.synchronize()
    return host(losses), host(d_lp), host(d_v)


@pytest.mark.parametrize("n_seq,T,start,eps", [(4, 512, 0, 0.2), (4, 512, 256, 0.2), (3, 77, 5, 0.1), (1, 1, 0, 0.2),
                                               (5, 3000, 100, 0.3), (2, 64, 10, 0.0)])
def test_ppo_loss_matches_oracle(n_seq, T, start, eps, dev):
    say("ppo_loss", n_seq, T, start, eps)
    lp_new, lp_old, A, V, R = _loss_inputs(n_seq * 1000 + T + start, n_seq, T)
    losses, d_lp, d_v = _run_loss(dev, lp_new, lp_old, A, V, R, n_seq, T, start, eps)
    e = ppo_loss_ref(lp_new, lp_old, A, V, R, n_seq, T, start, eps)
    for i, k in enumerate(("pg_loss", "v_loss")):
        assert abs(losses[i] - e[k]) <= 1e-4 * max(abs(e[k]), 1e-3), (k, losses[i], e[k])
    # the clipped fraction is a count: equal except where fp32 rounding moves rho across a clip bound
    assert abs(losses[2] - e["clip_frac"]) <= 2.0 / (n_seq * (T - start))
    assert_rel(d_lp, e["d_lp"], "d_lp")
    assert_rel(d_v, e["d_v"], "d_v")
    assert np.all(d_lp.reshape(n_seq, T)[:, :start] == 0) and np.all(d_v.reshape(n_seq, T)[:, :start] == 0)


def test_ppo_loss_clip_cases_and_determinism(dev):
    """The four sides of the clip on single-token sequences, and identical bits on a second run."""
    say("ppo_loss clip cases")
    rho = np.array([1.5, 0.5, 0.5, 1.5, 1.0], np.float64)
    A = np.array([1.0, 1.0, -1.0, -1.0, 2.0], np.float32)
    lp_old = np.zeros(5, np.float32)
    lp_new = np.log(rho).astype(np.float32)
    z = np.zeros(5, np.float32)
    losses, d_lp, _ = _run_loss(dev, lp_new, lp_old, A, z, z, 5, 1, 0, 0.2)
    # objective per token: 1.2, 0.5, -0.8, -1.5, 2.0 -> mean 0.28; unclipped gradient where active
    assert abs(losses[0] + 0.28) < 1e-6
    np.testing.assert_allclose(d_lp, [0.0, -0.1, 0.0, 0.3, -0.4], rtol=0, atol=1e-6)
    assert abs(losses[2] - 0.4) < 1e-7
    lp_new, lp_old, A, V, R = _loss_inputs(77, 4, 512)
    a = _run_loss(dev, lp_new, lp_old, A, V, R, 4, 512, 0, 0.2)
    b = _run_loss(dev, lp_new, lp_old, A, V, R, 4, 512, 0, 0.2)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
