"""A seeded sweep of shapes over every GPU entry point against the float64 oracle: row counts from one row to several
row tiles, ragged K and N, every rank class (0, odd ranks, each padded rank and its neighbours), vocabularies from
one column upward.  The shapes are drawn once from a fixed seed, so every run checks the same cases and a failure
names its shape.  Covered: the single, workspace, grouped and multi-input linears, the fused scoring pass, the
epilogue over logits, the backward with the transpose, the value head with the advantage step, and the PPO losses."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import (gae_ref, lora_linear_backward_ref, lora_linear_multi_ref, lora_linear_ref, ppo_loss_ref,
                    ppo_rewards_ref, score_head_ref, score_logits_ref, value_head_ref)
from gpu_helpers import assert_abs, assert_rel, dev_bf16, host, say
from gpu_helpers import dev as to_dev

pytestmark = pytest.mark.gpu

RANKS = [0, 1, 7, 15, 16, 17, 31, 32, 33, 63, 64, 65, 100, 127, 128]
_rng = np.random.Generator(np.random.PCG64(20230901))


def _rows(lo=1, hi=600):
    return int(np.exp(_rng.uniform(np.log(lo), np.log(hi + 1)))) if _rng.random() < 0.8 else int(_rng.integers(1, 17))


def _mult8(lo, hi):
    return 8 * int(_rng.integers(max(1, lo // 8), hi // 8 + 1))


LINEAR = [(_rows(), _mult8(8, 3000), int(_rng.integers(1, 1500)), int(_rng.choice(RANKS))) for _ in range(30)]
SCORE = [(int(_rng.integers(1, 6)), int(_rng.integers(1, 131)), _mult8(8, 1024), int(_rng.integers(1, 3001)),
          int(_rng.choice(RANKS))) for _ in range(12)]
BACKWARD = [(_rows(), _mult8(8, 2000), _mult8(8, 1200), int(_rng.choice(RANKS))) for _ in range(12)]
LOGITS = [(int(_rng.integers(1, 65)), int(_rng.integers(1, 5001))) for _ in range(8)]


def _rank_for(M):
    # above 16 rows the no-workspace calls take ranks up to 64 (a larger rank asks for the workspace call)
    r = int(_rng.choice(RANKS))
    return r if M <= 16 or r <= 64 else int(_rng.choice([v for v in RANKS if v <= 64]))


GROUP = []
for _ in range(6):
    _M = _rows(1, 300)
    GROUP.append((int(_rng.integers(1, 9)), _M, _mult8(8, 1500), int(_rng.integers(1, 700)), _rank_for(_M)))
MULTI = []
for _ in range(6):
    _M = _rows(1, 300)
    MULTI.append((_M, _mult8(8, 1500), int(_rng.integers(1, 700)), _rank_for(_M), int(_rng.integers(0, 5)),
                  bool(_rng.random() < 0.7)))
ADVANTAGE = []
for _ in range(6):
    _T = int(_rng.integers(1, 701))
    ADVANTAGE.append((int(_rng.integers(1, 7)), _T, _mult8(8, 2048), int(_rng.integers(0, _T)),
                      float(_rng.choice([1.0, 0.99])), float(_rng.choice([0.0, 0.95, 1.0]))))
LOSS = []
for _ in range(6):
    _T = int(_rng.integers(1, 1500))
    LOSS.append((int(_rng.integers(1, 7)), _T, int(_rng.integers(0, _T)), float(_rng.choice([0.1, 0.2, 0.3]))))


@pytest.mark.parametrize("M,K,N,r", LINEAR)
def test_linear_sweep(M, K, N, r, dev):
    import torch
    say("sweep linear", M, K, N, r)
    c = WL.gen_linear(5000 + M * 7 + K + N + r, M, K, N, r)
    x, W = dev_bf16(c.x, dev), dev_bf16(c.W, dev)
    A = dev_bf16(c.A, dev) if r else None
    B = dev_bf16(c.B, dev) if r else None
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    nan = float("nan")
    plain_ok = M <= 16 or r <= 64  # above, the in-tile update does not fit: hydra_lora_linear asks for a workspace
    if plain_ok:
        y_off, y_on = torch.full((M, N), nan, device=dev), torch.full((M, N), nan, device=dev)
        H.hydra_lora_linear(x, W, A, B, c.s, y_off, y_on)
        torch.cuda.synchronize()
        assert_rel(host(y_off), e_off, "y_off")
        assert_rel(host(y_on), e_on, "y_on")
    else:
        with pytest.raises(H.HydraError):
            H.hydra_lora_linear(x, W, A, B, c.s, torch.empty((M, N), device=dev), torch.empty((M, N), device=dev))
    y_off, y_on = torch.full((M, N), nan, device=dev), torch.full((M, N), nan, device=dev)
    H.hydra_lora_linear_ws(x, W, A, B, c.s, y_off, y_on)
    torch.cuda.synchronize()
    assert_rel(host(y_off), e_off, "ws y_off")
    assert_rel(host(y_on), e_on, "ws y_on")


@pytest.mark.parametrize("n_seq,seq_len,K,V,r", SCORE)
def test_score_sweep(n_seq, seq_len, K, V, r, dev):
    import torch
    say("sweep score", n_seq, seq_len, K, V, r)
    s = WL.gen_score_head(6000 + n_seq * seq_len + K + V + r, n_seq, seq_len, K, V, r)
    A = dev_bf16(s.A, dev) if r else None
    B = dev_bf16(s.B, dev) if r else None
    out = {k: torch.full((s.M,), float("nan"), device=dev) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
    reward = torch.full((s.n_seq,), float("nan"), device=dev)
    H.hydra_score(dev_bf16(s.h, dev), dev_bf16(s.W_lm, dev), A, B, s.s, torch.from_numpy(s.ids).to(dev),
                  dev_bf16(s.w_rm, dev), s.n_seq, s.seq_len, out["lp_on"], out["lp_off"], out["kl"], reward=reward,
                  lse_on=out["lse_on"], lse_off=out["lse_off"])
    torch.cuda.synchronize()
    e = score_head_ref(s.h, s.W_lm, s.A, s.B, s.s, s.ids, s.w_rm, s.n_seq, s.seq_len)
    for k, v in out.items():
        assert_abs(host(v), e[k], k)
    assert_rel(host(reward), e["reward"], "reward")


@pytest.mark.parametrize("M,K,N,r", BACKWARD)
def test_backward_sweep(M, K, N, r, dev):
    import torch
    say("sweep backward", M, K, N, r)
    case = WL.gen_backward(7000 + M * 3 + K + N + r, M, K, N, r)
    c = case.lin
    x, dy = dev_bf16(c.x, dev), dev_bf16(case.dy, dev)
    A = dev_bf16(c.A, dev) if r else None
    B = dev_bf16(c.B, dev) if r else None
    Wd = dev_bf16(c.W, dev)
    Wt = torch.empty((K, N), dtype=Wd.dtype, device=dev)
    H.hydra_transpose_bf16(Wd, Wt)
    nan = float("nan")
    dx = torch.full((M, K), nan, device=dev)
    dA = torch.full((r, K), nan, device=dev) if r else None
    dB = torch.full((N, r), nan, device=dev) if r else None
    H.hydra_lora_linear_backward(x, Wt, A, B, c.s, dy, dx, dA, dB)
    torch.cuda.synchronize()
    e_dx, e_dA, e_dB = lora_linear_backward_ref(c.x, c.W, c.A, c.B, c.s, case.dy)
    assert_rel(host(dx), e_dx, "dx")
    if r:
        assert_rel(host(dA), e_dA, "dA")
        assert_rel(host(dB), e_dB, "dB")


@pytest.mark.parametrize("M,V", LOGITS)
def test_score_logits_sweep(M, V, dev):
    import torch
    say("sweep score_logits", M, V)
    on, off, ids = WL.gen_logits(8000 + M + V, M, V)
    res = {k: torch.full((M,), float("nan"), device=dev) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
    H.hydra_score_logits(to_dev(on, dev), to_dev(off, dev), to_dev(ids.astype(np.int32), dev), res["lp_on"],
                         res["lp_off"], res["kl"], res["lse_on"], res["lse_off"])
    torch.cuda.synchronize()
    e = score_logits_ref(on, off, ids)
    for k, v in res.items():
        assert_abs(host(v), e[k], k)


@pytest.mark.parametrize("G,M,K,N,r", GROUP)
def test_group_sweep(G, M, K, N, r, dev):
    """G linears of one shape in one call, each against the oracle."""
    import torch
    say("sweep group", G, M, K, N, r)
    cs = [WL.gen_linear(9000 + 97 * g + M + K + N + r, M, K, N, r, s=1.0 + 0.5 * g) for g in range(G)]
    nan = float("nan")
    y_offs = [torch.full((M, N), nan, device=dev) for _ in cs]
    y_ons = [torch.full((M, N), nan, device=dev) for _ in cs]
    H.hydra_lora_linear_group([dev_bf16(c.x, dev) for c in cs], [dev_bf16(c.W, dev) for c in cs],
                              [dev_bf16(c.A, dev) if r else None for c in cs],
                              [dev_bf16(c.B, dev) if r else None for c in cs], [c.s for c in cs], y_offs, y_ons)
    torch.cuda.synchronize()
    for g, c in enumerate(cs):
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(host(y_offs[g]), e_off, f"y_off[{g}]")
        assert_rel(host(y_ons[g]), e_on, f"y_on[{g}]")


@pytest.mark.parametrize("M,K,N,r,n_on,with_off", MULTI)
def test_multi_sweep(M, K, N, r, n_on, with_off, dev):
    """One W for a LoRA-off input and n_on LoRA-on inputs with their own adapters."""
    import torch
    if n_on == 0 and not with_off:
        with_off = True
    say("sweep multi", M, K, N, r, n_on, with_off)
    c = WL.gen_multi(9500 + M + K + N + r + n_on, M, K, N, r, n_on, with_off, scales=(2.0, -0.5, 1.0, 3.0))
    nan = float("nan")
    y_off = torch.full((M, N), nan, device=dev) if with_off else None
    y_ons = [torch.full((M, N), nan, device=dev) for _ in range(n_on)]
    H.hydra_lora_linear_multi(dev_bf16(c.x_off, dev) if with_off else None, dev_bf16(c.W, dev),
                              [dev_bf16(x, dev) for x in c.x_on], [dev_bf16(a, dev) if r else None for a in c.A],
                              [dev_bf16(b, dev) if r else None for b in c.B], c.s, y_off, y_ons)
    torch.cuda.synchronize()
    e_off, e_ons = lora_linear_multi_ref(c.x_off, c.W, c.x_on, c.A if r else [None] * n_on,
                                         c.B if r else [None] * n_on, c.s)
    if with_off:
        assert_rel(host(y_off), e_off, "y_off")
    for a in range(n_on):
        assert_rel(host(y_ons[a]), e_ons[a], f"y_on[{a}]")


@pytest.mark.parametrize("n_seq,T,K,start,gamma,lam", ADVANTAGE)
def test_advantage_sweep(n_seq, T, K, start, gamma, lam, dev):
    """The value head, then per-token rewards, GAE advantages and returns."""
    import torch
    say("sweep advantages", n_seq, T, K, start, gamma, lam)
    c = WL.gen_advantages(9900 + n_seq * T + K + start, n_seq, T, K, start=start, gamma=gamma, lam=lam)
    M = n_seq * T
    vals = torch.full((M,), float("nan"), device=dev)
    H.hydra_value_head(dev_bf16(c.h, dev), dev_bf16(c.w_v, dev), vals)
    adv, ret, rew = (torch.full((M,), float("nan"), device=dev) for _ in range(3))
    H.hydra_ppo_advantages(to_dev(c.kl, dev), to_dev(c.reward, dev), vals, n_seq, T, adv, ret, rewards=rew,
                           start=start, beta=c.beta, gamma=gamma, lam=lam)
    torch.cuda.synchronize()
    e_vals = value_head_ref(c.h, c.w_v)
    assert_rel(host(vals), e_vals, "values")
    e_rew = ppo_rewards_ref(c.kl, c.reward, n_seq, T, start, c.beta)
    e_adv, e_ret = gae_ref(e_rew, e_vals, n_seq, T, start, gamma, lam)
    assert_rel(host(rew), e_rew, "rewards")
    assert_rel(host(adv), e_adv, "advantages")
    assert_rel(host(ret), e_ret, "returns")


@pytest.mark.parametrize("n_seq,T,start,eps", LOSS)
def test_ppo_loss_sweep(n_seq, T, start, eps, dev):
    """The clipped surrogate and value losses and their per-token gradients."""
    import torch
    say("sweep ppo_loss", n_seq, T, start, eps)
    rng = np.random.default_rng(9990 + n_seq * T + start)
    M = n_seq * T
    lp_old = -rng.uniform(0.5, 6.0, M).astype(np.float32)
    lp_new = (lp_old + rng.normal(0, 0.3, M)).astype(np.float32)
    A, V = rng.normal(0, 1, M).astype(np.float32), rng.normal(0, 1, M).astype(np.float32)
    R = (V + rng.normal(0, 0.5, M)).astype(np.float32)
    losses = torch.full((3,), float("nan"), device=dev)
    d_lp, d_v = torch.full((M,), float("nan"), device=dev), torch.full((M,), float("nan"), device=dev)
    H.hydra_ppo_loss(*(to_dev(v, dev) for v in (lp_new, lp_old, A, V, R)), n_seq, T, losses, d_lp, d_v,
                     start=start, eps=eps)
    torch.cuda.synchronize()
    e = ppo_loss_ref(lp_new, lp_old, A, V, R, n_seq, T, start, eps)
    got = host(losses)
    for i, k in enumerate(("pg_loss", "v_loss")):
        assert abs(got[i] - e[k]) <= 1e-4 * max(abs(e[k]), 1e-3), (k, got[i], e[k])
    assert abs(got[2] - e["clip_frac"]) <= 2.0 / (n_seq * (T - start))
    assert_rel(host(d_lp), e["d_lp"], "d_lp")
    assert_rel(host(d_v), e["d_v"], "d_v")
