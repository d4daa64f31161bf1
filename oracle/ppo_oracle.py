"""Plain float64 CPU oracle for the PPO advantage step that follows scoring.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library and imports nothing from it.

What is computed, and where the paper defines it
------------------------------------------------
* The critic's per-token values V(x, y) from its scalar head on the critic's
  hidden states (Sec. 2, "Stage 3: PPO": V is trained on the returns and used
  by generalized advantage estimation; App. A, Alg. 2: the critic-LoRA pass
  over the generated sequences yields the values).  Reading: no
  bias, ``V[t] = <h_crit[t], w_v>``.
* The per-token PPO reward: the KL penalty with weight beta (App. B: beta =
  0.02) on every scored token, plus the sequence's reward-model score on its
  last token (App. A, Alg. 2: the advantage step combines the reward and the
  reference log-probabilities).  Reading: ``r_t = -beta * KL_t`` for response tokens
  ``t >= start``, ``r_{T-1} += reward``; tokens before ``start`` carry none.
* Generalized advantage estimation with gamma and lambda (Sec. 2, "Stage 3:
  PPO", citing GAE; App. B: gamma = 1.0, lambda = 0.95): the TD residual
  ``delta_t = r_t + gamma V_{t+1} - V_t`` (``V_T = 0``: the episode ends with
  the sequence), the advantage ``A_t = sum_{l >= 0} (gamma lambda)^l
  delta_{t+l}`` over the rest of the sequence, the return ``A_t + V_t``.
  Positions before ``start`` get advantage and return 0.

* The PPO losses of the update stage (Sec. 2, "Stage 3: PPO": the clipped
  surrogate objective on the probability ratio of the new and old policy,
  and the critic's squared-error loss on the returns).  Readings: the
  ratio is ``exp(lp_new - lp_old)`` of the sampled tokens' log-probabilities;
  the clip range eps is a parameter (the paper names it without a value);
  both losses are means over the response tokens (``t >= start``) of all
  sequences; the value loss is ``(V - R)^2 / 2`` without clipping; where the
  clipped and unclipped terms are equal the unclipped term's gradient is used.

Every function is the plain definition.  ``gae_ref`` evaluates the sum over
the rest of the sequence for every position (no recurrence), so it checks a
recursive or scanned evaluation independently.

Pins: see ``tests/test_oracle_ppo_pins.py`` (Fraction brute force, the lambda = 1
telescoping closed form, lambda = 0, constant-residual geometric series, the
one-step recurrence as a property).
"""
from __future__ import annotations

import numpy as np

from .hydra_oracle import bf16_to_f64

__all__ = ["value_head_ref", "ppo_rewards_ref", "gae_ref", "ppo_loss_ref"]


def value_head_ref(h, w_v) -> np.ndarray:
    """V[m] = sum_k h[m, k] * w_v[k] in float64 on the decoded bf16 inputs."""
    H = bf16_to_f64(h)
    w = bf16_to_f64(w_v)
    return H @ w


def ppo_rewards_ref(kl, reward, n_seq: int, seq_len: int, start: int, beta: float) -> np.ndarray:
    """Per-token PPO reward [n_seq * seq_len]: -beta * KL on tokens t >= start, plus
    the sequence's reward on its last token."""
    K = np.asarray(kl, dtype=np.float64).reshape(n_seq, seq_len)
    R = np.asarray(reward, dtype=np.float64).reshape(n_seq)
    r = np.zeros((n_seq, seq_len))
    r[:, start:] = -beta * K[:, start:]
    r[:, seq_len - 1] += R
    return r.reshape(-1)


def gae_ref(rewards, values, n_seq: int, seq_len: int, start: int, gamma: float, lam: float):
    """(advantages, returns) [n_seq * seq_len] by the definition
    A_t = sum_{l=0}^{T-1-t} (gamma lam)^l delta_{t+l}, delta_t = r_t + gamma V_{t+1} - V_t."""
    r = np.asarray(rewards, dtype=np.float64).reshape(n_seq, seq_len)
    V = np.asarray(values, dtype=np.float64).reshape(n_seq, seq_len)
    V_next = np.concatenate([V[:, 1:], np.zeros((n_seq, 1))], axis=1)
    delta = r + gamma * V_next - V
    c = gamma * lam
    A = np.zeros((n_seq, seq_len))
    for t in range(start, seq_len):
        w = c ** np.arange(seq_len - t, dtype=np.float64)
        A[:, t] = delta[:, t:] @ w
    ret = np.zeros_like(A)
    ret[:, start:] = A[:, start:] + V[:, start:]
    return A.reshape(-1), ret.reshape(-1)


def ppo_loss_ref(lp_new, lp_old, adv, v_new, returns, n_seq: int, seq_len: int, start: int, eps: float):
    """Clipped surrogate and value losses over the response tokens, and their gradients.

    Returns a dict with
      pg_loss   = -(1/n) sum_t min(rho_t A_t, clip(rho_t, 1 - eps, 1 + eps) A_t),  rho_t = exp(lp_new_t - lp_old_t)
      v_loss    = (1/n) sum_t (V_t - R_t)^2 / 2
      clip_frac = (1/n) #{t : the clipped term is strictly smaller}
      d_lp[t]   = d pg_loss / d lp_new_t  (-rho_t A_t / n where the unclipped term is the minimum, else 0)
      d_v[t]    = d v_loss / d V_t        ((V_t - R_t) / n)
    with n = n_seq * (seq_len - start); positions before start contribute nothing (gradient 0).
    """
    shape = (n_seq, seq_len)
    ln = np.asarray(lp_new, np.float64).reshape(shape)
    lo = np.asarray(lp_old, np.float64).reshape(shape)
    A = np.asarray(adv, np.float64).reshape(shape)
    V = np.asarray(v_new, np.float64).reshape(shape)
    R = np.asarray(returns, np.float64).reshape(shape)
    mask = np.zeros(shape, dtype=bool)
    mask[:, start:] = True
    n = n_seq * (seq_len - start)
    rho = np.exp(ln - lo)
    unclipped = rho * A
    clipped = np.clip(rho, 1.0 - eps, 1.0 + eps) * A
    obj = np.minimum(unclipped, clipped)
    pg_loss = -obj[mask].sum() / n
    d_lp = np.where(mask & (unclipped <= clipped), -unclipped / n, 0.0)
    v_loss = 0.5 * ((V - R)[mask] ** 2).sum() / n
    d_v = np.where(mask, (V - R) / n, 0.0)
    clip_frac = (clipped < unclipped)[mask].sum() / n
    return dict(pg_loss=float(pg_loss), v_loss=float(v_loss), clip_frac=float(clip_frac),
                d_lp=d_lp.reshape(-1), d_v=d_v.reshape(-1))
