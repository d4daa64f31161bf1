"""Plain float64 CPU oracle for the Hydra-PPO hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers or tables) and imports nothing from it.

What is computed, and where the paper defines it
------------------------------------------------
* LoRA on every linear layer of the actor and critic (Sec. 2, "Stage 3: PPO",
  last paragraph).  The paper cites LoRA without printing its formula; the
  reading used here is ``y_on = x W^T + s (x A^T) B^T`` with an explicit scale
  ``s`` (W stored output-major ``[N x K]``, A ``[r x K]``, B ``[N x r]``).
* Dynamic LoRA: the reference / reward model is the same network with LoRA
  "turned off", ``LO(.)``, i.e. ``y_off = x W^T`` on the same frozen W
  (Sec. 3, "Dynamic LoRA" paragraph; "Stage 2: Hydra-PPO" paragraph for the
  two adapter sets over one base).
* The two heads of pi^hydra: a causal-LM head over the vocabulary and a
  scalar reward head on the same input (Sec. 3, opening paragraph).
* Reference log-probabilities and reward from the LoRA-off model
  (App. A, Alg. 1 and Alg. 2, the LoRA-off scoring step); log-probability of
  the sampled token under a temperature-1 softmax; the per-token KL penalty
  estimate ``lp_on - lp_off`` whose weight beta = 0.02 (App. B, PPO common
  parameters) is applied downstream, not here.

Every function is the plain definition: one library matmul per product, then
explicit row-wise max / exp / sum / log in float64.  No blocking, fusion or
reordering beyond a row split of the matmul to bound memory.

Pins: see ``tests/test_oracle_pins.py`` (Fraction brute force, merged-weight
invariant, closed forms of the log-softmax, KL identities, library
cross-checks).  No function here is "parity unpinned".
"""
from __future__ import annotations

import math
from typing import Optional, Tuple

import numpy as np

__all__ = [
    "lora_linear_backward_ref",
    "lora_linear_multi_ref",
    "bf16_to_f64",
    "lora_linear_ref",
    "log_softmax_gather_ref",
    "score_logits_ref",
    "reward_ref",
    "score_head_ref",
    "score_head_two_input_ref",
]

_ROW_BLOCK = 256


def bf16_to_f64(u16) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) to float64.  Every bf16 value is exact in float64."""
    u = np.asarray(u16, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _mm(X: np.ndarray, Yt: np.ndarray) -> np.ndarray:
    """X @ Yt.T in float64, split by rows of X only (bounded memory)."""
    out = np.empty((X.shape[0], Yt.shape[0]), dtype=np.float64)
    for i in range(0, X.shape[0], _ROW_BLOCK):
        out[i:i + _ROW_BLOCK] = X[i:i + _ROW_BLOCK] @ Yt.T
    return out


def lora_linear_ref(x, W, A, B, s: float) -> Tuple[np.ndarray, np.ndarray]:
    """LoRA-switchable linear (Sec. 2 Stage 3 LoRA-PPO; Sec. 3 Dynamic LoRA).

    x: [M x K] bf16 bits, W: [N x K], A: [r x K], B: [N x r], s: scale.
    Returns (y_off, y_on) in float64:
      y_off = X W^T                    (LoRA off, LO(.): reference / reward role)
      y_on  = X W^T + s (X A^T) B^T    (LoRA on: actor or critic role)
    """
    X = bf16_to_f64(x)
    Wd = bf16_to_f64(W)
    Ad = bf16_to_f64(A)
    Bd = bf16_to_f64(B)
    y_off = _mm(X, Wd)
    T = _mm(X, Ad)                      # [M x r]
    y_on = y_off + float(s) * _mm(T, Bd)
    return y_off, y_on


def lora_linear_backward_ref(x, W, A, B, s: float, dy):
    """Gradients of the LoRA-on output with the base weight frozen (the PPO update
    stage trains only the adapters: Sec. 2 Stage 3, LoRA on all linears; Table 1
    update latency).  For y_on = X W^T + s (X A^T) B^T and an upstream gradient dY
    of y_on (all bf16 bits but dY, which may be bf16 bits or float):
      dX = dY W + s (dY B) A          [M x K]
      dA = s (dY B)^T X               [r x K]
      dB = s dY^T (X A^T)             [N x r]
    in float64 (each is the plain chain rule of the forward definition).
    """
    X = bf16_to_f64(x)
    Wd = bf16_to_f64(W)
    Ad = bf16_to_f64(A)
    Bd = bf16_to_f64(B)
    dY = bf16_to_f64(dy) if np.asarray(dy).dtype == np.uint16 else np.asarray(dy, np.float64)
    U = dY @ Bd                       # [M x r]
    T = _mm(X, Ad)                    # [M x r]
    dX = dY @ Wd + float(s) * (U @ Ad)
    dA = float(s) * (U.T @ X)
    dB = float(s) * (dY.T @ T)
    return dX, dA, dB


def lora_linear_multi_ref(x_off, W, x_ons, As, Bs, ss):
    """One frozen W serving several passes (App. A, Alg. 2: the actor pass with the
    actor adapter, the critic pass with the critic adapter, the reference / reward
    passes with LoRA off, all over the same base weights; Sec. 3 Dynamic LoRA).

    x_off: [M x K] bf16 bits or None; x_ons[a]: [M x K]; As[a]: [r x K]; Bs[a]: [N x r].
    Returns (y_off or None, [y_on[a]]) in float64:
      y_off   = X_off W^T
      y_on[a] = X_on[a] W^T + s[a] (X_on[a] A[a]^T) B[a]^T
    Each pass is its own plain product; sharing the reads of W is a property of
    the kernel, not of what is computed.
    """
    Wd = bf16_to_f64(W)
    y_off = None if x_off is None else _mm(bf16_to_f64(x_off), Wd)
    y_ons = []
    for x, A, B, s in zip(x_ons, As, Bs, ss):
        X = bf16_to_f64(x)
        y = _mm(X, Wd)
        if A is not None and np.asarray(A).size:
            y = y + float(s) * _mm(_mm(X, bf16_to_f64(A)), bf16_to_f64(B))
        y_ons.append(y)
    return y_off, y_ons


def log_softmax_gather_ref(z, ids) -> Tuple[np.ndarray, np.ndarray]:
    """Sampled-token log-probability under a temperature-1 softmax over the vocabulary.

    For each row i: m = max_v z[i, v]; S = sum_v exp(z[i, v] - m);
    lse = m + ln S; lp = z[i, t_i] - lse.  A token id outside [0, V) yields NaN.
    Returns (lp, lse), float64 [M].
    """
    z = np.asarray(z, dtype=np.float64)
    ids = np.asarray(ids, dtype=np.int64)
    M, V = z.shape
    lp = np.empty(M, dtype=np.float64)
    lse = np.empty(M, dtype=np.float64)
    for i in range(M):
        row = z[i]
        m = row.max()
        S = np.exp(row - m).sum()
        lse[i] = m + math.log(S)
        t = int(ids[i])
        lp[i] = row[t] - lse[i] if 0 <= t < V else math.nan
    return lp, lse


def score_logits_ref(logits_on, logits_off, ids):
    """Scoring epilogue on materialised logits (App. A, Alg. 2 reference log-probabilities).

    Returns dict(lp_on, lp_off, kl, lse_on, lse_off) with kl = lp_on - lp_off,
    the per-token sampled KL estimate (beta is applied downstream).
    """
    lp_on, lse_on = log_softmax_gather_ref(logits_on, ids)
    lp_off, lse_off = log_softmax_gather_ref(logits_off, ids)
    return dict(lp_on=lp_on, lp_off=lp_off, kl=lp_on - lp_off, lse_on=lse_on, lse_off=lse_off)


def reward_ref(h, w_rm, n_seq: int, seq_len: int, rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Scalar reward head on the last token of each sequence (Sec. 2 Stage 2; Sec. 3 two heads).

    reward[b] = sum_k H[b*seq_len + seq_len - 1, k] * w_rm[k]; no bias, no
    normalisation.  ``rows`` (optional) are the row indices of ``h`` when only
    a subset of the hidden rows is passed.
    """
    H = bf16_to_f64(h)
    w = bf16_to_f64(w_rm)
    out = np.empty(n_seq, dtype=np.float64)
    for b in range(n_seq):
        want = b * seq_len + seq_len - 1
        idx = want if rows is None else int(np.nonzero(np.asarray(rows) == want)[0][0])
        out[b] = float(H[idx] @ w)
    return out


def score_head_ref(h, W_lm, A, B, s: float, ids, w_rm=None, n_seq: int = 0, seq_len: int = 0,
                   rows: Optional[np.ndarray] = None):
    """Two-head PPO scoring pass (Sec. 3 two heads; App. A Alg. 2 critic / LoRA-off steps).

    Logits are the CLM head applied with LoRA on (actor) and off (reference),
    then the sampled-token log-softmax of each, their difference, and the
    reward head on each sequence's last token.  ``rows`` selects a subset of
    token rows (``h`` and ``ids`` are then already that subset); the reward is
    computed only when every sequence's last row is among them.
    """
    z_off, z_on = lora_linear_ref(h, W_lm, A, B, s)
    res = score_logits_ref(z_on, z_off, ids)
    if w_rm is not None and n_seq > 0:
        lasts = [b * seq_len + seq_len - 1 for b in range(n_seq)]
        if rows is None or all(l in set(int(v) for v in rows) for l in lasts):
            res["reward"] = reward_ref(h, w_rm, n_seq, seq_len, rows)
    return res


def score_head_two_input_ref(h_act, h_off, W_lm, A, B, s: float, ids, w_rm=None, n_seq: int = 0, seq_len: int = 0):
    """Two-head scoring with each pass's own final hidden states (App. A, Alg. 2: the actor pass runs with the
    actor's adapter and the reference / reward pass with LoRA off, over the same sequences; in a multi-layer
    model their hidden states differ; Sec. 3 Dynamic LoRA: the reward model is the LoRA-off network).

      z_on  = H_act W_lm^T + s (H_act A^T) B^T   (the actor's logits: LoRA on the CLM head too)
      z_off = H_off W_lm^T                        (the reference logits: LoRA off)
      lp_on, lp_off, lse_on, lse_off, kl = lp_on - lp_off as in score_logits_ref;
      reward[b] = <H_off[b*seq_len + seq_len - 1], w_rm>  (the reward head on the LoRA-off pass).
    """
    _, z_on = lora_linear_ref(h_act, W_lm, A, B, s)
    z_off = _mm(bf16_to_f64(h_off), bf16_to_f64(W_lm))
    res = score_logits_ref(z_on, z_off, ids)
    if w_rm is not None and n_seq > 0:
        res["reward"] = reward_ref(h_off, w_rm, n_seq, seq_len)
    return res
