"""GPU parity of hydra_score_two_input: the actor pass's log-probabilities from its own hidden states with the CLM
head's LoRA, the reference log-probabilities and the reward from the LoRA-off pass's, one launch over both inputs,
against the oracle."""
import math

import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import reward_ref, score_head_two_input_ref
from gpu_helpers import assert_abs, assert_rel, dev as to_dev, dev_bf16, host, row_chunks, say

pytestmark = pytest.mark.gpu

KEYS = ("lp_on", "lp_off", "kl", "lse_on", "lse_off")


def _run(c, device, h_act=None, ids=None, B=None):
    import torch
    h_act = c.h_act if h_act is None else h_act
    ids = c.ids if ids is None else ids
    B = c.B if B is None else B
    out = {k: torch.full((c.M,), float("nan"), device=device) for k in KEYS}
    out["reward"] = torch.full((c.n_seq,), float("nan"), device=device)
    err = torch.zeros(1, dtype=torch.int32, device=device)
    ws = torch.full((H.hydra_score_workspace_bytes(c.M, c.V),), 0xFF, dtype=torch.uint8, device=device)
    H.hydra_score_two_input(dev_bf16(h_act, device), dev_bf16(c.h, device), dev_bf16(c.W_lm, device),
                            dev_bf16(c.A, device) if c.r else None, dev_bf16(B, device) if c.r else None, c.s,
                            to_dev(ids.astype(np.int32), device), dev_bf16(c.w_rm, device), c.n_seq, c.seq_len,
                            out["lp_on"], out["lp_off"], out["kl"], reward=out["reward"], lse_on=out["lse_on"],
                            lse_off=out["lse_off"], workspace=ws, err_flag=err)
    torch.cuda.synchronize()
    res = {k: host(v) for k, v in out.items()}
    res["err"] = int(host(err)[0])
    return res


def _check_every_row(c, g, h_act=None, B=None):
    h_act = c.h_act if h_act is None else h_act
    B = c.B if B is None else B
    for rows in row_chunks(c.M):
        e = score_head_two_input_ref(h_act[rows], c.h[rows], c.W_lm, c.A, B, c.s, c.ids[rows])
        for k in KEYS:
            assert_abs(g[k][rows], e[k], f"{k} rows {rows[0]}..{rows[-1]}")
    assert_rel(g["reward"], reward_ref(c.h, c.w_rm, c.n_seq, c.seq_len), "reward")


@pytest.mark.parametrize("n_seq,seq_len,K,V,r", [
    (2, 64, 256, 1000, 16), (3, 37, 264, 1003, 8), (1, 300, 512, 4096, 0), (2, 130, 256, 777, 128),
    (4, 70, 1032, 2500, 32),
])
def test_score_two_input_matches_oracle(n_seq, seq_len, K, V, r, dev):
    """Ragged row tiles (the two inputs' tiles interleave), ragged vocabulary tiles, every rank class."""
    say("score two-input", n_seq, seq_len, K, V, r)
    c = WL.gen_score_two_input(6000 + K + V + r, n_seq, seq_len, K, V, r)
    g = _run(c, dev)
    _check_every_row(c, g)
    assert g["err"] == 0


def test_score_two_input_equal_inputs_have_the_one_input_bits(dev):
    """h_act == h_off: every output has the bits of hydra_score (same tiles, same reduction order)."""
    import torch
    say("score two-input equal inputs")
    c = WL.gen_score_two_input(6100, 3, 90, 264, 1100, 16)
    g2 = _run(c, dev, h_act=c.h)
    out = {k: torch.full((c.M,), float("nan"), device=dev) for k in KEYS}
    reward = torch.full((c.n_seq,), float("nan"), device=dev)
    H.hydra_score(dev_bf16(c.h, dev), dev_bf16(c.W_lm, dev), dev_bf16(c.A, dev), dev_bf16(c.B, dev), c.s,
                  to_dev(c.ids.astype(np.int32), dev), dev_bf16(c.w_rm, dev), c.n_seq, c.seq_len, out["lp_on"],
                  out["lp_off"], out["kl"], reward=reward, lse_on=out["lse_on"], lse_off=out["lse_off"])
    torch.cuda.synchronize()
    for k in KEYS:
        assert np.array_equal(g2[k], host(out[k])), k
    assert np.array_equal(g2["reward"], host(reward))


def test_score_two_input_b_zero_and_bad_token(dev):
    """B = 0: lp_on is the log-softmax of h_act W^T alone; an out-of-range token gives NaN and the error flag."""
    say("score two-input B=0, bad token")
    c = WL.gen_score_two_input(6200, 2, 40, 256, 900, 16)
    Bz = np.zeros_like(c.B)
    g = _run(c, dev, B=Bz)
    _check_every_row(c, g, B=Bz)
    ids = c.ids.copy()
    ids[5] = c.V
    gb = _run(c, dev, ids=ids)
    assert gb["err"] == 1 and math.isnan(gb["lp_on"][5]) and math.isnan(gb["kl"][5])
    assert not math.isnan(gb["lp_on"][4])


def test_score_two_input_full_size_every_row(dev):
    """The Llama-7B heads at M = 2048 tokens (4 x 512), K = 4096, V = 32000, r = 16, with the two passes' own hidden
    states: every row and every reward against the oracle."""
    c = WL.make("two_input_score")
    say("score two-input full", c.M, c.K, c.V, c.r)
    g = _run(c, dev)
    _check_every_row(c, g)
    assert g["err"] == 0
