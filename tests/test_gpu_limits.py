"""GPU parity at the largest sizes the C ABI accepts, where 32-bit buffer ranges and offsets are tightest:
K = 2^21 (the inner dimension of every linear path, the rank-128 pre-pass and the backward), and a vocabulary of
V = 2^21 (the fused scoring head and the epilogue over materialised logits)."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import lora_linear_backward_ref, lora_linear_ref, score_head_ref, score_logits_ref
from gpu_helpers import assert_abs, assert_rel, dev_bf16, host, say
from gpu_helpers import dev as to_dev

pytestmark = pytest.mark.gpu

KMAX = 1 << 21
VMAX = 1 << 21


@pytest.mark.parametrize("M,r,ws", [(1, 16, False), (17, 16, False), (17, 128, True), (40, 64, True)])
def test_linear_at_largest_k(M, r, ws, dev):
    """Decode (M = 1), the dual GEMM (M = 17) and the pre-pass GEMM (rank 128, and rank 64 with a ragged row tile)
    with K = 2^21."""
    import torch
    say("linear K=2^21", M, r, ws)
    c = WL.gen_linear(610 + M + r, M, KMAX, 8, r)
    x, W, A, B = (dev_bf16(a, dev) for a in (c.x, c.W, c.A, c.B))
    y_off = torch.full((c.M, c.N), float("nan"), device=dev)
    y_on = torch.full((c.M, c.N), float("nan"), device=dev)
    if ws:
        H.hydra_lora_linear_ws(x, W, A, B, c.s, y_off, y_on)
    else:
        H.hydra_lora_linear(x, W, A, B, c.s, y_off, y_on)
    torch.cuda.synchronize()
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert_rel(host(y_off), e_off, "y_off")
    assert_rel(host(y_on), e_on, "y_on")


def test_backward_at_largest_k(dev):
    """dx, dA, dB with K = 2^21 (x rows of 4 MB; the dx GEMM writes 2^21 columns)."""
    import torch
    say("backward K=2^21")
    case = WL.gen_backward(620, 33, KMAX, 8, 16)
    c = case.lin
    x, A, B, dy = (dev_bf16(a, dev) for a in (c.x, c.A, c.B, case.dy))
    Wt = torch.empty((c.K, c.N), dtype=torch.int16, device=dev)
    H.hydra_transpose_bf16(dev_bf16(c.W, dev), Wt)
    dx = torch.full((c.M, c.K), float("nan"), device=dev)
    dA = torch.full((c.r, c.K), float("nan"), device=dev)
    dB = torch.full((c.N, c.r), float("nan"), device=dev)
    H.hydra_lora_linear_backward(x, Wt, A, B, c.s, dy, dx, dA, dB)
    torch.cuda.synchronize()
    e_dx, e_dA, e_dB = lora_linear_backward_ref(c.x, c.W, c.A, c.B, c.s, case.dy)
    assert_rel(host(dx), e_dx, "dx")
    assert_rel(host(dA), e_dA, "dA")
    assert_rel(host(dB), e_dB, "dB")


def test_score_at_largest_vocabulary(dev):
    """The fused two-head pass with V = 2^21 (8192 column tiles merged per row) at rank 16."""
    import torch
    say("score V=2^21")
    s = WL.gen_score_head(630, 2, 3, 64, VMAX, 16)
    out = {k: torch.full((s.M,), float("nan"), device=dev) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
    reward = torch.full((s.n_seq,), float("nan"), device=dev)
    H.hydra_score(dev_bf16(s.h, dev), dev_bf16(s.W_lm, dev), dev_bf16(s.A, dev), dev_bf16(s.B, dev), s.s,
                  torch.from_numpy(s.ids).to(dev), dev_bf16(s.w_rm, dev), s.n_seq, s.seq_len, out["lp_on"],
                  out["lp_off"], out["kl"], reward=reward, lse_on=out["lse_on"], lse_off=out["lse_off"])
    torch.cuda.synchronize()
    e = score_head_ref(s.h, s.W_lm, s.A, s.B, s.s, s.ids, s.w_rm, s.n_seq, s.seq_len)
    for k, v in out.items():
        assert_abs(host(v), e[k], k)
    assert_rel(host(reward), e["reward"], "reward")


def test_score_logits_at_largest_vocabulary(dev):
    """The epilogue over materialised logits with V = 2^21 per row (8 MB per row)."""
    import torch
    say("score_logits V=2^21")
    on, off, ids = WL.gen_logits(640, 3, VMAX)
    res = {k: torch.full((3,), float("nan"), device=dev) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
    H.hydra_score_logits(to_dev(on, dev), to_dev(off, dev), to_dev(ids.astype(np.int32), dev), res["lp_on"],
                         res["lp_off"], res["kl"], res["lse_on"], res["lse_off"])
    torch.cuda.synchronize()
    e = score_logits_ref(on, off, ids)
    for k, v in res.items():
        assert_abs(host(v), e[k], k)
