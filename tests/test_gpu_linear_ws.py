"""GPU parity of hydra_lora_linear_ws (the MFMA GEMM taking its LoRA update from the pre-pass workspace) and of
the paper's rank 128 on every linear path, against the float64 oracle."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import lora_linear_ref
from gpu_helpers import DESIGN_REL, assert_rel, dev_bf16, host, rel_err, say

pytestmark = pytest.mark.gpu

WS_SHAPES = [
    # (M, K, N, r): GEMM rows past 16 with ragged row / column tiles and K tails, every padded rank up to 128
    # (r = 100 pads to 128), rank 0, and decode rows (M <= 16, the workspace is not used) at rank 128,
    # including 8 < M <= 16 (rank 128 runs those rows in two halves).
    (17, 64, 256, 8), (33, 520, 300, 16), (130, 72, 513, 1), (257, 1024, 700, 33), (64, 128, 96, 64),
    (300, 2048, 1200, 100), (130, 520, 300, 128), (129, 8, 255, 128), (200, 64, 256, 0),
    (4, 4096, 256, 128), (12, 1032, 77, 128), (16, 512, 512, 128), (1, 64, 40, 128),
]


def _run(c, device, ws=True, want_off=True, fill=None):
    import torch
    x, W = dev_bf16(c.x, device), dev_bf16(c.W, device)
    A = dev_bf16(c.A, device) if c.r > 0 else None
    B = dev_bf16(c.B, device) if c.r > 0 else None
    y_off = torch.full((c.M, c.N), float("nan"), device=device) if want_off else None
    y_on = torch.full((c.M, c.N), float("nan"), device=device)
    if ws:
        need = H.hydra_lora_linear_workspace_bytes(c.M, c.N, c.r)
        buf = torch.full((max(need, 1),), 0 if fill is None else fill, dtype=torch.uint8, device=device)
        H.hydra_lora_linear_ws(x, W, A, B, c.s, y_off, y_on, workspace=buf)
    else:
        H.hydra_lora_linear(x, W, A, B, c.s, y_off, y_on)
    torch.cuda.synchronize()
    return (host(y_off) if want_off else None), host(y_on)


@pytest.mark.parametrize("M,K,N,r", WS_SHAPES)
def test_linear_ws_matches_oracle(M, K, N, r, dev):
    say("linear_ws", M, K, N, r)
    c = WL.gen_linear(900 + M + r, M, K, N, r)
    y_off, y_on = _run(c, dev)
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert_rel(y_off, e_off, "y_off")
    assert_rel(y_on, e_on, "y_on")
    if r <= 64 or M <= 16:
        # same LoRA-off bits as the call without a workspace; y_on to the rounding of T
        p_off, p_on = _run(c, dev, ws=False)
        assert np.array_equal(y_off, p_off)
        assert rel_err(y_on, p_on) <= DESIGN_REL


def test_linear_ws_y_on_only_and_workspace_contents(dev):
    """y_on alone, and a workspace full of NaN bit patterns: the pre-pass overwrites what it reads."""
    say("linear_ws y_on only")
    c = WL.gen_linear(950, 160, 520, 300, 128)
    _, a_on = _run(c, dev, want_off=False, fill=0xFF)
    _, b_on = _run(c, dev, want_off=False, fill=0)
    assert np.array_equal(a_on, b_on)
    _, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert_rel(a_on, e_on, "y_on")


def test_linear_ws_b_zero_is_lora_off(dev):
    """B = 0: the update slabs add exact zeros, so y_on has the bits of y_off."""
    say("linear_ws B = 0")
    c = WL.gen_linear(951, 130, 256, 300, 128)
    c.B = np.zeros_like(c.B)
    y_off, y_on = _run(c, dev)
    assert np.array_equal(y_off, y_on)


def test_linear_ws_rank128_gate_projection_every_row(dev):
    """The Llama-7B gate projection (4096 -> 11008) over 2048 tokens at the paper's rank 128, every row."""
    say("linear_ws gate r=128 full size")
    c = WL.gen_linear(952, 2048, 4096, 11008, 128)
    y_off, y_on = _run(c, dev)
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert_rel(y_off, e_off, "y_off")
    assert_rel(y_on, e_on, "y_on")


@pytest.mark.parametrize("proj", ["q", "fc1", "fc2"])
def test_opt13b_layer_rank128_full_size(proj, dev):
    """OPT-1.3b at the paper's rank 128 (App. B), mini-batch 8 x 512 = 4096 tokens: 2048 -> 2048, 2048 -> 8192 and
    8192 -> 2048 through the pre-pass GEMM; every row of both outputs is compared with the oracle."""
    say("opt13b layer r128", proj)
    c = {x.name: x for x in WL.make("opt13b_layer_r128")}[proj]
    y_off, y_on = _run(c, dev)
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert_rel(y_off, e_off, "y_off")
    assert_rel(y_on, e_on, "y_on")
