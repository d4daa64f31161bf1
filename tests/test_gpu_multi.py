"""GPU parity of hydra_lora_linear_multi (one W for a LoRA-off input and several LoRA-on inputs with their own
adapters) against the float64 oracle, and bit-for-bit against the single-input calls."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import lora_linear_multi_ref
from gpu_helpers import assert_rel, dev_bf16, host, row_chunks, say

pytestmark = pytest.mark.gpu

CASES = [
    # (M, K, N, r, n_on, with_off): stacked rows in one pass of W (<= 8), in several passes, rank 0, the
    # per-input paths (M > 8: decode MFMA kernel, M > 16: GEMM), ragged K / N, every padded-rank class.
    (4, 4096, 512, 16, 2, True), (4, 520, 300, 16, 1, True), (1, 64, 40, 8, 3, True), (8, 1032, 77, 32, 1, True),
    (3, 136, 33, 0, 2, False), (2, 4104, 130, 64, 4, True), (5, 256, 96, 16, 0, True), (4, 11008, 64, 16, 2, True),
    (12, 520, 300, 16, 2, True), (64, 512, 256, 16, 2, True),
    # above 16 rows (one GEMM per input): ragged rows and columns, four adapters, rank 64, no LoRA-off input,
    # rank 0
    (300, 520, 300, 16, 4, True), (130, 72, 513, 64, 2, True), (200, 264, 520, 32, 3, False),
    (257, 1024, 700, 0, 2, True),
]


def _run_multi(c, device):
    import torch
    x_off = dev_bf16(c.x_off, device) if c.x_off is not None else None
    W = dev_bf16(c.W, device)
    xs = [dev_bf16(x, device) for x in c.x_on]
    As = [dev_bf16(a, device) if c.r else None for a in c.A]
    Bs = [dev_bf16(b, device) if c.r else None for b in c.B]
    y_off = torch.full((c.M, c.N), float("nan"), device=device) if x_off is not None else None
    y_ons = [torch.full((c.M, c.N), float("nan"), device=device) for _ in xs]
    H.hydra_lora_linear_multi(x_off, W, xs, As, Bs, c.s, y_off, y_ons)
    torch.cuda.synchronize()
    return (None if y_off is None else host(y_off)), [host(t) for t in y_ons]


def _run_single(x, W, A, B, s, device, want_off):
    import torch
    M, N = x.shape[0], W.shape[0]
    y_off = torch.full((M, N), float("nan"), device=device) if want_off else None
    y_on = torch.full((M, N), float("nan"), device=device) if A is not None or not want_off else None
    H.hydra_lora_linear(dev_bf16(x, device), dev_bf16(W, device), None if A is None else dev_bf16(A, device),
                        None if B is None else dev_bf16(B, device), s, y_off, y_on)
    torch.cuda.synchronize()
    return (None if y_off is None else host(y_off)), (None if y_on is None else host(y_on))


@pytest.mark.parametrize("M,K,N,r,n_on,with_off", CASES)
def test_multi_matches_oracle_and_single_calls(M, K, N, r, n_on, with_off, dev):
    say("multi", M, K, N, r, n_on, with_off)
    c = WL.gen_multi(700 + M * 7 + n_on, M, K, N, r, n_on, with_off, scales=(2.0, 0.5, -1.0, 1.5))
    g_off, g_ons = _run_multi(c, dev)
    e_off, e_ons = lora_linear_multi_ref(c.x_off, c.W, c.x_on, c.A if r else [None] * n_on,
                                         c.B if r else [None] * n_on, c.s)
    if with_off:
        assert_rel(g_off, e_off, "y_off")
        s_off, _ = _run_single(c.x_off, c.W, None, None, 0.0, dev, want_off=True)
        assert np.array_equal(g_off, s_off), "y_off differs from the single LoRA-off call"
    for a in range(n_on):
        assert_rel(g_ons[a], e_ons[a], f"y_on[{a}]")
        A, B = (c.A[a], c.B[a]) if r else (None, None)
        _, s_on = _run_single(c.x_on[a], c.W, A, B, c.s[a], dev, want_off=False)
        assert np.array_equal(g_ons[a], s_on), f"y_on[{a}] differs from the single LoRA-on call"


def test_multi_adapters_do_not_leak(dev):
    """Swapping the two adapters swaps nothing else: each y_on depends on its own input and adapter only."""
    say("multi adapter swap")
    c = WL.gen_multi(790, 4, 1032, 200, 16, 2)
    g_off, g = _run_multi(c, dev)
    c2 = WL.MultiCase("swap", c.W, c.x_off, c.x_on[::-1], c.A[::-1], c.B[::-1], c.s[::-1])
    g2_off, g2 = _run_multi(c2, dev)
    assert np.array_equal(g_off, g2_off)
    assert np.array_equal(g[0], g2[1]) and np.array_equal(g[1], g2[0])


def test_decode_multi_full_size(dev):
    """The decode workload: one 4096 x 4096 projection for the reference, actor and critic passes at M = 4."""
    c = WL.make("decode_multi")
    say("decode_multi", c.M, c.K, c.N, c.r, len(c.x_on))
    g_off, g_ons = _run_multi(c, dev)
    e_off, e_ons = lora_linear_multi_ref(c.x_off, c.W, c.x_on, c.A, c.B, c.s)
    assert_rel(g_off, e_off, "y_off")
    for a in range(len(g_ons)):
        assert_rel(g_ons[a], e_ons[a], f"y_on[{a}]")


def test_prefill_multi_full_size_every_row(dev):
    """One 4096 x 4096 projection over 2048 tokens for the LoRA-off, actor and critic passes (three inputs): every
    row against the oracle, and the bits of the single-input calls."""
    M, K, N, r = 2048, 4096, 4096, 16
    say("prefill multi", M, K, N, r)
    c = WL.gen_multi(991, M, K, N, r, 2, True, scales=(2.0, -1.0))
    g_off, g_ons = _run_multi(c, dev)
    e_off, e_ons = lora_linear_multi_ref(c.x_off, c.W, c.x_on, c.A, c.B, c.s)
    assert_rel(g_off, e_off, "y_off")
    s_off, _ = _run_single(c.x_off, c.W, None, None, 0.0, dev, want_off=True)
    assert np.array_equal(g_off, s_off), "y_off differs from the single LoRA-off call"
    for a in range(2):
        assert_rel(g_ons[a], e_ons[a], f"y_on[{a}]")
        _, s_on = _run_single(c.x_on[a], c.W, c.A[a], c.B[a], c.s[a], dev, want_off=False)
        assert np.array_equal(g_ons[a], s_on), f"y_on[{a}] differs from the single LoRA-on call"


def _run_multi_ws(c, device):
    import torch
    x_off = dev_bf16(c.x_off, device) if c.x_off is not None else None
    W = dev_bf16(c.W, device)
    xs = [dev_bf16(x, device) for x in c.x_on]
    As = [dev_bf16(a, device) if c.r else None for a in c.A]
    Bs = [dev_bf16(b, device) if c.r else None for b in c.B]
    y_off = torch.full((c.M, c.N), float("nan"), device=device) if x_off is not None else None
    y_ons = [torch.full((c.M, c.N), float("nan"), device=device) for _ in xs]
    ws = torch.full((H.hydra_lora_linear_multi_workspace_bytes(c.M, c.N, c.r),), 0xA5, dtype=torch.uint8,
                    device=device)
    H.hydra_lora_linear_multi_ws(x_off, W, xs, As, Bs, c.s, y_off, y_ons, workspace=ws)
    torch.cuda.synchronize()
    return (None if y_off is None else host(y_off)), [host(t) for t in y_ons]


@pytest.mark.parametrize("M,K,N,r,n_on,with_off", [
    (130, 520, 300, 128, 2, True), (48, 264, 136, 100, 3, False), (4, 1032, 200, 128, 2, True),
    (64, 512, 256, 16, 2, True),
])
def test_multi_ws_matches_oracle_and_single_calls(M, K, N, r, n_on, with_off, dev):
    """Rank 128 above 16 rows through the pre-pass GEMM (each adapter in turn over one workspace, filled with junk
    first): the oracle's result, and the bits of hydra_lora_linear_ws per adapter; the decode and rank-16 shapes
    take the plain multi-input call (its bits)."""
    import torch
    say("multi_ws", M, K, N, r, n_on, with_off)
    c = WL.gen_multi(900 + M * 7 + n_on, M, K, N, r, n_on, with_off, scales=(2.0, 0.5, -1.0, 1.5))
    g_off, g_ons = _run_multi_ws(c, dev)
    e_off, e_ons = lora_linear_multi_ref(c.x_off, c.W, c.x_on, c.A, c.B, c.s)
    if with_off:
        assert_rel(g_off, e_off, "y_off")
    for a in range(n_on):
        assert_rel(g_ons[a], e_ons[a], f"y_on[{a}]")
    pre = M > 16 and r > 64
    if pre:
        W = dev_bf16(c.W, dev)
        for a in range(n_on):
            y = torch.full((M, N), float("nan"), device=dev)
            ws = torch.empty(H.hydra_lora_linear_workspace_bytes(M, N, r), dtype=torch.uint8, device=dev)
            H.hydra_lora_linear_ws(dev_bf16(c.x_on[a], dev), W, dev_bf16(c.A[a], dev), dev_bf16(c.B[a], dev), c.s[a],
                                   None, y, workspace=ws)
            torch.cuda.synchronize()
            assert np.array_equal(g_ons[a], host(y)), f"y_on[{a}] differs from hydra_lora_linear_ws"
    else:
        p_off, p_ons = _run_multi(c, dev)
        if with_off:
            assert np.array_equal(g_off, p_off)
        for a in range(n_on):
            assert np.array_equal(g_ons[a], p_ons[a]), a


def test_multi_ws_opt13b_full_size_every_row(dev):
    """OPT-1.3b's q projection at the paper's rank 128 over a PPO mini-batch of 8 x 512 tokens, for the LoRA-off,
    actor and critic passes, each with its own input: every row against the oracle."""
    M, K, N, r = 4096, 2048, 2048, 128
    say("multi_ws opt13b", M, K, N, r)
    c = WL.gen_multi(990, M, K, N, r, 2, True, scales=(2.0, 2.0))
    g_off, g_ons = _run_multi_ws(c, dev)
    for rows in row_chunks(M):
        e_off, e_ons = lora_linear_multi_ref(c.x_off[rows], c.W, [x[rows] for x in c.x_on], c.A, c.B, c.s)
        assert_rel(g_off[rows], e_off, f"y_off rows {rows[0]}..")
        for a in range(2):
            assert_rel(g_ons[a][rows], e_ons[a], f"y_on[{a}] rows {rows[0]}..")
