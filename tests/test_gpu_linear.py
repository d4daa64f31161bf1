"""GPU parity of hydra_lora_linear (both kernels) against the float64 oracle."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import lora_linear_ref
from gpu_helpers import assert_rel, dev_bf16, host, say

pytestmark = pytest.mark.gpu


def _run(c, device, want_off=True, want_on=True, s=None, B=None):
    import torch
    s = c.s if s is None else s
    B = c.B if B is None else B
    x, W = dev_bf16(c.x, device), dev_bf16(c.W, device)
    A = dev_bf16(c.A, device) if c.r > 0 else None
    Bt = dev_bf16(B, device) if c.r > 0 else None
    y_off = torch.full((c.M, c.N), float("nan"), device=device) if want_off else None
    y_on = torch.full((c.M, c.N), float("nan"), device=device) if want_on else None
    H.hydra_lora_linear(x, W, A, Bt, s, y_off, y_on)
    torch.cuda.synchronize()
    return (host(y_off) if want_off else None), (host(y_on) if want_on else None)


SHAPES = [
    # (M, K, N, r): decode kernel (M <= 16) and MFMA GEMM (M > 16), ragged
    # rows / columns / K tails, every padded-rank class, rank 0.
    (1, 64, 40, 8), (3, 520, 300, 16), (4, 4096, 256, 16), (16, 512, 512, 8), (16, 72, 1000, 64),
    (5, 136, 33, 1), (7, 256, 20, 0), (2, 8, 17, 33), (6, 520, 300, 64), (8, 4104, 130, 32), (12, 1032, 77, 16),
    (17, 64, 256, 8), (33, 520, 300, 16), (128, 512, 256, 16), (130, 72, 513, 1), (257, 1024, 700, 33),
    (200, 64, 256, 0), (64, 128, 96, 64), (300, 2048, 1200, 17), (129, 8, 255, 16),
    # decode shapes whose x rows span several LDS segments (K > 4096, or K > 2048 at M > 4)
    (4, 11008, 96, 16), (2, 8200, 50, 64), (1, 4096, 300, 32), (8, 2056, 70, 8),
]


@pytest.mark.parametrize("M,K,N,r", SHAPES)
def test_linear_matches_oracle(M, K, N, r, dev):
    seed = 1000 + M + 7 * K + 13 * N + r
    say("lora_linear", dict(M=M, K=K, N=N, r=r, seed=seed))
    c = WL.gen_linear(seed, M, K, N, r, s=2.0)
    y_off, y_on = _run(c, dev)
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert_rel(y_off, e_off, "y_off")
    assert_rel(y_on, e_on, "y_on")


@pytest.mark.parametrize("M", [4, 64])
def test_linear_single_outputs(M, dev):
    say("lora_linear single outputs", M)
    c = WL.gen_linear(77, M, 256, 300, 16)
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    off_only, _ = _run(c, dev, want_on=False)
    _, on_only = _run(c, dev, want_off=False)
    assert_rel(off_only, e_off, "y_off only")
    assert_rel(on_only, e_on, "y_on only")
    both_off, both_on = _run(c, dev)
    assert np.array_equal(off_only, both_off) and np.array_equal(on_only, both_on)


@pytest.mark.parametrize("M", [4, 200])
def test_lora_off_identities_are_bitwise(M, dev):
    """B = 0 or s = 0 turns LoRA off: y_on must equal y_off bit for bit."""
    say("lora_linear B=0 / s=0", M)
    c = WL.gen_linear(78, M, 512, 384, 16)
    off, on = _run(c, dev, B=np.zeros_like(c.B))
    assert np.array_equal(off, on)
    off2, on2 = _run(c, dev, s=0.0)
    assert np.array_equal(off2, on2) and np.array_equal(off, off2)


@pytest.mark.parametrize("M", [4, 300])
def test_linear_deterministic(M, dev):
    say("lora_linear determinism", M)
    c = WL.gen_linear(79, M, 1024, 520, 16)
    a = _run(c, dev)
    b = _run(c, dev)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_adapter_selection_actor_vs_critic(dev):
    """Hydra-PPO: two adapter sets over one W; each call uses only the pair passed."""
    say("adapter selection")
    act = WL.gen_linear(80, 96, 256, 128, 16)
    crit = WL.gen_linear(81, 96, 256, 128, 16)
    c2 = WL.LinearCase("critic", act.x, act.W, crit.A, crit.B, 2.0)
    off_a, on_a = _run(act, dev)
    off_c, on_c = _run(c2, dev)
    assert np.array_equal(off_a, off_c)
    assert_rel(on_c, lora_linear_ref(act.x, act.W, crit.A, crit.B, 2.0)[1], "critic y_on")


def test_decode_qkvo_full(dev):
    """Decode step, batch 4: the four 4096x4096 attention projections, r = 16 (full oracle)."""
    cases = WL.make("decode_qkvo")
    for c in cases:
        say("decode", c.name, c.M, c.K, c.N, c.r)
        y_off, y_on = _run(c, dev)
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(y_off, e_off, f"{c.name} y_off")
        assert_rel(y_on, e_on, f"{c.name} y_on")


def test_prefill_layer_full_size_every_row(dev):
    """Prefill, M = 2048: all seven linears of one Llama-7B layer, r = 16, in the launch configuration the bench
    times; every row of both outputs is compared with the oracle."""
    cases = WL.make("prefill_layer")
    for c in cases:
        say("prefill", c.name, c.M, c.K, c.N, c.r)
        y_off, y_on = _run(c, dev)
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(y_off, e_off, f"{c.name} y_off")
        assert_rel(y_on, e_on, f"{c.name} y_on")


def _group_run(cases, device, want_on=None):
    import torch
    G = len(cases)
    want_on = want_on or [True] * G
    adapter = want_on
    xs = [dev_bf16(c.x, device) for c in cases]
    Ws = [dev_bf16(c.W, device) for c in cases]
    As = [dev_bf16(c.A, device) if (c.r and adapter[i]) else None for i, c in enumerate(cases)]
    Bs = [dev_bf16(c.B, device) if (c.r and adapter[i]) else None for i, c in enumerate(cases)]
    yo = [torch.full((c.M, c.N), float("nan"), device=device) for c in cases]
    yn = [torch.full((c.M, c.N), float("nan"), device=device) if want_on[i] else None for i, c in enumerate(cases)]
    H.hydra_lora_linear_group(xs, Ws, As, Bs, [c.s for c in cases], yo, yn)
    torch.cuda.synchronize()
    return [host(t) for t in yo], [None if t is None else host(t) for t in yn]


def test_group_decode_matches_single_calls_bitwise(dev):
    """The four decode projections in one grouped launch give exactly the single-call results."""
    cases = WL.make("decode_qkvo")
    say("group decode qkvo", len(cases))
    go, gn = _group_run(cases, dev)
    for i, c in enumerate(cases):
        so, sn = _run(c, dev)
        assert np.array_equal(go[i], so) and np.array_equal(gn[i], sn), c.name
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(gn[i], e_on, f"group {c.name} y_on")


def test_group_mixed_members(dev):
    """Members with different scales, one without an adapter (LoRA off only), ragged N."""
    say("group mixed members")
    base = [WL.gen_linear(90 + i, 3, 520, 300, 16, s=[2.0, 0.5, -1.0][i]) for i in range(3)]
    go, gn = _group_run(base, dev, want_on=[True, False, True])
    for i, c in enumerate(base):
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(go[i], e_off, f"member {i} y_off")
        if gn[i] is not None:
            assert_rel(gn[i], e_on, f"member {i} y_on")


@pytest.mark.parametrize("M", [1, 4, 8])
def test_group_lora_off_member_between_lora_members(dev, M):
    """At every decode row class, a LoRA-off member (no y_on, no adapter) sits between two members whose y_on
    gets the LoRA update; the update must touch only its own members."""
    say("group lora-off member", M)
    base = [WL.gen_linear(70 + i, M, 1032, 200, 16) for i in range(3)]
    go, gn = _group_run(base, dev, want_on=[True, False, True])
    assert gn[1] is None
    for i in range(3):
        e_off, e_on = lora_linear_ref(base[i].x, base[i].W, base[i].A, base[i].B, base[i].s)
        assert_rel(go[i], e_off, f"member {i} y_off")
        if i != 1:
            assert_rel(gn[i], e_on, f"member {i} y_on")


def test_group_gemm_path(dev):
    say("group M > 16")
    cases = [WL.gen_linear(95 + i, 130, 256, 300, 16) for i in range(2)]
    go, gn = _group_run(cases, dev)
    for i, c in enumerate(cases):
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(go[i], e_off, "y_off")
        assert_rel(gn[i], e_on, "y_on")


@pytest.mark.parametrize("M,K,N,r,G", [(300, 520, 300, 16, 3), (130, 72, 513, 64, 2), (17, 64, 256, 1, 8)])
def test_group_gemm_matches_single_calls_bitwise(M, K, N, r, G, dev):
    """At M > 16 (the dual GEMM) every member of a group call has the bits of its single call (ragged tiles,
    members with different scales, up to 8 members)."""
    say("group gemm", M, K, N, r, G)
    cases = [WL.gen_linear(400 + 10 * G + i, M, K, N, r, s=1.0 + 0.5 * i) for i in range(G)]
    go, gn = _group_run(cases, dev)
    for i, c in enumerate(cases):
        so, sn = _run(c, dev)
        assert np.array_equal(go[i], so) and np.array_equal(gn[i], sn), c.name
    e_off, e_on = lora_linear_ref(cases[-1].x, cases[-1].W, cases[-1].A, cases[-1].B, cases[-1].s)
    assert_rel(go[-1], e_off, "last member y_off")
    assert_rel(gn[-1], e_on, "last member y_on")


def test_group_gemm_lora_off_member(dev):
    """A member without an adapter and without y_on between two LoRA members, at M > 16."""
    say("group gemm lora-off member")
    base = [WL.gen_linear(480 + i, 200, 264, 520, 16) for i in range(3)]
    go, gn = _group_run(base, dev, want_on=[True, False, True])
    assert gn[1] is None
    for i in range(3):
        so, sn = _run(base[i], dev) if i != 1 else (None, None)
        if i != 1:
            assert np.array_equal(go[i], so) and np.array_equal(gn[i], sn)
        e_off, _ = lora_linear_ref(base[i].x, base[i].W, base[i].A, base[i].B, base[i].s)
        assert_rel(go[i], e_off, f"member {i} y_off")


@pytest.mark.parametrize("names", [("q", "k", "v"), ("gate", "up")])
def test_group_prefill_layer_full_size(names, dev):
    """The prefill layer's linears that share an input (q/k/v: 768 tiles, three rounds of the persistent launch;
    gate/up: 1376 tiles, a last round of 96) as one group call: each member has the bits of its single call, and
    every row of both outputs matches the oracle."""
    say("group prefill", names)
    cases = {c.name: c for c in WL.make("prefill_layer")}
    group = [cases[n] for n in names]
    go, gn = _group_run(group, dev)
    for i, c in enumerate(group):
        so, sn = _run(c, dev)
        assert np.array_equal(go[i], so) and np.array_equal(gn[i], sn), c.name
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(go[i], e_off, f"group {c.name} y_off")
        assert_rel(gn[i], e_on, f"group {c.name} y_on")


@pytest.mark.parametrize("M,K,N,r,G", [
    (1000, 136, 1040, 16, 8),   # 320 tiles: two rounds, the second of 64 (eight per XCD)
    (2050, 72, 1300, 9, 3),     # 306 tiles, a one-row last row tile; last round of 50 (not a multiple of 8)
    (520, 200, 2100, 32, 7),    # rank 32, 315 tiles
])
def test_group_gemm_several_rounds(M, K, N, r, G, dev):
    """More tiles than CUs: the persistent workgroups run several rounds, each one streaming the next tile's slabs
    through the ring while the current tile's epilogue runs; members alternate scales and one has no adapter."""
    say("group gemm rounds", M, K, N, r, G)
    cases = [WL.gen_linear(700 + 10 * G + i, M, K, N, r, s=[2.0, -0.5, 1.5][i % 3]) for i in range(G)]
    want_on = [i != 1 for i in range(G)]
    go, gn = _group_run(cases, dev, want_on=want_on)
    for i, c in enumerate(cases):
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(go[i], e_off, f"member {i} y_off")
        if want_on[i]:
            assert_rel(gn[i], e_on, f"member {i} y_on")
        else:
            assert gn[i] is None


def test_opt13b_decode_rank128_group(dev):
    """OPT-1.3b decode step: the generation batch of 6 rows through the four 2048 x 2048 attention projections at
    rank 128, one group call, each member against the oracle and against its single call."""
    cases = WL.make("opt13b_decode_r128")
    say("opt13b decode r128", len(cases))
    go, gn = _group_run(cases, dev)
    for i, c in enumerate(cases):
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(go[i], e_off, f"{c.name} y_off")
        assert_rel(gn[i], e_on, f"{c.name} y_on")
        so, sn = _run(c, dev)
        assert np.array_equal(go[i], so) and np.array_equal(gn[i], sn), c.name
