"""GPU parity of hydra_lora_linear_group_ws: the decode step in one launch (T = x A^T published by the first
workgroups, the LoRA update added by the workgroups that stream W), and the workspace group call at every row
class, against the oracle."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import lora_linear_ref
from gpu_helpers import assert_rel, dev_bf16, host, say

pytestmark = pytest.mark.gpu


def _inputs(cases, device, want_on=None):
    import torch
    G = len(cases)
    want_on = want_on or [True] * G
    t = dict(
        xs=[dev_bf16(c.x, device) for c in cases],
        Ws=[dev_bf16(c.W, device) for c in cases],
        As=[dev_bf16(c.A, device) if (c.r and want_on[i]) else None for i, c in enumerate(cases)],
        Bs=[dev_bf16(c.B, device) if (c.r and want_on[i]) else None for i, c in enumerate(cases)],
        ss=[c.s for c in cases],
        yo=[torch.full((c.M, c.N), float("nan"), device=device) for c in cases],
        yn=[torch.full((c.M, c.N), float("nan"), device=device) if want_on[i] else None
            for i, c in enumerate(cases)],
    )
    return t


def _call(t, ws):
    import torch
    H.hydra_lora_linear_group_ws(t["xs"], t["Ws"], t["As"], t["Bs"], t["ss"], t["yo"], t["yn"], workspace=ws)
    torch.cuda.synchronize()
    return [host(v).copy() for v in t["yo"]], [None if v is None else host(v).copy() for v in t["yn"]]


POISON = 1 << 31


def _keeper_runs(M, r, K):
    """Whether a single-launch decode call publishes T through the workspace (and so advances its generation): padded
    rank 32 and up, or rank 16 above 4 rows or above K = 2048; up to 4 rows, rank 0 needs no T and rank 16 with
    K <= 2048 forms T in every workgroup."""
    rp = 0 if r == 0 else 16 if r <= 16 else 32 if r <= 32 else 64 if r <= 64 else 128
    return M <= 8 and (rp >= 32 or (rp == 16 and (M > 4 or K > 2048)))


def _ctl(ws):
    """(bucket counts, generation word copies) of the workspace's 32 bucket lines (line 2 + q: a 64-bit word, low
    half the count, high half the generation word)."""
    c = host(ws[:H.HYDRA_GROUP_WS_CONTROL_BYTES]).view(np.uint32)
    lines = [2 * 32 + 32 * q for q in range(32)]
    return [int(c[i]) for i in lines], [int(c[i + 1]) for i in lines]


def _assert_generation(ws, launches, poisoned=False):
    """After a call: every copy of the generation word advanced to `launches`, and every count cleared.  (Once a
    keeper's wait has run out, a report can land after its clearing; the counts then stay unchecked, as the poison
    bit makes every later call form T itself until the workspace is zeroed.)"""
    counts, gens = _ctl(ws)
    if not poisoned:
        assert counts == [0] * 32, counts
    want = launches | (POISON if poisoned else 0)
    assert gens == [want] * 32, (gens[:4], want)


def _check(cases, go, gn, want_on=None):
    want_on = want_on or [True] * len(cases)
    for i, c in enumerate(cases):
        e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
        assert_rel(go[i], e_off, f"member {i} y_off")
        if want_on[i]:
            assert_rel(gn[i], e_on, f"member {i} y_on")
        else:
            assert gn[i] is None


@pytest.mark.parametrize("M,K,N,r,G", [
    (1, 512, 256, 16, 1), (2, 1032, 200, 8, 3), (4, 4096, 520, 16, 4), (3, 8200, 130, 32, 2),
    (6, 2048, 300, 128, 4), (8, 1000, 64, 64, 2), (5, 264, 33, 1, 8), (4, 520, 100, 0, 2),
])
def test_group_ws_decode_matches_oracle(M, K, N, r, G, dev):
    """One launch per call at M <= 8: every rank class (0, 1, 8, 16, 32, 64, 128), ragged K (segments of x
    past 4096, a K tail inside a chunk) and N (a partial 16-row block), up to 8 members."""
    say("group_ws decode", M, K, N, r, G)
    cases = [WL.gen_linear(1100 + 10 * G + i, M, K, N, r, s=[2.0, -0.5, 1.5][i % 3]) for i in range(G)]
    t = _inputs(cases, dev)
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn)
    # one launch: the counts are clear again and the generation has advanced by one where T is published
    _assert_generation(ws, 1 if _keeper_runs(M, r, K) else 0)


def test_group_ws_repeated_calls_reuse_the_workspace(dev):
    """Ten calls in a row on one workspace with changing inputs: each gives the oracle's result, and a repeated
    input gives the same bits."""
    import torch
    say("group_ws repeated")
    M, K, N, r, G = 4, 2048, 400, 16, 4
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    first = None
    for it in range(10):
        seed = 1200 + (it % 3)
        cases = [WL.gen_linear(seed * 10 + i, M, K, N, r) for i in range(G)]
        go, gn = _call(_inputs(cases, dev), ws)
        if it in (0, 1, 2):
            _check(cases, go, gn)
        if it == 0:
            first = (go, gn)
        if it in (3, 6, 9):  # seed 1200 again
            for i in range(G):
                assert np.array_equal(go[i], first[0][i]) and np.array_equal(gn[i], first[1][i])
    _assert_generation(ws, 10 if _keeper_runs(M, r, K) else 0)


def test_group_ws_members_without_adapter(dev):
    """A LoRA-off member (no y_on, no adapter) between members with adapters, and a member whose y_on has no
    adapter's update to wait for."""
    say("group_ws mixed members")
    cases = [WL.gen_linear(1300 + i, 4, 1024, 260, 16) for i in range(3)]
    want_on = [True, False, True]
    t = _inputs(cases, dev, want_on)
    ws = H.hydra_lora_linear_group_workspace(3, 4, 260, 16, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn, want_on)


@pytest.mark.parametrize("M,K,N,r", [(6, 4096, 2048, 128), (4, 4096, 4096, 16)])
def test_group_ws_wait_bound_fallback_same_bits(M, K, N, r, dev):
    """With the wait bound word set to one round, workgroups that find T (or, up to rank 64, a row's published
    LoRA-off output) not yet there form it themselves through the same routine: the bits are those of the default
    bound.  If the keeper's wait ran out too, the workspace stays poisoned (every later call forms them where they
    are used, same bits) until it is zeroed."""
    import torch
    say("group_ws wait bound", M, K, N, r)
    G = 4
    cases = [WL.gen_linear(1400 + i, M, K, N, r) for i in range(G)]
    t = _inputs(cases, dev)
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn)
    _assert_generation(ws, 1)
    bw = 4 * H.HYDRA_GROUP_WS_BOUND_WORD
    bound = ws[bw:bw + 4].view(torch.int32)  # the caller's wait bound word (0 selects the default)
    bound.fill_(1)
    go1, gn1 = _call(t, ws)
    for i in range(G):
        assert np.array_equal(go[i], go1[i]) and np.array_equal(gn[i], gn1[i]), i
    assert int(host(ws[bw:bw + 4].view(torch.int32))[0]) == 1  # the bound word is the caller's, not reset
    bound.fill_(0)
    poisoned = (_ctl(ws)[1][0] & POISON) != 0
    _assert_generation(ws, 2, poisoned)
    go2, gn2 = _call(t, ws)
    for i in range(G):
        assert np.array_equal(go[i], go2[i]) and np.array_equal(gn[i], gn2[i]), i
    _assert_generation(ws, 3, poisoned)  # poison is kept


def test_group_ws_poisoned_workspace_same_bits_until_zeroed(dev):
    """A workspace whose generation word carries the poison bit (what a keeper leaves when its bounded wait runs
    out, set here from the host): every call forms T in every workgroup and gives the bits of a normal call, the
    bit stays set, and zeroing the workspace restores normal calls."""
    import torch
    say("group_ws poisoned")
    M, K, N, r, G = 4, 2048, 1024, 32, 4
    cases = [WL.gen_linear(1450 + i, M, K, N, r) for i in range(G)]
    t = _inputs(cases, dev)
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn)
    words = ws[:H.HYDRA_GROUP_WS_CONTROL_BYTES].view(torch.int32)
    for q in range(32):
        words[2 * 32 + 32 * q + 1] = (1 | POISON) - (1 << 32)  # the same bits as a signed 32-bit value
    torch.cuda.synchronize()
    for it in range(2):
        go1, gn1 = _call(t, ws)
        for i in range(G):
            assert np.array_equal(go[i], go1[i]) and np.array_equal(gn[i], gn1[i]), (it, i)
        _assert_generation(ws, 2 + it, poisoned=True)
    ws.zero_()
    go2, gn2 = _call(t, ws)
    for i in range(G):
        assert np.array_equal(go[i], go2[i]) and np.array_equal(gn[i], gn2[i]), i
    _assert_generation(ws, 1)


@pytest.mark.parametrize("M,r", [(12, 16), (16, 128), (130, 16), (130, 128)])
def test_group_ws_above_decode_rows(M, r, dev):
    """9..16 rows (the small-M MFMA kernel; at rank 128 two single-launch halves) and the GEMM rows (rank 128 per
    member through the pre-pass GEMM, each over its own part of the workspace)."""
    say("group_ws rows", M, r)
    K, N, G = 520, 300, 3
    cases = [WL.gen_linear(1500 + 7 * M + i, M, K, N, r, s=1.0 + i) for i in range(G)]
    t = _inputs(cases, dev)
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn)
    # the single launch runs only at rank 128 up to 16 rows (once per row half)
    _assert_generation(ws, 2 if (M <= 16 and r > 64) else 0)


@pytest.mark.parametrize("r,G,off,b2", [(128, 3, None, False), (128, 8, None, False), (128, 3, 1, False),
                                        (100, 3, None, False), (128, 3, None, True)])
def test_group_ws_rank128_rows_same_bits_as_linear_ws(r, G, off, b2, dev):
    """Above 16 rows at padded rank 128 each member has a pre-pass workspace of its own: with every B of exactly 128
    columns the members' pre-passes share one pair of launches (also with a member without adapter), at rank 100 each
    member pads its B in turn, and so it does when one B is only 2-byte aligned (b2).  Either way every member's outputs carry the bits of hydra_lora_linear_ws on that
    member alone (the same K chunks, summed in the same order), and match the oracle."""
    import torch
    say("group_ws rank-128 rows", r, G, off, b2)
    M, K, N = 300, 520, 264
    want_on = [i != off for i in range(G)]
    cases = [WL.gen_linear(1700 + 11 * G + i, M, K, N, r, s=0.5 + i) for i in range(G)]
    t = _inputs(cases, dev, want_on)
    if b2:
        # member 1's B at a 2-byte offset inside a larger buffer (same values)
        buf = torch.empty(N * r + 8, dtype=t["Bs"][1].dtype, device=dev)
        t["Bs"][1] = buf[1:1 + N * r].view(N, r)
        t["Bs"][1].copy_(dev_bf16(cases[1].B, dev))
        assert t["Bs"][1].data_ptr() % 16 != 0
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn, want_on)
    for i in range(G):
        yo = torch.full((M, N), float("nan"), device=dev)
        yn = torch.full((M, N), float("nan"), device=dev) if want_on[i] else None
        H.hydra_lora_linear_ws(t["xs"][i], t["Ws"][i], t["As"][i], t["Bs"][i], t["ss"][i], yo, yn)
        torch.cuda.synchronize()
        assert np.array_equal(host(yo), go[i]), i
        if want_on[i]:
            assert np.array_equal(host(yn), gn[i]), i
    go2, gn2 = _call(t, ws)
    for i in range(G):
        assert np.array_equal(go[i], go2[i]) and (gn[i] is None or np.array_equal(gn[i], gn2[i])), i


@pytest.mark.parametrize("N", [16000, 20000])
def test_group_ws_output_region_limit(N, dev):
    """Up to rank 64 the stream workgroups publish their LoRA-off outputs in a region of fixed size
    (HYDRA_GROUP_WS_Y_BYTES, G x N x 8 rows x 8 bytes here): at N = 16000 they fit and the LoRA update runs at the
    tail of the launch, at N = 20000 they do not and the workgroups that stream W add it themselves.  Both match the
    oracle and advance the generation once."""
    say("group_ws output region", N)
    M, K, r, G = 8, 256, 16, 2
    assert (G * N * 8 * 8 <= H.HYDRA_GROUP_WS_Y_BYTES) == (N == 16000)
    cases = [WL.gen_linear(1650 + i, M, K, N, r) for i in range(G)]
    t = _inputs(cases, dev)
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn)
    _assert_generation(ws, 1)


def test_group_ws_decode_qkvo_full(dev):
    """The decode step of the Llama-7B attention projections (batch 4, 4096 x 4096, r = 16) as one call."""
    say("group_ws decode_qkvo")
    cases = WL.make("decode_qkvo")
    t = _inputs(cases, dev)
    ws = H.hydra_lora_linear_group_workspace(len(cases), 4, 4096, 16, dev)
    go, gn = _call(t, ws)
    _check(cases, go, gn)


@pytest.mark.parametrize("r", [16, 32])
def test_group_ws_graph_replays(r, dev):
    """Captured in a HIP graph and replayed three times with eager work between the replays: every replay has the
    bits of the eager call (at rank 32 every launch, replayed or eager, advances the workspace's generation; at rank
    16 the workgroups form T themselves)."""
    import torch
    say("group_ws graph", r)
    M, K, N, G = 4, 1024, 512, 4
    cases = [WL.gen_linear(1600 + i, M, K, N, r) for i in range(G)]
    t = _inputs(cases, dev)
    ws = H.hydra_lora_linear_group_workspace(G, M, N, r, dev)
    eo, en = _call(t, ws)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        H.hydra_lora_linear_group_ws(t["xs"], t["Ws"], t["As"], t["Bs"], t["ss"], t["yo"], t["yn"], workspace=ws)
    torch.cuda.synchronize()
    other = [WL.gen_linear(1700 + i, M, K, N, r) for i in range(G)]
    to = _inputs(other, dev)
    for rep in range(3):
        for v in t["yo"] + t["yn"]:
            v.fill_(float("nan"))
        _call(to, ws)  # eager work on the same workspace between the replays
        g.replay()
        torch.cuda.synchronize()
        for i in range(G):
            assert np.array_equal(host(t["yo"][i]), eo[i]) and np.array_equal(host(t["yn"][i]), en[i]), (rep, i)
    _assert_generation(ws, (1 + 3 * 2) if _keeper_runs(M, r, K) else 0)
