"""hydra_score_noalloc (the scoring pass with its workspace in the library's own device scratch) against hydra_score
with a caller workspace, through the C ABI: bit-identical outputs on consecutive calls of decreasing size, the
oracle's tolerances, and replays from a captured HIP graph."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import reward_ref, score_head_ref
from gpu_helpers import assert_abs, assert_rel, dev, dev_bf16, host, row_chunks, say

pytestmark = pytest.mark.gpu

KEYS = ("lp_on", "lp_off", "kl", "lse_on", "lse_off", "reward", "err")


def _inputs(c, device):
    import torch
    return dict(h=dev_bf16(c.h, device), W=dev_bf16(c.W_lm, device), A=dev_bf16(c.A, device),
                B=dev_bf16(c.B, device), ids=dev(c.ids.astype(np.int32), device), w_rm=dev_bf16(c.w_rm, device))


def _outputs(c, device):
    import torch
    out = {k: torch.full((c.M,), float("nan"), device=device) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
    out["reward"] = torch.full((c.n_seq,), float("nan"), device=device)
    out["err"] = torch.zeros(1, dtype=torch.int32, device=device)
    return out


def _call(c, t, o, noalloc, ws=None):
    args = (t["h"], t["W"], t["A"], t["B"], c.s, t["ids"], t["w_rm"], c.n_seq, c.seq_len, o["lp_on"], o["lp_off"],
            o["kl"])
    kw = dict(reward=o["reward"], lse_on=o["lse_on"], lse_off=o["lse_off"], err_flag=o["err"])
    if noalloc:
        H.hydra_score_noalloc(*args, **kw)
    else:
        H.hydra_score(*args, workspace=ws, **kw)


def _host(o):
    return {k: host(v).copy() for k, v in o.items()}


def test_score_noalloc_matches_workspace_call_twice(dev):
    """Two calls in a row on one GPU: the Llama-7B scoring pass (2048 x 32000, 21.5 MB of scratch), then a smaller
    ragged one; each has the bits of hydra_score with its own workspace and the oracle's tolerances."""
    import torch
    cases = [WL.make("two_head_score"), WL.gen_score_head(7002, 3, 37, 264, 1003, 24)]
    for i, c in enumerate(cases):
        say("score_noalloc call", i, c.M, c.K, c.V, c.r)
        t = _inputs(c, dev)
        ref = _outputs(c, dev)
        ws = torch.full((H.hydra_score_workspace_bytes(c.M, c.V),), 0xFF, dtype=torch.uint8, device=dev)
        _call(c, t, ref, noalloc=False, ws=ws)
        got = _outputs(c, dev)
        _call(c, t, got, noalloc=True)
        torch.cuda.synchronize()
        g, r = _host(got), _host(ref)
        for k in KEYS:
            assert np.array_equal(g[k], r[k]), f"call {i}: {k} differs from hydra_score"
        assert g["err"][0] == 0
        # the oracle's tolerances (every row of the small case; the first row block of the large one)
        for rows in row_chunks(c.M)[: (1 if c.M > 1024 else None)]:
            e = score_head_ref(c.h[rows], c.W_lm, c.A, c.B, c.s, c.ids[rows])
            for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off"):
                assert_abs(g[k][rows], e[k], f"call {i} {k}")
        assert_rel(g["reward"], reward_ref(c.h, c.w_rm, c.n_seq, c.seq_len), f"call {i} reward")


def test_score_noalloc_replays_in_a_hip_graph(dev):
    """Captured in a HIP graph (a caller that cannot allocate) and replayed three times with eager work between the
    replays: every replay has the bits of the eager call."""
    import torch
    c = WL.gen_score_head(7003, 2, 64, 256, 1000, 16)
    say("score_noalloc graph", c.M, c.K, c.V, c.r)
    t = _inputs(c, dev)
    o = _outputs(c, dev)
    _call(c, t, o, noalloc=True)
    torch.cuda.synchronize()
    eager = _host(o)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _call(c, t, o, noalloc=True)
    torch.cuda.synchronize()
    other = WL.gen_score_head(7004, 1, 40, 256, 777, 8)
    to, oo = _inputs(other, dev), _outputs(other, dev)
    for rep in range(3):
        for k, v in o.items():
            if k != "err":
                v.fill_(float("nan"))
        _call(other, to, oo, noalloc=True)  # eager work on the same scratch between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _host(o)
        for k in KEYS:
            assert np.array_equal(got[k], eager[k]), f"replay {rep}: {k}"
