"""Every entry point enqueues on the stream it is given: each call runs on a second stream (default priority) with
its outputs NaN-filled on that stream, only that stream is synchronised, and the results must have the bits of the
same call on the default stream."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from gpu_helpers import dev_bf16, host, say

pytestmark = pytest.mark.gpu


def _cases(dev):
    import torch
    nan = float("nan")

    def full(*shape):
        return torch.full(shape, nan, device=dev)

    def lin_inputs(c):
        return (dev_bf16(c.x, dev), dev_bf16(c.W, dev), dev_bf16(c.A, dev) if c.r else None,
                dev_bf16(c.B, dev) if c.r else None)

    cases = {}
    for name, (M, K, N, r) in {"linear_decode": (4, 512, 264, 16), "linear_prefill": (130, 520, 300, 16)}.items():
        c = WL.gen_linear(950 + M, M, K, N, r)
        x, W, A, B = lin_inputs(c)

        def run(st, c=c, x=x, W=W, A=A, B=B):
            o = {"y_off": full(c.M, c.N), "y_on": full(c.M, c.N)}
            H.hydra_lora_linear(x, W, A, B, c.s, o["y_off"], o["y_on"], stream=st)
            return o
        cases[name] = run

    cw = WL.gen_linear(953, 130, 256, 264, 128)
    xw, Ww, Aw, Bw = lin_inputs(cw)

    def run_ws(st):
        o = {"y_off": full(cw.M, cw.N), "y_on": full(cw.M, cw.N)}
        ws = torch.empty(H.hydra_lora_linear_workspace_bytes(cw.M, cw.N, cw.r), dtype=torch.uint8, device=dev)
        H.hydra_lora_linear_ws(xw, Ww, Aw, Bw, cw.s, o["y_off"], o["y_on"], workspace=ws, stream=st)
        return o
    cases["linear_ws_r128"] = run_ws

    grp = [WL.gen_linear(960 + i, 4, 512, 256, 16) for i in range(3)]
    gin = [lin_inputs(c) for c in grp]

    def run_group(st):
        o = {f"{k}{i}": full(c.M, c.N) for i, c in enumerate(grp) for k in ("off", "on")}
        H.hydra_lora_linear_group([g[0] for g in gin], [g[1] for g in gin], [g[2] for g in gin],
                                  [g[3] for g in gin], [c.s for c in grp], [o[f"off{i}"] for i in range(3)],
                                  [o[f"on{i}"] for i in range(3)], stream=st)
        return o
    cases["group"] = run_group

    mc = WL.gen_linear(970, 4, 512, 256, 16)
    xm, Wm, Am, Bm = lin_inputs(mc)
    x2 = dev_bf16(WL.gen_linear(971, 4, 512, 256, 16).x, dev)

    def run_multi(st):
        o = {"off": full(mc.M, mc.N), "on0": full(mc.M, mc.N), "on1": full(mc.M, mc.N)}
        H.hydra_lora_linear_multi(xm, Wm, [xm, x2], [Am, Am], [Bm, Bm], [mc.s, -mc.s], o["off"],
                                  [o["on0"], o["on1"]], stream=st)
        return o
    cases["multi"] = run_multi

    sc = WL.gen_score_head(980, 2, 64, 256, 1000, 16)
    h, Wl, As, Bs, w_rm = (dev_bf16(a, dev) for a in (sc.h, sc.W_lm, sc.A, sc.B, sc.w_rm))
    ids = torch.from_numpy(sc.ids).to(dev)

    def run_score(st):
        o = {k: full(sc.M) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
        o["reward"] = full(sc.n_seq)
        H.hydra_score(h, Wl, As, Bs, sc.s, ids, w_rm, sc.n_seq, sc.seq_len, o["lp_on"], o["lp_off"], o["kl"],
                      reward=o["reward"], lse_on=o["lse_on"], lse_off=o["lse_off"], stream=st)
        return o
    cases["score"] = run_score

    on, off, lids = WL.gen_logits(981, 6, 1000)
    lon, loff = torch.from_numpy(on).to(dev), torch.from_numpy(off).to(dev)
    lid = torch.from_numpy(lids.astype(np.int32)).to(dev)

    def run_logits(st):
        o = {k: full(6) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
        H.hydra_score_logits(lon, loff, lid, o["lp_on"], o["lp_off"], o["kl"], o["lse_on"], o["lse_off"], stream=st)
        return o
    cases["score_logits"] = run_logits

    rng = np.random.default_rng(982)
    n_seq, seq_len = 3, 40
    M = n_seq * seq_len

    def f32(*shape):
        return torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(dev)
    kl, rew, vals, lp_new = f32(M), f32(n_seq), f32(M), f32(M)
    lp_old = torch.from_numpy(-rng.uniform(0.5, 4.0, M).astype(np.float32)).to(dev)

    def run_adv(st):
        o = {"adv": full(M), "ret": full(M), "rewards": full(M), "losses": full(3), "d_lp": full(M),
             "d_v": full(M)}
        H.hydra_ppo_advantages(kl, rew, vals, n_seq, seq_len, o["adv"], o["ret"], rewards=o["rewards"], start=5,
                               stream=st)
        H.hydra_ppo_loss(lp_new, lp_old, o["adv"], vals, o["ret"], n_seq, seq_len, o["losses"], d_lp=o["d_lp"],
                         d_v=o["d_v"], start=5, stream=st)
        return o
    cases["advantages_and_loss"] = run_adv

    hv = dev_bf16(WL.gen_linear(983, 70, 520, 8, 0).x, dev)
    wv = dev_bf16(WL.gen_linear(984, 1, 520, 8, 0).x[0], dev)

    def run_value(st):
        o = {"values": full(70)}
        H.hydra_value_head(hv, wv, o["values"], stream=st)
        return o
    cases["value_head"] = run_value

    bw = WL.gen_backward(985, 130, 256, 264, 16)
    c = bw.lin
    xb, Wb, Ab, Bb = lin_inputs(c)
    dyb = dev_bf16(bw.dy, dev)

    def run_bwd(st):
        Wt = torch.empty((c.K, c.N), dtype=Wb.dtype, device=dev)
        H.hydra_transpose_bf16(Wb, Wt, stream=st)
        o = {"dx": full(c.M, c.K), "dA": full(c.r, c.K), "dB": full(c.N, c.r)}
        H.hydra_lora_linear_backward(xb, Wt, Ab, Bb, c.s, dyb, o["dx"], o["dA"], o["dB"], stream=st)
        o["Wt"] = Wt
        return o
    cases["transpose_and_backward"] = run_bwd
    return cases


def test_every_entry_point_runs_on_the_given_stream(dev):
    import torch
    cases = _cases(dev)
    torch.cuda.synchronize()
    side = torch.cuda.Stream(device=dev)
    for name, run in cases.items():
        say("stream", name)
        ref = run(None)
        torch.cuda.synchronize()
        ref = {k: host(v).copy() for k, v in ref.items()}
        with torch.cuda.stream(side):
            got = run(side)
        side.synchronize()
        for k, v in got.items():
            g = host(v)
            assert np.array_equal(g.view(np.uint8), ref[k].view(np.uint8)), f"{name}: {k} differs on a second stream"


def test_concurrent_calls_from_two_threads_on_two_streams(dev):
    """The library keeps no mutable state between calls: two host threads, each calling entry points on its own
    stream at the same time, get the bits of the calls made one after the other."""
    import threading

    import torch
    cases = _cases(dev)
    torch.cuda.synchronize()
    groups = [["score", "linear_prefill", "group", "advantages_and_loss"],
              ["transpose_and_backward", "linear_ws_r128", "multi", "score_logits", "value_head", "linear_decode"]]
    ref = {}
    for name in sum(groups, []):
        o = cases[name](None)
        torch.cuda.synchronize()
        ref[name] = {k: host(v).copy() for k, v in o.items()}
    say("two threads, two streams")
    streams = [torch.cuda.Stream(device=dev) for _ in groups]
    got = [dict() for _ in groups]
    errors = []
    start = threading.Barrier(len(groups))

    def worker(i):
        try:
            torch.cuda.set_device(dev)
            start.wait(timeout=30)
            with torch.cuda.stream(streams[i]):
                for _ in range(3):
                    for name in groups[i]:
                        got[i][name] = cases[name](streams[i])
            streams[i].synchronize()
        except BaseException as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(groups))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    for i, names in enumerate(groups):
        for name in names:
            for k, v in got[i][name].items():
                assert np.array_equal(host(v).view(np.uint8), ref[name][k].view(np.uint8)), f"{name}: {k}"
