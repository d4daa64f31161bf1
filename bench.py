"""Benchmark of the Hydra-PPO hot path on one MI355X.

One step is one pass of the whole path over one batch of 4 sequences x 512
tokens at Llama-7B shapes (hidden 4096, MLP 11008, vocabulary 32000, LoRA
rank 16, scale 2), i.e. the inference stage of one PPO iteration for one
decoder layer plus the heads:

  * decode: one generation step of the four attention projections, M = 4
    (hydra_lora_linear_group_ws: one bandwidth-bound launch), both LoRA-off and LoRA-on outputs;
  * prefill: the seven LoRA linears of a layer over all 2048 tokens
    (hydra_lora_linear, dual-output MFMA GEMM), both outputs;
  * score: the CLM head with LoRA on and off, sampled-token log-probabilities,
    per-token KL and the reward head over the 2048 tokens (hydra_score; the
    logits are never materialised).

Inputs are synthetic (seeded Gaussians, see workloads/) and already resident
in HBM when the timed region starts.  The timed region is K steps back to
back on the launch stream between two HIP events.  A parts pass afterwards
runs K more steps with an event at the start of each part (and at the step's
end), so each part's time covers its launches back to back plus one event's
overhead; a detail pass then brackets every launch with its own pair of events
(those figures include the events' own overhead, a few microseconds each).  The
decode step is one launch of hydra_lora_linear_group_ws (T = x A^T published by
its first workgroups, the LoRA update added by the workgroups that stream W).  The standalone scoring epilogue over
materialised logits (hydra_score_logits, 512 x 32000) is timed separately
(rotating four input sets so that the 256 MB last-level cache does not serve
it) and reported under "aux"; it is not part of the step.  So is the PPO
advantage step that follows scoring (hydra_value_head on the 2048 critic
hidden states, then hydra_ppo_advantages).

Prints one JSON line.  ``--gpus`` above 1 is refused: this path is built and
measured on a single GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "dual-path LoRA GEMM TFLOP/s + scoring tokens/s, % of MFMA/HBM roofline"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E
AUX_NAMES = ("score_logits", "single_linear", "ppo_advantages", "decode_multi", "lora_backward_layer",
             "opt13b_r128", "score_two_input")


def lin_flops(M, K, N, r):
    return 2.0 * M * K * N + 2.0 * M * K * r + 2.0 * M * r * N


def lin_bytes(M, K, N, r):
    return 2.0 * (M * K + N * K + r * K + N * r) + 2 * 4.0 * M * N


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=30,
                   help="untimed steps first: the clock settles over the first few tens of milliseconds")
    p.add_argument("--parts", default="decode,prefill,score",
                   help="comma list of step parts to run (profiling aid; the metric needs all three; "
                        "'advantages' adds the PPO advantage step, which is also timed under aux)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-aux", action="store_true")
    p.add_argument("--aux", default=",".join(AUX_NAMES),
                   help="comma list of the auxiliary measurements to run after the step (profiling aid)")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the CPU oracle sample")
    p.add_argument("--copy-bytes", type=int, default=0,
                   help="run one plain device-to-device copy of this many bytes before the steps "
                        "(calibrates FETCH_SIZE / WRITE_SIZE counters in a profiling run)")
    a = p.parse_args()
    unknown = [x for x in a.aux.split(",") if x and x not in AUX_NAMES]
    if unknown:
        p.error(f"unknown --aux entries {unknown}; known: {', '.join(AUX_NAMES)}")
    return a


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print(f"bench.py: --gpus {max(args.gpus, world)} refused: the path runs and is measured on one GPU "
              f"(the data-parallel sharding is described, not launched)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2309_00754_amd as H
    import workloads as WL

    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)
    H.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    parts = [p for p in args.parts.split(",") if p]
    aux_names = [a for a in args.aux.split(",") if a]

    def bf(u):
        return torch.from_numpy(np.ascontiguousarray(u).view(np.int16)).to(dev)

    t_gen = time.perf_counter()
    launches = []   # (part, label, fn, flops, bytes)
    host = {}

    if "decode" in parts:
        # the four attention projections of one decode step, one grouped launch
        host["decode"] = dec = WL.make("decode_qkvo")
        xd = bf(dec[0].x)
        gW = [bf(c.W) for c in dec]
        gA = [bf(c.A) for c in dec]
        gB = [bf(c.B) for c in dec]
        gyo = [torch.empty(c.M, c.N, device=dev) for c in dec]
        gyn = [torch.empty(c.M, c.N, device=dev) for c in dec]
        dws = H.hydra_lora_linear_group_workspace(len(dec), dec[0].M, dec[0].N, dec[0].r, dev)
        fn = (lambda: H.hydra_lora_linear_group_ws([xd] * len(dec), gW, gA, gB, [c.s for c in dec], gyo, gyn,
                                                   workspace=dws))
        launches.append(("decode", "qkvo", fn, sum(lin_flops(c.M, c.K, c.N, c.r) for c in dec),
                         sum(lin_bytes(c.M, c.K, c.N, c.r) for c in dec)))
    if "prefill" in parts:
        # the seven linears as a layer issues them: q/k/v share their input (one group call), then o, then
        # gate/up (one group call), then down; every call computes both outputs of each of its linears
        xs = {}
        host["prefill"] = WL.make("prefill_layer")
        dev_in = {}
        for c in host["prefill"]:
            if id(c.x) not in xs:
                xs[id(c.x)] = bf(c.x)
            dev_in[c.name] = (c, xs[id(c.x)], bf(c.W), bf(c.A), bf(c.B), torch.empty(c.M, c.N, device=dev),
                              torch.empty(c.M, c.N, device=dev))
        for names in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",)):
            mem = [dev_in[n] for n in names]
            if len(mem) == 1:
                c, x, W, A, B, yo, yn = mem[0]
                fn = (lambda x=x, W=W, A=A, B=B, s=c.s, yo=yo, yn=yn: H.hydra_lora_linear(x, W, A, B, s, yo, yn))
            else:
                fn = (lambda mem=mem: H.hydra_lora_linear_group([m[1] for m in mem], [m[2] for m in mem],
                                                                [m[3] for m in mem], [m[4] for m in mem],
                                                                [m[0].s for m in mem], [m[5] for m in mem],
                                                                [m[6] for m in mem]))
            launches.append(("prefill", "_".join(names), fn,
                             sum(lin_flops(m[0].M, m[0].K, m[0].N, m[0].r) for m in mem),
                             sum(lin_bytes(m[0].M, m[0].K, m[0].N, m[0].r) for m in mem)))
    sc = None
    if "score" in parts:
        sc = host["score"] = WL.make("two_head_score")
        h, Wl, A, B, w_rm = bf(sc.h), bf(sc.W_lm), bf(sc.A), bf(sc.B), bf(sc.w_rm)
        ids = torch.from_numpy(sc.ids).to(dev)
        M = sc.M
        lp_on, lp_off, kl = (torch.empty(M, device=dev) for _ in range(3))
        reward = torch.empty(sc.n_seq, device=dev)
        ws = torch.empty(H.hydra_score_workspace_bytes(M, sc.V), dtype=torch.uint8, device=dev)
        fn = (lambda: H.hydra_score(h, Wl, A, B, sc.s, ids, w_rm, sc.n_seq, sc.seq_len, lp_on, lp_off, kl,
                                    reward=reward, workspace=ws))
        fl = lin_flops(M, sc.K, sc.V, sc.r) + 2.0 * sc.n_seq * sc.K
        by = 2.0 * (M * sc.K + sc.V * sc.K + sc.r * sc.K + sc.V * sc.r + sc.K) + 4.0 * M + 3 * 4.0 * M + 4.0 * sc.n_seq
        launches.append(("score", "clm_rm_head", fn, fl, by))
    if "advantages" in parts:
        # the critic's value head on every token, then per-token rewards, GAE advantages and returns
        adv = host["advantages"] = WL.make("ppo_advantages")
        Ma = adv.M
        ha, wv = bf(adv.h), bf(adv.w_v)
        kl_a = torch.from_numpy(adv.kl).to(dev)
        rw_a = torch.from_numpy(adv.reward).to(dev)
        vals = torch.empty(Ma, device=dev)
        r_out, a_out, ret_out = (torch.empty(Ma, device=dev) for _ in range(3))
        launches.append(("advantages", "value_head", (lambda: H.hydra_value_head(ha, wv, vals)),
                         2.0 * Ma * adv.K, 2.0 * Ma * adv.K + 2.0 * adv.K + 4.0 * Ma))
        launches.append(("advantages", "gae",
                         (lambda: H.hydra_ppo_advantages(kl_a, rw_a, vals, adv.n_seq, adv.seq_len, a_out, ret_out,
                                                         rewards=r_out, start=adv.start, beta=adv.beta,
                                                         gamma=adv.gamma, lam=adv.lam)),
                         10.0 * Ma, 4.0 * Ma * 2 + 4.0 * adv.n_seq + 4.0 * Ma * 3))
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen

    if args.copy_bytes > 0:
        src = torch.full((args.copy_bytes,), 7, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    stream = torch.cuda.current_stream()

    part_order = []
    for l in launches:
        if l[0] not in part_order:
            part_order.append(l[0])

    def step(evs=None, per_launch=False):
        # evs: one event per part boundary (the part's first launch) plus a closing one; with per_launch, a
        # pair of events around every launch instead (a detail pass: each pair adds its own overhead)
        cur = None
        for i, (part, _, fn, _, _) in enumerate(launches):
            if evs is not None and per_launch:
                evs[i][0].record(stream)
            elif evs is not None and part != cur:
                evs[part_order.index(part)].record(stream)
                cur = part
            fn()
            if evs is not None and per_launch:
                evs[i][1].record(stream)
        if evs is not None and not per_launch:
            evs[-1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps

    def new_event():
        return torch.cuda.Event(enable_timing=True)

    # the timed region: K steps back to back on the launch stream, one event before and one after
    start, end = new_event(), new_event()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    start.record(stream)
    for k in range(K):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / K

    # parts pass, outside the timed region: K more steps with an event at each part boundary; per-part durations
    # (ms) averaged over them (each boundary event adds its own small overhead to the part it opens)
    evs = [[new_event() for _ in range(len(part_order) + 1)] for _ in range(K)]
    p0, p1 = new_event(), new_event()
    p0.record(stream)
    for k in range(K):
        step(evs[k])
    p1.record(stream)
    torch.cuda.synchronize()
    parts_pass_ms = p0.elapsed_time(p1) / K
    part_ms = {p: float(np.mean([evs[k][j].elapsed_time(evs[k][j + 1]) for k in range(K)]))
               for j, p in enumerate(part_order)}

    # detail pass, outside the timed region: each launch between its own pair of events
    KD = min(K, 10)
    devs = [[(new_event(), new_event()) for _ in launches] for _ in range(KD)]
    for k in range(KD):
        step(devs[k], per_launch=True)
    torch.cuda.synchronize()
    avg = np.array([[devs[k][i][0].elapsed_time(devs[k][i][1]) for i in range(len(launches))]
                    for k in range(KD)]).mean(0)

    comp = {}
    for part in part_order:
        idx = [i for i, l in enumerate(launches) if l[0] == part]
        t = part_ms[part] * 1e-3
        fl = sum(launches[i][3] for i in idx)
        by = sum(launches[i][4] for i in idx)
        d = dict(launches=len(idx), us=round(t * 1e6, 2), tflops=round(fl / t / 1e12, 2),
                 gbps=round(by / t / 1e9, 1))
        if part in ("decode", "advantages"):
            d["bound"] = "hbm"
            d["frac"] = round(by / t / 1e9 / PEAK_HBM_GBPS, 4)
        else:
            d["bound"] = "mfma"
            d["frac"] = round(fl / t / 1e12 / PEAK_BF16_TFLOPS, 4)
        if part == "score":
            d["tokens_per_s"] = round(sc.M / t, 1)
        d["per_launch_us"] = {launches[i][1]: round(float(avg[i]) * 1e3, 2) for i in idx}
        comp[part] = d

    total_flops = sum(l[3] for l in launches)
    value = total_flops / (ms_per_step * 1e-3) / 1e12

    # the dominant kernel: the part with the largest share of the step
    dom = max(comp, key=lambda p: comp[p]["us"])
    dcomp = comp[dom]
    if dcomp["bound"] == "hbm":
        roof = dict(bound="hbm", achieved=dcomp["gbps"], peak=PEAK_HBM_GBPS, unit="GB/s", frac=dcomp["frac"])
    else:
        roof = dict(bound="mfma", achieved=dcomp["tflops"], peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                    frac=dcomp["frac"])
    roof["kernel"] = {"prefill": "lora_gemm_kernel<16,false> (4 copy + 4 MFMA waves, 128x256 tiles)",
                      "score": "lora_t_part_kernel<16> + lora_t_finish_kernel<16> + score_gemm_kernel<16,false> + "
                               "score_combine_kernel",
                      "decode": "gemv_split_kernel<4,16> (q/k/v/o in one launch)",
                      "advantages": "value_head_kernel + gae_kernel"}[dom]
    tr = committed_traffic(dom)
    roof["traffic"] = None if tr is None else tr["bytes_per_launch"]
    if tr is not None:
        roof["traffic_detail"] = tr

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_with_part_events": round(parts_pass_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "hydra_ppo_inference_pass_llama7b_b4x512",
            "parts": parts,
            "batch": 4, "seq_len": 512, "hidden": 4096, "mlp": 11008, "vocab": 32000,
            "lora_rank": 16, "lora_scale": 2.0, "decode_rows": 4, "prefill_rows": 2048,
            "parallelism": "single_gpu",
        },
        "scoring_tokens_per_s": comp.get("score", {}).get("tokens_per_s"),
        "roofline": roof,
        "components": comp,
        "wall_s_timed": round(wall, 4),
        "input_gen_s": round(t_gen, 2),
    }

    if not args.no_aux:
        aux_fns = {"score_logits": bench_score_logits, "single_linear": bench_single_linear,
                   "ppo_advantages": bench_advantages,
                   "decode_multi": bench_decode_multi, "lora_backward_layer": bench_backward,
                   "opt13b_r128": bench_opt13b, "score_two_input": bench_score_two_input}
        out["aux"] = {name: aux_fns[name](torch, H, WL, dev) for name in aux_names}

    if not args.no_cpu_baseline:
        hi = gout = None
        if all(k in host for k in ("decode", "prefill", "score")):
            hi = (host["decode"], host["prefill"], host["score"])
            # the outputs of the last timed step, for the oracle's comparison on the sampled rows
            gout = dict(decode=[(a.cpu().numpy(), b.cpu().numpy()) for a, b in zip(gyo, gyn)],
                        prefill={n: (v[5].cpu().numpy(), v[6].cpu().numpy()) for n, v in dev_in.items()},
                        score=dict(lp_on=lp_on.cpu().numpy(), lp_off=lp_off.cpu().numpy(), kl=kl.cpu().numpy(),
                                   reward=reward.cpu().numpy()))
        out["cpu_baseline"] = cpu_baseline(args.cpu_seconds, hi, gout)

    print(json.dumps(out), flush=True)


def kernel_source_digest() -> str:
    """sha256 of the HIP sources the dominant kernels are built from."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2309_00754_amd", "csrc")
    for name in ("lora_gemm.hip", "hydra_device.h"):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def committed_traffic(part: str):
    """HBM bytes per launch of the dominant kernel, from the committed counter summary.

    profiles/traffic_<part>.txt holds FETCH_SIZE / WRITE_SIZE readings scaled by a
    plain copy of known size, and the digest of the kernel sources they were taken
    on; when the sources have changed since, the figure is stale and None is returned.
    """
    path = os.path.join(ROOT, "profiles", f"traffic_{part}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_digest():
        return None
    try:
        return {"bytes_per_launch": float(kv["hbm_bytes_per_launch"]),
                "read_bytes_per_launch": float(kv["read_bytes_per_launch"]),
                "write_bytes_per_launch": float(kv["write_bytes_per_launch"]),
                "algorithmic_bytes_per_launch": float(kv["algorithmic_bytes_per_launch"]),
                "source": os.path.relpath(path, ROOT)}
    except (KeyError, ValueError):
        return None


def bench_score_logits(torch, H, WL, dev, iters=20):
    """hydra_score_logits on 512 x 32000 fp32 logits (on and off), four rotating input sets."""
    on, off, ids = WL.make("score_logits")
    M, V = on.shape
    sets = []
    for i in range(4):
        sets.append((torch.from_numpy(on).to(dev) + 0.0 * i, torch.from_numpy(off).to(dev),
                     torch.from_numpy(ids).to(dev)))
    outs = [torch.empty(M, device=dev) for _ in range(3)]
    for i in range(3):
        a, b, t = sets[i % 4]
        H.hydra_score_logits(a, b, t, *outs)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    # blocks of back-to-back launches between one pair of events (per-launch event pairs would add a few
    # microseconds of their own to a 24 us kernel); the median block average
    blocks = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(iters):
            a, b, t = sets[i % 4]
            H.hydra_score_logits(a, b, t, *outs)
        e1.record(stream)
        torch.cuda.synchronize()
        blocks.append(e0.elapsed_time(e1) / iters)
    us = float(np.median(blocks)) * 1e3
    by = 2.0 * M * V * 4 + 4.0 * M + 3 * 4.0 * M
    return dict(rows=M, vocab=V, us=round(us, 2), gbps=round(by / us / 1e3, 1),
                frac_hbm=round(by / us / 1e3 / PEAK_HBM_GBPS, 4), tokens_per_s=round(M / us * 1e6, 1),
                note="average over blocks of 20 back-to-back launches (median of 5 blocks), 4 rotating input "
                     "sets (524 MB, more than the last-level cache)")


def bench_single_linear(torch, H, WL, dev, iters=200):
    """hydra_lora_linear on the small single linear (x [16 x 512], W [512 x 512], rank 8): launch-latency bound, so
    it is reported for completeness (no roofline).  Eager back-to-back calls are bound by the host (the binding's
    argument checks); the same calls captured in one HIP graph and replayed give the GPU-side time per call."""
    c = WL.make("single_linear")
    bf = (lambda u: torch.from_numpy(np.ascontiguousarray(u).view(np.int16)).to(dev))
    x, W, A, B = bf(c.x), bf(c.W), bf(c.A), bf(c.B)
    yo, yn = torch.empty(c.M, c.N, device=dev), torch.empty(c.M, c.N, device=dev)

    def calls():
        for _ in range(iters):
            H.hydra_lora_linear(x, W, A, B, c.s, yo, yn)

    stream = torch.cuda.current_stream()

    def per_call_us(fn):
        blocks = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            blocks.append(e0.elapsed_time(e1) / iters)
        return float(np.median(blocks)) * 1e3

    calls()
    torch.cuda.synchronize()
    eager = per_call_us(calls)
    side = torch.cuda.Stream(device=dev)
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        calls()
    stream.wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    graph = per_call_us(g.replay)
    fl = lin_flops(c.M, c.K, c.N, c.r)
    return dict(M=c.M, K=c.K, N=c.N, r=c.r, us_graph=round(graph, 2), us_eager=round(eager, 2),
                tflops_graph=round(fl / graph / 1e6, 3),
                note="one call = one launch of the small-M MFMA kernel (8 < M <= 16); median of 5 blocks of 200 "
                     "calls, eager (host-bound) and replayed from one captured HIP graph")


def bench_advantages(torch, H, WL, dev, iters=30):
    """The PPO advantage step after scoring: the critic value head on all 2048 tokens (K = 4096), then the
    per-token rewards, GAE advantages and returns (4 sequences x 512 tokens)."""
    adv = WL.make("ppo_advantages")
    M, K = adv.M, adv.K
    h = torch.from_numpy(adv.h.view(np.int16)).to(dev)
    w = torch.from_numpy(adv.w_v.view(np.int16)).to(dev)
    kl = torch.from_numpy(adv.kl).to(dev)
    rw = torch.from_numpy(adv.reward).to(dev)
    vals = torch.empty(M, device=dev)
    r_out, a_out, ret_out = (torch.empty(M, device=dev) for _ in range(3))

    # twenty sets of hidden states in rotation (320 MB, more than the 256 MB last-level cache), so that every
    # launch reads cold data; the extra sets are seeded N(0, 1) draws on the device, for timing only
    gen = torch.Generator(device=dev)
    gen.manual_seed(4096)
    hs = [h] + [torch.randn(M, K, generator=gen, device=dev).to(torch.bfloat16).view(torch.int16) for _ in range(19)]
    rot = [0]

    def vh():
        H.hydra_value_head(hs[rot[0] % len(hs)], w, vals)
        rot[0] += 1

    def gae():
        H.hydra_ppo_advantages(kl, rw, vals, adv.n_seq, adv.seq_len, a_out, ret_out, rewards=r_out, start=adv.start,
                               beta=adv.beta, gamma=adv.gamma, lam=adv.lam)

    # PPO losses of the update stage on the same tokens (new log-probabilities a small step from the old ones)
    rng = np.random.default_rng(5)
    lp_old = torch.from_numpy(-rng.uniform(0.5, 6.0, M).astype(np.float32)).to(dev)
    lp_new = lp_old + torch.from_numpy(rng.normal(0, 0.3, M).astype(np.float32)).to(dev)
    losses, d_lp, d_v = torch.empty(3, device=dev), torch.empty(M, device=dev), torch.empty(M, device=dev)

    def loss():
        H.hydra_ppo_loss(lp_new, lp_old, a_out, vals, ret_out, adv.n_seq, adv.seq_len, losses, d_lp=d_lp, d_v=d_v)

    # each launch repeated back to back between one pair of events on the launch stream
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e3

    H.hydra_value_head(h, w, vals)
    gae()
    t_vh, t_gae, t_loss = timed(vh), timed(gae), timed(loss)
    del hs
    vh_bytes = 2.0 * M * K + 2.0 * K + 4.0 * M
    gae_bytes = 4.0 * M * 2 + 4.0 * adv.n_seq + 4.0 * M * 3
    loss_bytes = 4.0 * M * 5 + 4.0 * M * 2 + 12.0
    return dict(tokens=M, K=K, value_head_us=round(t_vh, 2), value_head_gbps=round(vh_bytes / t_vh / 1e3, 1),
                value_head_frac_hbm=round(vh_bytes / t_vh / 1e3 / PEAK_HBM_GBPS, 4), gae_us=round(t_gae, 2),
                gae_bytes=int(gae_bytes), ppo_loss_us=round(t_loss, 2), ppo_loss_bytes=int(loss_bytes),
                note="average over back-to-back launches (launch gaps included); the value head reads twenty "
                     "rotating 16 MB sets of hidden states (cold); GAE and the losses read their few hundred KB hot")


def bench_decode_multi(torch, H, WL, dev, iters=20, sets=3):
    """One 4096 x 4096 decode projection serving three passes at M = 4 (reference with LoRA off, actor and
    critic with their adapters): one hydra_lora_linear_multi call against three hydra_lora_linear calls.
    Three weight sets rotate (402 MB, more than the last-level cache); each figure is the average over a
    block of back-to-back launches between one pair of events."""
    c = WL.make("decode_multi")
    bf = (lambda u: torch.from_numpy(np.ascontiguousarray(u).view(np.int16)).to(dev))
    Ws = [bf(c.W)] + [bf(WL.gen_multi(60 + i, 1, c.K, c.N, 0, 0).W) for i in range(sets - 1)]
    x_off, xs = bf(c.x_off), [bf(x) for x in c.x_on]
    As, Bs = [bf(a) for a in c.A], [bf(b) for b in c.B]
    y_off = torch.empty(c.M, c.N, device=dev)
    y_ons = [torch.empty(c.M, c.N, device=dev) for _ in xs]

    def multi(W):
        H.hydra_lora_linear_multi(x_off, W, xs, As, Bs, c.s, y_off, y_ons)

    def separate(W):
        H.hydra_lora_linear(x_off, W, None, None, 0.0, y_off, None)
        for a in range(len(xs)):
            H.hydra_lora_linear(xs[a], W, As[a], Bs[a], c.s[a], None, y_ons[a])

    stream = torch.cuda.current_stream()

    def timed(fn):
        for i in range(2 * sets):
            fn(Ws[i % sets])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(iters):
            fn(Ws[i % sets])
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e3

    t_multi, t_sep = timed(multi), timed(separate)
    passes = 1 + len(xs)
    by = passes * lin_bytes(c.M, c.K, c.N, c.r)   # what the passes move when each reads W itself
    return dict(passes=passes, M=c.M, K=c.K, N=c.N, r=c.r, multi_us=round(t_multi, 2), separate_us=round(t_sep, 2),
                speedup=round(t_sep / t_multi, 3), multi_pass_equiv_gbps=round(by / t_multi / 1e3, 1),
                note="multi stacks the 12 input rows into two reads of W (8 + 4 rows); separate reads W three "
                     "times; GB/s counts the bytes of three independent passes")


def bench_backward(torch, H, WL, dev, iters=5):
    """The update stage's backward through every linear of one Llama-7B layer at M = 2048, rank 16, W frozen
    (hydra_lora_linear_backward: dx, dA, dB).  W^T is made once beforehand (W does not change while the adapters
    train).  Each figure is the average over a block of back-to-back layer passes between one pair of events."""
    cases = WL.make("backward_layer")
    bf = (lambda u: torch.from_numpy(np.ascontiguousarray(u).view(np.int16)).to(dev))
    xs, calls, flops = {}, [], []
    for b in cases:
        c = b.lin
        if id(c.x) not in xs:
            xs[id(c.x)] = bf(c.x)
        W = bf(c.W)
        Wt = torch.empty((c.K, c.N), dtype=W.dtype, device=dev)
        H.hydra_transpose_bf16(W, Wt)
        del W
        A, B, dy = bf(c.A), bf(c.B), bf(b.dy)
        dx = torch.empty(c.M, c.K, device=dev)
        dA = torch.empty(c.r, c.K, device=dev)
        dB = torch.empty(c.N, c.r, device=dev)
        ws = torch.empty(H.hydra_lora_linear_backward_workspace_bytes(c.M, c.N, c.K, c.r), dtype=torch.uint8,
                         device=dev)
        x = xs[id(c.x)]
        calls.append((c.name, lambda x=x, Wt=Wt, A=A, B=B, s=c.s, dy=dy, dx=dx, dA=dA, dB=dB, ws=ws:
                      H.hydra_lora_linear_backward(x, Wt, A, B, s, dy, dx, dA, dB, workspace=ws)))
        # dx = dy W (2MNK) + s U A (2MrK); U = dy B (2MNr); T = x A^T (2MKr); dA (2rKM); dB (2NrM)
        flops.append(2.0 * c.M * c.N * c.K + 4.0 * c.M * c.N * c.r + 6.0 * c.M * c.K * c.r)
    stream = torch.cuda.current_stream()

    def timed(fns):
        for fn in fns:
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            for fn in fns:
                fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e3

    t_layer = timed([fn for _, fn in calls])
    per = {name: round(timed([fn]), 2) for name, fn in calls}
    fl = sum(flops)
    c0 = cases[0].lin
    return dict(M=c0.M, r=c0.r, layer_us=round(t_layer, 2), per_linear_us=per,
                tflops=round(fl / t_layer / 1e6, 2), frac_bf16_peak=round(fl / t_layer / 1e6 / PEAK_BF16_TFLOPS, 4),
                note="dx, dA and dB of the 7 linears; FLOPs = 2MNK + 4MNr + 6MKr per linear; W^T prepared once")


def bench_opt13b(torch, H, WL, dev, iters=5):
    """OPT-1.3b at the paper's LoRA rank 128: the six linears of a layer over a mini-batch of 8 x 512 tokens
    (hydra_lora_linear_ws: the pre-pass GEMM), the CLM head with V = 50272 plus the reward head over the same tokens
    (hydra_score), and a decode step of the generation batch of 6 through the four attention projections
    (hydra_lora_linear_group).  Each figure is the average over a block of back-to-back calls between one pair of
    events."""
    bf = (lambda u: torch.from_numpy(np.ascontiguousarray(u).view(np.int16)).to(dev))
    stream = torch.cuda.current_stream()

    def timed(fns):
        for fn in fns:
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            for fn in fns:
                fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e3

    out = {}
    # layer
    lay = WL.make("opt13b_layer_r128")
    xs, calls = {}, []
    for c in lay:
        if id(c.x) not in xs:
            xs[id(c.x)] = bf(c.x)
        x, W, A, B = xs[id(c.x)], bf(c.W), bf(c.A), bf(c.B)
        yo, yn = torch.empty(c.M, c.N, device=dev), torch.empty(c.M, c.N, device=dev)
        ws = torch.empty(H.hydra_lora_linear_workspace_bytes(c.M, c.N, c.r), dtype=torch.uint8, device=dev)
        calls.append((c.name, lambda x=x, W=W, A=A, B=B, s=c.s, yo=yo, yn=yn, ws=ws:
                      H.hydra_lora_linear_ws(x, W, A, B, s, yo, yn, workspace=ws)))
    t_layer = timed([fn for _, fn in calls])
    fl = sum(lin_flops(c.M, c.K, c.N, c.r) for c in lay)
    out["layer"] = dict(M=lay[0].M, r=lay[0].r, us=round(t_layer, 2), tflops=round(fl / t_layer / 1e6, 2),
                        frac_bf16_peak=round(fl / t_layer / 1e6 / PEAK_BF16_TFLOPS, 4),
                        per_linear_us={n: round(timed([fn]), 2) for n, fn in calls})
    # the same layer with the three projections that read the same input (q, k, v) in one hydra_lora_linear_group_ws
    # call: their pre-passes run together, then one GEMM each
    groups = {}
    for c, (_, fn) in zip(lay, calls):
        groups.setdefault((id(c.x), c.N, c.K) if c.name in ("q", "k", "v") else c.name, []).append((c, fn))
    gcalls = []
    for mem in groups.values():
        if len(mem) == 1:
            gcalls.append(mem[0][1])
            continue
        cs = [c for c, _ in mem]
        c0 = cs[0]
        gW, gA, gB = [bf(c.W) for c in cs], [bf(c.A) for c in cs], [bf(c.B) for c in cs]
        gyo = [torch.empty(c0.M, c0.N, device=dev) for _ in cs]
        gyn = [torch.empty(c0.M, c0.N, device=dev) for _ in cs]
        gws = H.hydra_lora_linear_group_workspace(len(cs), c0.M, c0.N, c0.r, dev)
        gcalls.append(lambda x=xs[id(c0.x)], n=len(cs), gW=gW, gA=gA, gB=gB, gs=[c.s for c in cs], gyo=gyo, gyn=gyn,
                      gws=gws: H.hydra_lora_linear_group_ws([x] * n, gW, gA, gB, gs, gyo, gyn, workspace=gws))
    t_grp = timed(gcalls)
    out["layer"].update(us_shared_input_grouped=round(t_grp, 2),
                        frac_bf16_peak_shared_input_grouped=round(fl / t_grp / 1e6 / PEAK_BF16_TFLOPS, 4))
    del calls, gcalls, groups, xs
    # scoring head
    sc = WL.make("opt13b_score_r128")
    h, Wl, A, B, w_rm = bf(sc.h), bf(sc.W_lm), bf(sc.A), bf(sc.B), bf(sc.w_rm)
    ids = torch.from_numpy(sc.ids).to(dev)
    lp_on, lp_off, kl = (torch.empty(sc.M, device=dev) for _ in range(3))
    reward = torch.empty(sc.n_seq, device=dev)
    ws = torch.empty(H.hydra_score_workspace_bytes(sc.M, sc.V), dtype=torch.uint8, device=dev)
    t_sc = timed([lambda: H.hydra_score(h, Wl, A, B, sc.s, ids, w_rm, sc.n_seq, sc.seq_len, lp_on, lp_off, kl,
                                        reward=reward, workspace=ws)])
    fl = lin_flops(sc.M, sc.K, sc.V, sc.r) + 2.0 * sc.n_seq * sc.K
    out["score"] = dict(M=sc.M, V=sc.V, r=sc.r, us=round(t_sc, 2), tflops=round(fl / t_sc / 1e6, 2),
                        frac_bf16_peak=round(fl / t_sc / 1e6 / PEAK_BF16_TFLOPS, 4),
                        tokens_per_s=round(sc.M / (t_sc * 1e-6), 1))
    del h, Wl, ws
    # decode step
    dec = WL.make("opt13b_decode_r128")
    xd = bf(dec[0].x)
    gW, gA, gB = [bf(c.W) for c in dec], [bf(c.A) for c in dec], [bf(c.B) for c in dec]
    gyo = [torch.empty(c.M, c.N, device=dev) for c in dec]
    gyn = [torch.empty(c.M, c.N, device=dev) for c in dec]
    # ten weight sets in rotation (336 MB, more than the 256 MB last-level cache); the extra sets are seeded
    # N(0, 1/K) draws on the device, for timing only
    gen = torch.Generator(device=dev)
    gen.manual_seed(1310)
    sets = [gW] + [[(torch.randn(c.N, c.K, generator=gen, device=dev) / np.sqrt(c.K)).to(torch.bfloat16)
                    .view(torch.int16) for c in dec] for _ in range(9)]
    dws = H.hydra_lora_linear_group_workspace(len(dec), dec[0].M, dec[0].N, dec[0].r, dev)
    calls = [lambda Ws=Ws: H.hydra_lora_linear_group_ws([xd] * len(dec), Ws, gA, gB, [c.s for c in dec], gyo, gyn,
                                                        workspace=dws)
             for Ws in sets]
    t_eager = timed(calls) / len(calls)
    # the eager calls are bound by the host at this size (~22 us of argument checks and marshalling per call against
    # a ~17 us kernel), so the GPU time per call comes from the same ten calls captured in a HIP graph and replayed
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            for fn in calls:
                fn()
    stream.wait_stream(side)
    torch.cuda.synchronize()
    t_dec = timed([graph.replay]) / len(calls)
    # the same ten calls without LoRA (y_off alone: the stream of W the one-launch form is built on), for scale
    nil = [None] * len(dec)
    off_calls = [lambda Ws=Ws: H.hydra_lora_linear_group_ws([xd] * len(dec), Ws, nil, nil, [c.s for c in dec], gyo,
                                                            nil, workspace=dws)
                 for Ws in sets]
    graph_off = torch.cuda.CUDAGraph()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph_off, stream=side):
            for fn in off_calls:
                fn()
    stream.wait_stream(side)
    torch.cuda.synchronize()
    t_off = timed([graph_off.replay]) / len(off_calls)
    by = sum(lin_bytes(c.M, c.K, c.N, c.r) for c in dec)
    by_off = sum(2 * (c.M * c.K + c.N * c.K) + 4 * c.M * c.N for c in dec)
    out["decode"] = dict(M=dec[0].M, r=dec[0].r, us=round(t_dec, 2), gbps=round(by / t_dec / 1e3, 1),
                         frac_hbm=round(by / t_dec / 1e3 / PEAK_HBM_GBPS, 4), eager_us=round(t_eager, 2),
                         lora_off_us=round(t_off, 2), lora_off_frac_hbm=round(by_off / t_off / 1e3 / PEAK_HBM_GBPS, 4),
                         note="four 2048 x 2048 projections per call (hydra_lora_linear_group_ws, one launch), ten "
                              "weight sets rotating (336 MB); us from a HIP-graph replay of the ten calls (the "
                              "eager calls are host-bound: eager_us); lora_off_us: the same calls without adapters "
                              "(W streamed for y_off alone)")
    del graph, graph_off
    return out


def bench_score_two_input(torch, H, WL, dev, iters=5):
    """The two-head scoring with each pass's own hidden states (hydra_score_two_input: the actor's rows with the
    head's LoRA, the LoRA-off rows for the reference log-probabilities and the reward) on the Llama-7B heads,
    2048 tokens, V = 32000, r = 16, beside the one-input call (hydra_score) on the same sizes.  The two-input call
    does the base product twice (once per input), so its FLOPs are about twice the one-input call's; the W_lm
    tiles are still read once per pair of row tiles.  Each figure is the average over a block of back-to-back
    calls between one pair of events."""
    bf = (lambda u: torch.from_numpy(np.ascontiguousarray(u).view(np.int16)).to(dev))
    stream = torch.cuda.current_stream()

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e3

    c = WL.make("two_input_score")
    ha, ho, Wl, A, B, w_rm = bf(c.h_act), bf(c.h), bf(c.W_lm), bf(c.A), bf(c.B), bf(c.w_rm)
    ids = torch.from_numpy(c.ids).to(dev)
    lp_on, lp_off, kl = (torch.empty(c.M, device=dev) for _ in range(3))
    reward = torch.empty(c.n_seq, device=dev)
    ws = torch.empty(H.hydra_score_workspace_bytes(c.M, c.V), dtype=torch.uint8, device=dev)
    t2 = timed(lambda: H.hydra_score_two_input(ha, ho, Wl, A, B, c.s, ids, w_rm, c.n_seq, c.seq_len, lp_on, lp_off,
                                               kl, reward=reward, workspace=ws))
    t1 = timed(lambda: H.hydra_score(ho, Wl, A, B, c.s, ids, w_rm, c.n_seq, c.seq_len, lp_on, lp_off, kl,
                                     reward=reward, workspace=ws))
    fl2 = 2 * 2.0 * c.M * c.K * c.V + 2.0 * c.M * c.K * c.r + 2.0 * c.M * c.r * c.V + 2.0 * c.n_seq * c.K
    fl1 = lin_flops(c.M, c.K, c.V, c.r) + 2.0 * c.n_seq * c.K
    return dict(M=c.M, K=c.K, V=c.V, r=c.r,
                two_input=dict(us=round(t2, 2), tflops=round(fl2 / t2 / 1e6, 2),
                               frac_bf16_peak=round(fl2 / t2 / 1e6 / PEAK_BF16_TFLOPS, 4),
                               tokens_per_s=round(c.M / (t2 * 1e-6), 1)),
                one_input=dict(us=round(t1, 2), tflops=round(fl1 / t1 / 1e6, 2),
                               frac_bf16_peak=round(fl1 / t1 / 1e6 / PEAK_BF16_TFLOPS, 4)))


def rel_err(got, ref):
    """max_i |g_i - o_i| / max(|o_i|, rms(o)): the error of an output relative to its own scale."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    denom = np.maximum(np.abs(ref), np.sqrt(np.mean(ref * ref)))
    return float(np.max(np.abs(got - ref) / np.where(denom == 0, 1.0, denom)))


def cpu_baseline(target_s: float, host_inputs=None, gpu_out=None):
    """The float64 oracle, as it stands, on a row sample of the same step (host cores); with gpu_out (the step's
    outputs on the host), also the largest error of the GPU outputs against the oracle on the sampled rows."""
    import oracle
    import workloads as WL

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))

    if host_inputs is None:
        host_inputs = (WL.make("decode_qkvo"), WL.make("prefill_layer"), WL.make("two_head_score"))
    dec, pre, sc = host_inputs

    last = {}

    def run(rows):
        fl = 0.0
        t0 = time.perf_counter()
        last["decode"] = [oracle.lora_linear_ref(c.x, c.W, c.A, c.B, c.s) for c in dec]
        fl += sum(lin_flops(c.M, c.K, c.N, c.r) for c in dec)
        last["prefill"] = {c.name: oracle.lora_linear_ref(c.x[:rows], c.W, c.A, c.B, c.s) for c in pre}
        fl += sum(lin_flops(rows, c.K, c.N, c.r) for c in pre)
        last["score"] = oracle.score_head_ref(sc.h[:rows], sc.W_lm, sc.A, sc.B, sc.s, sc.ids[:rows])
        last["reward"] = oracle.reward_ref(sc.h, sc.w_rm, sc.n_seq, sc.seq_len)
        fl += lin_flops(rows, sc.K, sc.V, sc.r) + 2.0 * sc.n_seq * sc.K
        return fl, time.perf_counter() - t0

    # time = a + b * rows: fit from two short runs, then size the sample
    _, t1 = run(16)
    _, t2 = run(64)
    b = max((t2 - t1) / 48.0, 1e-6)
    a = max(t1 - 16 * b, 0.0)
    rows = int(min(2048, max(64, (target_s - a) / b)))
    # whole steps (all rows) are repeated until the sample holds about target_s of CPU work, the count taken
    # from the first step's own time
    fl, t = run(rows)
    reps = 1
    while rows == 2048 and t + t / reps <= target_s:
        f_, t_ = run(rows)
        fl += f_
        t += t_
        reps += 1
    out = dict(value=round(fl / t / 1e12, 5), unit="TFLOP/s", cores=int(threads), kind="oracle",
               seconds=round(t, 2),
               sample=f"float64 oracle on {reps} step(s) with the 2048-token parts cut to their first {rows} rows "
                      f"(decode 4 x M=4 in full; prefill 7 linears and two-head scoring on {rows} rows)",
               host_cpus=len(os.sched_getaffinity(0)))
    if gpu_out is not None:
        # y and reward: relative to the output's scale; log-probabilities and KL: absolute (nats)
        err = {"decode_y_rel": max(max(rel_err(g[0], o[0]), rel_err(g[1], o[1]))
                                   for g, o in zip(gpu_out["decode"], last["decode"])),
               "prefill_y_rel": max(max(rel_err(gpu_out["prefill"][n][0][:rows], o[0]),
                                        rel_err(gpu_out["prefill"][n][1][:rows], o[1]))
                                    for n, o in last["prefill"].items()),
               "score_reward_rel": rel_err(gpu_out["score"]["reward"], last["reward"])}
        for k in ("lp_on", "lp_off", "kl"):
            err[f"score_{k}_abs"] = float(np.max(np.abs(gpu_out["score"][k][:rows].astype(np.float64)
                                                        - last["score"][k])))
        out["max_error_vs_oracle"] = {k: float(f"{v:.3e}") for k, v in err.items()}
        out["max_error_vs_oracle"]["rows"] = min([rows, sc.M] + [c.M for c in pre])
    out["single_thread"] = cpu_small_configs()
    return out


def cpu_small_configs():
    """The oracle on one thread for the two small configurations: the single linear (16 x 512 -> 512, r = 8) and
    the logits epilogue (512 x 32000 on and off); median of 3 runs after one warm-up."""
    import oracle
    import workloads as WL
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover
        return None
    lin = WL.make("single_linear")
    lon, loff, ids = WL.make("score_logits")

    def med(fn):
        fn()
        ts = []
        for _ in range(3):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return float(np.median(ts))

    with threadpool_limits(limits=1):
        t_lin = med(lambda: oracle.lora_linear_ref(lin.x, lin.W, lin.A, lin.B, lin.s))
        t_log = med(lambda: oracle.score_logits_ref(lon, loff, ids))
    return {"threads": 1,
            "single_linear_us": round(t_lin * 1e6, 1),
            "single_linear_tflops": round(lin_flops(lin.M, lin.K, lin.N, lin.r) / t_lin / 1e12, 6),
            "logits_epilogue_ms": round(t_log * 1e3, 2),
            "logits_epilogue_tokens_per_s": round(lon.shape[0] / t_log, 1)}


if __name__ == "__main__":
    main()
