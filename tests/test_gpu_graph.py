"""The whole path captured in one HIP graph (torch.cuda.CUDAGraph) and replayed: the library allocates nothing,
issues no memset or copy and keeps no state, so a serving loop can capture it.  Every replay must give the bits of
the eager calls; the replays are interleaved with eager work and synchronisations."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from gpu_helpers import dev_bf16, host, say

pytestmark = pytest.mark.gpu


def test_path_replays_in_a_hip_graph(dev):
    import torch
    say("graph capture: decode, prefill, ws r=128, score, advantages, ppo loss, backward")
    dec = WL.gen_linear(901, 4, 512, 256, 16)
    pre = WL.gen_linear(902, 160, 520, 300, 16)
    big = WL.gen_linear(903, 130, 256, 264, 128)
    sc = WL.gen_score_head(904, 2, 64, 256, 1000, 16)
    bw = WL.gen_backward(905, 130, 256, 264, 16)

    def lin_inputs(c):
        return dev_bf16(c.x, dev), dev_bf16(c.W, dev), dev_bf16(c.A, dev), dev_bf16(c.B, dev)

    xd, Wd, Ad, Bd = lin_inputs(dec)
    xp, Wp, Ap, Bp = lin_inputs(pre)
    xb, Wb, Ab, Bb = lin_inputs(big)
    ws_big = torch.empty(H.hydra_lora_linear_workspace_bytes(big.M, big.N, big.r), dtype=torch.uint8, device=dev)
    h, Wl, As, Bs, w_rm = (dev_bf16(a, dev) for a in (sc.h, sc.W_lm, sc.A, sc.B, sc.w_rm))
    ids = torch.from_numpy(sc.ids).to(dev)
    ws_sc = torch.empty(H.hydra_score_workspace_bytes(sc.M, sc.V), dtype=torch.uint8, device=dev)
    c = bw.lin
    xg, Ag, Bg, dyg = (dev_bf16(a, dev) for a in (c.x, c.A, c.B, bw.dy))
    Wt = torch.empty((c.K, c.N), dtype=torch.int16, device=dev)
    H.hydra_transpose_bf16(dev_bf16(c.W, dev), Wt)
    ws_bw = torch.empty(H.hydra_lora_linear_backward_workspace_bytes(c.M, c.N, c.K, c.r), dtype=torch.uint8,
                        device=dev)
    rng = np.random.default_rng(9)
    lp_old = torch.from_numpy(-rng.uniform(0.5, 4.0, sc.M).astype(np.float32)).to(dev)
    reward_in = torch.from_numpy(rng.standard_normal(sc.n_seq).astype(np.float32)).to(dev)
    values = torch.from_numpy(rng.standard_normal(sc.M).astype(np.float32)).to(dev)

    out = {
        "dec_off": torch.empty(dec.M, dec.N, device=dev), "dec_on": torch.empty(dec.M, dec.N, device=dev),
        "pre_off": torch.empty(pre.M, pre.N, device=dev), "pre_on": torch.empty(pre.M, pre.N, device=dev),
        "big_off": torch.empty(big.M, big.N, device=dev), "big_on": torch.empty(big.M, big.N, device=dev),
        "lp_on": torch.empty(sc.M, device=dev), "lp_off": torch.empty(sc.M, device=dev),
        "kl": torch.empty(sc.M, device=dev), "reward": torch.empty(sc.n_seq, device=dev),
        "adv": torch.empty(sc.M, device=dev), "ret": torch.empty(sc.M, device=dev),
        "losses": torch.empty(3, device=dev), "d_lp": torch.empty(sc.M, device=dev),
        "dx": torch.empty(c.M, c.K, device=dev), "dA": torch.empty(c.r, c.K, device=dev),
        "dB": torch.empty(c.N, c.r, device=dev),
    }

    def path():
        H.hydra_lora_linear(xd, Wd, Ad, Bd, dec.s, out["dec_off"], out["dec_on"])
        H.hydra_lora_linear(xp, Wp, Ap, Bp, pre.s, out["pre_off"], out["pre_on"])
        H.hydra_lora_linear_ws(xb, Wb, Ab, Bb, big.s, out["big_off"], out["big_on"], workspace=ws_big)
        H.hydra_score(h, Wl, As, Bs, sc.s, ids, w_rm, sc.n_seq, sc.seq_len, out["lp_on"], out["lp_off"],
                      out["kl"], reward=out["reward"], workspace=ws_sc)
        H.hydra_ppo_advantages(out["kl"], reward_in, values, sc.n_seq, sc.seq_len, out["adv"], out["ret"])
        H.hydra_ppo_loss(out["lp_on"], lp_old, out["adv"], values, out["ret"], sc.n_seq, sc.seq_len,
                         out["losses"], d_lp=out["d_lp"])
        H.hydra_lora_linear_backward(xg, Wt, Ag, Bg, c.s, dyg, out["dx"], out["dA"], out["dB"], workspace=ws_bw)

    path()
    torch.cuda.synchronize()
    eager = {k: host(v).copy() for k, v in out.items()}
    for k, v in eager.items():
        assert np.all(np.isfinite(v)), k

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        path()
    torch.cuda.synchronize()

    other = torch.empty(pre.M, pre.N, device=dev)
    H.hydra_lora_linear(xp, Wp, None, None, 0.0, other, None)
    torch.cuda.synchronize()
    other_eager = host(other).copy()
    for rep in range(3):
        for v in out.values():
            v.fill_(float("nan"))
        H.hydra_lora_linear(xp, Wp, None, None, 0.0, other, None)  # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in out.items():
            assert np.array_equal(host(v), eager[k]), f"replay {rep}: {k}"
    assert np.array_equal(host(other), other_eager)
