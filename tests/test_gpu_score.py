"""GPU parity of hydra_score (fused CLM-head scoring + reward head) and
hydra_score_logits (epilogue from materialised logits) against the oracle."""
import math

import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import reward_ref, score_head_ref, score_logits_ref
from gpu_helpers import assert_abs, assert_rel, dev, dev_bf16, host, row_chunks, say

pytestmark = pytest.mark.gpu


def _score(c, device, B=None, ids=None, s=None, with_lse=True):
    import torch
    B = c.B if B is None else B
    ids = c.ids if ids is None else ids
    s = c.s if s is None else s
    M = c.M
    out = {k: torch.full((M,), float("nan"), device=device) for k in ("lp_on", "lp_off", "kl")}
    if with_lse:
        out["lse_on"] = torch.full((M,), float("nan"), device=device)
        out["lse_off"] = torch.full((M,), float("nan"), device=device)
    out["reward"] = torch.full((c.n_seq,), float("nan"), device=device)
    err = torch.zeros(1, dtype=torch.int32, device=device)
    H.hydra_score(dev_bf16(c.h, device), dev_bf16(c.W_lm, device),
                  dev_bf16(c.A, device) if c.r else None, dev_bf16(B, device) if c.r else None, s,
                  dev(ids.astype(np.int32), device), dev_bf16(c.w_rm, device), c.n_seq, c.seq_len,
                  out["lp_on"], out["lp_off"], out["kl"], reward=out["reward"],
                  lse_on=out.get("lse_on"), lse_off=out.get("lse_off"), err_flag=err)
    torch.cuda.synchronize()
    res = {k: host(v) for k, v in out.items()}
    res["err"] = int(host(err)[0])
    return res


SCORE_SHAPES = [
    # (n_seq, seq_len, K, V, r): ragged row tiles, ragged vocabulary tiles
    # (V = 300 leaves a whole wave's half-tile past V), tiny V, every padded
    # rank (0, 16, 32, 64) with and without a ragged last column tile, several
    # 256-row tiles, K tails inside a 32-wide slab.
    (2, 100, 64, 1000, 8), (1, 7, 72, 300, 16), (3, 50, 128, 7, 1), (2, 64, 512, 2048, 64),
    (1, 129, 256, 513, 0), (4, 40, 1024, 4000, 33),
    (3, 200, 96, 1280, 24), (2, 256, 64, 512, 16), (1, 300, 40, 768, 0), (2, 150, 200, 777, 20),
    # the paper's rank 128 (and a rank that pads to it), ragged and whole vocabulary tiles
    (2, 100, 512, 1000, 128), (1, 260, 264, 512, 100),
]


@pytest.mark.parametrize("n_seq,seq_len,K,V,r", SCORE_SHAPES)
def test_score_matches_oracle(n_seq, seq_len, K, V, r, dev):
    seed = 2000 + n_seq * seq_len + K + V + r
    say("score", dict(n_seq=n_seq, seq_len=seq_len, K=K, V=V, r=r, seed=seed))
    c = WL.gen_score_head(seed, n_seq, seq_len, K, V, r)
    g = _score(c, dev)
    e = score_head_ref(c.h, c.W_lm, c.A, c.B, c.s, c.ids, c.w_rm, n_seq, seq_len)
    for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off"):
        assert_abs(g[k], e[k], k)
    assert_rel(g["reward"], e["reward"], "reward")
    assert g["err"] == 0


@pytest.mark.parametrize("K", [64, 8200])
def test_reward_with_a_two_byte_aligned_head_weight(K, dev):
    """The reward head's weight is only required to be 2-byte aligned: a w_rm one element into its allocation takes
    the 2-byte-load path of the reward dot product; at K = 8200 each thread's groups run over two rounds, the last
    with one group.  Same bits as with an aligned copy of the same weight, and the oracle's reward."""
    import torch
    say("reward, w_rm 2-byte aligned", K)
    c = WL.gen_score_head(2050 + K, 3, 5, K, 300, 16)
    h, W, A, B = (dev_bf16(a, dev) for a in (c.h, c.W_lm, c.A, c.B))
    ids = torch.from_numpy(c.ids.astype(np.int32)).to(dev)
    w_al = dev_bf16(c.w_rm, dev)
    w_buf = torch.zeros(K + 1, dtype=torch.int16, device=dev)
    w_buf[1:] = w_al
    w_odd = w_buf[1:]
    assert w_odd.data_ptr() % 16 == 2
    rewards = []
    for w in (w_al, w_odd):
        lp = [torch.empty(c.M, device=dev) for _ in range(3)]
        rw = torch.full((c.n_seq,), float("nan"), device=dev)
        H.hydra_score(h, W, A, B, c.s, ids, w, c.n_seq, c.seq_len, lp[0], lp[1], lp[2], reward=rw)
        torch.cuda.synchronize()
        rewards.append(host(rw))
    assert np.array_equal(rewards[0], rewards[1])
    assert_rel(rewards[1], reward_ref(c.h, c.w_rm, c.n_seq, c.seq_len), "reward")


def test_score_lora_off_gives_exact_zero_kl(dev):
    say("score B=0 / s=0 / r=0 -> KL == 0")
    c = WL.gen_score_head(2100, 2, 70, 256, 1500, 16)
    g = _score(c, dev, B=np.zeros_like(c.B))
    assert np.all(g["kl"] == 0.0) and np.array_equal(g["lp_on"], g["lp_off"])
    g2 = _score(c, dev, s=0.0)
    assert np.all(g2["kl"] == 0.0)


def test_score_out_of_range_token_sets_nan_and_flag(dev):
    say("score out-of-range token")
    c = WL.gen_score_head(2200, 2, 40, 128, 700, 8)
    ids = c.ids.copy()
    ids[3] = 700
    ids[50] = -5
    g = _score(c, dev, ids=ids)
    assert g["err"] == 1
    for k in ("lp_on", "lp_off", "kl"):
        assert math.isnan(g[k][3]) and math.isnan(g[k][50])
    ok = np.ones(80, bool)
    ok[[3, 50]] = False
    e = score_head_ref(c.h, c.W_lm, c.A, c.B, c.s, ids, c.w_rm, 2, 40)
    assert_abs(g["lp_on"][ok], e["lp_on"][ok], "lp_on (valid rows)")


def test_score_deterministic(dev):
    say("score determinism")
    c = WL.gen_score_head(2300, 2, 96, 256, 3000, 16)
    a = _score(c, dev)
    b = _score(c, dev)
    for k in ("lp_on", "lp_off", "kl", "reward"):
        assert np.array_equal(a[k], b[k])


def test_score_workspace_contents_do_not_matter(dev):
    """A workspace full of NaN bit patterns gives bit-identical results."""
    import torch
    say("score dirty workspace")
    c = WL.gen_score_head(2400, 3, 90, 160, 1100, 24)
    clean = _score(c, dev)
    ws = torch.full((H.hydra_score_workspace_bytes(c.M, c.V),), 0xFF, dtype=torch.uint8, device=dev)
    out = {k: torch.full((c.M,), float("nan"), device=dev) for k in ("lp_on", "lp_off", "kl")}
    H.hydra_score(dev_bf16(c.h, dev), dev_bf16(c.W_lm, dev), dev_bf16(c.A, dev), dev_bf16(c.B, dev), c.s,
                  torch.from_numpy(c.ids.astype(np.int32)).to(dev), dev_bf16(c.w_rm, dev), c.n_seq, c.seq_len,
                  out["lp_on"], out["lp_off"], out["kl"], workspace=ws)
    torch.cuda.synchronize()
    for k in ("lp_on", "lp_off", "kl"):
        assert np.array_equal(host(out[k]), clean[k]), k


def _assert_score_every_row(c, g):
    """Every row of lp_on, lp_off, kl and both lse against the oracle (evaluated in row blocks), and every reward."""
    for rows in row_chunks(c.M):
        e = score_head_ref(c.h[rows], c.W_lm, c.A, c.B, c.s, c.ids[rows])
        for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off"):
            assert_abs(g[k][rows], e[k], f"{k} rows {rows[0]}..{rows[-1]}")
    assert_rel(g["reward"], reward_ref(c.h, c.w_rm, c.n_seq, c.seq_len), "reward")


def test_two_head_score_full_size_every_row(dev):
    """M = 2048 tokens (4 x 512), K = 4096, V = 32000, r = 16: the full CLM head in the bench's launch
    configuration; every row and every reward compared with the oracle."""
    c = WL.make("two_head_score")
    say("two_head_score full", c.M, c.K, c.V, c.r)
    g = _score(c, dev)
    _assert_score_every_row(c, g)
    assert np.all(np.isfinite(g["lp_on"])) and np.all(np.isfinite(g["kl"]))
    # every row: the log-sum-exp dominates the sampled logit, so lp <= 0
    assert np.all(g["lp_on"] <= 1e-6) and np.all(g["lp_off"] <= 1e-6)
    assert g["err"] == 0


# ------------------------------------------------------------------ epilogue from logits

def _score_logits(on, off, ids, device):
    import torch
    M = on.shape[0]
    out = {k: torch.full((M,), float("nan"), device=device) for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")}
    err = torch.zeros(1, dtype=torch.int32, device=device)
    H.hydra_score_logits(dev(on, device), dev(off, device), dev(ids.astype(np.int32), device),
                         out["lp_on"], out["lp_off"], out["kl"], out["lse_on"], out["lse_off"], err_flag=err)
    torch.cuda.synchronize()
    res = {k: host(v) for k, v in out.items()}
    res["err"] = int(host(err)[0])
    return res


@pytest.mark.parametrize("M,V", [(1, 4), (5, 1003), (7, 1000), (3, 32000), (9, 5), (2, 70001)])
def test_score_logits_matches_oracle(M, V, dev):
    say("score_logits", M, V)
    on, off, ids = WL.gen_logits(3000 + M + V, M, V)
    g = _score_logits(on, off, ids, dev)
    e = score_logits_ref(on, off, ids)
    for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off"):
        assert_abs(g[k], e[k], k)


def test_score_logits_full_workload(dev):
    """The 512 x 32000 logits workload (4 sequences x 128 tokens), every row."""
    on, off, ids = WL.make("score_logits")
    say("score_logits full", on.shape)
    g = _score_logits(on, off, ids, dev)
    e = score_logits_ref(on, off, ids)
    for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off"):
        assert_abs(g[k], e[k], k)
    assert g["err"] == 0


def test_score_logits_identities(dev):
    say("score_logits identities")
    on, off, ids = WL.gen_logits(3100, 6, 2000)
    g = _score_logits(on, on.copy(), ids, dev)
    assert np.all(g["kl"] == 0.0)
    u = np.zeros((2, 32000), np.float32)
    gu = _score_logits(u, u.copy(), np.array([5, 31999]), dev)
    assert np.allclose(gu["lp_on"], -math.log(32000), atol=2e-6, rtol=0)
    ids2 = ids.copy()
    ids2[1] = 2000
    gb = _score_logits(on, off, ids2, dev)
    assert gb["err"] == 1 and math.isnan(gb["lp_on"][1]) and not math.isnan(gb["lp_on"][0])


def test_opt13b_score_rank128_every_row(dev):
    """OPT-1.3b's CLM head (K = 2048, V = 50272: a ragged last column tile) at rank 128 over 8 x 512 tokens, with the
    reward head; every row and every reward compared with the oracle."""
    c = WL.make("opt13b_score_r128")
    say("opt13b score r128", c.M, c.K, c.V, c.r)
    g = _score(c, dev)
    _assert_score_every_row(c, g)
    assert g["err"] == 0
