"""Seeded synthetic inputs for the Hydra-PPO scoring / LoRA-switchable-linear workloads.

This module only draws random numbers and encodes them; it holds none of the
method's arithmetic.  It is shared by the tests, ``bench.py`` and the smoke
check: the GPU path and the CPU oracle both receive exactly these arrays.

Storage conventions (the same ones the C-ABI uses):

* bf16 tensors are ``numpy.uint16`` bit patterns, rounded from float32 with
  round-to-nearest-even;
* a linear layer's frozen weight ``W`` is stored output-major, ``[N x K]``
  (the ``nn.Linear.weight`` layout), the LoRA down projection ``A`` is
  ``[r x K]`` and the up projection ``B`` is ``[N x r]``, so that
  ``y = x W^T + s (x A^T) B^T``;
* token ids are ``int32``.

Recipe (the paper's workload shapes are Llama-7B ones: hidden 4096, MLP 11008,
vocabulary 32000, batch 4 per GPU and 512-token sequences, and OPT-1.3b ones:
hidden 2048, MLP 8192, vocabulary 50272, generation batch 6 and mini-batch 8;
its datasets and weights are not available, so Gaussian stand-ins are drawn):

* one ``numpy.random.Generator(PCG64(seed))`` per workload, tensors drawn in
  the order listed by each generator, each as float64 standard normals in
  row chunks, scaled by its standard deviation, cast to float32, then rounded
  to bf16;
* activations ~ N(0, 1); base weights and LoRA-down ~ N(0, 1/K) with the
  layer's own K; LoRA-up ~ N(0, 1/r); the reward head ~ N(0, 1/K);
* token ids uniform in [0, V), drawn last;
* the PPO advantage step: critic hidden states ~ N(0, 1), value head
  ~ N(0, 1/K), per-token KL estimates ~ N(0, 0.1^2) (the spread of lp_on -
  lp_off when the LoRA-on and LoRA-off logits differ by N(0, 0.1^2) noise),
  sequence rewards ~ N(0, 1);
* the backward of the LoRA-switchable linear (update stage): the forward's
  inputs as above, then one upstream gradient dy [M x N] ~ N(0, 1) per linear.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

__all__ = [
    "f32_to_bf16",
    "bf16_bits_to_f32",
    "LinearCase",
    "gen_linear",
    "gen_linears",
    "gen_logits",
    "gen_score_head",
    "BackwardCase",
    "gen_backward",
    "gen_backward_layer",
    "AdvantageCase",
    "gen_advantages",
    "WORKLOADS",
    "DECODE_PROJ",
    "PREFILL_PROJ",
    "OPT13B_DECODE_PROJ",
    "OPT13B_PROJ",
]

_CHUNK_ELEMS = 1 << 22


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); returns uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        rounded[nan] = np.uint16(0x7FC0)
    return rounded


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    """Draw N(0, std^2) in row chunks, cast to float32, round to bf16."""
    shape = tuple(int(d) for d in shape)
    out = np.empty(shape, dtype=np.uint16)
    flat = out.reshape(-1)
    n = flat.size
    pos = 0
    while pos < n:
        cnt = min(_CHUNK_ELEMS, n - pos)
        v = rng.standard_normal(cnt, dtype=np.float64) * std
        flat[pos:pos + cnt] = f32_to_bf16(v.astype(np.float32))
        pos += cnt
    return out


@dataclasses.dataclass
class LinearCase:
    """One LoRA-switchable linear: x[M x K], W[N x K], A[r x K], B[N x r] (bf16 bits), scale s."""
    name: str
    x: np.ndarray
    W: np.ndarray
    A: np.ndarray
    B: np.ndarray
    s: float

    @property
    def M(self) -> int:
        return int(self.x.shape[0])

    @property
    def K(self) -> int:
        return int(self.x.shape[1])

    @property
    def N(self) -> int:
        return int(self.W.shape[0])

    @property
    def r(self) -> int:
        return int(self.A.shape[0])


def _lora_weights(rng, K: int, N: int, r: int):
    W = _normal_bf16(rng, (N, K), 1.0 / np.sqrt(K))
    A = _normal_bf16(rng, (r, K), 1.0 / np.sqrt(K))
    B = _normal_bf16(rng, (N, r), 1.0 / np.sqrt(r)) if r > 0 else np.zeros((N, 0), np.uint16)
    return W, A, B


def gen_linear(seed: int, M: int, K: int, N: int, r: int, s: float = 2.0, name: str = "linear") -> LinearCase:
    """Draw order: x, W, A, B."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = _normal_bf16(rng, (M, K), 1.0)
    W, A, B = _lora_weights(rng, K, N, r)
    return LinearCase(name, x, W, A, B, float(s))


# (name, K, N): the attention projections of one Llama-7B decoder layer.
DECODE_PROJ = [("q", 4096, 4096), ("k", 4096, 4096), ("v", 4096, 4096), ("o", 4096, 4096)]
# (name, K, N): every linear of one Llama-7B decoder layer.
PREFILL_PROJ = DECODE_PROJ + [("gate", 4096, 11008), ("up", 4096, 11008), ("down", 11008, 4096)]
# (name, K, N): every linear of one OPT-1.3b decoder layer (hidden 2048, MLP 8192); the attention projections
# alone for its decode step.
OPT13B_DECODE_PROJ = [("q", 2048, 2048), ("k", 2048, 2048), ("v", 2048, 2048), ("o", 2048, 2048)]
OPT13B_PROJ = OPT13B_DECODE_PROJ + [("fc1", 2048, 8192), ("fc2", 8192, 2048)]


def gen_linears(seed: int, M: int, proj, r: int, s: float = 2.0) -> List[LinearCase]:
    """Several linears sharing one activation per input width.

    Draw order: one x[M x K] per distinct K (in order of first appearance),
    then (W, A, B) for each projection in the listed order.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    xs: Dict[int, np.ndarray] = {}
    for _, K, _ in proj:
        if K not in xs:
            xs[K] = _normal_bf16(rng, (M, K), 1.0)
    cases = []
    for name, K, N in proj:
        W, A, B = _lora_weights(rng, K, N, r)
        cases.append(LinearCase(name, xs[K], W, A, B, float(s)))
    return cases


@dataclasses.dataclass
class BackwardCase:
    """Backward of one LoRA-switchable linear: its forward inputs and the upstream gradient dy [M x N] (bf16 bits)."""
    lin: LinearCase
    dy: np.ndarray


def gen_backward(seed: int, M: int, K: int, N: int, r: int, s: float = 2.0, name: str = "backward") -> BackwardCase:
    """Draw order: x, W, A, B (as gen_linear), then dy."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = _normal_bf16(rng, (M, K), 1.0)
    W, A, B = _lora_weights(rng, K, N, r)
    dy = _normal_bf16(rng, (M, N), 1.0)
    return BackwardCase(LinearCase(name, x, W, A, B, float(s)), dy)


def gen_backward_layer(seed: int, M: int, proj, r: int, s: float = 2.0) -> List[BackwardCase]:
    """The backward of every listed linear: the inputs of gen_linears (same draw order), then one dy per
    projection in the listed order."""
    rng = np.random.Generator(np.random.PCG64(seed))
    xs: Dict[int, np.ndarray] = {}
    for _, K, _ in proj:
        if K not in xs:
            xs[K] = _normal_bf16(rng, (M, K), 1.0)
    lins = []
    for name, K, N in proj:
        W, A, B = _lora_weights(rng, K, N, r)
        lins.append(LinearCase(name, xs[K], W, A, B, float(s)))
    return [BackwardCase(c, _normal_bf16(rng, (M, c.N), 1.0)) for c in lins]


def gen_logits(seed: int, M: int, V: int, noise_std: float = 0.1, logit_std: float = 2.0):
    """Materialised logits for the scoring epilogue alone.

    Draw order: logits_on ~ N(0, logit_std^2); noise ~ N(0, noise_std^2),
    logits_off = logits_on + noise (in float64, then float32); ids uniform.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    on64 = rng.standard_normal((M, V), dtype=np.float64) * logit_std
    noise = rng.standard_normal((M, V), dtype=np.float64) * noise_std
    logits_on = on64.astype(np.float32)
    logits_off = (logits_on.astype(np.float64) + noise).astype(np.float32)
    ids = rng.integers(0, V, size=M, dtype=np.int32)
    return logits_on, logits_off, ids


@dataclasses.dataclass
class MultiCase:
    """One W shared by a LoRA-off input and n_on LoRA-on inputs with their own adapters."""
    name: str
    W: np.ndarray                 # [N x K] bf16 bits
    x_off: Optional[np.ndarray]   # [M x K] or None
    x_on: List[np.ndarray]        # n_on x [M x K]
    A: List[np.ndarray]           # n_on x [r x K]
    B: List[np.ndarray]           # n_on x [N x r]
    s: List[float]

    @property
    def M(self) -> int:
        return (self.x_off if self.x_off is not None else self.x_on[0]).shape[0]

    @property
    def K(self) -> int:
        return self.W.shape[1]

    @property
    def N(self) -> int:
        return self.W.shape[0]

    @property
    def r(self) -> int:
        return self.A[0].shape[0] if self.A else 0


def gen_multi(seed: int, M: int, K: int, N: int, r: int, n_on: int, with_off: bool = True,
              scales=(2.0, 2.0, 2.0, 2.0), name: str = "multi") -> MultiCase:
    """Draw order: W, then x_off (when present), then (x_on, A, B) per adapter.  W, A ~ N(0, 1/K),
    B ~ N(0, 1/r), inputs ~ N(0, 1), as for the single linear."""
    rng = np.random.Generator(np.random.PCG64(seed))
    W = _normal_bf16(rng, (N, K), (1.0 / K) ** 0.5)
    x_off = _normal_bf16(rng, (M, K), 1.0) if with_off else None
    xs, As, Bs = [], [], []
    for _ in range(n_on):
        xs.append(_normal_bf16(rng, (M, K), 1.0))
        As.append(_normal_bf16(rng, (r, K), (1.0 / K) ** 0.5))
        Bs.append(_normal_bf16(rng, (N, r), (1.0 / max(r, 1)) ** 0.5))
    return MultiCase(name, W, x_off, xs, As, Bs, [float(v) for v in scales[:n_on]])


@dataclasses.dataclass
class ScoreCase:
    """Two-head scoring input: final hidden h[M x K], CLM head W_lm[V x K] + LoRA, RM head w_rm[K]."""
    h: np.ndarray
    W_lm: np.ndarray
    A: np.ndarray
    B: np.ndarray
    w_rm: np.ndarray
    ids: np.ndarray
    s: float
    n_seq: int
    seq_len: int

    @property
    def M(self) -> int:
        return int(self.h.shape[0])

    @property
    def K(self) -> int:
        return int(self.h.shape[1])

    @property
    def V(self) -> int:
        return int(self.W_lm.shape[0])

    @property
    def r(self) -> int:
        return int(self.A.shape[0])


def gen_score_head(seed: int, n_seq: int, seq_len: int, K: int, V: int, r: int, s: float = 2.0) -> ScoreCase:
    """Draw order: h, W_lm, A, B, w_rm, ids."""
    rng = np.random.Generator(np.random.PCG64(seed))
    M = n_seq * seq_len
    h = _normal_bf16(rng, (M, K), 1.0)
    W_lm, A, B = _lora_weights(rng, K, V, r)
    w_rm = _normal_bf16(rng, (K,), 1.0 / np.sqrt(K))
    ids = rng.integers(0, V, size=M, dtype=np.int32)
    return ScoreCase(h, W_lm, A, B, w_rm, ids, float(s), n_seq, seq_len)


@dataclasses.dataclass
class TwoInputScoreCase(ScoreCase):
    """Scoring with the actor pass's own final hidden states: h (inherited) is the LoRA-off pass's, h_act the actor
    pass's [M x K] bf16."""
    h_act: np.ndarray = None


def gen_score_two_input(seed: int, n_seq: int, seq_len: int, K: int, V: int, r: int,
                        s: float = 2.0) -> TwoInputScoreCase:
    """Draw order: the inputs of gen_score_head (h, W_lm, A, B, w_rm, ids), then h_act ~ N(0, 1)."""
    c = gen_score_head(seed, n_seq, seq_len, K, V, r, s)
    rng = np.random.Generator(np.random.PCG64(seed + (1 << 20)))
    h_act = _normal_bf16(rng, (c.M, K), 1.0)
    return TwoInputScoreCase(c.h, c.W_lm, c.A, c.B, c.w_rm, c.ids, c.s, c.n_seq, c.seq_len, h_act)


@dataclasses.dataclass
class AdvantageCase:
    """PPO advantage-step input: per-token KL kl[M] and sequence rewards reward[n_seq] (fp32), the critic's
    hidden states h[M x K] and value head w_v[K] (bf16); M = n_seq * seq_len, sequence-major."""
    kl: np.ndarray
    reward: np.ndarray
    h: np.ndarray
    w_v: np.ndarray
    n_seq: int
    seq_len: int
    start: int
    beta: float
    gamma: float
    lam: float

    @property
    def M(self) -> int:
        return self.n_seq * self.seq_len

    @property
    def K(self) -> int:
        return self.h.shape[1]


def gen_advantages(seed: int, n_seq: int, seq_len: int, K: int, start: int = 0, beta: float = 0.02,
                   gamma: float = 1.0, lam: float = 0.95) -> AdvantageCase:
    """Draw order: h, w_v, kl, reward."""
    rng = np.random.Generator(np.random.PCG64(seed))
    M = n_seq * seq_len
    h = _normal_bf16(rng, (M, K), 1.0)
    w_v = _normal_bf16(rng, (K,), 1.0 / np.sqrt(K))
    kl = (rng.standard_normal(M) * 0.1).astype(np.float32)
    reward = rng.standard_normal(n_seq).astype(np.float32)
    return AdvantageCase(kl, reward, h, w_v, n_seq, seq_len, start, float(beta), float(gamma), float(lam))


# The workloads, by what they are.  "seed" doubles as the workload index.
WORKLOADS = {
    "single_linear": dict(seed=0, M=16, K=512, N=512, r=8, s=2.0),
    "score_logits": dict(seed=1, n_seq=4, seq_len=128, V=32000),
    "decode_qkvo": dict(seed=2, M=4, proj=DECODE_PROJ, r=16, s=2.0),
    "prefill_layer": dict(seed=3, M=2048, proj=PREFILL_PROJ, r=16, s=2.0),
    "two_head_score": dict(seed=4, n_seq=4, seq_len=512, K=4096, V=32000, r=16, s=2.0),
    "ppo_advantages": dict(seed=5, n_seq=4, seq_len=512, K=4096, start=0, beta=0.02, gamma=1.0, lam=0.95),
    # one decode projection serving the reference (LoRA off), actor and critic passes (M = 4 each)
    "decode_multi": dict(seed=6, M=4, K=4096, N=4096, r=16, n_on=2),
    # the update stage's backward through every linear of one layer (W frozen, rank-16 adapters trained)
    "backward_layer": dict(seed=7, M=2048, proj=PREFILL_PROJ, r=16, s=2.0),
    # OPT-1.3b at the paper's LoRA rank 128: a layer over a mini-batch of 8 x 512 tokens, the CLM head (vocabulary
    # 50272) with the reward head over the same tokens, and a decode step of the generation batch of 6
    "opt13b_layer_r128": dict(seed=8, M=4096, proj=OPT13B_PROJ, r=128, s=2.0),
    "opt13b_score_r128": dict(seed=9, n_seq=8, seq_len=512, K=2048, V=50272, r=128, s=2.0),
    "opt13b_decode_r128": dict(seed=10, M=6, proj=OPT13B_DECODE_PROJ, r=128, s=2.0),
    # the Llama-7B two-head scoring pass with the actor pass's and the LoRA-off pass's own final hidden states
    "two_input_score": dict(seed=11, n_seq=4, seq_len=512, K=4096, V=32000, r=16, s=2.0),
}


def make(name: str, M: Optional[int] = None):
    """Materialise a workload by name (M overrides the row count where meaningful)."""
    w = WORKLOADS[name]
    if name == "single_linear":
        return gen_linear(w["seed"], M or w["M"], w["K"], w["N"], w["r"], w["s"], name)
    if name == "score_logits":
        return gen_logits(w["seed"], M or w["n_seq"] * w["seq_len"], w["V"])
    if name in ("decode_qkvo", "prefill_layer", "opt13b_layer_r128", "opt13b_decode_r128"):
        return gen_linears(w["seed"], M or w["M"], w["proj"], w["r"], w["s"])
    if name in ("two_head_score", "opt13b_score_r128"):
        return gen_score_head(w["seed"], w["n_seq"], w["seq_len"], w["K"], w["V"], w["r"], w["s"])
    if name == "two_input_score":
        return gen_score_two_input(w["seed"], w["n_seq"], w["seq_len"], w["K"], w["V"], w["r"], w["s"])
    if name == "decode_multi":
        return gen_multi(w["seed"], M or w["M"], w["K"], w["N"], w["r"], w["n_on"], name=name)
    if name == "backward_layer":
        return gen_backward_layer(w["seed"], M or w["M"], w["proj"], w["r"], w["s"])
    if name == "ppo_advantages":
        return gen_advantages(w["seed"], w["n_seq"], w["seq_len"], w["K"], w["start"], w["beta"], w["gamma"], w["lam"])
    raise KeyError(name)
