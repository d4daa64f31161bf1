"""Write the stored oracle samples under tests/golden/ (calls only oracle/ and the input generators).

Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import lora_linear_ref, score_logits_ref  # noqa: E402
import workloads as WL  # noqa: E402


def single_linear_samples():
    c = WL.make("single_linear")
    y_off, y_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    rng = np.random.default_rng(12345)
    idx = [(int(m), int(n)) for m, n in zip(rng.integers(0, c.M, 48), rng.integers(0, c.N, 48))]
    idx += [(0, 0), (c.M - 1, c.N - 1)]
    return {
        "what": "LoRA-switchable linear, 16x512x512, r=8, s=2, seed 0: sampled oracle outputs",
        "cite": "Sec. 2 Stage 3 (LoRA on all linears); Sec. 3 Dynamic LoRA (LO = LoRA off)",
        "samples": [{"m": m, "n": n, "y_off": float(y_off[m, n]), "y_on": float(y_on[m, n])} for m, n in idx],
        "row_sums_off": [float(v) for v in y_off.sum(1)],
        "row_sums_on": [float(v) for v in y_on.sum(1)],
    }


def score_logits_samples():
    on, off, ids = WL.gen_logits(1, 8, 32000)
    r = score_logits_ref(on, off, ids)
    return {
        "what": "scoring epilogue on the first 8 rows of the 512x32000 logits workload (seed 1)",
        "cite": "App. A Alg. 2 (reference log-probabilities from the LoRA-off model); App. B (KL weight beta)",
        "ids": [int(v) for v in ids],
        **{k: [float(v) for v in r[k]] for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off")},
    }


if __name__ == "__main__":
    for name, fn in (("single_linear_samples.json", single_linear_samples),
                     ("score_logits_rows8.json", score_logits_samples)):
        with open(os.path.join(HERE, name), "w") as f:
            json.dump(fn(), f, indent=1)
            f.write("\n")
        print("wrote", name)
