"""The oracle reproduces the stored samples and the closed forms under tests/golden/ (CPU only)."""
import json
import math
import os

import numpy as np

from oracle import lora_linear_ref, log_softmax_gather_ref, score_logits_ref
import workloads as WL

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_single_linear_samples():
    g = _load("single_linear_samples.json")
    c = WL.make("single_linear")
    y_off, y_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    for e in g["samples"]:
        assert y_off[e["m"], e["n"]] == e["y_off"] and y_on[e["m"], e["n"]] == e["y_on"]
    assert np.allclose(y_off.sum(1), g["row_sums_off"], rtol=1e-13, atol=1e-12)
    assert np.allclose(y_on.sum(1), g["row_sums_on"], rtol=1e-13, atol=1e-12)


def test_score_logits_rows():
    g = _load("score_logits_rows8.json")
    on, off, ids = WL.gen_logits(1, 8, 32000)
    assert list(ids) == g["ids"]
    r = score_logits_ref(on, off, ids)
    for k in ("lp_on", "lp_off", "kl", "lse_on", "lse_off"):
        assert np.allclose(r[k], g[k], rtol=0, atol=1e-12)


def test_closed_forms():
    g = _load("closed_forms.json")
    V = g["uniform_row"]["V"]
    lp, _ = log_softmax_gather_ref(np.zeros((1, V)), np.array([17], np.int32))
    assert abs(lp[0] - g["uniform_row"]["lp"]) < 1e-12
    z = np.array([g["two_class"]["z"]] * 2)
    lp, _ = log_softmax_gather_ref(z, np.array([0, 1], np.int32))
    assert np.allclose(lp, g["two_class"]["lp"], rtol=0, atol=1e-14)
    kb = g["kl_bump"]
    off = np.zeros((1, kb["V"]))
    on = off.copy()
    on[0, 4] += kb["bump"]
    r = score_logits_ref(on, off, np.array([4], np.int32))
    assert abs(r["kl"][0] - kb["kl"]) < 1e-13
    assert not math.isnan(r["kl"][0])
