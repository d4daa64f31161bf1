"""The Python binding's argument checks on device tensors: a tensor on the host, of another dtype, not contiguous
or of the wrong shape is refused with the matching exception before anything is launched (the outputs keep their
contents), and the accepted form runs and matches the oracle."""
import numpy as np
import pytest

import paper_2309_00754_amd as H
import workloads as WL
from oracle import lora_linear_ref
from gpu_helpers import assert_rel, dev_bf16, host, say

pytestmark = pytest.mark.gpu


def _case(device, M=24, K=264, N=136, r=8):
    import torch
    c = WL.gen_linear(2100, M, K, N, r, s=1.5)
    t = dict(x=dev_bf16(c.x, device), W=dev_bf16(c.W, device), A=dev_bf16(c.A, device), B=dev_bf16(c.B, device),
             y_off=torch.full((M, N), 7.0, device=device), y_on=torch.full((M, N), 7.0, device=device))
    return c, t


def _call(t):
    H.hydra_lora_linear(t["x"], t["W"], t["A"], t["B"], 1.5, t["y_off"], t["y_on"])


@pytest.mark.parametrize("what,exc", [
    ("host_x", ValueError), ("float_W", TypeError), ("strided_A", ValueError), ("short_B", ValueError),
    ("numpy_A", TypeError), ("half_y", TypeError), ("transposed_y", ValueError),
])
def test_bad_argument_is_refused_before_launch(what, exc, dev):
    import torch
    say("binding check", what)
    c, t = _case(dev)
    bad = dict(t)
    if what == "host_x":
        bad["x"] = t["x"].cpu()
    elif what == "float_W":
        bad["W"] = t["W"].view(torch.bfloat16).float()
    elif what == "strided_A":
        bad["A"] = torch.cat([t["A"], t["A"]], 1)[:, ::2]
    elif what == "short_B":
        bad["B"] = t["B"][:-1]
    elif what == "numpy_A":
        bad["A"] = c.A
    elif what == "half_y":
        bad["y_on"] = torch.zeros_like(t["y_on"], dtype=torch.float16)
    elif what == "transposed_y":
        bad["y_off"] = torch.zeros(t["y_off"].shape[1], t["y_off"].shape[0], device=dev).t()
    with pytest.raises(exc):
        _call(bad)
    torch.cuda.synchronize()
    assert (host(t["y_off"]) == 7.0).all() and (host(t["y_on"]) == 7.0).all()


def test_accepted_form_runs(dev):
    import torch
    c, t = _case(dev)
    _call(t)
    torch.cuda.synchronize()
    e_off, e_on = lora_linear_ref(c.x, c.W, c.A, c.B, c.s)
    assert_rel(host(t["y_off"]), e_off, "y_off")
    assert_rel(host(t["y_on"]), e_on, "y_on")
    # bf16 tensors are accepted as they are, not only their 16-bit integer views
    t2 = dict(t, x=t["x"].view(torch.bfloat16), W=t["W"].view(torch.bfloat16))
    t2["y_off"] = torch.full_like(t["y_off"], np.nan)
    t2["y_on"] = torch.full_like(t["y_on"], np.nan)
    _call(t2)
    torch.cuda.synchronize()
    assert np.array_equal(host(t2["y_off"]), host(t["y_off"])) and np.array_equal(host(t2["y_on"]), host(t["y_on"]))
