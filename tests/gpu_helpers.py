"""Helpers shared by the GPU tests: device transfer and the parity metrics."""
import sys

import numpy as np

# Tolerances stated for the path: relative 1e-2 on bf16-input / fp32-accumulate
# outputs (normwise, floored by the output's rms so that near-zero entries are
# judged against the output's scale), absolute 1e-3 on log-probabilities and KL.
REL_TOL = 1e-2
ABS_TOL_LP = 1e-3
# Tighter bound derived from the arithmetic (fp32 accumulation over K <= 11008
# bf16 products; LoRA term through a bf16 hi+lo split, ~2^-16 relative): a
# healthy kernel stays well below it, a dropped lo part or a wrong rounding
# does not.
DESIGN_REL = 2e-4
DESIGN_ABS_LP = 1e-4


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def row_chunks(M, size=512):
    """Row blocks [i, i + size) covering 0..M: the oracle is evaluated block by block on full-size cases so that
    its float64 intermediates stay small."""
    return [np.arange(i, min(i + size, M)) for i in range(0, M, size)]


def dev_bf16(u16, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).to(device)


def dev(arr, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def host(t):
    return t.detach().cpu().numpy()


def rel_err(got, ref):
    """max_i |g_i - o_i| / max(|o_i|, rms(o))."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    denom = np.maximum(np.abs(ref), rms)
    denom = np.where(denom == 0, 1.0, denom)
    return float(np.max(np.abs(got - ref) / denom)) if ref.size else 0.0


def assert_rel(got, ref, what):
    e = rel_err(got, ref)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    assert e <= REL_TOL, f"{what}: relative error {e:.3e} > {REL_TOL}"
    assert e <= DESIGN_REL, f"{what}: relative error {e:.3e} above the arithmetic bound {DESIGN_REL}"
    return e


def assert_abs(got, ref, what, finite=True):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if finite:
        assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    e = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    assert e <= ABS_TOL_LP, f"{what}: abs error {e:.3e} > {ABS_TOL_LP}"
    assert e <= DESIGN_ABS_LP, f"{what}: abs error {e:.3e} above the arithmetic bound {DESIGN_ABS_LP}"
    return e
