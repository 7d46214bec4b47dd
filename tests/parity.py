"""Parity helpers shared by the GPU tests.

Metric (per output vector): for each row of length d_head,
    err = max_c |gpu_c - ref_c| / max(max_c |ref_c|, 1e-6),
and the reported error is the maximum over rows. Gradient tests raise the
denominator floor to 1% of the tensor's largest row (floor_frac), since a
gradient row can cancel to zero while its terms do not. The bars are the paper-path
tolerances: 1e-4 for the fp32 path, 2e-2 for bf16.
"""

import sys

import numpy as np
import torch

TOL = {torch.float32: 1e-4, torch.bfloat16: 2e-2}


def to64(t) -> np.ndarray:
    if isinstance(t, torch.Tensor):
        return t.detach().float().cpu().numpy().astype(np.float64)
    return np.asarray(t, dtype=np.float64)


def rowwise_rel(gpu, ref, floor_frac: float = 0.0, abs_floor: float = 1e-6) -> float:
    """Row-wise relative error; with floor_frac > 0 a row's denominator is at
    least floor_frac times the largest row of the tensor (for gradients whose
    rows can cancel to zero, e.g. dQ~ of the first causal row, where only an
    absolute comparison at the tensor's scale is meaningful)."""
    g = to64(gpu).reshape(-1, np.shape(ref)[-1])
    r = to64(ref).reshape(-1, np.shape(ref)[-1])
    if g.shape[0] == 0:
        return 0.0
    num = np.max(np.abs(g - r), axis=1)
    rowmax = np.max(np.abs(r), axis=1)
    den = np.maximum(np.maximum(rowmax, floor_frac * float(np.max(rowmax))), abs_floor)
    return float(np.max(num / den))


def assert_parity(gpu, ref, dtype, what="", floor_frac: float = 0.0, abs_floor: float = 1e-6):
    err = rowwise_rel(gpu, ref, floor_frac, abs_floor)
    assert np.all(np.isfinite(to64(gpu))), f"{what}: non-finite output"
    assert err <= TOL[dtype], f"{what}: row-wise relative error {err:.3e} > {TOL[dtype]:.0e}"
    return err


def say(msg: str):
    """Name the case before a GPU step, so a failure can be traced."""
    print(msg, flush=True)
    sys.stdout.flush()
