"""Shared helpers of the test suite (no method arithmetic)."""

import numpy as np
import torch

# Tolerances on rel_err (max relative error, floored at the rms of the
# reference): bf16 2e-2, fp32 1e-5.
TOL = {"bf16": 2e-2, "f32": 1e-5}


def f64(t):
    """Exact fp64 copy of a CPU/GPU tensor (fp32 or bf16) or array."""
    if isinstance(t, torch.Tensor):
        return t.detach().float().cpu().numpy().astype(np.float64)
    return np.asarray(t, np.float64)


def rel_err(got, want):
    """max_i |g_i - o_i| / max(|o_i|, rms(o))."""
    g = f64(got)
    o = f64(want)
    if o.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(o * o)))
    floor = np.maximum(np.abs(o), rms if rms > 0 else 1e-300)
    return float(np.max(np.abs(g - o) / floor))


def has_gpu():
    return torch.cuda.is_available()
