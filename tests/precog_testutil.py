"""Shared helpers for the test suite (comparison metric, small input drawing)."""
from __future__ import annotations

import numpy as np


def err_rms(got, ref) -> float:
    """max_i |g_i - o_i| / max(|o_i|, rms(o)): elementwise relative error with
    a floor at the tensor's rms, so entries that cancel to near zero are
    judged against the tensor's scale rather than against themselves."""
    g = np.asarray(got, dtype=np.float64).ravel()
    o = np.asarray(ref, dtype=np.float64).ravel()
    if o.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(o * o)))
    floor = np.maximum(np.abs(o), rms if rms > 0 else 1e-300)
    return float(np.max(np.abs(g - o) / floor))


# Parity bars: fp32 inputs 1e-5; bf16 inputs with fp32 state 2e-3.
TOL_F32 = 1e-5
TOL_BF16 = 2e-3
