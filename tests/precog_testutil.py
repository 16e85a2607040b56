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


def oracle_rows(oracle, inp, rows, h0=None, want_y=True, nthreads=8):
    """fp64 oracle on a sample of (b, d) rows of a (possibly device-resident)
    scan problem.  Rows are independent (Eq. 1 is diagonal in the state), so
    each batch row's selected channels form a smaller problem of their own.
    Returns {(b, d): (y[L] or None, hT[N])}."""
    import torch

    by_b = {}
    for b, d in rows:
        by_b.setdefault(int(b), []).append(int(d))
    out = {}
    for b, ds in by_b.items():
        ds = sorted(set(ds))
        di = torch.tensor(ds, dtype=torch.long)

        def sel(t):
            if t is None:
                return None
            return t[b:b + 1].index_select(2, di.to(t.device)).cpu()

        sub_h0 = None
        if h0 is not None:
            sub_h0 = h0[b:b + 1].index_select(1, di.to(h0.device)).cpu()
        y, hT = oracle.scan(sel(inp["x"]), sel(inp["dt"]),
                            inp["A"].index_select(0, di.to(inp["A"].device)).cpu(),
                            inp["B"][b:b + 1].cpu(),
                            None if inp.get("C") is None else inp["C"][b:b + 1].cpu(),
                            sel(inp.get("z")),
                            None if inp.get("Dskip") is None else
                            inp["Dskip"].index_select(0, di.to(inp["Dskip"].device)).cpu(),
                            sub_h0, want_y=want_y, nthreads=nthreads)
        for j, d in enumerate(ds):
            out[(b, d)] = ((y[0, :, j] if y is not None else None), hT[0, j])
    return out


def sample_rows(B, D, count, seed):
    """Rows spread over the batch, always including the first and last
    channel and both sides of 64-lane wave boundaries."""
    g = np.random.default_rng(seed)
    rows = {(0, 0), (B - 1, D - 1), (0, min(63, D - 1)), (B - 1, min(64, D - 1))}
    while len(rows) < count:
        rows.add((int(g.integers(0, B)), int(g.integers(0, D))))
    return sorted(rows)
