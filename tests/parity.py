"""Comparison helpers for GPU-vs-oracle parity tests.

Tolerances (absolute, against the fp64 oracle on the same bf16 inputs):
  O:   max |err| <= 2e-2 and mean |err| <= 2e-3
  LSE: max |err| <= 1e-3
Rows the oracle marks empty (LSE = -inf) must come back as O = 0 exactly
and LSE = -inf.
"""
from __future__ import annotations

import numpy as np
import torch

O_MAX = 2e-2
O_MEAN = 2e-3
LSE_MAX = 1e-3


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").to(torch.float64).numpy()


def errors(o_gpu, lse_gpu, o_ref, lse_ref):
    o = to_f64(o_gpu) if isinstance(o_gpu, torch.Tensor) else np.asarray(o_gpu, np.float64)
    e = np.abs(o - o_ref)
    out = {"o_max": float(e.max()) if e.size else 0.0,
           "o_mean": float(e.mean()) if e.size else 0.0,
           "o_nan": int(np.isnan(o).sum())}
    if lse_gpu is not None:
        lg = to_f64(lse_gpu) if isinstance(lse_gpu, torch.Tensor) else np.asarray(lse_gpu)
        empty = np.isneginf(lse_ref)
        out["lse_empty_mismatch"] = int((np.isneginf(lg) != empty).sum())
        fin = ~empty
        out["lse_max"] = float(np.abs(lg[fin] - lse_ref[fin]).max()) if fin.any() else 0.0
        out["lse_nan"] = int(np.isnan(lg).sum())
        # empty rows must be exactly zero
        if empty.any():
            out["empty_o_nonzero"] = int((o[empty] != 0).sum())
    return out


def assert_parity(name, o_gpu, lse_gpu, o_ref, lse_ref, o_max=O_MAX, o_mean=O_MEAN,
                  lse_max=LSE_MAX):
    e = errors(o_gpu, lse_gpu, o_ref, lse_ref)
    print(f"[parity] {name}: {e}", flush=True)
    assert e["o_nan"] == 0, f"{name}: NaN in O"
    assert e["o_max"] <= o_max, f"{name}: max|err| O = {e['o_max']}"
    assert e["o_mean"] <= o_mean, f"{name}: mean|err| O = {e['o_mean']}"
    if lse_gpu is not None:
        assert e["lse_nan"] == 0, f"{name}: NaN in LSE"
        assert e["lse_empty_mismatch"] == 0, f"{name}: empty-row LSE mismatch"
        assert e["lse_max"] <= lse_max, f"{name}: max|err| LSE = {e['lse_max']}"
        assert e.get("empty_o_nonzero", 0) == 0, f"{name}: empty row with non-zero O"
    return e
