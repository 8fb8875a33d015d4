"""Comparison metrics used by the parity tests (test infrastructure only).

* ``max_abs_rel``: per tensor, max|x - y| / max(max|y|, floor), the
  max-abs-relative error gated at 1e-4 (fp32) and 2e-2 (bf16); ``floor``
  (default 1e-30) only matters for a reference that is identically zero.
* ``paper_pass_fraction``: the paper's element-wise mixed rule from its
  alignment study (Sec. 5.2), |x - y| <= tau_abs + tau_rel * max(|x|, |y|),
  with tau_abs = 1e-3 and tau_rel = 1e-2 for BF16; returns the fraction of
  elements that pass.
"""
import numpy as np


def max_abs_rel(x, y, floor: float = 1e-30) -> float:
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    if x.shape != y.shape:
        raise ValueError(f"shape mismatch {x.shape} vs {y.shape}")
    if x.size == 0:
        return 0.0
    return float(np.max(np.abs(x - y)) / max(float(np.max(np.abs(y))), floor))


def paper_pass_fraction(x, y, tau_abs: float = 1e-3, tau_rel: float = 1e-2) -> float:
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    if x.size == 0:
        return 1.0
    ok = np.abs(x - y) <= tau_abs + tau_rel * np.maximum(np.abs(x), np.abs(y))
    return float(np.mean(ok))
