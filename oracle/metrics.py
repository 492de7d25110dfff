"""Error metric used to compare a result with the oracle.

The tolerance is stated as a maximum relative error. The reading used
throughout is the infinity-norm relative error of a whole output tensor:
max_i |a_i - b_i| / max_i |b_i|, with b the oracle's value.
"""
import numpy as np


def max_rel_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.shape != ref.shape:
        raise ValueError(f"shape mismatch {got.shape} vs {ref.shape}")
    if ref.size == 0:
        return 0.0
    denom = float(np.max(np.abs(ref)))
    num = float(np.max(np.abs(got - ref)))
    if denom == 0.0:
        return num
    return num / denom
