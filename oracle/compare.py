"""Error measures for comparing computed node states with the oracle's.

The parity bound is a maximum relative error.  Element-wise |g - r| / |r| is
ill-posed where r is near zero, so the primary measure is normwise per state
vector: max over nodes v and over {h, c} of ||g_v - r_v||_inf / max(||r_v||_inf, 1e-6).
The element-wise form with a floor of 1e-3 on |r| is reported beside it.
"""
from __future__ import annotations

import numpy as np


def normwise_rel_err(got, ref, floor=1e-6, rows=None):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if rows is not None:
        got, ref = got[rows], ref[rows]
    if got.size == 0:
        return 0.0
    num = np.max(np.abs(got - ref), axis=1)
    den = np.maximum(np.max(np.abs(ref), axis=1), floor)
    return float(np.max(num / den))


def elementwise_rel_err(got, ref, floor=1e-3):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.size == 0:
        return 0.0
    return float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), floor)))


def state_rel_err(h, c, h_ref, c_ref, h_rows=None):
    """Normwise error over both states; h_rows restricts h to nodes that have one."""
    return max(normwise_rel_err(h, h_ref, rows=h_rows), normwise_rel_err(c, c_ref))
