"""Asynchronous aggregation of Algorithm 4 (the aggregation branch).

Test infrastructure (see package docstring).  For an arriving device-side
model with version t_k while the global version is t, the staleness is
s = t - t_k.  If s exceeds the maximum delay D the model is dropped and the
global model and version are left as they are.  Otherwise the mixing weight
is the staleness-discounted weight alpha / (s + 1) (with alpha = 1 this is
exactly the weight 1/(t - t_k + 1) of Algorithm 4; alpha = 0 switches
mixing off), the global model becomes w * local + (1 - w) * global, the
same rule is applied to the auxiliary model (the library treats theta_d and
the auxiliary parameters as one flat vector), and t is incremented.

The mix is computed in fp64 and rounded once to fp32.
"""
from __future__ import annotations

import numpy as np


def weight(alpha: float, staleness: int) -> float:
    return float(alpha) / (float(staleness) + 1.0)


def mix(global_vec, local_vec, alpha, staleness, max_delay=None):
    """Returns (new global fp32 vector, applied?)."""
    g = np.asarray(global_vec, dtype=np.float32)
    if max_delay is not None and staleness > max_delay:
        return g.copy(), False
    w = weight(alpha, staleness)
    g64 = g.astype(np.float64)
    l64 = np.asarray(local_vec, dtype=np.float32).astype(np.float64)
    out = w * l64 + (1.0 - w) * g64
    return out.astype(np.float32), True


def mix_sequence(global_vec, locals_, alphas, stalenesses, max_delay=None):
    """Several arrivals handled one after another in FIFO order, rounding to
    fp32 after each, exactly as repeated single aggregations would."""
    g = np.asarray(global_vec, dtype=np.float32).copy()
    applied = []
    for l, a, s in zip(locals_, alphas, stalenesses):
        g, ok = mix(g, l, a, s, max_delay)
        applied.append(ok)
    return g, applied
