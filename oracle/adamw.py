"""fp64 CPU oracle of one optimizer step: gradient clipping by the global L2
norm, then AdamW (Adam with decoupled weight decay).

TEST INFRASTRUCTURE ONLY.  Nothing in the library's product path imports,
links or calls this module; only the tests, the smoke check and the CPU
baseline leg of the benchmark do.

The Litespark report trains with AdamW (beta1 0.9, beta2 0.95, weight decay
0.01) and clips gradients at norm 1.0 (Section 2.5, optimizer settings, and Table 2).  The step, over
all parameters held in flat arrays, of which the first n_decay take weight
decay and the rest (RMSNorm gains) do not:

    norm  = sqrt(sum_i g_i^2)                       (over every parameter)
    c     = min(1, max_norm / (norm + 1e-6))
    g     = c g
    m     = beta1 m + (1 - beta1) g
    v     = beta2 v + (1 - beta2) g^2
    mhat  = m / (1 - beta1^t),   vhat = v / (1 - beta2^t)
    p     = p - lr wd p   (decayed parameters only)
    p     = p - lr mhat / (sqrt(vhat) + eps)

t counts steps from 1.  The 1e-6 in the clip coefficient and eps = 1e-8 are
the usual library conventions (the report gives neither).
"""
from __future__ import annotations

import numpy as np


def global_norm(grads: np.ndarray) -> float:
    """L2 norm of all gradients."""
    return float(np.sqrt(np.sum(grads * grads)))


def clip_coefficient(norm: float, max_norm: float) -> float:
    return min(1.0, max_norm / (norm + 1e-6))


def adamw_step(p: np.ndarray, g: np.ndarray, m: np.ndarray, v: np.ndarray, *, step: int, lr: float,
               beta1: float, beta2: float, eps: float, weight_decay: float, max_norm: float | None,
               n_decay: int | None = None):
    """One step on flat fp64 arrays.  Returns (p, m, v, norm) as new arrays;
    norm is the gradient norm before clipping.  max_norm None = no clipping;
    n_decay None = every parameter takes weight decay."""
    n = p.shape[0]
    nd = n if n_decay is None else n_decay
    norm = global_norm(g)
    if max_norm is not None:
        g = g * clip_coefficient(norm, max_norm)
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    p = p.copy()
    p[:nd] = p[:nd] - lr * weight_decay * p[:nd]
    p = p - lr * mhat / (np.sqrt(vhat) + eps)
    return p, m, v, norm
