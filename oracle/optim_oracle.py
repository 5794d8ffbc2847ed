"""fp64 oracle of the fused optimizer step: gradient-norm clipping, Adam and
the stochastic weight average (SWA).  TEST INFRASTRUCTURE ONLY (imported by
tests, the smoke check and the benchmark's CPU-baseline leg); the product
path never imports it, and it imports nothing from the product.

ScaleFold Section 3.3, "Adam and SWA Optimization" and "Gradient Clipping
Optimization": the paper fuses Adam, the SWA update that follows it and the
adjacent elementwise work into one kernel over all parameters, and computes
the gradient norm of the clipping step from packed buffers.  The arithmetic
is the standard one, written out per tensor in the order below:

  clipping:  norm  = sqrt(sum over every gradient element of g^2)
             scale = min(1, max_norm / (norm + 1e-6))
  Adam:      g  = grad * scale  (+ weight_decay * p when weight_decay != 0)
             m  = beta1 m + (1 - beta1) g
             v  = beta2 v + (1 - beta2) g^2
             p  = p - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
  SWA:       w  = swa_decay * w + (1 - swa_decay) * p        (with the updated p)

(swa_decay = n / (n + 1) gives the running mean of the first n + 1 iterates;
a constant close to 1 gives the exponential average AlphaFold training keeps.)
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

import numpy as np


def grad_norm_scale(grads: Sequence[np.ndarray], max_norm: float):
    """(norm, scale) of the clipping step over all gradient tensors."""
    total = 0.0
    for g in grads:
        g = np.asarray(g, dtype=np.float64)
        total += float(np.sum(g * g))
    norm = math.sqrt(total)
    return norm, min(1.0, max_norm / (norm + 1e-6))


def adam_swa_step(params: List[np.ndarray], grads: Sequence[np.ndarray], m: List[np.ndarray],
                  v: List[np.ndarray], swa: List[np.ndarray], *, lr: float, beta1: float, beta2: float,
                  eps: float, weight_decay: float, step: int, swa_decay: float, grad_scale: float = 1.0):
    """One step for every tensor; returns new (params, m, v, swa) lists (fp64)."""
    bc1 = 1.0 - beta1 ** step
    bc2 = 1.0 - beta2 ** step
    out_p, out_m, out_v, out_w = [], [], [], []
    for p, g, m_, v_, w in zip(params, grads, m, v, swa):
        p = np.asarray(p, np.float64)
        g = np.asarray(g, np.float64) * grad_scale
        if weight_decay:
            g = g + weight_decay * p
        m_ = beta1 * np.asarray(m_, np.float64) + (1.0 - beta1) * g
        v_ = beta2 * np.asarray(v_, np.float64) + (1.0 - beta2) * g * g
        p = p - lr * (m_ / bc1) / (np.sqrt(v_ / bc2) + eps)
        w = swa_decay * np.asarray(w, np.float64) + (1.0 - swa_decay) * p
        out_p.append(p)
        out_m.append(m_)
        out_v.append(v_)
        out_w.append(w)
    return out_p, out_m, out_v, out_w
