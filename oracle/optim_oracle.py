"""Optimizer of the coefficient values: plain fp64 reference.

TEST INFRASTRUCTURE ONLY (same rules as frameft_oracle: only tests/, smoke() and
bench.py's cpu_baseline may use it; it shares nothing with the HIP library).

The paper trains only the coefficient values of C with AdamW under a linear
learning-rate schedule with warmup (Appendix G, the hyperparameter tables of the
GLUE, image-classification and instruction-tuning experiments).  AdamW is Adam
with the weight decay decoupled from the gradient (Loshchilov and Hutter,
"Decoupled Weight Decay Regularization"): the decay shrinks the parameters
directly instead of being added to the gradient.  The steps below follow that
algorithm in the order common training frameworks use: decay with the step's
learning rate, then the bias-corrected Adam step.  The schedule is the usual
linear warmup from 0 to the base rate over the warmup steps, then linear decay
to 0 at the last step.
"""
from __future__ import annotations

import math

import numpy as np


def adamw_step(c, g, m, v, t, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0):
    """One AdamW step at step number t (1 for the first step) on fp64 copies of the arrays.

    Returns (c, m, v) after the step:
        c <- c (1 - lr * weight_decay)                      (decoupled decay)
        m <- beta1 m + (1 - beta1) g                        (first moment)
        v <- beta2 v + (1 - beta2) g^2                      (second moment)
        c <- c - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
    """
    if t < 1:
        raise ValueError("step numbers start at 1")
    c = np.asarray(c, dtype=np.float64) * (1.0 - lr * weight_decay)
    g = np.asarray(g, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    c = c - lr * m_hat / (np.sqrt(v_hat) + eps)
    return c, m, v


def warmup_steps(total_steps: int, warmup_ratio: float) -> int:
    """Warmup length for a ratio of the run (the tables give ratios 0.06 and 0.03), rounded up."""
    return int(math.ceil(total_steps * warmup_ratio))


def linear_warmup_lr(step: int, warmup: int, total: int, base_lr: float) -> float:
    """Learning rate of optimizer step `step` (0 for the first): rises linearly from 0 over
    `warmup` steps to base_lr, then falls linearly to 0 at step `total`."""
    if step < warmup:
        return base_lr * step / max(1, warmup)
    return base_lr * max(0.0, (total - step) / max(1, total - warmup))
