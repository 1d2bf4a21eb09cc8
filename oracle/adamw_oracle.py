"""Plain float64 CPU reference of the optimizer step of the reconstruction loop.

TEST INFRASTRUCTURE ONLY: only the test-suite may import it.  It shares no code with
the GPU path and imports nothing from it.

The paper trains the converter-introduced projections per layer with a gradient
method but names neither the optimizer nor its settings (Sec. 4.1).  The loop here
reads it as AdamW: Adam's bias-corrected first and second moments with the weight
decay decoupled from the gradient (applied to the weight itself, scaled by the
learning rate).  Written from that published definition, one step at a time:

    m_t = b1 m_{t-1} + (1 - b1) g_t
    v_t = b2 v_{t-1} + (1 - b2) g_t^2
    w_t = w_{t-1} - lr ( (m_t / (1 - b1^t)) / (sqrt(v_t / (1 - b2^t)) + eps) + wd w_{t-1} )
"""
from __future__ import annotations

import numpy as np


def adamw_step(w, g, m, v, step: int, lr: float, beta1: float = 0.9, beta2: float = 0.999,
               eps: float = 1e-8, weight_decay: float = 0.0):
    """One AdamW step (step counts from 1); returns the new (w, m, v), float64."""
    w = np.asarray(w, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m_new = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v_new = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m_new / (1.0 - beta1 ** step)
    v_hat = v_new / (1.0 - beta2 ** step)
    w_new = w - lr * (m_hat / (np.sqrt(v_hat) + eps) + weight_decay * w)
    return w_new, m_new, v_new
