"""Plain float64 CPU reference of calibration capture over a frozen attention stack.

TEST INFRASTRUCTURE ONLY: only the test-suite may import it.  It shares no code with
the GPU path and imports nothing from it.

Sec. 4.1 reconstructs each layer independently on cached layer inputs H^l taken from
the frozen original model.  The stand-in model here is an attention-only residual stack
(a reading: the paper's models also have MLPs, which are frozen and do not enter the
reconstruction of an attention layer):

    h^l     = x^l / sqrt(mean_d (x^l)^2 + eps)     (RMS normalisation, no gain)
    x^{l+1} = x^l + A^l_orig(h^l)                  (the frozen block's post-W_O output)

Calibration capture records h^0 .. h^{L-1}.
"""
from __future__ import annotations

import numpy as np

from .mla_recon_oracle import teacher_forward


def rms_norm(x, eps: float = 1e-6):
    """Each row of x over its last axis divided by its root mean square (float64)."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def capture(x0, layers, n_heads, n_kv_groups, scale, eps: float = 1e-6, round_fn=None):
    """Layer inputs h^0 .. h^{L-1} of the stack.  x0: [B, T, D] residual stream entering
    layer 0; layers: per-layer dicts with Wq, Wk, Wv, Wo, inv_freq (the frozen blocks).
    round_fn, when given, rounds each h^l to the storage precision before the layer uses it
    (the device stores the layer inputs in its storage dtype)."""
    x = np.asarray(x0, dtype=np.float64)
    hs = []
    for w in layers:
        h = rms_norm(x, eps)
        if round_fn is not None:
            h = round_fn(h)
        hs.append(h)
        x = x + teacher_forward(h, w["Wq"], w["Wk"], w["Wv"], w["Wo"], w["inv_freq"], n_heads,
                                n_kv_groups, scale)
    return hs
