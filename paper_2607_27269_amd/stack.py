"""Calibration capture over a frozen attention stack, then layer-by-layer reconstruction.

Sec. 4.1 reconstructs each attention layer independently on cached layer inputs H^l of the
frozen original model.  The stand-in model is an attention-only residual stack of frozen
GQA blocks (each drawn like a single-layer workload, its own seed):

    h^l = x^l / rms(x^l),   x^{l+1} = x^l + A^l_orig(h^l)

`capture` runs the frozen blocks (mla_recon_teacher_fwd) and the residual update with RMS
normalisation (mla_recon_residual_rmsnorm) to fill every layer's input; `reconstruct` then
trains each layer's converted block on its own input (DeviceStep.train: the single-call step
and AdamW).  Everything runs in the library's kernels; torch only holds device memory.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _lib as L
from . import synth
from .configs import LayerConfig
from .step import DeviceStep, _ptr


class ReconStack:
    def __init__(self, cfg: LayerConfig, n_layers: int, lengths=None, seed0: int = 100,
                 device: str = "cuda:0"):
        self.cfg = cfg
        self.layers = [DeviceStep(synth.make_workload(cfg, lengths=lengths, seed=seed0 + l),
                                  device=device) for l in range(n_layers)]
        # the residual stream entering layer 0: RMS-normalised tokens of its own seed
        x0 = synth.make_workload(cfg, seed=seed0 - 1, dtype="fp32").h
        self.x0 = torch.from_numpy(np.ascontiguousarray(x0.reshape(cfg.tokens, cfg.hidden),
                                                        dtype=np.float32)).to(device)
        self.x = self.x0.clone()

    @property
    def _dt(self) -> int:
        return L.MLA_FP32 if self.cfg.dtype == "fp32" else L.MLA_BF16

    def capture(self, eps: float = 1e-6):
        """Layer inputs h^0 .. h^{L-1} into each layer's DeviceStep (its `h`)."""
        c, n = self.cfg, len(self.layers)
        self.x.copy_(self.x0)
        first = self.layers[0]
        L.mla_recon_residual_rmsnorm(_ptr(self.x), None, _ptr(first.h), c.tokens, c.hidden,
                                     self._dt, eps, first.stream)
        for l in range(n - 1):
            cur, nxt = self.layers[l], self.layers[l + 1]
            cur.teacher_fwd()                       # A^l_orig(h^l) into cur.A_t
            L.mla_recon_residual_rmsnorm(_ptr(self.x), _ptr(cur.A_t), _ptr(nxt.h), c.tokens,
                                         c.hidden, self._dt, eps, cur.stream)

    def reconstruct(self, steps: int, lr: float, **adamw) -> list:
        """Train every layer's converted block on its captured input; per-layer losses."""
        return [layer.train(steps, lr, **adamw) for layer in self.layers]
