"""Calibration capture over a frozen attention stack, then layer-by-layer reconstruction.

Sec. 4.1 reconstructs each attention layer independently on cached layer inputs H^l of the
frozen original model.  The stand-in model is an attention-only residual stack of frozen
GQA blocks (each drawn like a single-layer workload, its own seed):

    h^l = x^l / rms(x^l),   x^{l+1} = x^l + A^l_orig(h^l)

`capture` runs the frozen blocks (mla_recon_teacher_fwd) and the residual update with RMS
normalisation (mla_recon_residual_rmsnorm) to fill every layer's input, for each calibration
minibatch (each its own residual stream entering layer 0); `reconstruct` then trains each
layer's converted block on its own inputs: over the minibatches (E_b of Eq. 11, the frozen
teacher's output computed once per minibatch) or, with one minibatch, the single-call step
and AdamW.  Everything runs in the library's kernels; torch only holds device memory.
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
                 device: str = "cuda:0", n_minibatches: int = 1):
        self.cfg = cfg
        self.layers = [DeviceStep(synth.make_workload(cfg, lengths=lengths, seed=seed0 + l),
                                  device=device) for l in range(n_layers)]
        # the residual stream entering layer 0 of minibatch k: RMS-normalised tokens of
        # seed seed0 - 1 - k
        self.x0 = []
        for k in range(n_minibatches):
            x0 = synth.hidden_states(cfg, synth.make_rng(seed0 - 1 - k))
            self.x0.append(torch.from_numpy(np.ascontiguousarray(
                x0.reshape(cfg.tokens, cfg.hidden), dtype=np.float32)).to(device))
        self.x = torch.empty_like(self.x0[0])
        # captured layer inputs: inputs[l][k] = h^l of minibatch k (storage dtype)
        self.inputs = [[l.h if k == 0 else torch.empty_like(l.h) for k in range(n_minibatches)]
                       for l in self.layers]

    @property
    def _dt(self) -> int:
        return L.MLA_FP32 if self.cfg.dtype == "fp32" else L.MLA_BF16

    def capture(self, eps: float = 1e-6):
        """Layer inputs h^0 .. h^{L-1} of every minibatch into inputs[l][k]; each layer's
        DeviceStep is left on its minibatch-0 input (its `h`)."""
        c, n = self.cfg, len(self.layers)
        for k, x0 in enumerate(self.x0):
            self.x.copy_(x0)
            first = self.layers[0]
            L.mla_recon_residual_rmsnorm(_ptr(self.x), None, _ptr(self.inputs[0][k]), c.tokens,
                                         c.hidden, self._dt, eps, first.stream)
            for l in range(n - 1):
                cur = self.layers[l]
                cur.set_minibatch(self.inputs[l][k])
                cur.teacher_fwd()                       # A^l_orig(h^l) into cur.A_t
                L.mla_recon_residual_rmsnorm(_ptr(self.x), _ptr(cur.A_t), _ptr(self.inputs[l + 1][k]),
                                             c.tokens, c.hidden, self._dt, eps, cur.stream)
        for l, layer in enumerate(self.layers):
            layer.set_minibatch(self.inputs[l][0])

    def reconstruct(self, steps: int, lr: float, **adamw) -> list:
        """Train every layer's converted block on its captured inputs; per-layer losses.
        With several minibatches, `steps` is the number of optimiser steps per layer, taken
        as whole passes over the minibatches (one step per minibatch)."""
        if len(self.x0) == 1:
            return [layer.train(steps, lr, **adamw) for layer in self.layers]
        epochs = max(1, steps // len(self.x0))
        return [layer.train_minibatches(self.inputs[l], epochs, lr, **adamw)
                for l, layer in enumerate(self.layers)]
