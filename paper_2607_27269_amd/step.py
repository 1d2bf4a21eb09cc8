"""Device buffers and call sequence of one reconstruction step (torch for memory/streams).

``DeviceStep`` uploads a synthetic workload once (hidden states, frozen teacher, student
weights, mask) and owns the outputs (A_t, A_s, loss, dA, gradients) and the workspace.
Its methods forward the tensors' device pointers and the current HIP stream to the C
ABI; all arithmetic happens in the library's kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _lib as L
from . import synth


def _dev_tensor(x: np.ndarray, dtype: str, device) -> torch.Tensor:
    if dtype == "bf16":
        bits = synth.bf16_bits(x).view(np.int16)
        return torch.from_numpy(np.ascontiguousarray(bits)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)


def _ptr(t):
    return None if t is None else t.data_ptr()


class DeviceStep:
    def __init__(self, wl: "synth.Workload", device: str = "cuda:0", grads: tuple = None,
                 ws_bytes: int | None = None):
        if not torch.cuda.is_available():
            raise RuntimeError("DeviceStep needs a ROCm GPU")
        L.lib()  # fail loudly if the HIP library is not built
        cfg = wl.cfg
        self.cfg = cfg
        self.dtype = cfg.dtype
        self.device = torch.device(device)
        self.ccfg = L.make_cfg(cfg)
        dev = self.device
        up = lambda a: None if a is None else _dev_tensor(a, self.dtype, dev)
        B, T, D = cfg.batch, cfg.seq, cfg.hidden
        self.h = up(wl.h.reshape(B * T, D))
        self.Wq, self.Wk, self.Wv, self.Wo = up(wl.Wq), up(wl.Wk), up(wl.Wv), up(wl.Wo)
        self.inv_freq_t = torch.from_numpy(wl.inv_freq_t.astype(np.float32)).to(dev)
        self.Wdq, self.Wuq, self.Wdkv_kr = up(wl.Wdq), up(wl.Wuq), up(wl.Wdkv_kr)
        self.Wuk, self.Wuv = up(wl.Wuk), up(wl.Wuv)
        self.inv_freq_s = torch.from_numpy(np.ascontiguousarray(wl.inv_freq_s, np.float32)).to(dev)
        self.mask = torch.from_numpy(np.ascontiguousarray(wl.mask.reshape(-1))).to(dev)
        tdt = torch.bfloat16 if self.dtype == "bf16" else torch.float32
        self.A_t = torch.zeros(B * T, D, dtype=torch.float32, device=dev)
        self.A_s = torch.zeros(B * T, D, dtype=torch.float32, device=dev)
        self.loss_buf = torch.zeros(2, dtype=torch.float32, device=dev)
        self.dA = torch.zeros(B * T, D, dtype=tdt, device=dev)
        want = grads or ("dWdq", "dWuq", "dWdkv_kr", "dWuk", "dWuv")
        self.grads = {}
        for name, W in (("dWdq", self.Wdq), ("dWuq", self.Wuq), ("dWdkv_kr", self.Wdkv_kr),
                        ("dWuk", self.Wuk), ("dWuv", self.Wuv)):
            if W is not None and name in want:
                self.grads[name] = torch.full(tuple(W.shape), float("nan"), dtype=torch.float32,
                                              device=dev)
        # the preferred workspace unless the caller asks for another size (a smaller one
        # runs the backward's attention in more chunks of sequences)
        self.ws_bytes = ws_bytes or L.mla_recon_workspace_size(self.ccfg)
        if self.ws_bytes == 0:
            raise L.MlaError(L.MLA_ERR_INVALID_ARG, L.last_error())
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.tw = L.TeacherW(_ptr(self.Wq), _ptr(self.Wk), _ptr(self.Wv), _ptr(self.Wo),
                             _ptr(self.inv_freq_t))
        self.sw = L.StudentW(_ptr(self.Wdq), _ptr(self.Wuq), _ptr(self.Wdkv_kr), _ptr(self.Wuk),
                             _ptr(self.Wuv), _ptr(self.inv_freq_s))
        self.sg = L.StudentGrads(*[_ptr(self.grads.get(n)) for n in
                                   ("dWdq", "dWuq", "dWdkv_kr", "dWuk", "dWuv")])

    @property
    def stream(self) -> int:
        return torch.cuda.current_stream(self.device).cuda_stream

    def teacher_fwd(self):
        L.mla_recon_teacher_fwd(self.ccfg, _ptr(self.h), self.tw, _ptr(self.A_t),
                                _ptr(self.ws), self.ws_bytes, self.stream)

    def student_fwd(self):
        L.mla_recon_student_fwd(self.ccfg, _ptr(self.h), self.sw, _ptr(self.Wo), _ptr(self.A_s),
                                _ptr(self.ws), self.ws_bytes, self.stream)

    def loss(self, A_s=None, A_t=None, mask=True, dA=True):
        A_s = self.A_s if A_s is None else A_s
        A_t = self.A_t if A_t is None else A_t
        L.mla_recon_loss(self.ccfg, _ptr(A_s), _ptr(A_t), _ptr(self.mask) if mask else None,
                         _ptr(self.loss_buf), _ptr(self.dA) if dA else None, _ptr(self.ws),
                         self.ws_bytes, self.stream)

    def bwd(self, dA=None):
        dA = self.dA if dA is None else dA
        L.mla_recon_bwd(self.ccfg, _ptr(self.h), self.sw, _ptr(self.Wo), _ptr(dA), self.sg,
                        _ptr(self.ws), self.ws_bytes, self.stream)

    def step(self):
        """One whole step: teacher forward, student forward, Eq. 11, backward."""
        self.teacher_fwd()
        self.student_fwd()
        self.loss()
        self.bwd()

    def fused_step(self, with_dA: bool = True):
        """The same step through mla_recon_step: W_O applied to o_s - o_t, A_t and A_s not
        formed (loss, the gradients and, with_dA, dL/dA_s)."""
        L.mla_recon_step(self.ccfg, _ptr(self.h), self.tw, self.sw, _ptr(self.mask),
                         _ptr(self.loss_buf), _ptr(self.dA) if with_dA else None, self.sg,
                         _ptr(self.ws), self.ws_bytes, self.stream)

    def capture_fused_step(self, with_dA: bool = False):
        """The single-call step recorded once as a HIP graph (torch.cuda.CUDAGraph): replay()
        launches the same kernels on the same buffers (h, weights, mask, workspace, outputs
        as they are at replay time) without the per-launch host work.  The library makes
        no allocation, synchronisation or memset inside a step, so the step is capturable;
        one eager call first does the library's one-time per-device queries."""
        self.fused_step(with_dA)
        torch.cuda.synchronize(self.device)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            self.fused_step(with_dA)
        torch.cuda.synchronize(self.device)
        return graph

    def teacher_cache(self):
        """Teacher forward up to its attention output (and W_O^T W_O), kept in the workspace."""
        L.mla_recon_teacher_cache(self.ccfg, _ptr(self.h), self.tw, _ptr(self.ws), self.ws_bytes,
                                  self.stream)

    def student_step(self, with_dA: bool = True):
        """The single-call step after the teacher, on the cached teacher output."""
        L.mla_recon_student_step(self.ccfg, _ptr(self.h), self.sw, _ptr(self.Wo), _ptr(self.mask),
                                 _ptr(self.loss_buf), _ptr(self.dA) if with_dA else None, self.sg,
                                 _ptr(self.ws), self.ws_bytes, self.stream)

    def rel_error(self):
        """loss[1] after fused_step / student_step: the relative error, from the teacher
        output the step left in the workspace (one more product)."""
        L.mla_recon_rel_error(self.ccfg, _ptr(self.Wo), _ptr(self.mask), _ptr(self.loss_buf),
                              _ptr(self.ws), self.ws_bytes, self.stream)

    # ---- optimizer (AdamW on the trainable projections, mla_recon_adamw) -----------------
    def init_optimizer(self):
        """fp32 master copies of the trainable weights and zero moments."""
        self.opt = []
        for gname, W in (("dWdq", self.Wdq), ("dWuq", self.Wuq), ("dWdkv_kr", self.Wdkv_kr),
                         ("dWuk", self.Wuk), ("dWuv", self.Wuv)):
            if W is None or gname not in self.grads:
                continue
            master = W.float().clone()
            self.opt.append((W, master, torch.zeros_like(master), torch.zeros_like(master),
                             self.grads[gname]))
        self.opt_steps = 0

    def optimizer_step(self, lr: float, beta1: float = 0.9, beta2: float = 0.999,
                       eps: float = 1e-8, weight_decay: float = 0.0):
        self.opt_steps += 1
        ts = [L.AdamwTensor(_ptr(master), _ptr(m), _ptr(v), _ptr(W), _ptr(g), master.numel())
              for (W, master, m, v, g) in self.opt]
        L.mla_recon_adamw(ts, L.MLA_FP32 if self.dtype == "fp32" else L.MLA_BF16,
                          self.opt_steps, lr, beta1, beta2, eps, weight_decay, self.stream)

    def train(self, steps: int, lr: float, **adamw) -> torch.Tensor:
        """`steps` optimizer steps on this minibatch (teacher recomputed each step, as Eq. 11
        is written); returns the loss before each update (host fp32 [steps])."""
        if not hasattr(self, "opt"):
            self.init_optimizer()
        losses = torch.empty(steps, dtype=torch.float32, device=self.device)
        for i in range(steps):
            self.fused_step(with_dA=False)
            losses[i] = self.loss_buf[0]
            self.optimizer_step(lr, **adamw)
        return losses.cpu()

    # ---- training over calibration minibatches (E_b of Eq. 11) ------------------------
    def set_minibatch(self, h: torch.Tensor, mask: torch.Tensor | None = None):
        """Run the following calls on another calibration minibatch already in HBM: h
        [B*T, D] in the storage dtype (referenced, not copied), mask [B*T] uint8 (copied;
        default all tokens valid)."""
        if h.shape != self.h.shape or h.dtype != self.h.dtype or h.device != self.h.device:
            raise ValueError("minibatch must match the layer's [B*T, D] shape, dtype and device")
        self.h = h
        if mask is None:
            self.mask.fill_(1)
        else:
            self.mask.copy_(mask.reshape(-1))

    def train_minibatches(self, minibatches, epochs: int, lr: float,
                          steps_per_minibatch: int = 1, masks=None, **adamw) -> torch.Tensor:
        """E_b of Eq. 11 by stochastic optimisation: `epochs` passes over the calibration
        minibatches in order; on each one the frozen teacher's output is computed once
        (mla_recon_teacher_cache), then `steps_per_minibatch` student steps
        (mla_recon_student_step), each followed by AdamW.  Returns the loss before each
        update (host fp32 [epochs * len(minibatches) * steps_per_minibatch])."""
        if not hasattr(self, "opt"):
            self.init_optimizer()
        n = epochs * len(minibatches) * steps_per_minibatch
        losses = torch.empty(n, dtype=torch.float32, device=self.device)
        i = 0
        for _ in range(epochs):
            for k, h in enumerate(minibatches):
                self.set_minibatch(h, None if masks is None else masks[k])
                self.teacher_cache()
                for _ in range(steps_per_minibatch):
                    self.student_step(with_dA=False)
                    losses[i] = self.loss_buf[0]
                    self.optimizer_step(lr, **adamw)
                    i += 1
        return losses.cpu()

    def eval_loss(self, h: torch.Tensor | None = None, mask: torch.Tensor | None = None) -> float:
        """Eq. 11 on a minibatch (e.g. a held-out one) without computing gradients."""
        if h is not None:
            self.set_minibatch(h, mask)
        none = L.StudentGrads(None, None, None, None, None)
        L.mla_recon_step(self.ccfg, _ptr(self.h), self.tw, self.sw, _ptr(self.mask),
                         _ptr(self.loss_buf), None, none, _ptr(self.ws), self.ws_bytes, self.stream)
        return float(self.loss_buf[0].cpu())

    def upload(self, x: np.ndarray, dtype: str | None = None) -> torch.Tensor:
        """A host array on this device in `dtype` (default the storage dtype); 3-d token
        arrays [B, T, D] become [B*T, D]."""
        if x.ndim == 3:
            x = x.reshape(-1, x.shape[-1])
        return _dev_tensor(x, dtype or self.dtype, self.device)

    def results(self) -> dict:
        torch.cuda.synchronize(self.device)
        B, T, D = self.cfg.batch, self.cfg.seq, self.cfg.hidden
        out = dict(A_t=self.A_t.double().cpu().numpy().reshape(B, T, D),
                   A_s=self.A_s.double().cpu().numpy().reshape(B, T, D),
                   loss=float(self.loss_buf[0]), rel=float(self.loss_buf[1]),
                   dA=self.dA.double().cpu().numpy().reshape(B, T, D))
        for k, v in self.grads.items():
            out[k] = v.double().cpu().numpy()
        return out
