"""ctypes binding of libmlarecon.so (include/mla_recon.h).

Argument marshalling only: every function forwards raw device pointers, sizes and the
HIP stream handle to the C ABI of the same name and raises on a non-zero status.  No
computation of the reconstruction step happens in Python.  The library must have been
built (``python -m paper_2607_27269_amd.build``); importing this module fails loudly
otherwise.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmlarecon.so")

MLA_OK = 0
MLA_ERR_INVALID_ARG = -1
MLA_ERR_UNSUPPORTED = -2
MLA_ERR_WORKSPACE = -3
MLA_ERR_HIP = -4
MLA_BF16 = 0
MLA_FP32 = 1
# static scratch of mla_recon_decode_noalloc (include/mla_recon.h)
MLA_DECODE_NOALLOC_SCRATCH_BYTES = 32 << 20

(KC_GEMM_NT, KC_GEMM_NN, KC_GEMM_TN, KC_ATTN_FWD, KC_ATTN_DKDV, KC_ATTN_DQ, KC_LOSS, KC_ELEM,
 KC_ATTN_DK) = range(9)
KCLASS_NAMES = {KC_GEMM_NT: "gemm_nt", KC_GEMM_NN: "gemm_nn", KC_GEMM_TN: "gemm_tn",
                KC_ATTN_FWD: "attn_fwd", KC_ATTN_DKDV: "attn_bwd_dkdv", KC_ATTN_DQ: "attn_bwd_dq",
                KC_LOSS: "loss", KC_ELEM: "elementwise", KC_ATTN_DK: "attn_bwd_dk"}
# kernel function(s) behind each timing class (as rocprofv3 names them)
KCLASS_KERNELS = {"gemm_nt": "gemm_mfma_persist_kernel<..., true, true, ...> (and the loss-epilogue gemm_mfma_kernel)",
                  "gemm_nn": "gemm_mfma_persist_kernel<..., true, false, ...>",
                  "gemm_tn": "gemm_mfma_persist_kernel<..., false, false, float> + splitk_reduce_kernel",
                  "attn_fwd": "attn_fwd_persist_kernel (or attn_fwd_mfma_kernel)",
                  "attn_bwd_dkdv": "attn_dv_mfma_kernel (or attn_dkdv_mfma_kernel)",
                  "attn_bwd_dq": "attn_ds_gemm_kernel<..., false, false, ...> (or attn_dq_mfma_kernel)",
                  "attn_bwd_dk": "attn_ds_gemm_persist_kernel<..., true, false, float>",
                  "loss": "mask_count_kernel + loss_main_kernel + loss_final_kernel",
                  "elementwise": "rope_table_kernel, rope_apply_kernel, attn_delta_kernel, dkpe_finish_kernel, "
                                 "kcat_kernel, attn_stats_t_kernel"}


class MlaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"mla_recon error {code}: {msg}")
        self.code = code


class Cfg(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seq", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_groups", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("q_rank", ctypes.c_int32),
                ("kv_rank", ctypes.c_int32), ("nope_dim", ctypes.c_int32),
                ("rope_dim", ctypes.c_int32), ("s_kv_groups", ctypes.c_int32),
                ("s_rope_groups", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("dtype", ctypes.c_int32)]


class TeacherW(ctypes.Structure):
    _fields_ = [("Wq", ctypes.c_void_p), ("Wk", ctypes.c_void_p), ("Wv", ctypes.c_void_p),
                ("Wo", ctypes.c_void_p), ("inv_freq", ctypes.c_void_p)]


class StudentW(ctypes.Structure):
    _fields_ = [("Wdq", ctypes.c_void_p), ("Wuq", ctypes.c_void_p), ("Wdkv_kr", ctypes.c_void_p),
                ("Wuk", ctypes.c_void_p), ("Wuv", ctypes.c_void_p), ("inv_freq", ctypes.c_void_p)]


class StudentGrads(ctypes.Structure):
    _fields_ = [("dWdq", ctypes.c_void_p), ("dWuq", ctypes.c_void_p),
                ("dWdkv_kr", ctypes.c_void_p), ("dWuk", ctypes.c_void_p),
                ("dWuv", ctypes.c_void_p)]


class ProfKernel(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_char_p), ("ms", ctypes.c_double), ("launches", ctypes.c_int64),
                ("alg_flops", ctypes.c_double), ("alg_bytes", ctypes.c_double)]


class AdamwTensor(ctypes.Structure):
    _fields_ = [("master", ctypes.c_void_p), ("m", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("w", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("n", ctypes.c_int64)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2607_27269_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
        P = ctypes.POINTER
        L.mla_recon_workspace_size.argtypes = [P(Cfg)]
        L.mla_recon_workspace_size.restype = sz
        L.mla_recon_workspace_size_min.argtypes = [P(Cfg)]
        L.mla_recon_workspace_size_min.restype = sz
        L.mla_recon_teacher_fwd.argtypes = [P(Cfg), vp, P(TeacherW), vp, vp, sz, vp]
        L.mla_recon_student_fwd.argtypes = [P(Cfg), vp, P(StudentW), vp, vp, vp, sz, vp]
        L.mla_recon_loss.argtypes = [P(Cfg), vp, vp, vp, vp, vp, vp, sz, vp]
        L.mla_recon_bwd.argtypes = [P(Cfg), vp, P(StudentW), vp, vp, P(StudentGrads), vp, sz, vp]
        L.mla_recon_step.argtypes = [P(Cfg), vp, P(TeacherW), P(StudentW), vp, vp, vp,
                                     P(StudentGrads), vp, sz, vp]
        L.mla_recon_teacher_cache.argtypes = [P(Cfg), vp, P(TeacherW), vp, sz, vp]
        L.mla_recon_residual_rmsnorm.argtypes = [vp, vp, vp, ctypes.c_int64, i32, i32,
                                                 ctypes.c_float, vp]
        L.mla_recon_decode_workspace_size.argtypes = [P(Cfg), i32]
        L.mla_recon_decode_workspace_size.restype = sz
        L.mla_recon_decode.argtypes = [P(Cfg), vp, vp, i32, vp, vp, vp, vp, vp, sz, vp]
        L.mla_recon_decode_noalloc.argtypes = [P(Cfg), vp, vp, i32, vp, vp, vp, vp, vp]
        L.mla_recon_prefill_workspace_size.argtypes = [P(Cfg)]
        L.mla_recon_prefill_workspace_size.restype = sz
        L.mla_recon_prefill.argtypes = [P(Cfg), vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.mla_recon_fold_uv_into_o.argtypes = [P(Cfg), vp, vp, vp, vp]
        L.mla_recon_adamw.argtypes = [P(AdamwTensor), i32, i32, i32, ctypes.c_float,
                                      ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                      ctypes.c_float, vp]
        L.mla_recon_student_step.argtypes = [P(Cfg), vp, P(StudentW), vp, vp, vp, vp,
                                             P(StudentGrads), vp, sz, vp]
        L.mla_recon_rel_error.argtypes = [P(Cfg), vp, vp, vp, vp, sz, vp]
        for f in ("mla_recon_teacher_fwd", "mla_recon_student_fwd", "mla_recon_loss",
                  "mla_recon_bwd", "mla_recon_step", "mla_recon_teacher_cache",
                  "mla_recon_student_step", "mla_recon_rel_error", "mla_recon_adamw",
                  "mla_recon_residual_rmsnorm",
                  "mla_recon_decode", "mla_recon_decode_noalloc", "mla_recon_prefill",
                  "mla_recon_fold_uv_into_o",
                  "mla_recon_prof_enable",
                  "mla_recon_prof_read"):
            getattr(L, f).restype = i32
        L.mla_recon_last_error.argtypes = []
        L.mla_recon_last_error.restype = ctypes.c_char_p
        L.mla_recon_prof_enable.argtypes = [i32, i32]
        L.mla_recon_prof_read.argtypes = [i32, P(ctypes.c_double), P(ctypes.c_int64),
                                          P(ctypes.c_double), P(ctypes.c_double)]
        L.mla_recon_prof_kernels.argtypes = [i32, P(ProfKernel), i32]
        L.mla_recon_prof_kernels.restype = i32
        _lib = L
    return _lib


def _check(rc: int):
    if rc != MLA_OK:
        raise MlaError(rc, lib().mla_recon_last_error().decode())


def mla_recon_last_error() -> str:
    return lib().mla_recon_last_error().decode()


last_error = mla_recon_last_error


def make_cfg(c) -> Cfg:
    """Cfg from a configs.LayerConfig (or any object with the same attributes)."""
    return Cfg(c.batch, c.seq, c.hidden, c.n_heads, c.n_kv_groups, c.head_dim, c.q_rank,
               c.kv_rank, c.nope_dim, c.rope_dim, c.s_kv_groups, c.s_rope_groups,
               float(c.softmax_scale), MLA_FP32 if c.dtype == "fp32" else MLA_BF16)


def mla_recon_workspace_size(cfg: Cfg) -> int:
    return int(lib().mla_recon_workspace_size(ctypes.byref(cfg)))


def mla_recon_workspace_size_min(cfg: Cfg) -> int:
    return int(lib().mla_recon_workspace_size_min(ctypes.byref(cfg)))


def mla_recon_teacher_fwd(cfg: Cfg, h: int, w: TeacherW, A_t: int, ws: int, ws_bytes: int,
                          stream: int) -> None:
    _check(lib().mla_recon_teacher_fwd(ctypes.byref(cfg), h, ctypes.byref(w), A_t, ws,
                                       ws_bytes, stream))


def mla_recon_student_fwd(cfg: Cfg, h: int, w: StudentW, Wo: int, A_s: int, ws: int,
                          ws_bytes: int, stream: int) -> None:
    _check(lib().mla_recon_student_fwd(ctypes.byref(cfg), h, ctypes.byref(w), Wo, A_s, ws,
                                       ws_bytes, stream))


def mla_recon_loss(cfg: Cfg, A_s: int, A_t: int, mask: int | None, loss: int, dA: int | None,
                   ws: int, ws_bytes: int, stream: int) -> None:
    _check(lib().mla_recon_loss(ctypes.byref(cfg), A_s, A_t, mask, loss, dA, ws, ws_bytes,
                                stream))


def mla_recon_bwd(cfg: Cfg, h: int, w: StudentW, Wo: int, dA: int, grads: StudentGrads,
                  ws: int, ws_bytes: int, stream: int) -> None:
    _check(lib().mla_recon_bwd(ctypes.byref(cfg), h, ctypes.byref(w), Wo, dA,
                               ctypes.byref(grads), ws, ws_bytes, stream))


def mla_recon_step(cfg: Cfg, h: int, tw: TeacherW, sw: StudentW, mask: int | None, loss: int,
                   dA: int, grads: StudentGrads, ws: int, ws_bytes: int, stream: int) -> None:
    _check(lib().mla_recon_step(ctypes.byref(cfg), h, ctypes.byref(tw), ctypes.byref(sw), mask,
                                loss, dA, ctypes.byref(grads), ws, ws_bytes, stream))


def mla_recon_teacher_cache(cfg: Cfg, h: int, tw: TeacherW, ws: int, ws_bytes: int,
                            stream: int) -> None:
    _check(lib().mla_recon_teacher_cache(ctypes.byref(cfg), h, ctypes.byref(tw), ws, ws_bytes,
                                         stream))


def mla_recon_student_step(cfg: Cfg, h: int, sw: StudentW, Wo: int, mask: int | None, loss: int,
                           dA: int | None, grads: StudentGrads, ws: int, ws_bytes: int,
                           stream: int) -> None:
    _check(lib().mla_recon_student_step(ctypes.byref(cfg), h, ctypes.byref(sw), Wo, mask, loss,
                                        dA, ctypes.byref(grads), ws, ws_bytes, stream))


def mla_recon_rel_error(cfg: Cfg, Wo: int, mask: int | None, loss: int, ws: int, ws_bytes: int,
                        stream: int) -> None:
    _check(lib().mla_recon_rel_error(ctypes.byref(cfg), Wo, mask, loss, ws, ws_bytes, stream))


def mla_recon_adamw(tensors: list, dtype: int, step: int, lr: float, beta1: float, beta2: float,
                    eps: float, weight_decay: float, stream: int) -> None:
    arr = (AdamwTensor * len(tensors))(*tensors)
    _check(lib().mla_recon_adamw(arr, len(tensors), dtype, step, lr, beta1, beta2, eps,
                                 weight_decay, stream))


def mla_recon_residual_rmsnorm(x: int, A: int | None, h: int, rows: int, hidden: int, dtype: int,
                               eps: float, stream: int) -> None:
    _check(lib().mla_recon_residual_rmsnorm(x, A, h, rows, hidden, dtype, eps, stream))


def mla_recon_decode_workspace_size(cfg: Cfg, max_len: int) -> int:
    return int(lib().mla_recon_decode_workspace_size(ctypes.byref(cfg), max_len))


def mla_recon_decode(cfg: Cfg, q: int, cache: int, max_len: int, lengths: int, Wuk: int,
                     Wuv: int, o: int, ws: int, ws_bytes: int, stream: int) -> None:
    _check(lib().mla_recon_decode(ctypes.byref(cfg), q, cache, max_len, lengths, Wuk, Wuv, o, ws,
                                  ws_bytes, stream))


def mla_recon_decode_noalloc(cfg: Cfg, q: int, cache: int, max_len: int, lengths: int, Wuk: int,
                             Wuv: int, o: int, stream: int) -> None:
    _check(lib().mla_recon_decode_noalloc(ctypes.byref(cfg), q, cache, max_len, lengths, Wuk,
                                          Wuv, o, stream))


def mla_recon_prefill_workspace_size(cfg: Cfg) -> int:
    return int(lib().mla_recon_prefill_workspace_size(ctypes.byref(cfg)))


def mla_recon_prefill(cfg: Cfg, q: int, cache: int, Wuk: int, Wuv: int, Wo: int, Wo_folded: int,
                      o: int, A: int, ws: int, ws_bytes: int, stream: int) -> None:
    _check(lib().mla_recon_prefill(ctypes.byref(cfg), q, cache, Wuk, Wuv, Wo, Wo_folded, o, A, ws,
                                   ws_bytes, stream))


def mla_recon_fold_uv_into_o(cfg: Cfg, Wo: int, Wuv: int, Wo_folded: int, stream: int) -> None:
    _check(lib().mla_recon_fold_uv_into_o(ctypes.byref(cfg), Wo, Wuv, Wo_folded, stream))


def mla_recon_prof_enable(kclass: int, on: bool) -> None:
    _check(lib().mla_recon_prof_enable(kclass, 1 if on else 0))


def mla_recon_prof_kernels(kclass: int) -> list:
    """Per-kernel split of class `kclass`'s record (not cleared): a list of dicts."""
    cap = 64
    arr = (ProfKernel * cap)()
    n = lib().mla_recon_prof_kernels(kclass, arr, cap)
    if n < 0:
        _check(n)
    return [dict(kernel=arr[i].kernel.decode(), ms=arr[i].ms, launches=arr[i].launches,
                 flops=arr[i].alg_flops, bytes=arr[i].alg_bytes) for i in range(min(n, cap))]


def mla_recon_prof_read(kclass: int):
    ms, n = ctypes.c_double(), ctypes.c_int64()
    fl, by = ctypes.c_double(), ctypes.c_double()
    _check(lib().mla_recon_prof_read(kclass, ctypes.byref(ms), ctypes.byref(n),
                                     ctypes.byref(fl), ctypes.byref(by)))
    return dict(ms=ms.value, launches=n.value, flops=fl.value, bytes=by.value)
