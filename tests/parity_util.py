"""Helpers shared by the GPU parity tests: run the oracle on a workload and compare."""
import numpy as np

import oracle as O

# Tolerances: relative Frobenius error per tensor (bf16 storage / fp32 check mode) and
# relative error of the Eq. 11 loss.
TOL = {"bf16": 2e-2, "fp32": 1e-5}
LOSS_TOL = 1e-3


def oracle_step(wl, dA=None):
    """The oracle's full step on a workload; with `dA` given, backpropagates that instead."""
    c = wl.cfg
    A_t = O.teacher_forward(wl.h, wl.Wq, wl.Wk, wl.Wv, wl.Wo, wl.inv_freq_t, c.n_heads,
                            c.n_kv_groups, c.softmax_scale)
    A_s, cache = O.student_forward(wl.h, wl.Wdq, wl.Wuq, wl.Wdkv_kr, wl.Wuk, wl.Wuv, wl.Wo,
                                   wl.inv_freq_s, n_heads=c.n_heads, s_kv_groups=c.s_kv_groups,
                                   s_rope_groups=c.s_rope_groups, nope_dim=c.nope_dim,
                                   rope_dim=c.rope_dim, scale=c.softmax_scale)
    L, rel, dA_ref = O.recon_loss(A_s, A_t, wl.mask)
    g = O.student_backward(cache, dA_ref if dA is None else dA)
    return dict(A_t=A_t, A_s=A_s, loss=L, rel=rel, dA=dA_ref, **g)


def rel_err(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(x - ref)
    if den == 0:
        return float(num)
    return float(num / den)


def compare(out, ref, names, tol, label=""):
    errs = {}
    for n in names:
        if ref.get(n) is None:
            continue
        assert np.all(np.isfinite(out[n])), f"{label}{n}: non-finite GPU values"
        errs[n] = rel_err(out[n], ref[n])
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"{label}relative errors above {tol}: {bad} (all: {errs})"
    return errs
