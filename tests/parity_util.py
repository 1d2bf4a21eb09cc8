"""Helpers shared by the GPU parity tests: run the oracle on a workload and compare."""
import numpy as np

import oracle as O

# Tolerances: relative Frobenius error per tensor (bf16 storage / fp32 check mode) and
# relative error of the Eq. 11 loss.  The same relative bound also holds for every block
# of a tensor (a head's rows of a weight gradient, a tile of tokens of an output), so that
# a defect confined to one head or one tile cannot hide under the norm of the rest.
TOL = {"bf16": 2e-2, "fp32": 1e-5}
LOSS_TOL = 1e-3
# A block whose reference norm is below this fraction of the tensor's RMS block norm is
# measured against that floor instead of its own norm (near-empty blocks, e.g. tokens a
# mask removed from dA, would otherwise turn rounding noise into a large relative error).
BLOCK_FLOOR = 0.05
TOKEN_TILE = 64


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


def row_blocks(name, shape, cfg):
    """Row ranges [(label, lo, hi)] of the blocks tensor `name` is checked by.

    Weight gradients split by head / group / latent block (rows of the [out, in] matrix);
    token-major outputs ([..., T, D] flattened to rows) split into tiles of TOKEN_TILE
    tokens.  None: the tensor has no block structure here."""
    rows = int(np.prod(shape[:-1]))
    if cfg is None:
        return None
    if name == "dWuq":
        step = cfg.nope_dim + cfg.rope_dim  # one head's [q^nope; q^rope] rows
        return [(f"head{i}", i * step, (i + 1) * step) for i in range(cfg.n_heads)]
    if name == "dWuk":
        return [(f"group{g}", g * cfg.nope_dim, (g + 1) * cfg.nope_dim) for g in range(cfg.s_kv_groups)]
    if name == "dWuv":
        return [(f"group{g}", g * cfg.head_dim, (g + 1) * cfg.head_dim) for g in range(cfg.s_kv_groups)]
    if name == "dWdkv_kr":
        out = [(f"ckv{r}", r, min(r + 64, cfg.kv_rank)) for r in range(0, cfg.kv_rank, 64)]
        out += [(f"kpe{g}", cfg.kv_rank + g * cfg.rope_dim, cfg.kv_rank + (g + 1) * cfg.rope_dim)
                for g in range(cfg.s_rope_groups)]
        return out
    if name == "dWdq":
        return [(f"rows{r}", r, min(r + 128, rows)) for r in range(0, rows, 128)]
    if name in ("A_t", "A_s", "dA"):
        return [(f"tok{r}", r, min(r + TOKEN_TILE, rows)) for r in range(0, rows, TOKEN_TILE)]
    return None


def block_errors(x, ref, blocks):
    """Relative error of each row block against max(its norm, BLOCK_FLOOR x RMS block norm)."""
    x = np.asarray(x, dtype=np.float64).reshape(-1, np.shape(ref)[-1])
    ref = np.asarray(ref, dtype=np.float64).reshape(x.shape)
    norms = np.array([np.linalg.norm(ref[lo:hi]) for _, lo, hi in blocks])
    floor = BLOCK_FLOOR * float(np.sqrt(np.mean(norms ** 2)))
    errs = {}
    for (label, lo, hi), n in zip(blocks, norms):
        den = max(n, floor)
        num = float(np.linalg.norm(x[lo:hi] - ref[lo:hi]))
        errs[label] = num / den if den > 0 else num
    return errs


def compare(out, ref, names, tol, label="", cfg=None):
    """Relative Frobenius error of each tensor <= tol; with `cfg`, also of each of its
    blocks (row_blocks).  Returns the whole-tensor errors."""
    errs = {}
    bad = {}
    for n in names:
        if ref.get(n) is None:
            continue
        assert np.all(np.isfinite(out[n])), f"{label}{n}: non-finite GPU values"
        errs[n] = rel_err(out[n], ref[n])
        if not errs[n] <= tol:
            bad[n] = errs[n]
        blocks = row_blocks(n, np.shape(ref[n]), cfg)
        if blocks:
            be = block_errors(out[n], ref[n], blocks)
            worst = max(be, key=be.get)
            if not be[worst] <= tol:
                bad[f"{n}[{worst}]"] = be[worst]
    assert not bad, f"{label}relative errors above {tol}: {bad} (whole tensors: {errs})"
    return errs
