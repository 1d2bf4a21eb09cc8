"""Seeded synthetic inputs for the functional-reconstruction step.

The paper trains on cached layer inputs of real draft models (Sec. 4.1) that
were converted by TransMLA or MHA2MLA (Sec. 4.2).  None of that is available,
so this module draws stand-ins with the same shapes and structure:

* calibration hidden states H_b (Sec. 4.1): RMS-normalised Gaussian tokens,
  optionally with a few outlier channels scaled up before normalisation;
* the frozen original block (Eq. 1, output projection W_O): Gaussian weights
  with standard deviation 1/sqrt(fan_in);
* RoPE frequencies of R_t (Sec. 3.1): rotate-half pairs (p, p + d/2) with
  inverse frequency theta^(-2p/d);
* an initial converted MLA block C(theta_orig) (Sec. 4.2): a keep/drop RoPE
  routing of the original keys (the representative routing of Eq. 8), a
  truncated-SVD factorisation of the stacked non-positional key / value map
  (the rank condition of Eq. 6-7) and of the query map, plus small Gaussian
  noise;
* the valid-token mask M_b (Sec. 4.1) as right padding.

Everything is generated in float64 from ``numpy.random.Generator(PCG64(seed))``
and then rounded to the storage precision (bf16 with round-to-nearest-even, or
fp32).  The returned float64 arrays hold exactly the rounded values, so the
oracle and the GPU path see identical inputs.  This module contains none of the
reconstruction step's own arithmetic (no attention, loss or gradient): it only
produces inputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .configs import LayerConfig

# ----------------------------------------------------------------------------
# rounding helpers (storage formats)
# ----------------------------------------------------------------------------


def to_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bit patterns (uint16), via fp32, round-to-nearest-even."""
    f = to_f32(x)
    u = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    rounding = ((u >> 16) & 1) + 0x7FFF
    r = ((u + rounding) >> 16).astype(np.uint16)
    r[nan] = 0x7FC0
    return r


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage dtype; return them as float64."""
    if dtype == "bf16":
        return bf16_to_f64(bf16_bits(x))
    if dtype == "fp32":
        return to_f32(x).astype(np.float64)
    if dtype == "fp64":
        return np.asarray(x, dtype=np.float64)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------
# the workload bundle
# ----------------------------------------------------------------------------


@dataclass
class Workload:
    cfg: LayerConfig
    h: np.ndarray            # [B, T, D]
    mask: np.ndarray         # [B, T] uint8
    Wq: np.ndarray           # [H*dk, D]
    Wk: np.ndarray           # [G*dk, D]
    Wv: np.ndarray           # [G*dk, D]
    Wo: np.ndarray           # [D, H*dk]
    inv_freq_t: np.ndarray   # [dk/2] float64 holding fp32 values
    Wdq: np.ndarray | None   # [r_q, D] or None when r_q == 0
    Wuq: np.ndarray          # [H*(d_nope+d_rope), r_q or D]
    Wdkv_kr: np.ndarray      # [r_kv + G_r*d_rope, D]
    Wuk: np.ndarray          # [G_kv*d_nope, r_kv]
    Wuv: np.ndarray          # [G_kv*dk, r_kv]
    inv_freq_s: np.ndarray   # [G_r, d_rope/2] float64 holding fp32 values
    kept_pairs: np.ndarray = field(default=None)  # [G_r, d_rope/2] teacher pair index of each student pair

    def teacher_weights(self):
        return dict(Wq=self.Wq, Wk=self.Wk, Wv=self.Wv, Wo=self.Wo, inv_freq=self.inv_freq_t)

    def student_weights(self):
        return dict(Wdq=self.Wdq, Wuq=self.Wuq, Wdkv_kr=self.Wdkv_kr, Wuk=self.Wuk,
                    Wuv=self.Wuv, inv_freq=self.inv_freq_s)


def make_rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


# ----------------------------------------------------------------------------
# pieces
# ----------------------------------------------------------------------------


def hidden_states(cfg: LayerConfig, rng: np.random.Generator, perm=None) -> np.ndarray:
    """RMS-normalised Gaussian tokens with optional outlier channels (the first
    cfg.outlier_channels entries of `perm`, drawn here when not given)."""
    h = rng.standard_normal((cfg.batch, cfg.seq, cfg.hidden))
    if perm is None:
        perm = rng.permutation(cfg.hidden)
    if cfg.outlier_channels:
        h[..., perm[: cfg.outlier_channels]] *= cfg.outlier_scale
    h /= np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + 1e-6)
    return h


def rope_inv_freq(dim: int, theta: float) -> np.ndarray:
    """Inverse frequencies of rotate-half pairs (p, p + dim/2), rounded to fp32."""
    p = np.arange(dim // 2, dtype=np.float64)
    return to_f32(theta ** (-2.0 * p / dim)).astype(np.float64)


def gaussian(rng, shape, std):
    return rng.standard_normal(shape) * std


def right_padding_mask(batch: int, seq: int, lengths) -> np.ndarray:
    m = np.zeros((batch, seq), dtype=np.uint8)
    for b, n in enumerate(lengths):
        m[b, : int(n)] = 1
    return m


def low_rank_split(M: np.ndarray, rank: int):
    """Balanced rank-`rank` truncated-SVD factors (U S^1/2, S^1/2 V^T) of M.

    Small matrices use numpy's SVD; large ones use the eigendecomposition of
    the smaller Gram matrix (same subspace, much faster).  Returns
    (up [m, rank], down [rank, n]).
    """
    m, n = M.shape
    rank = int(rank)
    if m * n <= (1 << 22) or rank > min(m, n) // 2 and min(m, n) <= 1024:
        U, s, Vt = np.linalg.svd(M, full_matrices=False)
        k = min(rank, s.size)
        up = U[:, :k] * np.sqrt(s[:k])
        down = np.sqrt(s[:k])[:, None] * Vt[:k]
    elif m >= n:
        w, V = np.linalg.eigh(M.T @ M)
        idx = np.argsort(w)[::-1][:rank]
        s = np.sqrt(np.maximum(w[idx], 1e-300))
        Vr = V[:, idx]
        down = np.sqrt(s)[:, None] * Vr.T
        up = (M @ Vr) / np.sqrt(s)[None, :]
        k = rank
    else:
        w, U = np.linalg.eigh(M @ M.T)
        idx = np.argsort(w)[::-1][:rank]
        s = np.sqrt(np.maximum(w[idx], 1e-300))
        Ur = U[:, idx]
        up = Ur * np.sqrt(s)[None, :]
        down = (Ur.T @ M) / np.sqrt(s)[:, None]
        k = rank
    if k < rank:   # pad with zero directions so the shapes match the config
        up = np.concatenate([up, np.zeros((m, rank - k))], axis=1)
        down = np.concatenate([down, np.zeros((rank - k, n))], axis=0)
    return up, down


def _pair_rows(pairs: np.ndarray, dk: int) -> np.ndarray:
    """Rows of a rotate-half head (first halves, then second halves) for `pairs`."""
    pairs = np.asarray(pairs, dtype=np.int64)
    return np.concatenate([pairs, pairs + dk // 2])


def select_kept_pairs(cfg: LayerConfig, Wq: np.ndarray, Wk: np.ndarray) -> np.ndarray:
    """Teacher rotary pairs that each student rope group keeps.

    Shared positional key (G_r < G): the first d_rope/2 pairs.  Per-group
    positional keys (G_r == G): the d_rope/2 pairs with the largest product of
    query and key weight norms, ties to the lower index (a weight-only
    stand-in for a partial-RoPE frequency selection).
    """
    dk, nr = cfg.head_dim, cfg.rope_dim // 2
    half = dk // 2
    if cfg.s_rope_groups < cfg.n_kv_groups:
        return np.tile(np.arange(nr), (cfg.s_rope_groups, 1))
    assert cfg.s_rope_groups == cfg.n_kv_groups
    out = np.zeros((cfg.s_rope_groups, nr), dtype=np.int64)
    hpg = cfg.n_heads // cfg.n_kv_groups
    for g in range(cfg.n_kv_groups):
        k = Wk[g * dk:(g + 1) * dk]
        kn = np.sqrt(np.sum(k[:half] ** 2, axis=1) + np.sum(k[half:] ** 2, axis=1))
        qn = np.zeros(half)
        for i in range(g * hpg, (g + 1) * hpg):
            q = Wq[i * dk:(i + 1) * dk]
            qn += np.sqrt(np.sum(q[:half] ** 2, axis=1) + np.sum(q[half:] ** 2, axis=1))
        score = qn * kn
        order = np.lexsort((np.arange(half), -score))   # descending score, then index
        out[g] = np.sort(order[:nr])
    return out


def student_init(cfg: LayerConfig, Wq, Wk, Wv, inv_freq_t, rng, noise_std: float = 1e-3):
    """Initial converted MLA block from the frozen teacher (float64, unrounded).

    Returns (Wdq | None, Wuq, Wdkv_kr, Wuk, Wuv, inv_freq_s, kept_pairs).
    """
    H, G, dk, D = cfg.n_heads, cfg.n_kv_groups, cfg.head_dim, cfg.hidden
    Gkv, Gr, dn, dr = cfg.s_kv_groups, cfg.s_rope_groups, cfg.nope_dim, cfg.rope_dim
    if Gkv != G:
        raise ValueError("the initialiser maps student KV groups one to one onto teacher groups")
    if H % Gr or Gr > G and Gr != G:
        raise ValueError("unsupported rope grouping")
    half = dk // 2
    kept = select_kept_pairs(cfg, Wq, Wk)
    shared = Gr < G
    if shared and dn != dk:
        raise ValueError("a shared positional key keeps all d_k non-positional rows")
    if not shared and dn != dk - dr:
        raise ValueError("per-group positional keys split d_k into d_nope + d_rope")
    heads_per_rg = H // Gr
    hpg = H // G

    Wkr = np.zeros((Gr * dr, D))
    for r in range(Gr):
        rows = _pair_rows(kept[r], dk)
        groups = sorted({i // hpg for i in range(r * heads_per_rg, (r + 1) * heads_per_rg)})
        Wkr[r * dr:(r + 1) * dr] = np.mean([Wk[g * dk:(g + 1) * dk][rows] for g in groups], axis=0)

    knope = []
    for g in range(G):
        Wkg = Wk[g * dk:(g + 1) * dk]
        r = (g * hpg) // heads_per_rg
        rows = _pair_rows(kept[r], dk)
        if shared:
            k = Wkg.copy()
            k[rows] -= Wkr[r * dr:(r + 1) * dr]
        else:
            drop = np.setdiff1d(np.arange(half), kept[r])
            k = Wkg[_pair_rows(drop, dk)]
        knope.append(k)
    kv_stack = np.concatenate(knope + [Wv], axis=0)          # [G*dn + G*dk, D]
    up, Wdkv = low_rank_split(kv_stack, cfg.kv_rank)
    Wuk, Wuv = up[: G * dn], up[G * dn:]

    qrows = []
    for i in range(H):
        Wqi = Wq[i * dk:(i + 1) * dk]
        r = i // heads_per_rg
        rows = _pair_rows(kept[r], dk)
        if shared:
            qn = Wqi
        else:
            drop = np.setdiff1d(np.arange(half), kept[r])
            qn = Wqi[_pair_rows(drop, dk)]
        qrows += [qn, Wqi[rows]]
    q_stack = np.concatenate(qrows, axis=0)                  # [H*(dn+dr), D]
    if cfg.q_rank:
        Wuq, Wdq = low_rank_split(q_stack, cfg.q_rank)
    else:
        Wuq, Wdq = q_stack, None

    inv_freq_s = np.stack([inv_freq_t[kept[r]] for r in range(Gr)])
    Wdkv_kr = np.concatenate([Wdkv, Wkr], axis=0)
    if noise_std:
        if Wdq is not None:
            Wdq = Wdq + gaussian(rng, Wdq.shape, noise_std)
        Wuq = Wuq + gaussian(rng, Wuq.shape, noise_std)
        Wdkv_kr = Wdkv_kr + gaussian(rng, Wdkv_kr.shape, noise_std)
        Wuk = Wuk + gaussian(rng, Wuk.shape, noise_std)
        Wuv = Wuv + gaussian(rng, Wuv.shape, noise_std)
    return Wdq, Wuq, Wdkv_kr, Wuk, Wuv, inv_freq_s, kept


def make_workload(cfg: LayerConfig, lengths=None, dtype: str | None = None,
                  noise_std: float = 1e-3, inv_freq_t: np.ndarray | None = None,
                  seed: int | None = None) -> Workload:
    """Draw one full synthetic workload for `cfg`.

    Draw order: h, outlier permutation, W_Q, W_K, W_V, W_O, then the noise of
    W_DQ, W_UQ, [W_DKV; W_KR], W_UK, W_UV.  `lengths` gives right-padding
    valid lengths per sequence (default: all tokens valid).
    """
    dtype = dtype or cfg.dtype
    rng = make_rng(cfg.seed if seed is None else seed)
    D, H, G, dk = cfg.hidden, cfg.n_heads, cfg.n_kv_groups, cfg.head_dim
    h = hidden_states(cfg, rng)
    Wq = gaussian(rng, (H * dk, D), 1.0 / np.sqrt(D))
    Wk = gaussian(rng, (G * dk, D), 1.0 / np.sqrt(D))
    Wv = gaussian(rng, (G * dk, D), 1.0 / np.sqrt(D))
    Wo = gaussian(rng, (D, H * dk), 1.0 / np.sqrt(H * dk))
    if inv_freq_t is None:
        inv_freq_t = rope_inv_freq(dk, cfg.rope_theta)
    Wdq, Wuq, Wdkv_kr, Wuk, Wuv, inv_freq_s, kept = student_init(
        cfg, Wq, Wk, Wv, inv_freq_t, rng, noise_std)
    if lengths is None:
        mask = np.ones((cfg.batch, cfg.seq), dtype=np.uint8)
    else:
        mask = right_padding_mask(cfg.batch, cfg.seq, lengths)
    r = lambda x: None if x is None else round_to(x, dtype)
    return Workload(cfg=cfg, h=r(h), mask=mask, Wq=r(Wq), Wk=r(Wk), Wv=r(Wv), Wo=r(Wo),
                    inv_freq_t=to_f32(inv_freq_t).astype(np.float64),
                    Wdq=r(Wdq), Wuq=r(Wuq), Wdkv_kr=r(Wdkv_kr), Wuk=r(Wuk), Wuv=r(Wuv),
                    inv_freq_s=to_f32(inv_freq_s).astype(np.float64), kept_pairs=kept)


def outlier_permutation(cfg: LayerConfig, seed: int | None = None) -> np.ndarray:
    """The channel permutation make_workload(cfg, seed=seed) draws (its first
    cfg.outlier_channels entries are the outlier channels of that layer's inputs)."""
    rng = make_rng(cfg.seed if seed is None else seed)
    rng.standard_normal((cfg.batch, cfg.seq, cfg.hidden))
    return rng.permutation(cfg.hidden)


def calibration_minibatches(cfg: LayerConfig, n: int, seed: int, dtype: str | None = None,
                            base_seed: int | None = None) -> list:
    """`n` more calibration minibatches [B, T, D] for the layer of make_workload(cfg,
    seed=base_seed): fresh tokens (minibatch k from seed + k) with the same outlier
    channels, rounded to the storage dtype.  They stand in for further batches of cached
    layer inputs of the same model."""
    perm = outlier_permutation(cfg, base_seed)
    return [round_to(hidden_states(cfg, make_rng(seed + k), perm), dtype or cfg.dtype)
            for k in range(n)]


def random_outputs(cfg: LayerConfig, seed: int, dtype: str = "fp32", scale: float = 1.0):
    """Two seeded [B, T, D] arrays standing in for A_MLA and A_orig (loss tests)."""
    rng = make_rng(seed)
    At = gaussian(rng, (cfg.batch, cfg.seq, cfg.hidden), scale)
    As = At + gaussian(rng, At.shape, 0.3 * scale)
    return round_to(As, dtype), round_to(At, dtype)


def random_upstream(cfg: LayerConfig, seed: int, dtype: str, rows=None, scale: float = 1e-3):
    """Seeded upstream gradient dL/dA [B, T, D]; `rows` = list of (b, t) kept non-zero."""
    rng = make_rng(seed)
    dA = gaussian(rng, (cfg.batch, cfg.seq, cfg.hidden), scale)
    if rows is not None:
        keep = np.zeros((cfg.batch, cfg.seq), dtype=bool)
        for b, t in rows:
            keep[b, t] = True
        dA[~keep] = 0.0
    return round_to(dA, dtype)
