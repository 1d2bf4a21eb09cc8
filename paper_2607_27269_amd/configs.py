"""Shape registry for the functional-reconstruction step.

Each entry describes one attention layer: the frozen original GQA/MHA block
(Sec. 3.1, Eq. 1-4: hidden size D, H query heads, G KV groups, head dim d_k)
and the converted MLA block that is reconstructed against it (Sec. 3.2, Eq. 5:
latent rank r, decoupled positional key; Sec. 4.1: the query and KV
projections the converter introduces).  The five shapes are the synthetic
stand-ins for the paper's draft models (Sec. 5.1: Llama/Qwen drafts); no
trained weight or calibration text is used anywhere.

This module holds no arithmetic of the method; it only names sizes.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass


@dataclass(frozen=True)
class LayerConfig:
    name: str
    dtype: str            # "fp32" (check mode) or "bf16"
    batch: int            # B sequences per calibration minibatch
    seq: int              # T tokens per sequence
    hidden: int           # D
    n_heads: int          # H
    n_kv_groups: int      # G (teacher); G == H is the MHA case
    head_dim: int         # d_k (teacher key and value width)
    rope_theta: float     # teacher RoPE base
    q_rank: int           # r_q; 0 means the query is not factorised (q = W_UQ h)
    kv_rank: int          # r (the KV latent rank of Eq. 5)
    nope_dim: int         # d_nope: student per-head non-positional q/k width
    rope_dim: int         # d_rope: student per-head rotary q/k width (even)
    s_kv_groups: int      # G_kv: student groups of non-positional keys/values
    s_rope_groups: int    # G_r: heads of the decoupled positional key k^PE
    outlier_channels: int = 0
    outlier_scale: float = 1.0
    seed: int = 0

    # ---- derived sizes -------------------------------------------------
    @property
    def tokens(self) -> int:
        return self.batch * self.seq

    @property
    def v_dim(self) -> int:          # student value width equals the teacher's d_k
        return self.head_dim

    @property
    def qk_dim(self) -> int:         # student per-head logit width d_nope + d_rope
        return self.nope_dim + self.rope_dim

    @property
    def softmax_scale(self) -> float:
        # Both logits are divided by sqrt(d_k) of the teacher (Eq. 2 and Eq. 8).
        return 1.0 / float(self.head_dim) ** 0.5

    @property
    def kv_out(self) -> int:         # rows of [W_DKV; W_KR]
        return self.kv_rank + self.s_rope_groups * self.rope_dim

    def replace(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)

    # ---- algorithmic work, counted as 2*M*N*K per product; causal attention
    # counts T(T+1)/2 (query, key) pairs per (sequence, head) ----------------
    def flops(self) -> dict:
        N, D, H, G, dk = self.tokens, self.hidden, self.n_heads, self.n_kv_groups, self.head_dim
        rq, rkv, dn, dr, dv = self.q_rank, self.kv_rank, self.nope_dim, self.rope_dim, self.v_dim
        gkv, gr = self.s_kv_groups, self.s_rope_groups
        dqk = dn + dr
        pairs = self.batch * H * self.seq * (self.seq + 1) / 2.0
        f = {}
        f["T1_qkv_proj"] = 2.0 * N * D * (H + 2 * G) * dk
        f["T3_attn_fwd"] = 2.0 * pairs * (dk + dk)
        f["T4_wo"] = 2.0 * N * (H * dk) * D
        q_in = D if rq == 0 else rq
        f["S1_q_path"] = (2.0 * N * D * rq if rq else 0.0) + 2.0 * N * q_in * H * dqk
        f["S2_kv_down"] = 2.0 * N * D * self.kv_out
        f["S3_up_proj"] = 2.0 * N * rkv * gkv * (dn + dv)
        f["S4_attn_fwd"] = 2.0 * pairs * (dqk + dv)
        f["S5_wo"] = 2.0 * N * (H * dv) * D
        f["B1_dO"] = 2.0 * N * D * H * dv
        # dV = P^T dO, dP = dO V^T, dQ = dS K, dK = dS^T Q
        f["B2_attn_bwd"] = 2.0 * pairs * (dv + dv + dqk + dqk)
        f["B3_up_bwd"] = 2.0 * 2.0 * N * rkv * gkv * (dn + dv)
        f["B4_down_bwd"] = 2.0 * N * D * self.kv_out
        f["B5_q_bwd"] = 2.0 * N * q_in * H * dqk * (2.0 if rq else 1.0) + (2.0 * N * rq * D if rq else 0.0)
        return f

    def total_flops(self) -> float:
        return float(sum(self.flops().values()))


CONFIGS = {
    0: LayerConfig("tiny-gqa-fp32", "fp32", batch=2, seq=64, hidden=256, n_heads=4,
                   n_kv_groups=2, head_dim=64, rope_theta=1e4, q_rank=128, kv_rank=128,
                   nope_dim=64, rope_dim=32, s_kv_groups=2, s_rope_groups=1),
    1: LayerConfig("qwen2.5-0.5b-layer", "bf16", batch=8, seq=2048, hidden=896, n_heads=14,
                   n_kv_groups=2, head_dim=64, rope_theta=1e6, q_rank=512, kv_rank=256,
                   nope_dim=64, rope_dim=32, s_kv_groups=2, s_rope_groups=1,
                   outlier_channels=4, outlier_scale=20.0),
    2: LayerConfig("llama-3.2-1b-layer", "bf16", batch=8, seq=2048, hidden=2048, n_heads=32,
                   n_kv_groups=8, head_dim=64, rope_theta=5e5, q_rank=1024, kv_rank=512,
                   nope_dim=64, rope_dim=64, s_kv_groups=8, s_rope_groups=1,
                   outlier_channels=4, outlier_scale=20.0),
    3: LayerConfig("llama-3-8b-layer", "bf16", batch=4, seq=4096, hidden=4096, n_heads=32,
                   n_kv_groups=8, head_dim=128, rope_theta=5e5, q_rank=1536, kv_rank=512,
                   nope_dim=128, rope_dim=64, s_kv_groups=8, s_rope_groups=1,
                   outlier_channels=8, outlier_scale=30.0),
    4: LayerConfig("mha-partial-rope-layer", "bf16", batch=4, seq=4096, hidden=4096, n_heads=32,
                   n_kv_groups=32, head_dim=128, rope_theta=1e4, q_rank=0, kv_rank=1024,
                   nope_dim=112, rope_dim=16, s_kv_groups=32, s_rope_groups=32,
                   outlier_channels=8, outlier_scale=30.0),
}


def get(idx: int) -> LayerConfig:
    return CONFIGS[idx]


def shrink(cfg: LayerConfig, batch: int, seq: int, **kw) -> LayerConfig:
    """Same layer shape with fewer / shorter sequences (parity-test sizes)."""
    return cfg.replace(batch=batch, seq=seq, **kw)
