"""Plain float64 CPU reference of decoding with the reconstructed MLA block in absorbed form.

TEST INFRASTRUCTURE ONLY: only the test-suite may import it.  It shares no code with
the GPU path and imports nothing from it.

After reconstruction the MLA block keeps, per token, only the latent c^KV_j and the
rotated positional key k^PE_j (Eq. 5's cache).  A new query attends to that cache without
forming k^nope or v: since k^nope_{g,j} = W_UK[g] c_j and v_{g,j} = W_UV[g] c_j,

    q^nope_i . k^nope_{g,j} = (W_UK[g]^T q^nope_i) . c_j      (the absorbed query)
    sum_j p_ij v_{g,j}      = W_UV[g] (sum_j p_ij c_j),

so head i attends with [W_UK[g]^T q^nope_i ; q^rope_i] against [c_j ; k^PE_{r(i),j}] and
its output is W_UV[g] applied to the attention-weighted latent.  g = i // (H / G_kv),
r = i // (H / G_r).
"""
from __future__ import annotations

import numpy as np


def absorbed_decode(q, cache, lengths, Wuk, Wuv, *, n_heads, s_kv_groups, s_rope_groups,
                    nope_dim, rope_dim, scale):
    """o [B, H, d_v] of one query token per sequence over its first lengths[b] cache rows.

    q: [B, H, d_nope + d_rope] (rope part rotated at the query's position);
    cache: [B, L, r_kv + G_r d_rope] = [c^KV | rotated k^PE]; Wuk [G_kv d_nope, r_kv];
    Wuv [G_kv d_v, r_kv]."""
    q = np.asarray(q, dtype=np.float64)
    cache = np.asarray(cache, dtype=np.float64)
    B, H = q.shape[0], n_heads
    dn, dr, Gkv, Gr = nope_dim, rope_dim, s_kv_groups, s_rope_groups
    r_kv = Wuk.shape[1]
    dv = Wuv.shape[0] // Gkv
    Wuk = np.asarray(Wuk, dtype=np.float64)
    Wuv = np.asarray(Wuv, dtype=np.float64)
    out = np.zeros((B, H, dv))
    for b in range(B):
        n = int(lengths[b])
        if n == 0:                     # an empty cache attends to nothing: o = 0 (reading)
            continue
        c = cache[b, :n, :r_kv]
        for i in range(H):
            g, r = i // (H // Gkv), i // (H // Gr)
            q_abs = Wuk[g * dn:(g + 1) * dn].T @ q[b, i, :dn]
            kpe = cache[b, :n, r_kv + r * dr:r_kv + (r + 1) * dr]
            s = (c @ q_abs + kpe @ q[b, i, dn:]) * scale
            p = np.exp(s - s.max())
            p /= p.sum()
            out[b, i] = Wuv[g * dv:(g + 1) * dv] @ (p @ c)
    return out
