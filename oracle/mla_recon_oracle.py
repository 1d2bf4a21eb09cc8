"""Plain float64 CPU oracle of the end-to-end functional-reconstruction step.

TEST INFRASTRUCTURE ONLY.  This module is the correctness reference for the
HIP implementation; only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark may import it.  It shares no code with the GPU path and
imports nothing from it.

What it computes (paper: "Beyond KV Reconstruction: Functional Reconstruction
for MLA Draft Models in Speculative Decoding"):

* teacher: the frozen GQA block, Eq. 1 (projections q = W^Q_i h, k = W^K_g h,
  v = W^V_g h), Sec. 3.1 (RoPE rotation R_t, relative rotation R_tj), Eq. 2-4
  (scaled causal softmax attention), then the fixed output projection W_O
  (Sec. 4.1, A^l is the attention output after W_O);
* student: the converted MLA block, Eq. 5 (latent c = W^DKV h, stacked
  [k^nope; v] = W^UKV c, small positional key k^PE), the low-rank query
  (c^Q = W_DQ h, q = W_UQ c^Q: the converter-introduced query projection of
  Sec. 4, DeepSeek-V2 style), RoPE on the positional query/key, the same
  causal softmax and the same frozen W_O;
* loss: Eq. 11, ||M (A_MLA - sg[A_orig])||_F^2 / (D sum_t M_t), over one
  minibatch with all its tokens flattened;
* backward: hand-derived gradients of Eq. 11 with respect to the
  converter-introduced projections only (Sec. 4: W_O and the teacher are
  frozen, the teacher path is under stop-gradient, the hidden states are data).

Everything is a direct definition: attention is materialised T x T per
(sequence, head), softmax subtracts the row maximum, and there is no tiling,
fusion or reordering.  numpy's matmul is the only library primitive used.

Conventions (readings where the paper is silent):
* RoPE is the rotate-half form: pair p couples dims (p, p + d/2) and rotates
  by angle t * inv_freq[p]; positions restart at 0 in every sequence.
* Both logits are scaled by 1/sqrt(d_k) of the teacher (Eq. 2, Eq. 8).
* Causal mask includes the diagonal (Eq. 3 sums u <= t); the valid-token mask
  M only enters the loss (Eq. 11).
* The student query of head i is [q^nope_i; q^rope_i]; its key is
  [k^nope_{g_kv(i)}; k^PE_{r(i)}] with g_kv(i) = i // (H/G_kv) and
  r(i) = i // (H/G_r); its value is v_{g_kv(i)}.
* An all-invalid mask gives L = 0 and dA = 0.

Parity pins: every function here is checked in tests/test_oracle_pins.py
against the paper's exact statements (zero loss at full rank, Eq. 6-7; the
logit-error identity, Eq. 8; MHA as G = H), closed forms (RoPE as complex
rotation, relativity of R_tj), a library routine (torch's causal
scaled-dot-product attention), finite differences and autograd for the
backward, and a hand-computed value of Eq. 11 (tests/golden).
"""
from __future__ import annotations

import numpy as np

# ----------------------------------------------------------------------------
# RoPE (Sec. 3.1): R_t rotates pair p by angle t * inv_freq[p]
# ----------------------------------------------------------------------------


def rope_tables(inv_freq: np.ndarray, T: int, pos_offset: int = 0):
    """cos/sin of t * inv_freq[p] for positions pos_offset .. pos_offset+T-1."""
    t = np.arange(T, dtype=np.float64) + float(pos_offset)
    ang = t[:, None] * np.asarray(inv_freq, dtype=np.float64)[None, :]
    return np.cos(ang), np.sin(ang)


def rope_apply(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """R_t x for x of shape [T, ..., d]; cos/sin of shape [T, d/2]."""
    half = x.shape[-1] // 2
    shape = (cos.shape[0],) + (1,) * (x.ndim - 2) + (half,)
    c, s = cos.reshape(shape), sin.reshape(shape)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def rope_apply_transpose(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """R_t^T x (the inverse rotation), same shapes as rope_apply."""
    return rope_apply(x, cos, -sin)


# ----------------------------------------------------------------------------
# scaled causal softmax attention, Eq. 2-4, for one (sequence, head)
# ----------------------------------------------------------------------------


def causal_softmax(S: np.ndarray) -> np.ndarray:
    """Row-wise softmax over u <= t (Eq. 3); entries above the diagonal are 0."""
    T = S.shape[0]
    allowed = np.tril(np.ones((T, S.shape[1]), dtype=bool))
    Sm = np.where(allowed, S, -np.inf)
    Sm = Sm - Sm.max(axis=1, keepdims=True)
    E = np.exp(Sm)
    return E / E.sum(axis=1, keepdims=True)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float):
    """o_t = sum_{j<=t} softmax_j(q_t . k_j * scale) v_j.  q,k: [T,d], v: [T,dv].

    The inputs are already rotated, so q_t . k_j equals q^T R_tj k of Eq. 2.
    Returns (o [T, dv], P [T, T]).
    """
    S = (q @ k.T) * scale
    P = causal_softmax(S)
    return P @ v, P


# ----------------------------------------------------------------------------
# teacher: frozen GQA block + W_O (Eq. 1-4, Sec. 4.1)
# ----------------------------------------------------------------------------


def teacher_forward(h, Wq, Wk, Wv, Wo, inv_freq, n_heads, n_kv_groups, scale, pos_offset=0):
    """A_orig(h) = W_O concat_i o_i.  h: [B, T, D] -> A: [B, T, D]."""
    h = np.asarray(h, dtype=np.float64)
    B, T, D = h.shape
    H, G = n_heads, n_kv_groups
    dk = Wq.shape[0] // H
    cos, sin = rope_tables(inv_freq, T, pos_offset)
    A = np.zeros((B, T, Wo.shape[0]))
    for b in range(B):
        q = (h[b] @ Wq.T).reshape(T, H, dk)
        k = (h[b] @ Wk.T).reshape(T, G, dk)
        v = (h[b] @ Wv.T).reshape(T, G, dk)
        q, k = rope_apply(q, cos, sin), rope_apply(k, cos, sin)
        o = np.zeros((T, H, dk))
        for i in range(H):
            g = i // (H // G)                       # g(i): group of query head i
            o[:, i], _ = causal_attention(q[:, i], k[:, g], v[:, g], scale)
        A[b] = o.reshape(T, H * dk) @ Wo.T
    return A


# ----------------------------------------------------------------------------
# student: converted MLA block + the same frozen W_O (Eq. 5, Sec. 4)
# ----------------------------------------------------------------------------


def student_logits(q_nope, q_rope, k_nope, k_pe, cos, sin, scale):
    """S_tj = ([q^nope_t; R_t q^rope_t] . [k^nope_j; R_j k^PE_j]) * scale for one head."""
    qh = np.concatenate([q_nope, rope_apply(q_rope, cos, sin)], axis=-1)
    kh = np.concatenate([k_nope, rope_apply(k_pe, cos, sin)], axis=-1)
    return (qh @ kh.T) * scale


def teacher_logits(q, k, cos, sin, scale):
    """S_tj = q_t^T R_tj k_j * scale (Eq. 2) for one head."""
    return (rope_apply(q, cos, sin) @ rope_apply(k, cos, sin).T) * scale


def student_forward(h, Wdq, Wuq, Wdkv_kr, Wuk, Wuv, Wo, inv_freq, *, n_heads, s_kv_groups,
                    s_rope_groups, nope_dim, rope_dim, scale, pos_offset=0):
    """A_MLA(h) and the intermediates the backward needs.

    c^Q = h W_DQ^T (h itself when W_DQ is None), q = c^Q W_UQ^T per head
    [q^nope; q^rope]; [c^KV | k^PE] = h [W_DKV; W_KR]^T; k^nope = c^KV W_UK^T,
    v = c^KV W_UV^T (Eq. 5); q^rope and k^PE are rotated with their rope
    group's frequencies inv_freq[r] ([G_r, d_rope/2]).
    """
    h = np.asarray(h, dtype=np.float64)
    B, T, D = h.shape
    H, Gkv, Gr, dn, dr = n_heads, s_kv_groups, s_rope_groups, nope_dim, rope_dim
    dqk = dn + dr
    r_kv = Wdkv_kr.shape[0] - Gr * dr
    dv = Wuv.shape[0] // Gkv
    inv_freq = np.asarray(inv_freq, dtype=np.float64).reshape(Gr, dr // 2)
    tables = [rope_tables(inv_freq[r], T, pos_offset) for r in range(Gr)]
    cache = dict(h=h, Wdq=Wdq, Wuq=Wuq, Wdkv_kr=Wdkv_kr, Wuk=Wuk, Wuv=Wuv, Wo=Wo,
                 tables=tables, H=H, Gkv=Gkv, Gr=Gr, dn=dn, dr=dr, dv=dv, r_kv=r_kv,
                 scale=scale, seq=[])
    A = np.zeros((B, T, Wo.shape[0]))
    for b in range(B):
        cQ = h[b] if Wdq is None else h[b] @ Wdq.T
        q = (cQ @ Wuq.T).reshape(T, H, dqk)
        ckv_kpe = h[b] @ Wdkv_kr.T
        ckv = ckv_kpe[:, :r_kv]
        kpe = ckv_kpe[:, r_kv:].reshape(T, Gr, dr)
        knope = (ckv @ Wuk.T).reshape(T, Gkv, dn)
        v = (ckv @ Wuv.T).reshape(T, Gkv, dv)
        # rotated query / key per head, assembled as [nope ; rope]
        qh = np.zeros((T, H, dqk))
        kh = np.zeros((T, H, dqk))
        o = np.zeros((T, H, dv))
        for i in range(H):
            g, r = i // (H // Gkv), i // (H // Gr)
            cos, sin = tables[r]
            qh[:, i, :dn] = q[:, i, :dn]
            qh[:, i, dn:] = rope_apply(q[:, i, dn:], cos, sin)
            kh[:, i, :dn] = knope[:, g]
            kh[:, i, dn:] = rope_apply(kpe[:, r], cos, sin)
            o[:, i], _ = causal_attention(qh[:, i], kh[:, i], v[:, g], scale)
        A[b] = o.reshape(T, H * dv) @ Wo.T
        cache["seq"].append(dict(cQ=cQ, ckv=ckv, qh=qh, kh=kh, v=v, o=o))
    return A, cache


# ----------------------------------------------------------------------------
# loss, Eq. 11
# ----------------------------------------------------------------------------


def recon_loss(A_s, A_t, mask):
    """(L, rel, dL/dA_s).

    L   = sum (M (A_s - A_t))^2 / (D sum M)          (Eq. 11; A_t under stop-gradient)
    rel = sum (M (A_s - A_t))^2 / sum (M A_t)^2       (relative diagnostic)
    dA  = 2 M (A_s - A_t) / (D sum M)
    """
    A_s = np.asarray(A_s, dtype=np.float64)
    A_t = np.asarray(A_t, dtype=np.float64)
    D = A_s.shape[-1]
    M = np.asarray(mask, dtype=np.float64)[..., None]
    E = M * (A_s - A_t)
    sse = float(np.sum(E * E))
    den = float(np.sum(M)) * D
    ref = float(np.sum((M * A_t) ** 2))
    if den == 0.0:
        return 0.0, 0.0, np.zeros_like(A_s)
    # a zero teacher energy is the only degenerate denominator; a NaN one propagates
    rel = (0.0 if sse == 0 else np.inf) if ref == 0 else sse / ref
    return sse / den, rel, 2.0 * E / den


# ----------------------------------------------------------------------------
# backward of Eq. 11 into the converter-introduced projections
# ----------------------------------------------------------------------------


def student_backward(cache, dA):
    """Gradients of L w.r.t. W_DQ, W_UQ, [W_DKV; W_KR], W_UK, W_UV.

    dO = dA W_O (W_O frozen: no dW_O), then per (sequence, head) the softmax
    attention backward: dV += P^T dO, dP = dO V^T, dS = P (dP - rowsum(P dP)),
    dQ = scale dS K, dK = scale dS^T Q; the rotary halves are rotated back with
    R^T, gradients of shared keys/values are summed over the heads that read
    them, and the chain continues through Eq. 5 and the query projection.
    The hidden states are data (no dh).
    """
    h = cache["h"]
    B, T, D = h.shape
    H, Gkv, Gr, dn, dr, dv = (cache[k] for k in ("H", "Gkv", "Gr", "dn", "dr", "dv"))
    dqk = dn + dr
    scale = cache["scale"]
    Wo, Wuq, Wuk, Wuv, Wdq = cache["Wo"], cache["Wuq"], cache["Wuk"], cache["Wuv"], cache["Wdq"]
    g = dict(dWuq=np.zeros_like(Wuq), dWdkv_kr=np.zeros_like(cache["Wdkv_kr"]),
             dWuk=np.zeros_like(Wuk), dWuv=np.zeros_like(Wuv),
             dWdq=None if Wdq is None else np.zeros_like(Wdq))
    dA = np.asarray(dA, dtype=np.float64)
    for b in range(B):
        s = cache["seq"][b]
        dO = (dA[b] @ Wo).reshape(T, H, dv)
        dq = np.zeros((T, H, dqk))
        dknope = np.zeros((T, Gkv, dn))
        dkpe = np.zeros((T, Gr, dr))
        dvv = np.zeros((T, Gkv, dv))
        for i in range(H):
            gi, r = i // (H // Gkv), i // (H // Gr)
            cos, sin = cache["tables"][r]
            qh, kh, vv = s["qh"][:, i], s["kh"][:, i], s["v"][:, gi]
            P = causal_softmax((qh @ kh.T) * scale)
            dvv[:, gi] += P.T @ dO[:, i]
            dP = dO[:, i] @ vv.T
            dS = P * (dP - np.sum(P * dP, axis=1, keepdims=True))
            dqh = scale * (dS @ kh)
            dkh = scale * (dS.T @ qh)
            dq[:, i, :dn] = dqh[:, :dn]
            dq[:, i, dn:] = rope_apply_transpose(dqh[:, dn:], cos, sin)
            dknope[:, gi] += dkh[:, :dn]
            dkpe[:, r] += rope_apply_transpose(dkh[:, dn:], cos, sin)
        dq = dq.reshape(T, H * dqk)
        dknope = dknope.reshape(T, Gkv * dn)
        dvv = dvv.reshape(T, Gkv * dv)
        ckv, cQ = s["ckv"], s["cQ"]
        g["dWuk"] += dknope.T @ ckv
        g["dWuv"] += dvv.T @ ckv
        dckv = dknope @ Wuk + dvv @ Wuv
        g["dWdkv_kr"] += np.concatenate([dckv, dkpe.reshape(T, Gr * dr)], axis=1).T @ h[b]
        g["dWuq"] += dq.T @ cQ
        if Wdq is not None:
            dcQ = dq @ Wuq
            g["dWdq"] += dcQ.T @ h[b]
    return g


# ----------------------------------------------------------------------------
# one whole step
# ----------------------------------------------------------------------------


def reconstruction_step(h, mask, teacher: dict, student: dict, *, n_heads, n_kv_groups,
                        s_kv_groups, s_rope_groups, nope_dim, rope_dim, scale):
    """teacher fwd -> student fwd -> Eq. 11 -> gradients.  Returns a dict."""
    A_t = teacher_forward(h, teacher["Wq"], teacher["Wk"], teacher["Wv"], teacher["Wo"],
                          teacher["inv_freq"], n_heads, n_kv_groups, scale)
    A_s, cache = student_forward(h, student["Wdq"], student["Wuq"], student["Wdkv_kr"],
                                 student["Wuk"], student["Wuv"], teacher["Wo"],
                                 student["inv_freq"], n_heads=n_heads,
                                 s_kv_groups=s_kv_groups, s_rope_groups=s_rope_groups,
                                 nope_dim=nope_dim, rope_dim=rope_dim, scale=scale)
    L, rel, dA = recon_loss(A_s, A_t, mask)
    grads = student_backward(cache, dA)
    return dict(A_t=A_t, A_s=A_s, loss=L, rel=rel, dA=dA, **grads)
