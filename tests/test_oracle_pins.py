"""Pins of the float64 oracle against what the paper and mathematics fix.

Each test names the passage it follows.  None of them compares the oracle
with itself: the references are exact identities of the paper (Eq. 6-8,
MHA as G = H), closed forms (RoPE as complex rotation, relativity of R_tj),
torch's own causal attention, finite differences and autograd, and a value
of Eq. 11 computed by hand.
"""
import json
import os

import numpy as np
import pytest

import oracle as O
from paper_2607_27269_amd import configs, synth

HERE = os.path.dirname(os.path.abspath(__file__))


def tiny_cfg(**kw):
    base = configs.LayerConfig("pin", "fp64", batch=2, seq=24, hidden=256, n_heads=4,
                               n_kv_groups=2, head_dim=64, rope_theta=1e4, q_rank=256,
                               kv_rank=256, nope_dim=64, rope_dim=32, s_kv_groups=2,
                               s_rope_groups=1)
    return base.replace(**kw)


def run_student(wl, cfg, pos_offset=0):
    s = wl.student_weights()
    A, cache = O.student_forward(wl.h, s["Wdq"], s["Wuq"], s["Wdkv_kr"], s["Wuk"], s["Wuv"],
                                 wl.Wo, s["inv_freq"], n_heads=cfg.n_heads,
                                 s_kv_groups=cfg.s_kv_groups, s_rope_groups=cfg.s_rope_groups,
                                 nope_dim=cfg.nope_dim, rope_dim=cfg.rope_dim,
                                 scale=cfg.softmax_scale, pos_offset=pos_offset)
    return A, cache


def run_teacher(wl, cfg, pos_offset=0):
    return O.teacher_forward(wl.h, wl.Wq, wl.Wk, wl.Wv, wl.Wo, wl.inv_freq_t, cfg.n_heads,
                             cfg.n_kv_groups, cfg.softmax_scale, pos_offset)


# ---------------------------------------------------------------------------
# P1: Eq. 6-7 -- at full latent rank with identical RoPE handling the student
# reproduces the teacher exactly, so Eq. 11 is zero.
# ---------------------------------------------------------------------------

def _zero_loss_case(case):
    if case == "Z0":   # shared positional key, RoPE off on both sides
        cfg = tiny_cfg()
        wl0 = synth.make_workload(cfg, dtype="fp64", noise_std=0.0)
        wl = synth.make_workload(cfg, dtype="fp64", noise_std=0.0,
                                 inv_freq_t=np.zeros_like(wl0.inv_freq_t))
    elif case == "Z1":  # per-group positional keys keeping every rotary pair
        cfg = tiny_cfg(nope_dim=0, rope_dim=64, s_rope_groups=2)
        wl = synth.make_workload(cfg, dtype="fp64", noise_std=0.0)
    else:               # per-group keys, subset kept, dropped pairs not rotated by the teacher
        cfg = tiny_cfg(nope_dim=48, rope_dim=16, s_rope_groups=2)
        wl0 = synth.make_workload(cfg, dtype="fp64", noise_std=0.0)
        kept = set(wl0.kept_pairs.ravel().tolist())
        assert np.all(wl0.kept_pairs[0] == wl0.kept_pairs[0])
        # one inv_freq table for the teacher: zero on pairs that no group keeps
        # and on pairs that only some groups keep (so every group sees R = I there)
        common = set(wl0.kept_pairs[0].tolist())
        for r in range(1, wl0.kept_pairs.shape[0]):
            common &= set(wl0.kept_pairs[r].tolist())
        f = wl0.inv_freq_t.copy()
        for p in range(f.size):
            if p not in common:
                f[p] = 0.0
        wl = synth.make_workload(cfg, dtype="fp64", noise_std=0.0, inv_freq_t=f)
        assert kept  # sanity
    return cfg, wl


@pytest.mark.parametrize("case", ["Z0", "Z1", "Z2"])
def test_P1_zero_loss_at_full_rank(case):
    cfg, wl = _zero_loss_case(case)
    A_t = run_teacher(wl, cfg)
    A_s, _ = run_student(wl, cfg)
    L, rel, dA = O.recon_loss(A_s, A_t, wl.mask)
    assert rel < 1e-20, rel
    assert L < 1e-20 * np.mean(A_t ** 2)


def test_P1_rank_deficit_leaves_residual():
    """Eq. 7: below the rank of the stacked K/V map the residual is non-zero."""
    cfg = tiny_cfg(kv_rank=32)
    wl0 = synth.make_workload(cfg, dtype="fp64", noise_std=0.0)
    wl = synth.make_workload(cfg, dtype="fp64", noise_std=0.0,
                             inv_freq_t=np.zeros_like(wl0.inv_freq_t))
    A_t = run_teacher(wl, cfg)
    A_s, _ = run_student(wl, cfg)
    L, rel, _ = O.recon_loss(A_s, A_t, wl.mask)
    assert rel > 1e-3


# ---------------------------------------------------------------------------
# P2: softmax rows (Eq. 3) sum to one over u <= t and vanish above the diagonal
# ---------------------------------------------------------------------------

def test_P2_causal_softmax_rows():
    rng = np.random.default_rng(1)
    S = rng.standard_normal((37, 37)) * 5
    P = O.causal_softmax(S)
    assert np.allclose(P.sum(axis=1), 1.0, atol=1e-14, rtol=0)
    assert np.all(P[np.triu_indices(37, 1)] == 0.0)
    assert np.all(P[np.tril_indices(37)] > 0)
    # first row attends only to itself
    assert P[0, 0] == 1.0
    # against the definition exp(s_tj) / sum_{u<=t} exp(s_tu), evaluated in long double
    t = 20
    e = np.exp(S[t, : t + 1].astype(np.longdouble))
    assert np.allclose(P[t, : t + 1], (e / e.sum()).astype(np.float64), rtol=1e-13, atol=0)


def test_P2_attention_vs_torch_sdpa():
    """Eq. 2-4 against torch's causal scaled_dot_product_attention (fp64, CPU)."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    T, d, dv = 33, 16, 12
    q, k, v = rng.standard_normal((T, d)), rng.standard_normal((T, d)), rng.standard_normal((T, dv))
    scale = 0.37
    o, _ = O.causal_attention(q, k, v, scale)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None], torch.from_numpy(k)[None, None],
        torch.from_numpy(v)[None, None], is_causal=True, scale=scale)[0, 0].numpy()
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-13)


def test_P2_teacher_vs_torch_sdpa_gqa():
    """Whole teacher (Eq. 1-4 + W_O) against an SDPA evaluation with repeated KV heads."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    cfg = tiny_cfg(seq=20)
    wl = synth.make_workload(cfg, dtype="fp64")
    A = run_teacher(wl, cfg)
    H, G, dk, T = cfg.n_heads, cfg.n_kv_groups, cfg.head_dim, cfg.seq
    h = torch.from_numpy(wl.h)
    ang = torch.arange(T, dtype=torch.float64)[:, None] * torch.from_numpy(wl.inv_freq_t)[None]
    rot = torch.polar(torch.ones_like(ang), ang)          # e^{i t w_p}

    def rope(x):  # rotate-half pairs as complex numbers z_p = x_p + i x_{p+d/2}
        z = torch.complex(x[..., : dk // 2], x[..., dk // 2:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    for b in range(cfg.batch):
        q = rope((h[b] @ torch.from_numpy(wl.Wq).T).reshape(T, H, dk))
        k = rope((h[b] @ torch.from_numpy(wl.Wk).T).reshape(T, G, dk))
        v = (h[b] @ torch.from_numpy(wl.Wv).T).reshape(T, G, dk)
        k = k.repeat_interleave(H // G, dim=1)
        v = v.repeat_interleave(H // G, dim=1)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           is_causal=True, scale=cfg.softmax_scale)
        ref = o.transpose(0, 1).reshape(T, H * dk) @ torch.from_numpy(wl.Wo).T
        assert np.allclose(A[b], ref.numpy(), rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------------------
# RoPE (Sec. 3.1): R_t as complex rotation; R_tj = R_t^T R_j depends on j - t only
# ---------------------------------------------------------------------------

def test_rope_is_complex_rotation():
    rng = np.random.default_rng(3)
    T, d = 11, 10
    x = rng.standard_normal((T, 3, d))
    f = rng.uniform(0, 2, d // 2)
    c, s = O.rope_tables(f, T, pos_offset=5)
    y = O.rope_apply(x, c, s)
    z = (x[..., : d // 2] + 1j * x[..., d // 2:]) * np.exp(1j * (np.arange(T) + 5)[:, None, None] * f)
    assert np.allclose(y, np.concatenate([z.real, z.imag], axis=-1), atol=1e-14)
    # R^T is the inverse and R is orthogonal
    assert np.allclose(O.rope_apply_transpose(y, c, s), x, atol=1e-14)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-14)
    # position 0 is the identity
    c0, s0 = O.rope_tables(f, 1)
    assert np.array_equal(O.rope_apply(x[:1], c0, s0), x[:1])


def test_P4_rope_relativity_teacher_and_student():
    """Shifting every position by a constant leaves A_orig and A_MLA unchanged."""
    cfg = tiny_cfg(seq=16)
    wl = synth.make_workload(cfg, dtype="fp64")
    for offset in (1, 1000):
        assert np.allclose(run_teacher(wl, cfg, offset), run_teacher(wl, cfg), rtol=1e-10, atol=1e-11)
        assert np.allclose(run_student(wl, cfg, offset)[0], run_student(wl, cfg)[0],
                           rtol=1e-10, atol=1e-11)


# ---------------------------------------------------------------------------
# P3: Eq. 8 -- exact logit-error decomposition of the keep/drop routing
# ---------------------------------------------------------------------------

def test_P3_logit_error_identity():
    rng = np.random.default_rng(4)
    T, dk = 9, 8
    q, dq = rng.standard_normal((T, dk)), 0.1 * rng.standard_normal((T, dk))
    kk, kd, dkk = rng.standard_normal((T, dk)), rng.standard_normal((T, dk)), 0.1 * rng.standard_normal((T, dk))
    f = rng.uniform(0.1, 1.0, dk // 2)
    c, s = O.rope_tables(f, T)
    scale = 1 / np.sqrt(dk)
    s_orig = O.teacher_logits(q, kk + kd, c, s, scale)
    # converted: nope path carries k^drop unrotated, rope path carries k^keep + dk
    s_conv = O.student_logits(q + dq, q + dq, kd, kk + dkk, c, s, scale)

    def Rtj(t, j):   # R_t^T R_j built from 2x2 blocks of angle (j - t) w_p
        R = np.zeros((dk, dk))
        h = dk // 2
        for p in range(h):
            a = (j - t) * f[p]
            R[p, p], R[p, p + h] = np.cos(a), -np.sin(a)
            R[p + h, p], R[p + h, p + h] = np.sin(a), np.cos(a)
        return R

    for t in range(T):
        for j in range(T):
            R = Rtj(t, j)
            rhs = scale * (q[t] @ R @ dkk[j] + q[t] @ (np.eye(dk) - R) @ kd[j]
                           + dq[t] @ R @ (kk[j] + dkk[j]) + dq[t] @ kd[j])
            assert abs((s_conv[t, j] - s_orig[t, j]) - rhs) < 1e-13


# ---------------------------------------------------------------------------
# P5: MHA is GQA with G = H (Sec. 3.1)
# ---------------------------------------------------------------------------

def test_P5_mha_equals_repeated_gqa():
    cfg = tiny_cfg(seq=12)
    wl = synth.make_workload(cfg, dtype="fp64")
    H, G, dk = cfg.n_heads, cfg.n_kv_groups, cfg.head_dim
    rep = lambda W: W.reshape(G, dk, -1).repeat(H // G, axis=0).reshape(H * dk, -1)
    A_gqa = run_teacher(wl, cfg)
    A_mha = O.teacher_forward(wl.h, wl.Wq, rep(wl.Wk), rep(wl.Wv), wl.Wo, wl.inv_freq_t, H, H,
                              cfg.softmax_scale)
    assert np.allclose(A_gqa, A_mha, rtol=1e-13, atol=1e-14)


def test_P5_student_per_head_groups_equal_shared():
    """Student with G_kv = G_r = H and replicated latent maps equals the grouped student."""
    cfg = tiny_cfg(seq=10)
    wl = synth.make_workload(cfg, dtype="fp64")
    H, Gkv, dn, dv, dr, rkv = cfg.n_heads, cfg.s_kv_groups, cfg.nope_dim, cfg.v_dim, cfg.rope_dim, cfg.kv_rank
    A, _ = run_student(wl, cfg)
    rep = lambda W, d, n: W.reshape(n, d, -1).repeat(H // n, axis=0).reshape(H * d, -1)
    Wkr = wl.Wdkv_kr[rkv:]
    Wdkv_kr = np.concatenate([wl.Wdkv_kr[:rkv], np.tile(Wkr, (H, 1))], axis=0)
    A2, _ = O.student_forward(wl.h, wl.Wdq, wl.Wuq, Wdkv_kr, rep(wl.Wuk, dn, Gkv),
                              rep(wl.Wuv, dv, Gkv), wl.Wo, np.tile(wl.inv_freq_s, (H, 1)),
                              n_heads=H, s_kv_groups=H, s_rope_groups=H, nope_dim=dn,
                              rope_dim=dr, scale=cfg.softmax_scale)
    assert np.allclose(A, A2, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------------------
# P8: Eq. 11 -- hand-computed value, masking, sign and gradient properties
# ---------------------------------------------------------------------------

def test_P8_loss_golden_by_hand():
    with open(os.path.join(HERE, "golden", "loss_eq11_tiny.json")) as f:
        g = json.load(f)
    L, rel, dA = O.recon_loss(np.array(g["A_s"], float), np.array(g["A_t"], float),
                              np.array(g["mask"], np.uint8))
    assert L == pytest.approx(g["loss"], rel=1e-15)
    assert rel == pytest.approx(g["rel"], rel=1e-15)
    assert np.allclose(dA, np.array(g["dA"]), rtol=1e-15, atol=0)


def test_P8_loss_properties():
    rng = np.random.default_rng(5)
    A_s, A_t = rng.standard_normal((3, 7, 5)), rng.standard_normal((3, 7, 5))
    mask = (rng.uniform(size=(3, 7)) < 0.6).astype(np.uint8)
    mask[0, 0] = 1
    L, rel, dA = O.recon_loss(A_s, A_t, mask)
    assert L > 0
    # zero iff equal on valid rows
    A2 = np.where(mask[..., None] == 1, A_t, A_s)
    assert O.recon_loss(A2, A_t, mask)[0] == 0.0
    # masked rows change neither the loss nor the gradient
    A3 = A_s + (1 - mask[..., None]) * 100.0
    L3, _, dA3 = O.recon_loss(A3, A_t, mask)
    assert L3 == L and np.array_equal(dA3, dA)
    # gradient by central differences in one coordinate
    b, t, d = np.argwhere(mask == 1)[0][0], np.argwhere(mask == 1)[0][1], 2
    e = 1e-6
    Ap, Am = A_s.copy(), A_s.copy()
    Ap[b, t, d] += e
    Am[b, t, d] -= e
    fd = (O.recon_loss(Ap, A_t, mask)[0] - O.recon_loss(Am, A_t, mask)[0]) / (2 * e)
    assert fd == pytest.approx(dA[b, t, d], rel=1e-7)
    # an all-invalid minibatch contributes nothing
    L0, rel0, dA0 = O.recon_loss(A_s, A_t, np.zeros_like(mask))
    assert L0 == 0.0 and not dA0.any()
    # relative error: a silent teacher on the valid rows is the only degenerate denominator
    # (0 when the student is silent too, else +inf); a NaN anywhere on a valid row is NaN
    Az = np.where(mask[..., None] == 1, 0.0, A_t)
    assert O.recon_loss(A_s, Az, mask)[1] == np.inf
    assert O.recon_loss(np.where(mask[..., None] == 1, 0.0, A_s), Az, mask)[1] == 0.0
    An = A_t.copy()
    An[b, t, 0] = np.nan
    Ln, reln, _ = O.recon_loss(A_s, An, mask)
    assert np.isnan(Ln) and np.isnan(reln)


# ---------------------------------------------------------------------------
# P6/P7: analytic gradients against finite differences and torch autograd
# ---------------------------------------------------------------------------

def fd_cfg(**kw):
    base = configs.LayerConfig("fd", "fp64", batch=2, seq=8, hidden=32, n_heads=4,
                               n_kv_groups=2, head_dim=8, rope_theta=100.0, q_rank=8,
                               kv_rank=8, nope_dim=8, rope_dim=4, s_kv_groups=2,
                               s_rope_groups=1)
    return base.replace(**kw)


def _loss_of(wl, cfg, A_t, student):
    A, _ = O.student_forward(wl.h, student["Wdq"], student["Wuq"], student["Wdkv_kr"],
                             student["Wuk"], student["Wuv"], wl.Wo, wl.inv_freq_s,
                             n_heads=cfg.n_heads, s_kv_groups=cfg.s_kv_groups,
                             s_rope_groups=cfg.s_rope_groups, nope_dim=cfg.nope_dim,
                             rope_dim=cfg.rope_dim, scale=cfg.softmax_scale)
    return O.recon_loss(A, A_t, wl.mask)[0]


@pytest.mark.parametrize("variant", ["shared_rope", "per_group_rope", "no_q_rank"])
def test_P7_gradients_vs_finite_differences(variant):
    if variant == "shared_rope":
        cfg = fd_cfg()
    elif variant == "per_group_rope":
        cfg = fd_cfg(nope_dim=4, rope_dim=4, s_rope_groups=2)
    else:
        cfg = fd_cfg(q_rank=0, n_kv_groups=4, s_kv_groups=4, s_rope_groups=4, nope_dim=4,
                     rope_dim=4)
    wl = synth.make_workload(cfg, dtype="fp64", lengths=[8, 5], noise_std=0.05)
    A_t = run_teacher(wl, cfg)
    A_s, cache = run_student(wl, cfg)
    L, _, dA = O.recon_loss(A_s, A_t, wl.mask)
    grads = O.student_backward(cache, dA)
    base = dict(Wdq=wl.Wdq, Wuq=wl.Wuq, Wdkv_kr=wl.Wdkv_kr, Wuk=wl.Wuk, Wuv=wl.Wuv)
    rng = np.random.default_rng(6)
    for name, W in base.items():
        if W is None:
            assert grads["d" + name] is None
            continue
        V = rng.standard_normal(W.shape)
        eps = 1e-6
        plus = dict(base, **{name: W + eps * V})
        minus = dict(base, **{name: W - eps * V})
        fd = (_loss_of(wl, cfg, A_t, plus) - _loss_of(wl, cfg, A_t, minus)) / (2 * eps)
        an = float(np.sum(grads["d" + name] * V))
        assert fd == pytest.approx(an, rel=1e-6, abs=1e-12), name


def test_P6_gradients_vs_torch_autograd():
    torch = pytest.importorskip("torch")
    cfg = fd_cfg(seq=12, hidden=48)
    wl = synth.make_workload(cfg, dtype="fp64", lengths=[12, 7], noise_std=0.05)
    A_t = run_teacher(wl, cfg)
    A_s, cache = run_student(wl, cfg)
    _, _, dA = O.recon_loss(A_s, A_t, wl.mask)
    grads = O.student_backward(cache, dA)

    H, Gkv, Gr, dn, dr, dv = (cfg.n_heads, cfg.s_kv_groups, cfg.s_rope_groups, cfg.nope_dim,
                              cfg.rope_dim, cfg.v_dim)
    B, T = cfg.batch, cfg.seq
    W = {k: torch.tensor(getattr(wl, k), requires_grad=True)
         for k in ("Wdq", "Wuq", "Wdkv_kr", "Wuk", "Wuv")}
    h = torch.from_numpy(wl.h)
    Wo = torch.from_numpy(wl.Wo)
    ang = torch.arange(T, dtype=torch.float64)[:, None] * torch.from_numpy(wl.inv_freq_s[0])[None]
    cz = torch.polar(torch.ones_like(ang), ang)

    def rope(x):
        z = torch.complex(x[..., : dr // 2], x[..., dr // 2:]) * cz[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    outs = []
    for b in range(B):
        q = (h[b] @ W["Wdq"].T @ W["Wuq"].T).reshape(T, H, dn + dr)
        ck = h[b] @ W["Wdkv_kr"].T
        rkv = cfg.kv_rank
        kn = (ck[:, :rkv] @ W["Wuk"].T).reshape(T, Gkv, dn).repeat_interleave(H // Gkv, 1)
        v = (ck[:, :rkv] @ W["Wuv"].T).reshape(T, Gkv, dv).repeat_interleave(H // Gkv, 1)
        kp = rope(ck[:, rkv:].reshape(T, Gr, dr)).repeat_interleave(H // Gr, 1)
        qq = torch.cat([q[..., :dn], rope(q[..., dn:])], -1)
        kk = torch.cat([kn, kp], -1)
        o = torch.nn.functional.scaled_dot_product_attention(
            qq.transpose(0, 1), kk.transpose(0, 1), v.transpose(0, 1), is_causal=True,
            scale=cfg.softmax_scale)
        outs.append(o.transpose(0, 1).reshape(T, H * dv) @ Wo.T)
    A = torch.stack(outs)
    M = torch.from_numpy(wl.mask.astype(np.float64))[..., None]
    L = ((M * (A - torch.from_numpy(A_t))) ** 2).sum() / (cfg.hidden * M.sum())
    L.backward()
    for k in W:
        assert np.allclose(grads["d" + k], W[k].grad.numpy(), rtol=1e-9, atol=1e-13), k


# ---------------------------------------------------------------------------
# P9: latent gauge -- an invertible change of latent basis leaves A_MLA unchanged
# ---------------------------------------------------------------------------

def test_P9_latent_gauge_invariance():
    cfg = tiny_cfg(seq=10, kv_rank=64, q_rank=96)
    wl = synth.make_workload(cfg, dtype="fp64")
    A, _ = run_student(wl, cfg)
    rng = np.random.default_rng(7)
    rkv = cfg.kv_rank
    S = np.eye(rkv) + 0.3 * rng.standard_normal((rkv, rkv))
    Si = np.linalg.inv(S)
    Sq = np.eye(cfg.q_rank) + 0.3 * rng.standard_normal((cfg.q_rank, cfg.q_rank))
    Wdkv_kr = wl.Wdkv_kr.copy()
    Wdkv_kr[:rkv] = S @ wl.Wdkv_kr[:rkv]
    A2, _ = O.student_forward(wl.h, Sq @ wl.Wdq, wl.Wuq @ np.linalg.inv(Sq), Wdkv_kr,
                              wl.Wuk @ Si, wl.Wuv @ Si, wl.Wo, wl.inv_freq_s,
                              n_heads=cfg.n_heads, s_kv_groups=cfg.s_kv_groups,
                              s_rope_groups=cfg.s_rope_groups, nope_dim=cfg.nope_dim,
                              rope_dim=cfg.rope_dim, scale=cfg.softmax_scale)
    assert np.allclose(A, A2, rtol=1e-9, atol=1e-10)


def test_stop_gradient_teacher_is_frozen():
    """Sec. 4: the gradient set is exactly the converter-introduced projections."""
    cfg = fd_cfg()
    wl = synth.make_workload(cfg, dtype="fp64")
    A_s, cache = run_student(wl, cfg)
    g = O.student_backward(cache, np.ones_like(A_s))
    assert set(g) == {"dWdq", "dWuq", "dWdkv_kr", "dWuk", "dWuv"}
