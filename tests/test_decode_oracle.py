"""Pin of the absorbed-form decode oracle: on the cache of a student forward, attending with
the absorbed query must give the naive block's output at the last cached token (Eq. 5's
factorisation of k^nope and v through the latent), for shared and per-head positional keys
and ragged lengths."""
import numpy as np
import pytest

import oracle as O
from paper_2607_27269_amd import configs, synth


@pytest.mark.parametrize("idx", [1, 4])
def test_absorbed_equals_naive_last_token(idx):
    cfg = configs.shrink(configs.get(idx), batch=2, seq=40)
    wl = synth.make_workload(cfg, dtype="fp64")
    s = wl.student_weights()
    _, cache = O.student_forward(wl.h, s["Wdq"], s["Wuq"], s["Wdkv_kr"], s["Wuk"], s["Wuv"], wl.Wo,
                                 s["inv_freq"], n_heads=cfg.n_heads, s_kv_groups=cfg.s_kv_groups,
                                 s_rope_groups=cfg.s_rope_groups, nope_dim=cfg.nope_dim,
                                 rope_dim=cfg.rope_dim, scale=cfg.softmax_scale)
    dn, dr, Gr, H = cfg.nope_dim, cfg.rope_dim, cfg.s_rope_groups, cfg.n_heads
    lengths = [40, 23]
    q = np.zeros((2, H, dn + dr))
    kv = np.zeros((2, 40, cfg.kv_rank + Gr * dr))
    want = np.zeros((2, H, cfg.head_dim))
    for b, n in enumerate(lengths):
        seq = cache["seq"][b]
        q[b] = seq["qh"][n - 1]
        kv[b, :, :cfg.kv_rank] = seq["ckv"]
        for r in range(Gr):              # head i of rope group r carries that group's key
            kv[b, :, cfg.kv_rank + r * dr:cfg.kv_rank + (r + 1) * dr] = seq["kh"][:, r * (H // Gr), dn:]
        want[b] = seq["o"][n - 1]        # causal: the last token attends to all n cached ones
    # the naive outputs at position n-1 only see the first n rows; rows past n are ignored
    kv[1, 23:] = 1e6
    got = O.absorbed_decode(q, kv, lengths, s["Wuk"], s["Wuv"], n_heads=H,
                            s_kv_groups=cfg.s_kv_groups, s_rope_groups=Gr, nope_dim=dn,
                            rope_dim=dr, scale=cfg.softmax_scale)
    np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-12)
