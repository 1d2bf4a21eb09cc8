"""Seeded input generator: shapes, determinism, rounding and the init recipe."""
import numpy as np
import pytest

from paper_2607_27269_amd import configs, synth


def test_bf16_round_to_nearest_even():
    # 1 + 2^-8 is exactly half-way between bf16 neighbours 1 and 1 + 2^-7 -> even (1.0)
    x = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.5, 0.0, 65504.0, 1e-40])
    r = synth.round_to(x, "bf16")
    assert r[0] == 1.0
    assert r[1] == 1.0 + 2 * 2.0 ** -7   # 1 + 3*2^-8 rounds up to the even neighbour
    assert r[2] == -2.5 and r[3] == 0.0
    bits = synth.bf16_bits(np.array([1.0, -2.0, np.nan]))
    assert bits[0] == 0x3F80 and bits[1] == 0xC000 and bits[2] == 0x7FC0


@pytest.mark.parametrize("idx", [0, 1])
def test_shapes_and_determinism(idx):
    cfg = configs.shrink(configs.get(idx), batch=2, seq=16)
    a = synth.make_workload(cfg)
    b = synth.make_workload(cfg)
    for name in ("h", "Wq", "Wk", "Wv", "Wo", "Wuq", "Wdkv_kr", "Wuk", "Wuv"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    D, H, G, dk = cfg.hidden, cfg.n_heads, cfg.n_kv_groups, cfg.head_dim
    assert a.h.shape == (2, 16, D)
    assert a.Wq.shape == (H * dk, D) and a.Wk.shape == (G * dk, D) and a.Wo.shape == (D, H * dk)
    assert a.Wuq.shape == (H * cfg.qk_dim, cfg.q_rank or D)
    assert a.Wdkv_kr.shape == (cfg.kv_out, D)
    assert a.Wuk.shape == (cfg.s_kv_groups * cfg.nope_dim, cfg.kv_rank)
    assert a.Wuv.shape == (cfg.s_kv_groups * cfg.v_dim, cfg.kv_rank)
    assert a.inv_freq_s.shape == (cfg.s_rope_groups, cfg.rope_dim // 2)
    # every token RMS-normalised (before rounding)
    rms = np.sqrt(np.mean(a.h ** 2, axis=-1))
    assert np.allclose(rms, 1.0, atol=2e-2 if cfg.dtype == "bf16" else 1e-6)
    if cfg.dtype == "bf16":
        assert np.array_equal(synth.round_to(a.h, "bf16"), a.h)


def test_mha_partial_rope_selection_is_per_head():
    cfg = configs.shrink(configs.get(4), batch=1, seq=8, hidden=256, n_heads=4, n_kv_groups=4,
                         s_kv_groups=4, s_rope_groups=4, kv_rank=64)
    wl = synth.make_workload(cfg)
    assert wl.kept_pairs.shape == (4, 8)
    for r in range(4):
        assert len(set(wl.kept_pairs[r].tolist())) == 8
        assert np.all(np.diff(wl.kept_pairs[r]) > 0)
        assert np.array_equal(wl.inv_freq_s[r], wl.inv_freq_t[wl.kept_pairs[r]])


def test_right_padding_mask():
    m = synth.right_padding_mask(3, 5, [5, 2, 0])
    assert m.tolist() == [[1] * 5, [1, 1, 0, 0, 0], [0] * 5]


def test_flop_model_matches_llama_8b_total():
    f = configs.get(3).total_flops()
    assert f == pytest.approx(6683.6e9, rel=2e-4)


def test_calibration_minibatches_share_outlier_channels():
    """Further calibration minibatches: new tokens, the base layer's outlier channels."""
    cfg = configs.shrink(configs.get(1), batch=2, seq=32)
    wl = synth.make_workload(cfg, dtype="fp32")
    more = synth.calibration_minibatches(cfg, 2, seed=10, dtype="fp32")
    perm = synth.outlier_permutation(cfg)
    k = cfg.outlier_channels
    assert k > 0
    for h in [wl.h] + more:
        rms = np.sqrt(np.mean(h.reshape(-1, cfg.hidden) ** 2, axis=0))
        assert set(np.argsort(rms)[-k:]) == set(perm[:k])
    assert not np.allclose(more[0], wl.h) and not np.allclose(more[0], more[1])
    again = synth.calibration_minibatches(cfg, 2, seed=10, dtype="fp32")
    assert all(np.array_equal(a, b) for a, b in zip(more, again))
