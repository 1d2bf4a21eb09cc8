"""Pins of the calibration-capture oracle (the stand-in for Sec. 4.1's cached layer inputs
of the frozen model): RMS normalisation by its defining property, and the residual stack
by the cases that reduce it to something known."""
import numpy as np

import oracle as O
from paper_2607_27269_amd import configs, synth


def test_rms_norm_unit_rms_and_direction():
    x = np.random.default_rng(0).standard_normal((7, 96)) * 3.0
    h = O.rms_norm(x, eps=0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(h * h, axis=-1)), 1.0, rtol=1e-12)
    # same direction: h is a positive multiple of x in every row
    cos = np.sum(h * x, -1) / (np.linalg.norm(h, axis=-1) * np.linalg.norm(x, axis=-1))
    np.testing.assert_allclose(cos, 1.0, rtol=1e-12)
    # eps enters under the root: a zero row stays zero
    assert not O.rms_norm(np.zeros((1, 8)), eps=1e-6).any()


def _layers(cfg, n, zero_wo=False):
    out = []
    for l in range(n):
        wl = synth.make_workload(cfg, seed=100 + l, dtype="fp64")
        out.append(dict(Wq=wl.Wq, Wk=wl.Wk, Wv=wl.Wv, Wo=0 * wl.Wo if zero_wo else wl.Wo,
                        inv_freq=wl.inv_freq_t))
    return out, synth.make_workload(cfg, seed=99, dtype="fp64").h


def test_capture_with_silent_blocks_repeats_the_first_input():
    # W_O = 0: every block adds nothing, so every layer sees rms_norm(x^0)
    cfg = configs.shrink(configs.get(1), batch=1, seq=16)
    layers, x0 = _layers(cfg, 3, zero_wo=True)
    hs = O.capture(x0, layers, cfg.n_heads, cfg.n_kv_groups, cfg.softmax_scale)
    for h in hs:
        np.testing.assert_allclose(h, O.rms_norm(x0), rtol=1e-13, atol=1e-15)


def test_capture_first_two_layers_by_hand():
    # h^0 = rms(x^0); h^1 = rms(x^0 + A^0(h^0)), with A^0 the frozen block itself
    cfg = configs.shrink(configs.get(1), batch=1, seq=16)
    layers, x0 = _layers(cfg, 2)
    hs = O.capture(x0, layers, cfg.n_heads, cfg.n_kv_groups, cfg.softmax_scale)
    w = layers[0]
    a0 = O.teacher_forward(O.rms_norm(x0), w["Wq"], w["Wk"], w["Wv"], w["Wo"], w["inv_freq"],
                           cfg.n_heads, cfg.n_kv_groups, cfg.softmax_scale)
    np.testing.assert_allclose(hs[1], O.rms_norm(x0 + a0), rtol=1e-12, atol=1e-14)
