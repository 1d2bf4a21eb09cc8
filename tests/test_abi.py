"""The C ABI library: symbols, workspace sizing and argument validation (no GPU needed).

Every check here returns before the library touches the GPU: validation happens before
any launch, so these calls are safe on a machine without a device.
"""
import ctypes
import os
import re

import pytest

from paper_2607_27269_amd import _lib as L
from paper_2607_27269_amd import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mla_recon.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH),
                                reason="libmlarecon.so not built (run __graft_entry__.build())")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mla_recon_\w+)\s*\(", text)))


def test_exports_every_declared_function():
    names = header_functions()
    assert {"mla_recon_teacher_fwd", "mla_recon_student_fwd", "mla_recon_loss",
            "mla_recon_bwd", "mla_recon_step", "mla_recon_teacher_cache",
            "mla_recon_student_step", "mla_recon_rel_error", "mla_recon_adamw",
            "mla_recon_residual_rmsnorm",
            "mla_recon_decode", "mla_recon_decode_workspace_size",
            "mla_recon_workspace_size", "mla_recon_workspace_size_min",
            "mla_recon_last_error"} <= set(names)
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_python_binding_names_match_header():
    for n in header_functions():
        assert hasattr(L, n), n


@pytest.mark.parametrize("idx", [0, 1, 2, 3, 4])
def test_workspace_size_positive(idx):
    c = L.make_cfg(configs.get(idx))
    ws = L.mla_recon_workspace_size(c)
    assert ws > 0 and ws % 256 == 0
    # monotone in the number of tokens
    c2 = L.make_cfg(configs.shrink(configs.get(idx), batch=1, seq=64))
    assert L.mla_recon_workspace_size(c2) < ws


@pytest.mark.parametrize("idx", [1, 3, 4])
def test_workspace_chunks(idx):
    """The backward's dS^T buffer holds one chunk of sequences: the minimum workspace has
    room for one sequence's, the preferred one for the whole batch's when that fits 16 GiB,
    else for as many sequences as fit; one sequence beyond 16 GiB is unsupported."""
    cfg = configs.get(idx)
    H, T = cfg.n_heads, cfg.seq
    ld = (T + 63) // 64 * 64
    ds_seq = H * ld * ld * 2    # square planes of 32 x 32 tiles
    pref = L.mla_recon_workspace_size(L.make_cfg(cfg))
    lo = L.mla_recon_workspace_size_min(L.make_cfg(cfg))
    assert 0 < lo < pref
    assert pref - lo >= (cfg.batch - 1) * ds_seq
    # a batch whose dS^T exceeds 16 GiB: the preferred workspace stops at the cap
    nb = 2 * (16 << 30) // ds_seq + 1
    big = cfg.replace(batch=nb)
    assert nb * ds_seq > (16 << 30)
    wbig = L.mla_recon_workspace_size(L.make_cfg(big))
    assert 0 < wbig < L.mla_recon_workspace_size_min(L.make_cfg(big)) + (16 << 30) + (1 << 30)
    # fp32 check mode stores no dS^T: one size
    f32 = L.make_cfg(configs.shrink(cfg, batch=2, seq=64).replace(dtype="fp32"))
    assert L.mla_recon_workspace_size(f32) == L.mla_recon_workspace_size_min(f32) > 0
    # one sequence whose dS^T alone exceeds 16 GiB
    long = L.make_cfg(cfg.replace(batch=1, seq=32768))
    assert L.mla_recon_workspace_size(long) == 0 and L.mla_recon_workspace_size_min(long) == 0


def bad(**kw):
    base = configs.shrink(configs.get(1), batch=1, seq=64)
    return L.make_cfg(base.replace(**kw))


@pytest.mark.parametrize("kw,code", [
    (dict(n_heads=15), L.MLA_ERR_INVALID_ARG),        # H % G != 0
    (dict(rope_dim=36), L.MLA_ERR_INVALID_ARG),       # not a multiple of 8
    (dict(head_dim=60), L.MLA_ERR_INVALID_ARG),
    (dict(batch=0), L.MLA_ERR_INVALID_ARG),
    (dict(q_rank=-8), L.MLA_ERR_INVALID_ARG),
    (dict(s_rope_groups=7, n_heads=14), L.MLA_ERR_UNSUPPORTED),   # G_kv % G_r != 0
])
def test_invalid_configs_rejected(kw, code):
    c = bad(**kw)
    assert L.mla_recon_workspace_size(c) == 0
    w = L.TeacherW(1, 1, 1, 1, 1)
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_teacher_fwd(c, 1, w, 1, 256, 1 << 40, None)
    assert e.value.code == code
    assert L.last_error()


def test_null_pointers_and_small_workspace_rejected():
    cfg = configs.shrink(configs.get(1), batch=1, seq=64)
    c = L.make_cfg(cfg)
    ws = L.mla_recon_workspace_size(c)
    w = L.TeacherW(1, 1, 1, 1, 1)
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_teacher_fwd(c, None, w, 1, 256, ws, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_teacher_fwd(c, 1, w, 1, 256, ws - 1, None)
    assert e.value.code == L.MLA_ERR_WORKSPACE
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_teacher_fwd(c, 1, w, 1, 257, ws, None)     # misaligned
    assert e.value.code == L.MLA_ERR_WORKSPACE
    sw = L.StudentW(None, 1, 1, 1, 1, 1)                           # W_DQ missing, q_rank > 0
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_student_fwd(c, 1, sw, 1, 1, 256, ws, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_loss(c, 1, 1, None, None, None, 256, ws, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG
    g = L.StudentGrads(1, None, None, None, None)
    c0 = L.make_cfg(cfg.replace(q_rank=0))
    with pytest.raises(L.MlaError) as e:   # dW_DQ requested without a W_DQ
        L.mla_recon_bwd(c0, 1, L.StudentW(None, 1, 1, 1, 1, 1), 1, 1, g, 256, 1 << 40, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG


def test_step_arguments_validated():
    cfg = configs.shrink(configs.get(1), batch=1, seq=64)
    c = L.make_cfg(cfg)
    ws = L.mla_recon_workspace_size(c)
    tw = L.TeacherW(1, 1, 1, 1, 1)
    sw = L.StudentW(1, 1, 1, 1, 1, 1)
    g = L.StudentGrads(1, 1, 1, 1, 1)
    for args, code in [
        ((c, 1, tw, sw, None, None, 256, g, 256, ws, None), L.MLA_ERR_INVALID_ARG),   # no loss
        ((L.make_cfg(cfg.replace(q_rank=0)), 1, tw, L.StudentW(None, 1, 1, 1, 1, 1), None, 256,
          None, g, 256, ws, None), L.MLA_ERR_INVALID_ARG),                            # dWdq, no W_DQ
        ((c, 1, tw, sw, None, 256, 264, g, 256, ws, None), L.MLA_ERR_INVALID_ARG),    # dA align
        ((c, 1, L.TeacherW(1, 1, 1, None, 1), sw, None, 256, 256, g, 256, ws, None),
         L.MLA_ERR_INVALID_ARG),                                                      # no W_O
        ((c, 1, tw, sw, None, 256, 256, g, 256, ws - 1, None), L.MLA_ERR_WORKSPACE),
    ]:
        with pytest.raises(L.MlaError) as e:
            L.mla_recon_step(*args)
        assert e.value.code == code, (args, L.last_error())


def test_cached_teacher_arguments_validated():
    cfg = configs.shrink(configs.get(1), batch=1, seq=64)
    c = L.make_cfg(cfg)
    ws = L.mla_recon_workspace_size(c)
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_teacher_cache(c, 1, L.TeacherW(1, 1, 1, None, 1), 256, ws, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_teacher_cache(c, 1, L.TeacherW(1, 1, 1, 1, 1), 256, ws - 1, None)
    assert e.value.code == L.MLA_ERR_WORKSPACE
    sw, g = L.StudentW(1, 1, 1, 1, 1, 1), L.StudentGrads(1, 1, 1, 1, 1)
    with pytest.raises(L.MlaError) as e:                                       # no W_O
        L.mla_recon_student_step(c, 1, sw, None, None, 256, None, g, 256, ws, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG
    with pytest.raises(L.MlaError) as e:                                       # no loss
        L.mla_recon_student_step(c, 1, sw, 1, None, None, None, g, 256, ws, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG
    for args, code in (((c, None, None, 256, 256, ws, None), L.MLA_ERR_INVALID_ARG),  # no W_O
                       ((c, 1, None, None, 256, ws, None), L.MLA_ERR_INVALID_ARG),    # no loss
                       ((c, 1, None, 256, 256, ws - 1, None), L.MLA_ERR_WORKSPACE)):
        with pytest.raises(L.MlaError) as e:
            L.mla_recon_rel_error(*args)
        assert e.value.code == code, args


def test_adamw_arguments_validated():
    ok = L.AdamwTensor(256, 512, 768, 1024, 1280, 100)
    cases = [
        (([ok], L.MLA_BF16, 0, 1e-3, 0.9, 0.999, 1e-8, 0.0), "step 0"),
        (([ok], L.MLA_BF16, 1, 1e-3, 1.0, 0.999, 1e-8, 0.0), "beta1 = 1"),
        (([ok], L.MLA_BF16, 1, 1e-3, 0.9, 0.999, 0.0, 0.0), "eps = 0"),
        (([ok], L.MLA_BF16, 1, -1.0, 0.9, 0.999, 1e-8, 0.0), "negative lr"),
        (([ok], 7, 1, 1e-3, 0.9, 0.999, 1e-8, 0.0), "dtype"),
        (([ok] * 9, L.MLA_BF16, 1, 1e-3, 0.9, 0.999, 1e-8, 0.0), "too many tensors"),
        (([L.AdamwTensor(256, 512, 768, 1024, None, 100)], L.MLA_BF16, 1, 1e-3, 0.9, 0.999,
          1e-8, 0.0), "NULL grad"),
        (([L.AdamwTensor(256, 512, 776, 1024, 1280, 100)], L.MLA_BF16, 1, 1e-3, 0.9, 0.999,
          1e-8, 0.0), "misaligned"),
        (([L.AdamwTensor(256, 512, 768, 1024, 1280, -1)], L.MLA_BF16, 1, 1e-3, 0.9, 0.999,
          1e-8, 0.0), "negative size"),
    ]
    for args, why in cases:
        with pytest.raises(L.MlaError) as e:
            L.mla_recon_adamw(*args, None)
        assert e.value.code == L.MLA_ERR_INVALID_ARG, why


def test_residual_rmsnorm_arguments_validated():
    for args in [(256, None, 512, -1, 64, L.MLA_BF16, 1e-6),      # negative rows
                 (256, None, 512, 4, 0, L.MLA_BF16, 1e-6),        # zero width
                 (256, None, 512, 4, 64, 9, 1e-6),                # dtype
                 (256, None, 512, 4, 64, L.MLA_FP32, -1.0),       # eps
                 (None, None, 512, 4, 64, L.MLA_FP32, 1e-6)]:     # NULL x
        with pytest.raises(L.MlaError) as e:
            L.mla_recon_residual_rmsnorm(*args, None)
        assert e.value.code == L.MLA_ERR_INVALID_ARG


def test_decode_configuration_checked():
    c3 = L.make_cfg(configs.get(3))
    assert L.mla_recon_decode_workspace_size(c3, 4096) > 0
    assert L.mla_recon_decode_workspace_size(c3, 0) == 0                    # no cache
    assert L.mla_recon_decode_workspace_size(L.make_cfg(configs.get(4)), 64) == 0   # G_r = H
    assert L.mla_recon_decode_workspace_size(L.make_cfg(configs.get(0)), 64) == 0   # fp32
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_decode(c3, 256, 256, 64, 256, 256, 256, 256, 256, 1, None)  # small ws
    assert e.value.code == L.MLA_ERR_WORKSPACE
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_decode(c3, None, 256, 64, 256, 256, 256, 256, 256, 1 << 30, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG


def test_prof_class_validation():
    with pytest.raises(L.MlaError):
        L.mla_recon_prof_read(99)


def test_decode_noalloc_rejects_before_any_launch():
    """Validation of the allocation-free decode happens on the host before any HIP call:
    an invalid or oversized call returns its error here, without a GPU."""
    cfg = configs.get(3)
    big = L.make_cfg(cfg.replace(batch=512, seq=4096))
    assert L.mla_recon_decode_workspace_size(big, 4096) > L.MLA_DECODE_NOALLOC_SCRATCH_BYTES
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_decode_noalloc(big, 256, 256, 4096, 256, 256, 256, 256, None)
    assert e.value.code == L.MLA_ERR_UNSUPPORTED and "static buffer" in L.last_error()
    small = L.make_cfg(cfg.replace(batch=4, seq=64))
    with pytest.raises(L.MlaError) as e:  # NULL output
        L.mla_recon_decode_noalloc(small, 256, 256, 64, 256, 256, 256, 0, None)
    assert e.value.code == L.MLA_ERR_INVALID_ARG
    with pytest.raises(L.MlaError) as e:  # two positional keys: not an MQA problem
        L.mla_recon_decode_noalloc(L.make_cfg(configs.get(4).replace(batch=4)), 256, 256, 64, 256,
                                   256, 256, 256, None)
    assert e.value.code == L.MLA_ERR_UNSUPPORTED
