"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Inputs are seeded synthetic workloads (paper_2607_27269_amd.synth) shaped like the five
layer configurations, shortened to sizes the oracle finishes in seconds while still
spanning several attention/GEMM tiles and a ragged tail.  Right-padding masks exercise
Eq. 11's M.  Tolerances: 2e-2 relative (Frobenius) for bf16 outputs and gradients, 1e-5
in the fp32 check mode, 1e-3 relative on the loss.
"""
import sys

import numpy as np
import pytest

from paper_2607_27269_amd import configs, synth
from parity_util import LOSS_TOL, TOL, compare, oracle_step, rel_err

pytestmark = pytest.mark.gpu

GRADS = ("dWdq", "dWuq", "dWdkv_kr", "dWuk", "dWuv")

CASES = {
    # name: (config index, batch, seq, valid lengths or None)
    "cfg0_full_fp32": (0, 2, 64, None),
    "cfg0_ragged_fp32": (0, 2, 77, [77, 40]),
    "cfg0_bf16": (0, 2, 64, None),
    "cfg1_ragged": (1, 2, 200, [200, 131]),
    "cfg2_short": (2, 1, 192, None),
    "cfg3_short": (3, 1, 136, [100]),
    "cfg4_short": (4, 1, 130, None),
    # more than one 256-key block of the dV / dS^T kernel, ragged last block
    "cfg1_long": (1, 2, 300, [300, 263]),
    "cfg3_long": (3, 1, 520, [517]),
    # token counts that are whole 256-row tiles: the projections and W_O products run on the
    # four-wavefront NT kernel (its persistent walk, the masked dO epilogue)
    "cfg3_tiles": (3, 1, 512, [400]),
    "cfg2_tiles": (2, 2, 256, [256, 180]),
}


def make_case(name):
    idx, B, T, lengths = CASES[name]
    cfg = configs.shrink(configs.get(idx), batch=B, seq=T)
    if name == "cfg0_bf16":
        cfg = cfg.replace(dtype="bf16")
    return cfg, synth.make_workload(cfg, lengths=lengths)


@pytest.mark.parametrize("name", list(CASES))
def test_step_parity(name):
    from paper_2607_27269_amd.step import DeviceStep
    print(f"[parity] case={name}", flush=True)
    cfg, wl = make_case(name)
    ref = oracle_step(wl)
    dev = DeviceStep(wl)
    dev.step()
    out = dev.results()
    tol = TOL[cfg.dtype]
    errs = compare(out, ref, ("A_t", "A_s") + GRADS, tol, label=f"{name}: ", cfg=cfg)
    assert abs(out["loss"] - ref["loss"]) <= LOSS_TOL * abs(ref["loss"]), (out["loss"], ref["loss"])
    assert abs(out["rel"] - ref["rel"]) <= LOSS_TOL * abs(ref["rel"]), (out["rel"], ref["rel"])
    print(f"[parity] {name} loss={out['loss']:.6e} ref={ref['loss']:.6e} errs={errs}", flush=True)


FUSED_CASES = ("cfg0_ragged_fp32", "cfg0_bf16", "cfg1_ragged", "cfg3_short", "cfg4_short",
               "cfg1_long", "cfg3_long", "cfg3_tiles", "cfg2_tiles")


@pytest.mark.parametrize("with_dA", [True, False])
@pytest.mark.parametrize("name", FUSED_CASES)
def test_fused_step_parity(name, with_dA):
    """mla_recon_step (W_O applied to o_s - o_t; without dA through W_O^T W_O) against the
    oracle's separate post-W_O outputs: the loss, dL/dA_s and the weight gradients."""
    import math
    from paper_2607_27269_amd.step import DeviceStep
    print(f"[parity] fused case={name} with_dA={with_dA}", flush=True)
    cfg, wl = make_case(name)
    ref = oracle_step(wl)
    dev = DeviceStep(wl)
    dev.fused_step(with_dA)
    out = dev.results()
    tol = TOL[cfg.dtype]
    errs = compare(out, ref, (("dA",) if with_dA else ()) + GRADS, tol, label=f"fused {name}: ", cfg=cfg)
    assert abs(out["loss"] - ref["loss"]) <= LOSS_TOL * abs(ref["loss"]), (out["loss"], ref["loss"])
    assert math.isnan(out["rel"])
    # the relative error on request (one more product over the teacher output in ws)
    dev.rel_error()
    rel = dev.loss_buf.double().cpu().numpy()
    assert rel[0] == np.float32(out["loss"])
    assert abs(rel[1] - ref["rel"]) <= LOSS_TOL * abs(ref["rel"]), (rel[1], ref["rel"])
    # the separate path on the same device state gives the same loss
    dev.step()
    again = dev.results()
    assert abs(again["loss"] - out["loss"]) <= LOSS_TOL * abs(ref["loss"])
    print(f"[parity] fused {name} loss={out['loss']:.6e} ref={ref['loss']:.6e} errs={errs}",
          flush=True)


@pytest.mark.parametrize("name", ("cfg0_ragged_fp32", "cfg1_ragged", "cfg3_short"))
def test_cached_teacher_parity(name):
    """mla_recon_teacher_cache once, then mla_recon_student_step twice (without, then with
    dA): both match the oracle, and the two steps give bitwise equal gradients."""
    import torch
    from paper_2607_27269_amd.step import DeviceStep
    print(f"[parity] cached teacher case={name}", flush=True)
    cfg, wl = make_case(name)
    ref = oracle_step(wl)
    dev = DeviceStep(wl)
    dev.teacher_cache()
    dev.student_step(with_dA=False)
    first = dev.results()
    dev.student_step(with_dA=True)
    second = dev.results()
    tol = TOL[cfg.dtype]
    dev.rel_error()
    rel = float(dev.loss_buf[1].cpu())
    assert abs(rel - ref["rel"]) <= LOSS_TOL * abs(ref["rel"]), (rel, ref["rel"])
    for out, names in ((first, GRADS), (second, ("dA",) + GRADS)):
        compare(out, ref, names, tol, label=f"cached {name}: ", cfg=cfg)
        assert abs(out["loss"] - ref["loss"]) <= LOSS_TOL * abs(ref["loss"]), (out["loss"], ref["loss"])
    if cfg.dtype == "fp32":
        for n in GRADS:
            if n in first:
                assert np.array_equal(first[n], second[n]), n
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_loss_kernel_parity(dtype):
    """Eq. 11 kernel alone on seeded A_s, A_t with a ragged mask (oracle in fp64)."""
    import torch
    from paper_2607_27269_amd.step import DeviceStep
    import oracle as O
    cfg = configs.shrink(configs.get(1), batch=3, seq=333).replace(dtype=dtype)
    wl = synth.make_workload(cfg, lengths=[333, 200, 0])
    dev = DeviceStep(wl)
    As, At = synth.random_outputs(cfg, seed=11, dtype="fp32")
    tA_s = dev.upload(As.reshape(-1, cfg.hidden), "fp32")
    tA_t = dev.upload(At.reshape(-1, cfg.hidden), "fp32")
    dev.loss(tA_s, tA_t)
    torch.cuda.synchronize()
    L, rel, dA = O.recon_loss(As, At, wl.mask)
    got = dev.loss_buf.double().cpu().numpy()
    assert abs(got[0] - L) <= 1e-6 * L and abs(got[1] - rel) <= 1e-6 * rel
    gdA = dev.dA.double().cpu().numpy().reshape(dA.shape)
    assert rel_err(gdA, dA) <= (4e-3 if dtype == "bf16" else 1e-6)
    assert not gdA[2].any() and not gdA[1, 200:].any()        # masked rows: zero gradient
    # the same inputs twice: bitwise identical (fixed reduction order)
    first = dev.loss_buf.clone()
    dev.loss(tA_s, tA_t)
    torch.cuda.synchronize()
    assert torch.equal(first, dev.loss_buf)
    # all-invalid mask
    dev.mask.zero_()
    dev.loss(tA_s, tA_t)
    torch.cuda.synchronize()
    assert float(dev.loss_buf[0]) == 0.0 and not dev.dA.any()


@pytest.mark.parametrize("name", ("cfg1_ragged", "cfg3_long"))
def test_chunked_backward_parity(name):
    """The smallest workspace (one sequence per pass of the backward's attention) gives the
    oracle's gradients, and the same as the preferred workspace up to rounding order."""
    from paper_2607_27269_amd import _lib as L
    from paper_2607_27269_amd.step import DeviceStep
    cfg, wl = make_case(name)
    if cfg.batch < 2:
        cfg = cfg.replace(batch=3)
        wl = synth.make_workload(cfg, lengths=[cfg.seq, cfg.seq - 3, 100])
    print(f"[parity] chunked backward case={name} B={cfg.batch}", flush=True)
    ref = oracle_step(wl)
    ws_min = L.mla_recon_workspace_size_min(L.make_cfg(cfg))
    assert ws_min < L.mla_recon_workspace_size(L.make_cfg(cfg))
    dev = DeviceStep(wl, ws_bytes=ws_min)
    for with_dA in (False, True):
        dev.fused_step(with_dA)
        out = dev.results()
        assert abs(out["loss"] - ref["loss"]) <= LOSS_TOL * abs(ref["loss"]), (out["loss"], ref["loss"])
        compare(out, ref, (("dA",) if with_dA else ()) + GRADS, TOL[cfg.dtype],
                label=f"chunked {name}: ", cfg=cfg)
    dev.step()
    out = dev.results()
    compare(out, ref, ("A_t", "A_s") + GRADS, TOL[cfg.dtype], label=f"chunked four-call {name}: ",
            cfg=cfg)
