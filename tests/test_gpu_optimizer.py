"""GPU parity of the optimizer step (mla_recon_adamw) and of the training loop built on the
single-call step, against the float64 oracles (AdamW as read for Sec. 4.1; Eq. 11 and its
backward)."""
import numpy as np
import pytest

from paper_2607_27269_amd import configs, synth
from parity_util import oracle_step

pytestmark = pytest.mark.gpu


def _bf16_round(x):
    """Round-to-nearest-even to bf16 (values as float64)."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_adamw_kernel_parity(dtype):
    """Three steps on three tensors (sizes with ragged tails) against the oracle."""
    import torch
    import oracle as O
    from paper_2607_27269_amd import _lib as L
    print(f"[optimizer] adamw dtype={dtype}", flush=True)
    rng = np.random.default_rng(5)
    sizes = (1000, 4099, 17)
    # the hyperparameters as the device receives them (fp32), given to both sides
    lr, b1, b2, eps, wd = (float(np.float32(x)) for x in (2e-3, 0.9, 0.999, 1e-8, 0.01))
    dev = torch.device("cuda:0")
    host = []
    for n in sizes:
        w = rng.standard_normal(n) * 0.05
        if dtype == "bf16":
            w = _bf16_round(w)
        host.append(dict(w=w, m=np.zeros(n), v=np.zeros(n)))
    tens = []
    for h in host:
        master = torch.tensor(h["w"], dtype=torch.float32, device=dev)
        wt = master.to(torch.bfloat16 if dtype == "bf16" else torch.float32).clone()
        tens.append(dict(master=master, m=torch.zeros_like(master), v=torch.zeros_like(master),
                         w=wt, g=torch.empty_like(master)))
    for step in (1, 2, 3):
        for h, t in zip(host, tens):
            g = (rng.standard_normal(len(h["w"])) * 1e-3).astype(np.float32)
            t["g"].copy_(torch.from_numpy(g))
            h["w"], h["m"], h["v"] = O.adamw_step(h["w"], g.astype(np.float64), h["m"], h["v"],
                                                  step, lr, b1, b2, eps, wd)
        L.mla_recon_adamw([L.AdamwTensor(t["master"].data_ptr(), t["m"].data_ptr(),
                                         t["v"].data_ptr(), t["w"].data_ptr(), t["g"].data_ptr(),
                                         t["master"].numel()) for t in tens],
                          L.MLA_FP32 if dtype == "fp32" else L.MLA_BF16, step, lr, b1, b2, eps,
                          wd, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        for h, t in zip(host, tens):
            master = t["master"].double().cpu().numpy()
            # fp32 arithmetic against fp64: a few units of fp32 rounding, relative to each
            # array's scale (the moment updates can cancel)
            for got, ref in ((master, h["w"]), (t["m"].double().cpu().numpy(), h["m"]),
                             (t["v"].double().cpu().numpy(), h["v"])):
                np.testing.assert_allclose(got, ref, rtol=2e-6, atol=2e-6 * np.abs(ref).max())
            # the stored weight is the kernel's master, rounded (bit-exact)
            want = _bf16_round(master) if dtype == "bf16" else master
            assert np.array_equal(t["w"].double().cpu().numpy(), want)


def _oracle_train(wl, steps, lr, adamw, schedule=None):
    """The oracle loop: Eq. 11 step, then AdamW on fp64 masters; the forward uses the
    weights in storage precision (bf16-rounded masters), as the device loop does.  With a
    schedule, step t runs on the hidden states schedule[t] (all tokens valid)."""
    import oracle as O
    names = ("Wdq", "Wuq", "Wdkv_kr", "Wuk", "Wuv")
    gnames = {"Wdq": "dWdq", "Wuq": "dWuq", "Wdkv_kr": "dWdkv_kr", "Wuk": "dWuk", "Wuv": "dWuv"}
    master = {n: np.asarray(getattr(wl, n), dtype=np.float64).copy() for n in names
              if getattr(wl, n) is not None}
    mom = {n: (np.zeros_like(w), np.zeros_like(w)) for n, w in master.items()}
    losses = []
    for t in range(1, steps + 1):
        for n, w in master.items():
            setattr(wl, n, _bf16_round(w) if wl.cfg.dtype == "bf16" else w)
        if schedule is not None:
            wl.h = schedule[t - 1]
            wl.mask = np.ones(wl.h.shape[:2], dtype=np.uint8)
        ref = oracle_step(wl)
        losses.append(ref["loss"])
        for n in master:
            master[n], m, v = O.adamw_step(master[n], ref[gnames[n]], *mom[n], t, lr, **adamw)
            mom[n] = (m, v)
    return np.array(losses)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_training_loop_parity(dtype):
    """Four steps of the device loop (single-call step + AdamW) against the oracle loop."""
    from paper_2607_27269_amd.step import DeviceStep
    print(f"[optimizer] loop dtype={dtype}", flush=True)
    cfg = configs.shrink(configs.get(1), batch=2, seq=96).replace(dtype=dtype)
    f32 = lambda x: float(np.float32(x))
    lr, adamw = f32(1e-3), dict(beta1=f32(0.9), beta2=f32(0.999), eps=f32(1e-8), weight_decay=0.0)
    dev = DeviceStep(synth.make_workload(cfg, lengths=[96, 70]))
    got = dev.train(4, lr, **adamw).numpy().astype(np.float64)
    want = _oracle_train(synth.make_workload(cfg, lengths=[96, 70]), 4, lr, adamw)
    print(f"[optimizer] losses device {got} oracle {want}", flush=True)
    # first step: the single-call step's own bound; later steps add the drift of
    # storage-precision weights (fp32 check mode: fp32 rounding only)
    tol = 1e-3 if dtype == "bf16" else 1e-5
    assert abs(got[0] - want[0]) <= tol * want[0]
    assert np.all(np.abs(got - want) <= 10 * tol * want)
    assert got[-1] < got[0]


def test_training_reduces_loss():
    """Twenty AdamW steps on one minibatch lower Eq. 11 (the method's purpose)."""
    from paper_2607_27269_amd.step import DeviceStep
    print("[optimizer] loss decrease", flush=True)
    cfg = configs.shrink(configs.get(1), batch=2, seq=256)
    dev = DeviceStep(synth.make_workload(cfg))
    losses = dev.train(20, 1e-3).numpy()
    print(f"[optimizer] losses {losses}", flush=True)
    assert np.all(np.isfinite(losses))
    assert losses[-1] < 0.7 * losses[0]


@pytest.mark.parametrize("dtype,per", [("fp32", 1), ("bf16", 2)])
def test_minibatch_loop_parity(dtype, per):
    """E_b of Eq. 11 over four calibration minibatches: the teacher output cached once per
    minibatch, `per` student steps on it, AdamW after each; the device losses follow the
    oracle loop on the same schedule (two epochs)."""
    from paper_2607_27269_amd.step import DeviceStep
    print(f"[optimizer] minibatch loop dtype={dtype} steps per minibatch={per}", flush=True)
    cfg = configs.shrink(configs.get(1), batch=2, seq=64).replace(dtype=dtype)
    f32 = lambda x: float(np.float32(x))
    lr, adamw = f32(1e-3), dict(beta1=f32(0.9), beta2=f32(0.999), eps=f32(1e-8), weight_decay=0.0)
    wl = synth.make_workload(cfg)
    hs = [wl.h] + synth.calibration_minibatches(cfg, 3, seed=500)
    dev = DeviceStep(wl)
    tb = [dev.upload(h) for h in hs]
    got = dev.train_minibatches(tb, 2, lr, steps_per_minibatch=per, **adamw).numpy().astype(np.float64)
    schedule = [h for _ in range(2) for h in hs for _ in range(per)]
    want = _oracle_train(synth.make_workload(cfg), len(schedule), lr, adamw, schedule=schedule)
    print(f"[optimizer] losses device {got} oracle {want}", flush=True)
    tol = 1e-3 if dtype == "bf16" else 1e-5
    assert abs(got[0] - want[0]) <= tol * want[0]
    assert np.all(np.abs(got - want) <= 10 * tol * want)
    # the minibatches differ: so do their losses at the first pass
    assert len({round(float(x), 7) for x in got[: 4 * per: per]}) == 4


def test_minibatch_training_lowers_heldout_loss():
    """Training over four calibration minibatches lowers Eq. 11 on a fifth, held-out one."""
    from paper_2607_27269_amd.step import DeviceStep
    print("[optimizer] held-out loss", flush=True)
    cfg = configs.shrink(configs.get(1), batch=2, seq=256)
    wl = synth.make_workload(cfg)
    dev = DeviceStep(wl)
    train = [dev.upload(h) for h in [wl.h] + synth.calibration_minibatches(cfg, 3, seed=600)]
    held = dev.upload(synth.calibration_minibatches(cfg, 1, seed=700)[0])
    before = dev.eval_loss(held)
    losses = dev.train_minibatches(train, 5, 1e-3).numpy()
    after = dev.eval_loss(held)
    print(f"[optimizer] held-out loss {before:.4e} -> {after:.4e}; train {losses[0]:.4e} -> {losses[-1]:.4e}",
          flush=True)
    assert np.all(np.isfinite(losses)) and np.isfinite(after)
    assert after < 0.8 * before
