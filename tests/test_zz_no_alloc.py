"""The allocation-free decoding entry point (mla_recon_decode_noalloc) against the one that
takes a workspace (mla_recon_decode), through the C ABI: two calls in a row on the same
GPU, the second with a smaller batch and cache (so it runs on the scratch the first call
left behind), each compared bitwise with mla_recon_decode on the same inputs; a batch whose
scratch exceeds the static buffer is rejected without launching anything."""
import numpy as np
import pytest

from paper_2607_27269_amd import configs

pytestmark = pytest.mark.gpu


def _inputs(cfg, B, T, lengths, seed):
    import torch
    H, dn, dr, rkv, dv, G = (cfg.n_heads, cfg.nope_dim, cfg.rope_dim, cfg.kv_rank, cfg.head_dim,
                             cfg.s_kv_groups)
    g = torch.Generator(device="cuda").manual_seed(seed)
    bf = torch.bfloat16
    q = (torch.randn(B, H, dn + dr, device="cuda", generator=g) * 0.5).to(bf)
    kv = torch.randn(B, T, rkv + dr, device="cuda", generator=g).to(bf)
    wuk = (torch.randn(G * dn, rkv, device="cuda", generator=g) / dn ** 0.5).to(bf)
    wuv = (torch.randn(G * dv, rkv, device="cuda", generator=g) / rkv ** 0.5).to(bf)
    lens = torch.tensor(lengths, dtype=torch.int32, device="cuda")
    return q, kv, wuk, wuv, lens


def _both(cfg, B, T, lengths, seed):
    import torch
    from paper_2607_27269_amd import _lib as L
    c = L.make_cfg(cfg.replace(batch=B, seq=T))
    q, kv, wuk, wuv, lens = _inputs(cfg, B, T, lengths, seed)
    H, dv = cfg.n_heads, cfg.head_dim
    stream = torch.cuda.current_stream().cuda_stream
    wsb = L.mla_recon_decode_workspace_size(c, T)
    assert 0 < wsb <= L.MLA_DECODE_NOALLOC_SCRATCH_BYTES, (wsb, L.last_error())
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    ref = torch.full((B, H, dv), float("nan"), dtype=torch.bfloat16, device="cuda")
    L.mla_recon_decode(c, q.data_ptr(), kv.data_ptr(), T, lens.data_ptr(), wuk.data_ptr(),
                       wuv.data_ptr(), ref.data_ptr(), ws.data_ptr(), wsb, stream)
    got = torch.full((B, H, dv), float("nan"), dtype=torch.bfloat16, device="cuda")
    L.mla_recon_decode_noalloc(c, q.data_ptr(), kv.data_ptr(), T, lens.data_ptr(),
                               wuk.data_ptr(), wuv.data_ptr(), got.data_ptr(), stream)
    torch.cuda.synchronize()
    return ref, got


def test_decode_noalloc_matches_decode():
    import torch
    cfg = configs.get(3)
    # first call: the benchmark's decoding shape, ragged lengths (chunks left empty)
    B1, T1 = 64, 4096
    l1 = [T1] * B1
    l1[5], l1[20], l1[33], l1[63] = 1, 1000, T1 - 1, 0
    print(f"[noalloc] call 1: B={B1} T={T1}", flush=True)
    ref, got = _both(cfg, B1, T1, l1, seed=11)
    assert torch.isfinite(got.float()).all()
    assert torch.equal(ref, got)
    # second call, smaller: fewer sequences, shorter cache, on the scratch call 1 left
    B2, T2 = 6, 333
    l2 = [333, 1, 0, 200, 32, 331]
    print(f"[noalloc] call 2: B={B2} T={T2}", flush=True)
    ref, got = _both(cfg, B2, T2, l2, seed=12)
    assert torch.equal(ref, got)
    assert not got[2].float().any()  # empty cache: zero output


def test_decode_noalloc_rejects_large_batch():
    import torch
    from paper_2607_27269_amd import _lib as L
    cfg = configs.get(3)
    B, T = 512, 4096
    c = L.make_cfg(cfg.replace(batch=B, seq=T))
    assert L.mla_recon_decode_workspace_size(c, T) > L.MLA_DECODE_NOALLOC_SCRATCH_BYTES
    o = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(L.MlaError) as e:
        L.mla_recon_decode_noalloc(c, o.data_ptr(), o.data_ptr(), T, o.data_ptr(), o.data_ptr(),
                                   o.data_ptr(), o.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert e.value.code == L.MLA_ERR_UNSUPPORTED
