"""Host-side helpers of bench.py: the mapping from rocprofv3 kernel names to the names the
library's instrumentation records (the agreement check of the profiles relies on it)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_rocprof_label_per_kernel_family():
    import bench
    ns = "void mla::(anonymous namespace)::"
    cases = {
        ns + "gemm_nt4_persist_kernel<256, unsigned short>(mla::(anonymous namespace)::GemmDev)":
            "gemm_nt4_persist_kernel<256,256,NT,bf16>",
        ns + "gemm_nt4_persist_kernel<192, float>(mla::(anonymous namespace)::GemmDev)":
            "gemm_nt4_persist_kernel<256,192,NT,fp32>",
        ns + "gemm_mfma_persist_kernel<256, 256, 2, 4, false, false, float, 64, 2>(GemmDev)":
            "gemm_mfma_persist_kernel<256,256,TN,fp32>",
        ns + "gemm_mfma_persist_kernel<256, 192, 4, 2, true, false, unsigned short, 64, 2>(GemmDev)":
            "gemm_mfma_persist_kernel<256,192,NN,bf16>",
        ns + "gemm_mfma_kernel<256, 256, 2, 4, true, true, unsigned short, 64, 2>(GemmDev)":
            "gemm_mfma_kernel(masked loss)<256,256,NT,bf16>",
        ns + "attn_ds_gemm_kernel<256, 192, 4, 2, false, false, unsigned short, 32, 4>(GemmDev)":
            "attn_ds_gemm_kernel<256,192,dQ,bf16>",
        "void mla::attn::(anonymous namespace)::attn_fwd_persist_kernel<192, 128, true, 4>(mla::attn::AttnDev)":
            "attn_fwd_persist_kernel<192,128,lse>",
        "void mla::attn::(anonymous namespace)::attn_dv_mfma_kernel<192, 128>(mla::attn::BwdDev)":
            "attn_dv_mfma_kernel<192,128>",
        "mla::rope_apply8_kernel(unsigned short*, int, int, int, long, long, int, int, int, float const*, float const*, float)":
            "rope_apply8_kernel",
    }
    for name, want in cases.items():
        assert bench.rocprof_label(name) == want, (name, bench.rocprof_label(name))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr)
