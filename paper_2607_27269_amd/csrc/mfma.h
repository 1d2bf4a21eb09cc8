// bf16 matrix-core (MFMA) kernels for gfx950; see gemm_mfma.hip and attn_mfma.hip.
#pragma once
#include "kernels.h"

namespace mla {
size_t gemm_mfma_scratch_elems(const Gemm& g);
hipError_t gemm_mfma(const Gemm& g, float* scratch, size_t scratch_elems, hipStream_t s);
bool attn_mfma_supported(int dqk, int dv);
hipError_t attn_fwd_mfma(const Attn& a, hipStream_t s);
hipError_t attn_bwd_mfma(const AttnBwd& w, hipStream_t s);
}  // namespace mla
