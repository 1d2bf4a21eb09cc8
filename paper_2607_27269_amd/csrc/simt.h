// fp32 check-mode (vector-ALU) kernels; see simt.hip.
#pragma once
#include "kernels.h"

namespace mla {
hipError_t gemm_simt(const Gemm& g, hipStream_t s);
bool attn_simt_supported(int dqk, int dv);
hipError_t attn_fwd_simt(const Attn& a, hipStream_t s);
hipError_t attn_bwd_simt(const AttnBwd& w, hipStream_t s);
hipError_t attn_delta(const AttnBwd& w, hipStream_t s);
}  // namespace mla
