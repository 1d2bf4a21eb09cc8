// Kernel selection: bf16 storage runs the MFMA kernels, fp32 (check mode) the vector-ALU
// kernels.  Also owns the per-launch FLOP/byte accounting of the instrumentation.
#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "mfma.h"
#include "simt.h"

namespace mla {

size_t gemm_scratch_elems(const Gemm& g) {
  return g.in_t == DT_BF16 ? gemm_mfma_scratch_elems(g) : 0;
}

hipError_t gemm(const Gemm& g, float* scratch, size_t scratch_elems, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  double flops = 2.0 * g.M * g.N * (double)g.K;
  double bytes = ((double)g.M * g.K + (double)g.N * g.K) * dsize(g.in_t) +
                 (double)g.M * g.N * dsize(g.c_t) * (g.beta != 0.f ? 2.0 : 1.0);
  const int kc = g.a_kmajor ? (g.b_kmajor ? KC_GEMM_NT : KC_GEMM_NN) : KC_GEMM_TN;
  // the matrix-core path brackets its product and its split-K sum separately
  if (g.in_t == DT_BF16) return gemm_mfma(g, scratch, scratch_elems, s, kc, flops, bytes);
  prof_begin(kc, s);
  hipError_t e = gemm_simt(g, s);
  prof_end(kc, s, flops, bytes, KLABEL("gemm_simt_kernel"));
  return e;
}

size_t gemm_masked_sse_parts(const Gemm& g) { return gemm_mfma_masked_sse_parts(g); }

hipError_t gemm_masked_sse(const Gemm& g, const float* scale, const uint8_t* mask,
                           const void* ref, int64_t ldref, double* part, int* nparts,
                           hipStream_t s) {
  double flops = 2.0 * g.M * g.N * (double)g.K;
  double bytes = ((double)g.M * g.K + (double)g.N * g.K) * dsize(g.in_t) +
                 (double)g.M * g.N * dsize(g.c_t) * ((ref ? 1.0 : 0.0) + (g.C ? 1.0 : 0.0)) +
                 (mask ? (double)g.M : 0.0);
  prof_begin(KC_GEMM_NT, s);
  const char* kname = nullptr;
  hipError_t e = gemm_mfma_masked_sse(g, scale, mask, ref, ldref, part, nparts, s, &kname);
  prof_end(KC_GEMM_NT, s, flops, bytes, kname);
  return e;
}

hipError_t gemm_masked_scale(const Gemm& g, const float* scale, const uint8_t* mask,
                             double* part, hipStream_t s) {
  double flops = 2.0 * g.M * g.N * (double)g.K;
  double bytes = ((double)g.M * g.K + (double)g.N * g.K) * dsize(g.in_t) +
                 (double)g.M * g.N * dsize(g.c_t) + (mask ? (double)g.M : 0.0);
  prof_begin(KC_GEMM_NT, s);
  const char* kname = nullptr;
  hipError_t e = gemm_mfma_masked_scale(g, scale, mask, part, s, &kname);
  prof_end(KC_GEMM_NT, s, flops, bytes, kname);
  return e;
}

static double causal_pairs(const Attn& a) {
  return (double)a.B * a.H * (double)a.T * (a.T + 1) / 2.0;
}

hipError_t attn_fwd(const Attn& a, hipStream_t s) {
  double flops = 2.0 * causal_pairs(a) * (a.dqk + a.dv);
  double N = (double)a.B * a.T;
  double bytes = N * a.H * (a.dqk + a.dv) * dsize(a.t) + N * a.H * (a.lse ? 4.0 : 0.0);
  if (a.o_diff) bytes += 2.0 * N * a.H * a.dv * dsize(a.t);
  const bool mfma = a.t == DT_BF16 && attn_mfma_supported(a.dqk, a.dv);
  // the query rotation on load exists on the matrix-core path only
  if (a.q_cos && (!mfma || a.q_roff != 0 || 2 * a.q_np != a.dqk || a.dqk % 32))
    return hipErrorInvalidValue;
  prof_begin(KC_ATTN_FWD, s);
  const char* kname = nullptr;
  hipError_t e = mfma ? attn_fwd_mfma(a, s, &kname) : attn_fwd_simt(a, s);
  prof_end(KC_ATTN_FWD, s, flops, bytes, mfma ? kname : KLABEL("attn_fwd_simt_kernel"));
  // the matrix-core kernel writes o_diff itself; the vector-ALU kernels leave it to a pass
  if (e == hipSuccess && a.o_diff && !mfma)
    e = sub_elementwise(a.O, a.o_ref, a.o_diff, (int64_t)N * a.H * a.dv, a.t, s);
  return e;
}

hipError_t attn_bwd(const AttnBwd& w, hipStream_t s) {
  const Attn& a = w.f;
  if (a.t == DT_BF16 && attn_mfma_supported(a.dqk, a.dv)) return attn_bwd_mfma(w, s);
  // vector-ALU path: one bracket for the whole backward
  double flops = 2.0 * causal_pairs(a) * (2.0 * a.dv + 2.0 * a.dqk);
  double N = (double)a.B * a.T;
  double bytes = N * a.H * (a.dqk + 2.0 * a.dv) * dsize(a.t) + N * a.H * (8.0 + 4.0 * a.dqk);
  prof_begin(KC_ATTN_DKDV, s);
  hipError_t e = attn_bwd_simt(w, s);
  prof_end(KC_ATTN_DKDV, s, flops, bytes, KLABEL("attn_dq_simt_kernel + attn_dkv_simt_kernel"));
  return e;
}

double attn_causal_pairs(const Attn& a) { return causal_pairs(a); }

int attn_bwd_chunk_seqs(int B, int H, int T, int dqk, int dv, DType t) {
  if (t != DT_BF16 || !attn_mfma_supported(dqk, dv)) return 0;
  const size_t limit = (size_t)16 << 30;
  const size_t one = attn_ds_bytes(1, H, T);
  if (one > limit) return -1;
  const size_t per = one - attn_ds_bytes(0, H, T);  // without the scratch rows
  const size_t fit = (limit - attn_ds_bytes(0, H, T)) / per;
  return (int)std::min<size_t>((size_t)B, fit);
}

}  // namespace mla
