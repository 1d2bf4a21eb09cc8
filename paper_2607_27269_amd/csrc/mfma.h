// bf16 matrix-core (MFMA) kernels for gfx950 (gemm_mfma.hip, attn_fwd.hip, attn_bwd.hip).
#pragma once
#include "kernels.h"

namespace mla {
size_t gemm_mfma_scratch_elems(const Gemm& g);
// Timed as class kc with the given algorithmic FLOPs / bytes (the split-K sum, if any, as
// an elementwise launch of its own).
hipError_t gemm_mfma(const Gemm& g, float* scratch, size_t scratch_elems, hipStream_t s, int kc,
                     double flops, double bytes);
// C = scale[0] mask[m] X[m, n] with X = A B^T (mask null = all rows) and part[t] = the sum
// over output tile t of mask[m] X[m, n]^2, or of mask[m] X[m, n] ref[m, n] (bf16, row
// stride ldref) when ref is given, in a fixed order; *nparts = the number of tiles (at most
// gemm_mfma_masked_sse_parts).  Both operands K-contiguous, no split-K.
size_t gemm_mfma_masked_sse_parts(const Gemm& g);
hipError_t gemm_mfma_masked_sse(const Gemm& g, const float* scale, const uint8_t* mask,
                                const void* ref, int64_t ldref, double* part, int* nparts,
                                hipStream_t s, const char** kernel);
// C = scale[0] X[m, n] on rows with mask[m] != 0 (mask null = all rows) and 0 on the other
// rows, X = A B^T (bf16 operands, both K-contiguous): the four-wavefront product with that
// epilogue where it applies, else the masked-loss kernel (its tile sums go to part, at
// least gemm_mfma_masked_sse_parts(g) values, and are not used).
hipError_t gemm_mfma_masked_scale(const Gemm& g, const float* scale, const uint8_t* mask,
                                  double* part, hipStream_t s, const char** kernel);
// Batch entry z of a batched causal GEMM uses A + z sA, B + (z / zdiv) sB1 +
// ((z % zdiv) / bdiv) sB2 and C + (z / zdiv) sC1 + (z % zdiv) sC2 (elements).  Row m of C
// sums k < min(K, end of m's 256-row tile) (rev = 0; A M-contiguous, bf16 C) or
// k >= start of m's tile (rev = 1; A K-contiguous, fp32 C), so A must hold zeros for the
// excluded side of the diagonal inside a tile; that K range is summed kgroups times, the
// j-th on A + j sAk and B + j sBk.  B is N-contiguous; rows m >= mstore are not written.
// A (a dS^T plane, key r x query c) is stored in 32 x 32 tiles: element (r, c) at
// ((r / 32) (lda / 32) + c / 32) 1024 + (r % 32) 32 + c % 32, lda a multiple of 32 (r is
// the K index for rev = 0 and the M index for rev = 1).
struct GemmBatch {
  int nbatch, zdiv, bdiv, mstore, rev, kgroups;
  int64_t sA, sB1, sB2, sC1, sC2, sAk, sBk;
  // k-major A only: columns n < split_n go to c_lo in bf16 (row stride ldc_lo, batch
  // strides sC1_lo, sC2_lo), the others to C in fp32 at column n - split_n (0: plain C)
  int split_n = 0;
  void* c_lo = nullptr;
  int64_t ldc_lo = 0, sC1_lo = 0, sC2_lo = 0;
};
hipError_t gemm_mfma_causal(const Gemm& g, const GemmBatch& bt, hipStream_t s);
bool attn_mfma_supported(int dqk, int dv);
hipError_t attn_fwd_mfma(const Attn& a, hipStream_t s, const char** kernel);
hipError_t attn_bwd_mfma(const AttnBwd& w, hipStream_t s);
}  // namespace mla
