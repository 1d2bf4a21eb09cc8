// Internal launch interface between the C ABI (api.cpp) and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include <mutex>

namespace mla {

enum DType { DT_BF16 = 0, DT_F32 = 1 };
inline size_t dsize(DType t) { return t == DT_BF16 ? 2 : 4; }

// Timing classes: one per kernel family (a GEMM layout, an attention kernel, ...).
enum KClass {
  KC_GEMM_NT = 0,      // C = A B^T, both operands K-contiguous (projections)
  KC_GEMM_NN = 1,      // B N-contiguous (data gradients)
  KC_GEMM_TN = 2,      // both operands M/N-contiguous (weight gradients, split-K)
  KC_ATTN_FWD = 3,     // causal attention forward
  KC_ATTN_DKDV = 4,    // attention backward: dK, dV
  KC_ATTN_DQ = 5,      // attention backward: dQ
  KC_LOSS = 6,         // Eq. 11 loss and gradient
  KC_ELEM = 7,         // RoPE tables / rotation, softmax-backward row term, dk^PE finishing
  KC_ATTN_DK = 8,      // attention backward: dK (GEMM over the stored dS^T)
  KC_COUNT = 9
};

// Timing instrumentation hooks (implemented in api.cpp).  prof_end also records the
// algorithmic FLOPs / bytes of the bracketed launch and the name of its kernel (a string
// that lives as long as the process, e.g. from KLABEL).
void prof_begin(int kclass, hipStream_t s);
void prof_end(int kclass, hipStream_t s, double flops, double bytes, const char* kernel = nullptr);

// A stable name for the kernel of one launch site, formatted once per site (and per
// template instance of the enclosing function).
#define KLABEL(...)                                                                      \
  ([&]() -> const char* {                                                                \
    static char kl_buf_[112];                                                            \
    static std::once_flag kl_once_;                                                      \
    std::call_once(kl_once_, [&] { snprintf(kl_buf_, sizeof(kl_buf_), __VA_ARGS__); });  \
    return kl_buf_;                                                                      \
  }())

// C[m, n] = alpha * sum_k A(m, k) B(n, k) + beta * C[m, n]
//   A(m, k) = A[m*lda + k] if a_kmajor else A[k*lda + m]
//   B(n, k) = B[n*ldb + k] if b_kmajor else B[k*ldb + n]
struct Gemm {
  int M, N, K;
  const void* A; int64_t lda; bool a_kmajor;
  const void* B; int64_t ldb; bool b_kmajor;
  void* C; int64_t ldc;
  DType in_t, c_t;
  float alpha, beta;
  // optional second output: rows m >= m2 are stored at C2 + (m - m2) * ldc instead (bf16
  // operands, beta = 0; the product then always goes through the split-K partials)
  void* C2 = nullptr;
  int m2 = 0;
};
// Scratch (fp32 elements) a GEMM of this shape needs for split-K partials.
size_t gemm_scratch_elems(const Gemm& g);
hipError_t gemm(const Gemm& g, float* scratch, size_t scratch_elems, hipStream_t s);

// Per-head strided view: element (n, i, d) at ptr[n*tok + (i / div)*head + d].
struct HeadView {
  const void* p; int64_t tok; int64_t head; int div;
};

// Causal attention over B sequences of T tokens, H query heads.  The logit width is
// dqk; key dims [0, dnope) come from Ka and [dnope, dqk) from Kb (d = dnope + e reads
// Kb element e).  Q, Ka, Kb, V are already rotated where RoPE applies.
struct Attn {
  int B, T, H, dqk, dnope, dv;
  HeadView Q, Ka, Kb, V;
  void* O; int64_t o_tok;   // O[n*o_tok + i*dv + d]
  float* lse;               // [N, H] (natural-log units) or null in the forward
  float scale;
  DType t;
  // forward only, optional: o_diff = O - o_ref (same layout as O, storage dtype), from the
  // rounded O
  const void* o_ref = nullptr;
  void* o_diff = nullptr;
  // forward only, optional (bf16 matrix-core path): Q is rotated on load as a whole, pairs
  // (p, p + q_np) with q_np = dqk / 2 and fp32 tables [T][q_np] (R_t of the rotate-half
  // convention); q_roff must be 0
  const float* q_cos = nullptr;
  const float* q_sin = nullptr;
  int q_roff = 0, q_np = 0;
};
hipError_t attn_fwd(const Attn& a, hipStream_t s);

struct AttnBwd {
  Attn f;                    // forward operands; f.O and f.lse are inputs here
  const void* dO;            // [N, H*dv], row stride H*dv
  float* delta;              // scratch [N, H]
  float* dq_acc;             // scratch [N, H, dqk] fp32 (vector-ALU path)
  void* dq;                  // out [N, H*dqk]: dQ with the rotary block [dnope, dqk) rotated
  int rdiv;                  //   back by R^T using the tables of rope group i / rdiv
  const float* cos_t;        //   ([G_r][T][(dqk-dnope)/2] fp32)
  const float* sin_t;
  void* dKa; int64_t dka_tok;  // [N, ...]: group g's d_nope grads at dKa[n*dka_tok + g*dnope]
  void* dV;  int64_t dv_tok;   // group g's value grads at dV[n*dv_tok + g*dv]
  float* dkb_part;           // [Gka, N, dqk - dnope] fp32 partial grads of the Kb part per Ka group
  int n_ka_groups;           // number of Ka groups (heads i / f.Ka.div)
  // Matrix-core path: dS^T is stored in bf16 by the dV kernel as B'*H planes of ds_ld x
  // ds_ld in 32 x 32 tiles (ds_ld = T rounded up to 64) for B' = attn_bwd_chunk_seqs
  // sequences at a time;
  // dQ = scale dS K is a batched causal GEMM against the keys gathered as kcat
  // [B' T][n_ka_groups][dqk], and dK = scale dS^T Q a GEMM whose epilogue writes dKa (bf16)
  // and dkb_part (fp32) directly.
  void* dsT;                 // attn_ds_bytes(B', f.H, f.T) bytes
  void* kcat;                // B' T * n_ka_groups * dqk bf16
  float* statT;              // attn_stats_bytes(B', f.H, f.T)
  int chunk_seqs;            // B' (>= 1, at most attn_bwd_chunk_seqs)
  // optional (bf16, dv % 8 == 0): with loss_ref [N, H*dv] (row stride H*dv) set, the delta
  // pass also leaves in loss_part[attn_delta_parts(N * H)] the fixed-order partial sums of
  // dO . loss_ref, one per workgroup
  const void* loss_ref = nullptr;
  double* loss_part = nullptr;
};
int64_t attn_delta_parts(int64_t rows);
// Row stride and size of the stored dS^T of the matrix-core backward.
int64_t attn_ds_ld(int T);
size_t attn_ds_bytes(int B, int H, int T);
int attn_stats_tpad(int T);
size_t attn_stats_bytes(int B, int H, int T);
// Sequences per chunk of the matrix-core backward (whose dS^T buffer holds at most
// 16 GiB): 0 when the backward stores no dS^T (vector-ALU path), -1 when one sequence's
// dS^T alone exceeds the limit (unsupported).
int attn_bwd_chunk_seqs(int B, int H, int T, int dqk, int dv, DType t);
hipError_t attn_bwd(const AttnBwd& a, hipStream_t s);
// (sequence, head, query, key) pairs with key <= query: B H T (T+1) / 2
double attn_causal_pairs(const Attn& a);

// RoPE -------------------------------------------------------------------------------
// cos/sin tables [G][T][npairs] fp32 from inv_freq [G][npairs] fp32 (angles in fp64).
hipError_t rope_tables(const float* inv_freq, int G, int T, int npairs, float* cos_t,
                       float* sin_t, hipStream_t s);
// In-place rotation of x[n*tok + h*head + off + {p, p + npairs}] for heads h < nheads,
// tokens n < N (position n % T), with the tables of group h / div; R^T when inverse.
// npairs must be a multiple of 4.
hipError_t rope_apply(void* x, DType t, int N, int T, int nheads, int64_t tok, int64_t head,
                      int off, int npairs, int div, const float* cos_t, const float* sin_t,
                      hipStream_t s, bool inverse = false);

// Backward finishing ----------------------------------------------------------------------
// dq[n, i, :] = dq_acc with the rotary block [dnope, dqk) rotated back by R^T (tables of
// rope group i / rdiv), written in storage dtype with row stride H*dqk.
hipError_t dq_finish(const float* dq_acc, void* dq, DType t, int N, int T, int H, int dqk,
                     int dnope, int rdiv, const float* cos_t, const float* sin_t, hipStream_t s);
// dk^PE of rope group r = R^T sum of the partials of Ka groups r*per .. r*per+per-1,
// written to out[n*out_tok + r*drope + e] in storage dtype.
hipError_t dkpe_finish(const float* part, void* out, DType t, int64_t out_tok, int N, int T,
                       int Gr, int per, int drope, const float* cos_t, const float* sin_t,
                       hipStream_t s);

// Eq. 11 with the masked squared differences summed per GEMM tile (gemm_masked_sse):
// loss_prepare counts the valid tokens and stores the gradient scale 2 / (D count), which
// loss_scale points to (device fp32); loss_from_parts then writes loss[0] = L from the
// tile sums (fixed order) and loss[1] = NaN.  Both loss paths keep the fp64 sum of squared
// masked differences in the scratch, for loss_rel_from_parts.
hipError_t loss_prepare(const uint8_t* mask, int64_t N, int D, void* scratch, hipStream_t s);
const float* loss_scale(const void* scratch);
hipError_t loss_from_parts(const double* part, int nparts, int D, float* loss,
                           void* scratch, hipStream_t s);
// The relative error of the last loss computed with this scratch: loss[1] = (its sum of
// squared masked differences) / ref, ref = the fixed-order sum of part[i * stride],
// i < nparts (tile sums of M A_t^2).  loss[1] = 0 when nothing is valid or both are 0,
// +inf when only ref is 0.
hipError_t loss_rel_from_parts(const double* part, int nparts, int stride, float* loss,
                               const void* scratch, hipStream_t s);
// fp32 check mode: the same from A_t [N, D] fp32 (masked sum of squares, fixed order).
hipError_t loss_rel_fp32(const float* A_t, const uint8_t* mask, int64_t N, int D, float* loss,
                         void* scratch, hipStream_t s);
// C = scale[0] mask[m] X[m, n] in C's dtype (C may be NULL: not stored), X = A B^T, and
// part[t] = the sum over output
// tile t of mask[m] X[m, n]^2, or of mask[m] X[m, n] ref[m, n] with ref (bf16, row stride
// ldref) given (bf16 operands, both K-contiguous); *nparts tiles, at most
// gemm_masked_sse_parts(g).
size_t gemm_masked_sse_parts(const Gemm& g);
hipError_t gemm_masked_sse(const Gemm& g, const float* scale, const uint8_t* mask,
                           const void* ref, int64_t ldref, double* part, int* nparts,
                           hipStream_t s);
// C = scale[0] X[m, n] on rows with mask[m] != 0 and 0 on the others, X = A B^T (bf16
// operands and C, both operands K-contiguous; no tile sums: part, of
// gemm_masked_sse_parts(g) values, is scratch).
hipError_t gemm_masked_scale(const Gemm& g, const float* scale, const uint8_t* mask,
                             double* part, hipStream_t s);

// AdamW (decoupled weight decay) on up to ADAMW_MAX tensors: fp32 master weights, moments
// and gradient; w (dtype wt) receives the rounded master weights.  16-byte aligned arrays.
constexpr int ADAMW_MAX = 8;
struct AdamwTensor {
  float* master; float* m; float* v; void* w; const float* g; int64_t n;
};
hipError_t adamw_step(const AdamwTensor* t, int count, DType wt, float lr, float beta1,
                      float beta2, float eps, float weight_decay, int step, hipStream_t s);

// Calibration capture: x[n] += A[n] (A may be null), then h[n] = x[n] / sqrt(mean(x[n]^2)
// + eps) in dtype t; N rows of D fp32 values.
hipError_t residual_rmsnorm(float* x, const float* A, void* h, int64_t N, int D, DType t, float eps,
                            hipStream_t s);

// Decoding with the reconstructed block in absorbed form (one query token per sequence,
// single positional key): see decode.hip.
struct Decode {
  int B, H, dn, dr, rkv, dv, hpg;  // hpg = heads per KV group
  const void* q;                   // [B][H][dn + dr] bf16, rope part rotated
  const void* cache;               // [B][Lmax][ldc] bf16: [c^KV | k^PE]
  int Lmax, ldc;
  const int32_t* len;              // [B] device
  const void* Wuk;                 // [G_kv dn][rkv]
  const void* Wuv;                 // [G_kv dv][rkv]
  float scale;
  void* o;                         // [B][H][dv] bf16, or null (no W_UV product)
  void* ws;                        // decode_ws_bytes
  // prefill: B counts query rows, row b is token b % tps of sequence b / tps and attends to
  // that sequence's first b % tps + 1 cache rows (len unused); 0 = decoding
  int tps = 0;
  void* lat_out = nullptr;         // optional [B][H][rkv] bf16: the attention-weighted latent
};
bool decode_supported(int DK, int DVL);
size_t decode_ws_bytes(int B, int H, int DK, int DVL, int Lmax);
// The static scratch of the allocation-free entry point: its size, and its address on the
// current device (looked up once per device).
size_t decode_scratch_bytes();
hipError_t decode_scratch(void** out);
hipError_t decode_attention(const Decode& d, hipStream_t s);

// out = a - b elementwise over n elements of dtype t (fp32 arithmetic)
hipError_t sub_elementwise(const void* a, const void* b, void* out, int64_t n, DType t,
                           hipStream_t s);

// Eq. 11 from dO = 2 M Y / (D sum M) and o_s - o_t: L = sum(dO . (o_s - o_t)) / 2 (the
// fixed-order sum of the nparts partials of the delta pass); loss[1] = NaN, the squared-error
// sum kept for loss_rel_from_parts
hipError_t loss_from_dot(const double* part, int64_t nparts, int D, float* loss, void* scratch,
                         hipStream_t s);

// Loss (Eq. 11) -------------------------------------------------------------------------
// scratch: at least loss_scratch_bytes(); loss[0] = L, loss[1] = relative error.  With
// A_t == nullptr, A_s holds the difference A_s - A_t and loss[1] is NaN.
size_t loss_scratch_bytes();
hipError_t recon_loss(const float* A_s, const float* A_t, const uint8_t* mask, int64_t N, int D,
                      float* loss, void* dA, DType t, void* scratch, hipStream_t s);

}  // namespace mla
