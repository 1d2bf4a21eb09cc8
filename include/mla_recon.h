/*
 * mla_recon.h -- C ABI of the MI355X (gfx950) end-to-end functional-reconstruction step.
 *
 * The objective of Sec. 4.1 (Eq. 11) of "Beyond KV Reconstruction: Functional
 * Reconstruction for MLA Draft Models in Speculative Decoding": the layer's output after
 * the shared, frozen W_O is computed twice on the same hidden states, once by the
 * original GQA/MHA attention and once by its MLA conversion, and the masked squared
 * difference is minimised over the MLA side's new projections.  One step is four calls,
 * all enqueued on the caller's HIP stream:
 *
 *   mla_recon_teacher_fwd  A_orig = W_O . GQA(h)                       (Eq. 1-4, Sec. 4.1)
 *   mla_recon_student_fwd  A_MLA  = W_O . MLA(h)                       (Eq. 5, Sec. 4)
 *   mla_recon_loss         L = ||M (A_MLA - sg[A_orig])||^2 / (D sum M), dL/dA_MLA (Eq. 11)
 *   mla_recon_bwd          dL/d{W_DQ, W_UQ, [W_DKV; W_KR], W_UK, W_UV}  (Sec. 4: only the
 *                          converter-introduced query and KV projections are trained;
 *                          W_O and the teacher are frozen; h is data)
 *
 * Conventions shared by every call
 *  - Pointers named h, W*, A_*, dA, mask, loss, inv_freq, dW* and ws are DEVICE pointers
 *    owned by the caller; `cfg` and the small structs below are HOST pointers read during
 *    the call only.  The library never allocates or frees memory on these paths and
 *    keeps no state between calls except the thread-local last-error text and the
 *    optional timing instrumentation below.
 *  - Matrices are row-major; a weight W[out, in] maps x -> W x (a row of activations
 *    X[tokens, in] maps to X W^T).  Tokens are flattened as n = b*T + t.
 *  - Storage dtype (cfg->dtype): MLA_BF16 -> h, all weights and dA are bf16 (raw 16-bit
 *    patterns); MLA_FP32 (check mode) -> they are fp32.  A_t, A_s, loss, inv_freq and all
 *    weight gradients are fp32 in both modes.  Arithmetic accumulates in fp32.
 *  - RoPE (Sec. 3.1): rotate-half pairs (p, p + d/2) of a head are rotated by the angle
 *    t * inv_freq[p], t = 0 .. T-1 restarting in every sequence.  Both logits use
 *    cfg->softmax_scale (1/sqrt(d_k) of the teacher, as in Eq. 2 and Eq. 8).
 *  - Causal attention includes the diagonal (Eq. 3, u <= t); sequences never attend to
 *    each other.  The mask M enters only the loss (Eq. 11).
 *  - Every call validates all arguments before enqueueing anything; on error it returns a
 *    negative mla_status, enqueues nothing and sets mla_recon_last_error().  On success it
 *    returns MLA_OK after only enqueueing work (no host synchronisation).
 *  - Workspace: ws is 256-byte aligned and holds at least mla_recon_workspace_size_min(cfg)
 *    bytes; mla_recon_workspace_size(cfg) is the preferred size.  A smaller workspace only
 *    makes the bf16 backward run its attention in more chunks of sequences (the dS^T
 *    buffer at the end of ws holds as many whole sequences as fit, at most 16 GiB of
 *    them); results are the same.  mla_recon_student_fwd stores the activations
 *    mla_recon_bwd needs in ws, so the same ws and ws_bytes, unmodified, must be passed
 *    from student_fwd to bwd.  teacher_fwd and loss only use scratch parts of ws that
 *    student_fwd/bwd do not keep.
 *  - Calls that share one ws (or overlapping outputs) must not run concurrently.
 */
#ifndef MLA_RECON_H
#define MLA_RECON_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MLA_OK = 0,
  MLA_ERR_INVALID_ARG = -1,  /* NULL required pointer, bad dimension or grouping        */
  MLA_ERR_UNSUPPORTED = -2,  /* valid for the method but not for these kernels          */
  MLA_ERR_WORKSPACE = -3,    /* ws too small or misaligned                              */
  MLA_ERR_HIP = -4           /* a HIP runtime call or launch failed                     */
} mla_status;

typedef enum { MLA_BF16 = 0, MLA_FP32 = 1 } mla_dtype;

/* Layer shape.  Teacher (Eq. 1): D = hidden, H query heads, G KV groups (G == H is MHA),
 * head width d_k (keys and values).  Student (Eq. 5 + decoupled RoPE): query latent rank
 * r_q (0 = no query factorisation: q = W_UQ h), KV latent rank r_kv, per-head logit width
 * d_nope + d_rope, value width d_k, G_kv groups of non-positional keys/values and G_r
 * positional keys k^PE (head i uses group i / (H/G_kv) and rope key i / (H/G_r)).
 * Requirements: all sizes >= 1 except q_rank, nope_dim >= 0; H % G == H % G_kv == H % G_r
 * == 0; d_k and d_rope even; hidden, head_dim, q_rank, kv_rank, nope_dim, rope_dim
 * multiples of 8; G_kv a multiple of G_r.  Attention widths: the teacher's (d_k, d_k) and
 * the student's (d_nope + d_rope, d_k) must be one of (64,64), (96,64), (128,64),
 * (128,128), (192,128) (matrix-core kernels) or, through the vector-ALU kernels, (64,32),
 * (32,32), (16,16), (12,8), (8,8); MLA_ERR_UNSUPPORTED otherwise.  Any seq >= 1.  In
 * bf16 the backward stores dS^T (2 bytes per (head, key, query) of a sequence) for as
 * many whole sequences as fit in 16 GiB at a time (the workspace holds one such chunk);
 * a single sequence with n_heads * seq^2 * 2 bytes above 16 GiB is MLA_ERR_UNSUPPORTED. */
typedef struct {
  int32_t batch, seq, hidden;               /* B, T, D                                    */
  int32_t n_heads, n_kv_groups, head_dim;   /* H, G, d_k                                  */
  int32_t q_rank, kv_rank;                  /* r_q (0 allowed), r_kv                      */
  int32_t nope_dim, rope_dim;               /* d_nope (0 allowed), d_rope                 */
  int32_t s_kv_groups, s_rope_groups;       /* G_kv, G_r                                  */
  float softmax_scale;                      /* multiplies both teacher and student logits */
  int32_t dtype;                            /* mla_dtype                                  */
} mla_recon_cfg;

/* Frozen original block.  Wq [H*d_k, D], Wk and Wv [G*d_k, D] (group g owns rows
 * g*d_k .. g*d_k+d_k-1, head i owns rows i*d_k ..), Wo [D, H*d_k].  inv_freq: fp32
 * [d_k/2], the RoPE inverse frequency of each rotate-half pair. */
typedef struct {
  const void *Wq, *Wk, *Wv, *Wo;
  const float *inv_freq;
} mla_teacher_w;

/* Converted MLA block.  Wdq [r_q, D] (NULL iff q_rank == 0); Wuq [H*(d_nope+d_rope),
 * r_q or D], each head's rows ordered non-positional then rotary; Wdkv_kr
 * [r_kv + G_r*d_rope, D] = W^DKV stacked over the positional-key projection W^KR;
 * Wuk [G_kv*d_nope, r_kv]; Wuv [G_kv*d_k, r_kv].  inv_freq: fp32 [G_r, d_rope/2]. */
typedef struct {
  const void *Wdq, *Wuq, *Wdkv_kr, *Wuk, *Wuv;
  const float *inv_freq;
} mla_student_w;

/* Weight gradients, fp32, same shapes as the weights; overwritten, not accumulated.
 * A NULL pointer leaves that projection frozen (its gradient is not computed). */
typedef struct {
  float *dWdq, *dWuq, *dWdkv_kr, *dWuk, *dWuv;
} mla_student_grads;

/* Preferred bytes of workspace for `cfg` (the backward's attention in one pass when its
 * dS^T fits 16 GiB), and the minimum (one sequence per pass); 0 if cfg is invalid. */
size_t mla_recon_workspace_size(const mla_recon_cfg *cfg);
size_t mla_recon_workspace_size_min(const mla_recon_cfg *cfg);

/* Teacher forward (Eq. 1-4 and the frozen W_O, Sec. 4.1).
 * h [B, T, D] (storage dtype); writes A_t [B, T, D] fp32 = the post-W_O attention
 * output of the original block.  Uses only scratch regions of ws. */
int mla_recon_teacher_fwd(const mla_recon_cfg *cfg, const void *h, const mla_teacher_w *w,
                          float *A_t, void *ws, size_t ws_bytes, void *hip_stream);

/* Student forward (Eq. 5; low-rank query; decoupled RoPE; Eq. 2-4; the teacher's W_O).
 * h [B, T, D]; Wo = the teacher's [D, H*d_k] (frozen, shared); writes A_s [B, T, D]
 * fp32 and keeps the activations the backward needs in ws. */
int mla_recon_student_fwd(const mla_recon_cfg *cfg, const void *h, const mla_student_w *w,
                          const void *Wo, float *A_s, void *ws, size_t ws_bytes,
                          void *hip_stream);

/* Eq. 11 on one minibatch (all B*T tokens flattened) and its gradient.
 * A_s, A_t [B, T, D] fp32; mask [B, T] uint8 (nonzero = valid) or NULL = all valid.
 * Writes loss[0] = L = sum(M (A_s - A_t))^2 / (D sum M), loss[1] = the relative error
 * sum(M (A_s - A_t))^2 / sum(M A_t)^2 (device fp32 [2]), and dA [B, T, D] (storage
 * dtype) = 2 M (A_s - A_t) / (D sum M).  An all-invalid mask gives L = 0 and dA = 0.
 * The reduction order is fixed: results are bitwise reproducible.  dA may be NULL
 * (loss only). */
int mla_recon_loss(const mla_recon_cfg *cfg, const float *A_s, const float *A_t,
                   const uint8_t *mask, float *loss, void *dA, void *ws, size_t ws_bytes,
                   void *hip_stream);

/* Backward of L through the student (Sec. 4: stop-gradient on the teacher, W_O frozen,
 * no gradient for h).  dA [B, T, D] (storage dtype) is dL/dA_s, e.g. from
 * mla_recon_loss; h, w and Wo must be the ones given to the preceding student_fwd, and
 * ws must still hold what it stored.  Writes the requested gradients (fp32). */
int mla_recon_bwd(const mla_recon_cfg *cfg, const void *h, const mla_student_w *w,
                  const void *Wo, const void *dA, const mla_student_grads *grads, void *ws,
                  size_t ws_bytes, void *hip_stream);

/* One whole reconstruction step: teacher forward, student forward, Eq. 11 and the
 * backward, as the four calls above make it, with one difference: A_t and A_s are not
 * formed.  Both blocks end in the same frozen W_O (Sec. 4.1), so A_s - A_t =
 * (o_s - o_t) W_O^T, the only quantity Eq. 11 and its gradient depend on; the step
 * forms o_s - o_t (storage dtype) and applies W_O to it.  tw->Wo is that shared W_O.
 * mask [B, T] uint8 or NULL (all valid).  Writes loss[0] = L (device fp32; loss[1] = NaN:
 * the relative error needs sum M A_t^2, which mla_recon_rel_error adds on request) and the
 * requested gradients (fp32, overwritten).
 * dA: NULL, or [B, T, D] (storage dtype, 16-byte aligned) that receives dL/dA_s.  Without
 * dA (bf16), the backward's dL/do_s = dA W_O is taken as 2 M Y / (D sum M) with
 * Y = (o_s - o_t) W_O^T W_O, and each token's squared error as its row of Y dotted with
 * its row of o_s - o_t: W_O^T W_O is formed (every call) and one [B T, H d_k] x
 * [H d_k, H d_k] product replaces the two [B T, D] x [D, H d_k] ones.  ws as for the
 * other calls. */
int mla_recon_step(const mla_recon_cfg *cfg, const void *h, const mla_teacher_w *tw,
                   const mla_student_w *sw, const uint8_t *mask, float *loss, void *dA,
                   const mla_student_grads *grads, void *ws, size_t ws_bytes, void *hip_stream);

/* The single-call step with the teacher cached (the frozen block's output depends only on
 * h and frozen weights, so it can be reused across steps on the same minibatch).
 * mla_recon_teacher_cache runs the teacher forward up to its attention output o_t (and,
 * bf16, W_O^T W_O) into ws; mla_recon_student_step then does everything mla_recon_step
 * does after the teacher, as often as wanted, for the same h, teacher weights and ws
 * (which keeps the cache until a call other than mla_recon_student_step uses it).  Wo is
 * the teacher's W_O; other arguments as for mla_recon_step. */
int mla_recon_teacher_cache(const mla_recon_cfg *cfg, const void *h, const mla_teacher_w *tw,
                            void *ws, size_t ws_bytes, void *hip_stream);
int mla_recon_student_step(const mla_recon_cfg *cfg, const void *h, const mla_student_w *sw,
                           const void *Wo, const uint8_t *mask, float *loss, void *dA,
                           const mla_student_grads *grads, void *ws, size_t ws_bytes,
                           void *hip_stream);

/* The relative error of the single-call step (the diagnostic loss[1] of mla_recon_loss:
 * sum(M (A_s - A_t))^2 / sum(M A_t)^2, Eq. 11's numerator over the teacher's masked
 * energy).  Call it after mla_recon_step or mla_recon_student_step, on the same stream,
 * with the same cfg, mask and ws and before any other call uses ws: it reads the teacher
 * output o_t and the step's fp64 sum of squared differences that the step left in ws, and
 * writes loss[1] (device fp32 [2]; loss[0] is not touched).  Wo is the teacher's W_O
 * [D, H*d_k].  Costs one [B T, H d_k] x [H d_k, D] product (A_t = o_t W_O^T, not stored
 * in bf16 mode), which is why the step leaves it out.  loss[1] = 0 for an all-invalid
 * mask, +inf when only sum(M A_t)^2 is 0. */
int mla_recon_rel_error(const mla_recon_cfg *cfg, const void *Wo, const uint8_t *mask,
                        float *loss, void *ws, size_t ws_bytes, void *hip_stream);

/* Optimizer step of the reconstruction loop (Sec. 4.1 trains the converter-introduced
 * projections but names no optimizer; this is AdamW: bias-corrected Adam moments, weight
 * decay decoupled from the gradient).  For each of `count` (1-8) tensors of n elements:
 *   m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2
 *   master -= lr ((m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 *                 + weight_decay master)
 *   w = master rounded to the storage dtype (round to nearest even for bf16).
 * master, m, v and grad are fp32, w is in `dtype`; all caller-owned device arrays, 16-byte
 * aligned, updated in place (fp32 arithmetic).  step counts from 1.  One launch. */
typedef struct {
  float *master, *m, *v;
  void *w;
  const float *grad;
  int64_t n;
} mla_adamw_tensor;
int mla_recon_adamw(const mla_adamw_tensor *tensors, int32_t count, int32_t dtype, int32_t step,
                    float lr, float beta1, float beta2, float eps, float weight_decay,
                    void *hip_stream);

/* Calibration capture over a frozen attention stack (Sec. 4.1 reconstructs each layer on
 * cached layer inputs of the frozen model; the stand-in model is an attention-only
 * residual stack: h^l = x^l / rms(x^l), x^{l+1} = x^l + A^l_orig(h^l)).  For each of `rows`
 * rows of `hidden` fp32 values: x += A (A may be NULL: no residual add), then
 * h = x / sqrt(mean(x^2) + eps) in `dtype` (the next layer's input, e.g. the h of
 * mla_recon_teacher_fwd).  x is updated in place; the row reduction has a fixed order. */
int mla_recon_residual_rmsnorm(float *x, const float *A, void *h, int64_t rows, int32_t hidden,
                               int32_t dtype, float eps, void *hip_stream);

/* Decoding with the reconstructed MLA block in absorbed form (Eq. 5's cache: per token the
 * latent c^KV and the rotated positional key; W_UK folded into the query, W_UV applied
 * after the attention-weighted latent).  One query token per sequence; cfg->batch
 * sequences; cfg gives H, G_kv, d_nope, d_rope, r_kv, d_k (= d_v) and the softmax scale;
 * cfg->seq is not used.  Requires bf16, a single positional key (s_rope_groups == 1) and
 * (r_kv + d_rope, r_kv) one of (576, 512), (288, 256), (160, 128), d_k 64 or 128 and at most
 * 65535 sequences; MLA_ERR_UNSUPPORTED otherwise.  W_UV is applied to the weighted latent
 * of each head on the matrix cores (the latent rounded to bf16).
 *   q       [B, H, d_nope + d_rope] bf16: the query token's [q^nope ; R_t q^rope]
 *   cache   [B, max_len, r_kv + d_rope] bf16: rows [c^KV_j | R_j k^PE_j], e.g. the
 *           [c^KV | k^PE] rows of the student forward
 *   lengths device int32 [B]: sequence b attends to its first lengths[b] rows (clamped to
 *           [0, max_len]; 0 rows give o = 0)
 *   Wuk [G_kv d_nope, r_kv], Wuv [G_kv d_k, r_kv] bf16 (the student's W_UK, W_UV)
 *   o       [B, H, d_k] bf16 out: the per-head attention outputs before W_O
 * q, cache, Wuv and ws 16-byte aligned; ws of mla_recon_decode_workspace_size bytes
 * (0 = unsupported or invalid cfg). */
size_t mla_recon_decode_workspace_size(const mla_recon_cfg *cfg, int32_t max_len);
int mla_recon_decode(const mla_recon_cfg *cfg, const void *q, const void *cache, int32_t max_len,
                     const int32_t *lengths, const void *Wuk, const void *Wuv, void *o, void *ws,
                     size_t ws_bytes, void *hip_stream);

/* mla_recon_decode without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops that decode one token per call, harnesses
 * that forbid allocation).  Same arguments and result as mla_recon_decode minus ws; the
 * scratch lives in a static buffer of MLA_DECODE_NOALLOC_SCRATCH_BYTES (32 MiB) that the
 * library holds on each GPU it runs on until the process ends, and this call allocates
 * nothing.  Returns MLA_ERR_UNSUPPORTED when mla_recon_decode_workspace_size(cfg, max_len)
 * exceeds that buffer (e.g. H = 32, r_kv = 512: up to about 100 sequences).  Every call on
 * one GPU uses the same buffer and overwrites what the previous call left there: calls that
 * may overlap on one GPU (concurrent streams, threads) race and must be serialised by the
 * caller. */
#define MLA_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int mla_recon_decode_noalloc(const mla_recon_cfg *cfg, const void *q, const void *cache,
                             int32_t max_len, const int32_t *lengths, const void *Wuk,
                             const void *Wuv, void *o, void *hip_stream);

/* Prefill in absorbed form: every token of cfg->batch sequences of cfg->seq tokens attends,
 * causally, to the latent cache of its own sequence (Eq. 5's rows [c^KV_j | R_j k^PE_j],
 * j <= t) with the absorbed query [W_UK^T q^nope ; q^rope]; the output is the block's
 * per-head attention output o = W_UV[g] (weighted latent) and/or its post-W_O output A
 * (the student side of Eq. 11), computed either as o W_O^T or, given the folded weights of
 * mla_recon_fold_uv_into_o, as (weighted latent) W_O'^T.  Same shape requirements as
 * mla_recon_decode, and at most 65535 tokens (batch * seq) per call.
 *   q     [B, T, H, d_nope + d_rope] bf16 (q^rope rotated by R_t)
 *   cache [B, T, r_kv + d_rope] bf16
 *   Wuk [G_kv d_nope, r_kv], Wuv [G_kv d_k, r_kv], Wo [D, H d_k] bf16; Wo_folded
 *   [D, H r_kv] bf16 or NULL
 *   o     [B, T, H, d_k] bf16 out, or NULL; A [B, T, D] fp32 out, or NULL (not both NULL;
 *   A needs Wo_folded, or Wo and Wuv; o needs Wuv)
 * q, cache, Wuv and ws 16-byte aligned; ws of mla_recon_prefill_workspace_size bytes. */
size_t mla_recon_prefill_workspace_size(const mla_recon_cfg *cfg);
int mla_recon_prefill(const mla_recon_cfg *cfg, const void *q, const void *cache, const void *Wuk,
                      const void *Wuv, const void *Wo, const void *Wo_folded, void *o, float *A,
                      void *ws, size_t ws_bytes, void *hip_stream);

/* W_UV folded into the frozen W_O (Eq. 5's value up-projection absorbed into the output
 * projection): Wo_folded[:, i r_kv + c] = sum_e Wo[:, i d_k + e] Wuv[g(i) d_k + e][c] for
 * every head i, bf16 [D, H r_kv].  With it the block's output is the attention-weighted
 * latent times Wo_folded^T.  (At r_kv > d_k the folded matrix is r_kv / d_k times larger
 * than W_O, so the unfolded products are cheaper per token; both are offered.) */
int mla_recon_fold_uv_into_o(const mla_recon_cfg *cfg, const void *Wo, const void *Wuv,
                             void *Wo_folded, void *hip_stream);

/* Text of the last error on the calling thread ("" if none). */
const char *mla_recon_last_error(void);

/* ---- timing instrumentation (not part of the method) --------------------------------
 * When enabled for a kernel class, every launch of that class made by the calls above is
 * bracketed by a pair of HIP events recorded on the launch stream.  mla_recon_prof_read
 * waits for those events, returns the summed kernel time (ms), the launch count and the
 * algorithmic FLOPs and HBM bytes those launches account for, and clears the record.
 * Classes: 0 GEMM C = A B^T, 1 GEMM with B N-contiguous, 2 GEMM with both operands
 * M/N-contiguous (weight gradients), 3 attention forward, 4 attention backward dV and
 * the stored dS^T, 5 attention backward dQ (a GEMM over dS^T), 6 loss, 7 elementwise
 * (RoPE, reductions, conversions, split-K sums), 8 attention backward dK (a GEMM over
 * dS^T).  Up to 4096 launches are recorded per class.
 * mla_recon_prof_kernels splits the same record by kernel (one entry per kernel function
 * and template instance, e.g. "gemm_mfma_persist_kernel<256,256,NT,bf16>"): it writes up
 * to cap entries, returns how many kernels the class ran (or a negative mla_status) and
 * leaves the record in place for mla_recon_prof_read.  The names are static strings. */
typedef struct {
  const char *kernel;
  double ms;            /* summed duration of its launches                                 */
  int64_t launches;
  double alg_flops;     /* algorithmic FLOPs of those launches                              */
  double alg_bytes;     /* algorithmic HBM bytes of those launches                          */
} mla_prof_kernel;
int mla_recon_prof_enable(int kernel_class, int on);
int mla_recon_prof_kernels(int kernel_class, mla_prof_kernel *out, int cap);
int mla_recon_prof_read(int kernel_class, double *total_ms, int64_t *launches,
                        double *alg_flops, double *alg_bytes);

#ifdef __cplusplus
}
#endif

#endif /* MLA_RECON_H */
