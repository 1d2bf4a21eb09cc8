// C ABI of the reconstruction step: argument validation, workspace layout and the launch
// sequence of each call (teacher forward, student forward, Eq. 11 loss, backward).
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "mla_recon.h"
#include "kernels.h"
#include "mfma.h"
#include "simt.h"

namespace mla {

// ---------------------------------------------------------------------------------------
// last error
// ---------------------------------------------------------------------------------------
static thread_local char g_err[512] = "";

static int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

#define HIP_TRY(expr)                                                                     \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return fail(MLA_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));            \
  } while (0)

// ---------------------------------------------------------------------------------------
// timing instrumentation
// ---------------------------------------------------------------------------------------
struct ProfClass {
  bool on = false;
  std::vector<hipEvent_t> ev;  // 2 per launch
  std::vector<const char*> kernel;  // per launch: its kernel's name
  std::vector<double> kflops, kbytes;  // per launch: its algorithmic FLOPs and bytes
  int used = 0;
  double flops = 0.0, bytes = 0.0;
};
static ProfClass g_prof[KC_COUNT];
static std::mutex g_prof_mu;
static constexpr int PROF_MAX = 4096;

void prof_begin(int k, hipStream_t s) {
  ProfClass& p = g_prof[k];
  if (!p.on || p.used >= PROF_MAX) return;
  (void)hipEventRecord(p.ev[2 * p.used], s);
}

void prof_end(int k, hipStream_t s, double flops, double bytes, const char* kernel) {
  ProfClass& p = g_prof[k];
  if (!p.on || p.used >= PROF_MAX) return;
  (void)hipEventRecord(p.ev[2 * p.used + 1], s);
  p.kernel[p.used] = kernel ? kernel : "unnamed";
  p.kflops[p.used] = flops;
  p.kbytes[p.used] = bytes;
  p.used++;
  p.flops += flops;
  p.bytes += bytes;
}

// ---------------------------------------------------------------------------------------
// configuration checks and workspace layout
// ---------------------------------------------------------------------------------------
struct Dims {
  int64_t B, T, N, D, H, G, dk, rq, rkv, dn, dr, dqk, dv, Gkv, Gr, kv_out;
  DType t;
  size_t ts;
};

static Dims dims_of(const mla_recon_cfg* c) {
  Dims d;
  d.B = c->batch; d.T = c->seq; d.N = d.B * d.T; d.D = c->hidden;
  d.H = c->n_heads; d.G = c->n_kv_groups; d.dk = c->head_dim;
  d.rq = c->q_rank; d.rkv = c->kv_rank; d.dn = c->nope_dim; d.dr = c->rope_dim;
  d.dqk = d.dn + d.dr; d.dv = d.dk; d.Gkv = c->s_kv_groups; d.Gr = c->s_rope_groups;
  d.kv_out = d.rkv + d.Gr * d.dr;
  d.t = c->dtype == MLA_FP32 ? DT_F32 : DT_BF16;
  d.ts = dsize(d.t);
  return d;
}

static bool attn_supported(const Dims& d, int dqk, int dv) {
  return attn_simt_supported(dqk, dv) || (d.t == DT_BF16 && attn_mfma_supported(dqk, dv));
}

static int check_cfg(const mla_recon_cfg* c) {
  if (!c) return fail(MLA_ERR_INVALID_ARG, "cfg is NULL");
  if (c->batch < 1 || c->seq < 1 || c->hidden < 1 || c->n_heads < 1 || c->n_kv_groups < 1 ||
      c->head_dim < 1 || c->kv_rank < 1 || c->rope_dim < 1 || c->s_kv_groups < 1 ||
      c->s_rope_groups < 1 || c->q_rank < 0 || c->nope_dim < 0)
    return fail(MLA_ERR_INVALID_ARG, "non-positive dimension in cfg");
  if (c->dtype != MLA_BF16 && c->dtype != MLA_FP32)
    return fail(MLA_ERR_INVALID_ARG, "unknown dtype %d", c->dtype);
  if (c->n_heads % c->n_kv_groups || c->n_heads % c->s_kv_groups || c->n_heads % c->s_rope_groups)
    return fail(MLA_ERR_INVALID_ARG, "n_heads must be a multiple of n_kv_groups, s_kv_groups and s_rope_groups");
  if (c->head_dim % 2 || c->rope_dim % 2)
    return fail(MLA_ERR_INVALID_ARG, "head_dim and rope_dim must be even");
  if (!(c->softmax_scale > 0.f) || c->softmax_scale > 1e30f)
    return fail(MLA_ERR_INVALID_ARG, "softmax_scale must be positive and finite");
  if (c->hidden % 8 || c->head_dim % 8 || c->q_rank % 8 || c->kv_rank % 8 || c->nope_dim % 8 ||
      c->rope_dim % 8)
    return fail(MLA_ERR_INVALID_ARG, "hidden, head_dim, q_rank, kv_rank, nope_dim, rope_dim must be multiples of 8");
  if (c->s_kv_groups % c->s_rope_groups)
    return fail(MLA_ERR_UNSUPPORTED, "s_kv_groups must be a multiple of s_rope_groups");
  Dims d = dims_of(c);
  if ((double)d.N * d.H * d.dqk >= 9.0e18)
    return fail(MLA_ERR_INVALID_ARG, "problem too large");
  if (!attn_supported(d, (int)d.dk, (int)d.dk))
    return fail(MLA_ERR_UNSUPPORTED, "teacher head_dim %d not supported by the attention kernels", c->head_dim);
  if (!attn_supported(d, (int)d.dqk, (int)d.dv))
    return fail(MLA_ERR_UNSUPPORTED, "student logit width %d with value width %d not supported", (int)d.dqk, (int)d.dv);
  if (attn_bwd_chunk_seqs((int)d.B, (int)d.H, (int)d.T, (int)d.dqk, (int)d.dv, d.t) < 0)
    return fail(MLA_ERR_UNSUPPORTED, "attention backward: one sequence's dS^T (%d heads x %d^2 tokens) exceeds 16 GiB",
                c->n_heads, c->seq);
  return MLA_OK;
}

static size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  // teacher scratch
  size_t t_cos, t_sin, t_qkv, t_o;
  // student state kept from student_fwd to bwd
  size_t s_cos, s_sin, s_cq, s_q, s_ckv, s_knope, s_v, s_o, s_lse;
  // backward scratch
  size_t b_do, b_delta, b_dqacc, b_dq, b_dkv, b_dkpe, b_dckv, b_dcq, b_split, b_ds, b_kcat;
  size_t b_statT;
  size_t b_ds_bytes;
  size_t b_split_elems;
  // loss scratch; the single-call step's per-tile sums (bf16) or A_s - A_t (fp32), its
  // W_O^T W_O (bf16) and, in fp32, its dA when the caller passes none
  size_t l_scr, l_diff, l_gram, l_da, l_dot;
  int chunk;  // sequences per chunk of the backward's dS^T
  size_t total;
};

static std::vector<Gemm> bwd_gemm_shapes(const Dims& d);
static Gemm mk(int M, int N, int K, const void* A, int64_t lda, bool ak, const void* B,
               int64_t ldb, bool bk, void* C, int64_t ldc, DType in_t, DType c_t,
               float beta = 0.f);

// Workspace layout.  The matrix-core backward's dS^T and per-token scratch come last and
// are sized for `chunk` sequences at a time (<= the 16 GiB cap): every other offset is
// independent of the chunk, so any workspace between the minimum (one sequence) and the
// preferred size (the largest chunk) serves, and the backward runs ceil(B / chunk) chunks.
static Layout layout_of(const Dims& d, int chunk) {
  Layout L;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o += al(bytes); return r; };
  const size_t ts = d.ts, N = d.N;
  L.t_cos = take(d.T * (d.dk / 2) * 4);
  L.t_sin = take(d.T * (d.dk / 2) * 4);
  L.t_qkv = take(N * (d.H + 2 * d.G) * d.dk * ts);
  L.t_o = take(N * d.H * d.dk * ts);
  L.s_cos = take(d.Gr * d.T * (d.dr / 2) * 4);
  L.s_sin = take(d.Gr * d.T * (d.dr / 2) * 4);
  L.s_cq = take(N * d.rq * ts);
  L.s_q = take(N * d.H * d.dqk * ts);
  L.s_ckv = take(N * d.kv_out * ts);
  L.s_knope = take(N * d.Gkv * d.dn * ts);
  L.s_v = take(N * d.Gkv * d.dv * ts);
  L.s_o = take(N * d.H * d.dv * ts);
  L.s_lse = take(N * d.H * 4);
  L.b_do = take(N * d.H * d.dv * ts);
  L.b_delta = take(N * d.H * 4);
  L.b_dqacc = take(d.t == DT_F32 ? N * d.H * d.dqk * 4 : 0);
  L.b_dq = take(N * d.H * d.dqk * ts);
  L.b_dkv = take(N * d.Gkv * (d.dn + d.dv) * ts);
  L.b_dkpe = take(d.Gkv * N * d.dr * 4);
  L.b_dckv = take(N * d.kv_out * ts);
  L.b_dcq = take(N * d.rq * ts);
  size_t se = 0;
  for (const Gemm& g : bwd_gemm_shapes(d)) se = std::max(se, gemm_scratch_elems(g));
  L.b_split_elems = se;
  L.b_split = take(se * 4);
  L.l_scr = take(loss_scratch_bytes());
  const int HV = (int)(d.H * d.dv);
  L.l_diff = take(d.t == DT_F32 ? N * d.D * 4
                                 : std::max(gemm_masked_sse_parts(mk((int)N, (int)d.D, HV, nullptr, 0,
                                                                     true, nullptr, 0, true, nullptr,
                                                                     0, d.t, d.t)),
                                            gemm_masked_sse_parts(mk((int)N, HV, HV, nullptr, 0,
                                                                     true, nullptr, 0, true, nullptr,
                                                                     0, d.t, d.t))) * 8);
  L.l_gram = take(d.t == DT_BF16 ? (size_t)HV * HV * 2 : 0);
  L.l_da = take(d.t == DT_F32 ? N * d.D * 4 : 0);
  // partial sums of dO . (o_s - o_t) left by the backward's delta pass (single call, bf16)
  L.l_dot = take(d.t == DT_BF16 ? (size_t)attn_delta_parts((int64_t)N * d.H) * 8 : 0);
  // the backward's dS^T chunk and its per-token scratch
  L.chunk = chunk;
  const size_t ctok = (size_t)chunk * d.T;
  L.b_ds_bytes = chunk ? attn_ds_bytes(chunk, (int)d.H, (int)d.T) : 0;
  L.b_ds = take(L.b_ds_bytes);
  L.b_kcat = take(ctok * d.Gkv * d.dqk * ts);
  L.b_statT = take(chunk ? attn_stats_bytes(chunk, (int)d.H, (int)d.T) : 0);
  L.total = o;
  return L;
}

// largest chunk of sequences the backward may use (0: no dS^T on this path)
static int max_chunk(const Dims& d) {
  return std::max(0, attn_bwd_chunk_seqs((int)d.B, (int)d.H, (int)d.T, (int)d.dqk, (int)d.dv, d.t));
}

// the layout for a workspace of ws_bytes: the largest chunk that fits (at least one
// sequence when the path has a chunk at all)
static Layout layout_for(const Dims& d, size_t ws_bytes) {
  int hi = max_chunk(d);
  if (hi <= 1) return layout_of(d, hi);
  int lo = 1;
  while (lo < hi) {  // largest c in [1, hi] with total(c) <= ws_bytes
    const int mid = lo + (hi - lo + 1) / 2;
    if (layout_of(d, mid).total <= ws_bytes) lo = mid; else hi = mid - 1;
  }
  return layout_of(d, lo);
}

static int check_ws(const mla_recon_cfg* cfg, void* ws, size_t ws_bytes, Layout* L) {
  const Dims d = dims_of(cfg);
  *L = layout_for(d, ws_bytes);
  if (!ws) return fail(MLA_ERR_INVALID_ARG, "workspace is NULL");
  if ((uintptr_t)ws % 256) return fail(MLA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < L->total)
    return fail(MLA_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes (minimum)", ws_bytes, L->total);
  return MLA_OK;
}

static inline char* at(void* ws, size_t off) { return (char*)ws + off; }

static Gemm mk(int M, int N, int K, const void* A, int64_t lda, bool ak, const void* B,
               int64_t ldb, bool bk, void* C, int64_t ldc, DType in_t, DType c_t,
               float beta) {
  Gemm g;
  g.M = M; g.N = N; g.K = K; g.A = A; g.lda = lda; g.a_kmajor = ak; g.B = B; g.ldb = ldb;
  g.b_kmajor = bk; g.C = C; g.ldc = ldc; g.in_t = in_t; g.c_t = c_t; g.alpha = 1.f; g.beta = beta;
  return g;
}

// Shapes (only M, N, K, layouts and types matter) of the backward GEMMs, for scratch sizing.
static std::vector<Gemm> bwd_gemm_shapes(const Dims& d) {
  std::vector<Gemm> v;
  const int N = (int)d.N;
  v.push_back(mk((int)(d.Gkv * d.dn), (int)d.rkv, N, 0, 0, false, 0, 0, false, 0, 0, d.t, DT_F32));
  v.push_back(mk((int)(d.Gkv * d.dv), (int)d.rkv, N, 0, 0, false, 0, 0, false, 0, 0, d.t, DT_F32));
  // dW_UK and dW_UV as one product (rows of both), summed into the two outputs
  v.push_back(mk((int)(d.Gkv * (d.dn + d.dv)), (int)d.rkv, N, 0, 0, false, 0, 0, false, 0, 0, d.t, DT_F32));
  v.back().C2 = reinterpret_cast<void*>(uintptr_t{256});  // any non-null pointer: the
                                                           // two-output form (always partials)
  v.back().m2 = (int)(d.Gkv * d.dn);
  v.push_back(mk((int)d.kv_out, (int)d.D, N, 0, 0, false, 0, 0, false, 0, 0, d.t, DT_F32));
  v.push_back(mk((int)(d.H * d.dqk), (int)(d.rq ? d.rq : d.D), N, 0, 0, false, 0, 0, false, 0, 0, d.t, DT_F32));
  if (d.rq) v.push_back(mk((int)d.rq, (int)d.D, N, 0, 0, false, 0, 0, false, 0, 0, d.t, DT_F32));
  return v;
}

}  // namespace mla

using namespace mla;

// ---------------------------------------------------------------------------------------
// the C ABI
// ---------------------------------------------------------------------------------------
extern "C" {

const char* mla_recon_last_error(void) { return g_err; }

size_t mla_recon_workspace_size(const mla_recon_cfg* cfg) {
  if (check_cfg(cfg) != MLA_OK) return 0;
  const Dims d = dims_of(cfg);
  return layout_of(d, max_chunk(d)).total;
}

size_t mla_recon_workspace_size_min(const mla_recon_cfg* cfg) {
  if (check_cfg(cfg) != MLA_OK) return 0;
  const Dims d = dims_of(cfg);
  return layout_of(d, std::min(1, max_chunk(d))).total;
}

// Teacher forward up to the attention output o_t (ws region t_o); with A_t also the frozen
// output projection.
static int teacher_impl(const mla_recon_cfg* cfg, const Layout& L, const void* h,
                        const mla_teacher_w* w, float* A_t, void* ws, hipStream_t s) {
  const Dims d = dims_of(cfg);
  const int N = (int)d.N, D = (int)d.D, H = (int)d.H, G = (int)d.G, dk = (int)d.dk;
  const int64_t ld_qkv = (H + 2 * G) * (int64_t)dk;
  float* cs = (float*)at(ws, L.t_cos);
  float* sn = (float*)at(ws, L.t_sin);
  char* qkv = at(ws, L.t_qkv);
  char* o = at(ws, L.t_o);
  const size_t ts = d.ts;

  HIP_TRY(rope_tables(w->inv_freq, 1, (int)d.T, dk / 2, cs, sn, s));
  // Eq. 1: q = W^Q h, k = W^K h, v = W^V h  (columns [Q | K | V] of one buffer)
  HIP_TRY(gemm(mk(N, H * dk, D, h, D, true, w->Wq, D, true, qkv, ld_qkv, d.t, d.t), nullptr, 0, s));
  HIP_TRY(gemm(mk(N, G * dk, D, h, D, true, w->Wk, D, true, qkv + (size_t)H * dk * ts, ld_qkv, d.t, d.t), nullptr, 0, s));
  HIP_TRY(gemm(mk(N, G * dk, D, h, D, true, w->Wv, D, true, qkv + (size_t)(H + G) * dk * ts, ld_qkv, d.t, d.t), nullptr, 0, s));
  // R_t on queries and keys (Sec. 3.1); on the matrix-core path the attention kernel rotates
  // the queries as it loads them (the teacher's rotated queries are not needed elsewhere)
  const bool q_on_load = d.t == DT_BF16 && attn_mfma_supported(dk, dk) && dk % 32 == 0;
  if (!q_on_load)
    HIP_TRY(rope_apply(qkv, d.t, N, (int)d.T, H, ld_qkv, dk, 0, dk / 2, H, cs, sn, s));
  HIP_TRY(rope_apply(qkv + (size_t)H * dk * ts, d.t, N, (int)d.T, G, ld_qkv, dk, 0, dk / 2, G, cs, sn, s));
  // Eq. 2-4: causal softmax attention, head i reads KV group i / (H/G)
  Attn a;
  a.B = (int)d.B; a.T = (int)d.T; a.H = H; a.dqk = dk; a.dnope = dk; a.dv = dk;
  a.Q = HeadView{qkv, ld_qkv, dk, 1};
  a.Ka = HeadView{qkv + (size_t)H * dk * ts, ld_qkv, dk, H / G};
  a.Kb = HeadView{nullptr, 0, 0, 1};
  a.V = HeadView{qkv + (size_t)(H + G) * dk * ts, ld_qkv, dk, H / G};
  a.O = o; a.o_tok = (int64_t)H * dk; a.lse = nullptr; a.scale = cfg->softmax_scale; a.t = d.t;
  if (q_on_load) {
    a.q_cos = cs; a.q_sin = sn; a.q_roff = 0; a.q_np = dk / 2;
  }
  HIP_TRY(attn_fwd(a, s));
  // the fixed output projection: A = concat_i o_i W_O^T
  if (A_t)
    HIP_TRY(gemm(mk(N, D, H * dk, o, (int64_t)H * dk, true, w->Wo, (int64_t)H * dk, true, A_t, D, d.t, DT_F32), nullptr, 0, s));
  return MLA_OK;
}

int mla_recon_teacher_fwd(const mla_recon_cfg* cfg, const void* h, const mla_teacher_w* w,
                          float* A_t, void* ws, size_t ws_bytes, void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!h || !w || !A_t || !w->Wq || !w->Wk || !w->Wv || !w->Wo || !w->inv_freq)
    return fail(MLA_ERR_INVALID_ARG, "teacher_fwd: NULL pointer argument");
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  return teacher_impl(cfg, L, h, w, A_t, ws, (hipStream_t)hip_stream);
}

static bool student_w_ok(const mla_recon_cfg* cfg, const mla_student_w* w) {
  return w && w->Wuq && w->Wdkv_kr && w->Wuv && w->inv_freq && (cfg->q_rank == 0 || w->Wdq) &&
         (cfg->nope_dim == 0 || w->Wuk);
}

// Student forward up to the attention output o_s (kept in ws for the backward); then
// A_s = o_s W_O^T when A_s is given, and o_diff = o_s - o_ref (storage dtype, same layout)
// when o_diff is given.
static int student_impl(const mla_recon_cfg* cfg, const Layout& L, const void* h,
                        const mla_student_w* w, const void* Wo, float* A_s, const void* o_ref,
                        void* o_diff, void* ws, hipStream_t s) {
  const Dims d = dims_of(cfg);
  const int N = (int)d.N, D = (int)d.D, H = (int)d.H, T = (int)d.T;
  const int rq = (int)d.rq, rkv = (int)d.rkv, dn = (int)d.dn, dr = (int)d.dr, dqk = (int)d.dqk;
  const int dv = (int)d.dv, Gkv = (int)d.Gkv, Gr = (int)d.Gr, kv_out = (int)d.kv_out;
  const size_t ts = d.ts;
  float* cs = (float*)at(ws, L.s_cos);
  float* sn = (float*)at(ws, L.s_sin);
  char* cq = at(ws, L.s_cq);
  char* q = at(ws, L.s_q);
  char* ckv = at(ws, L.s_ckv);
  char* knope = at(ws, L.s_knope);
  char* v = at(ws, L.s_v);
  char* o = at(ws, L.s_o);
  float* lse = (float*)at(ws, L.s_lse);

  HIP_TRY(rope_tables(w->inv_freq, Gr, T, dr / 2, cs, sn, s));
  // low-rank query: c^Q = W_DQ h, q = W_UQ c^Q  (q = W_UQ h when r_q = 0)
  const void* qin = h;
  int qk = D;
  if (rq > 0) {
    HIP_TRY(gemm(mk(N, rq, D, h, D, true, w->Wdq, D, true, cq, rq, d.t, d.t), nullptr, 0, s));
    qin = cq;
    qk = rq;
  }
  HIP_TRY(gemm(mk(N, H * dqk, qk, qin, qk, true, w->Wuq, qk, true, q, (int64_t)H * dqk, d.t, d.t), nullptr, 0, s));
  // Eq. 5: [c^KV | k^PE] = [W^DKV; W^KR] h, [k^nope; v] = W^UKV c^KV
  HIP_TRY(gemm(mk(N, kv_out, D, h, D, true, w->Wdkv_kr, D, true, ckv, kv_out, d.t, d.t), nullptr, 0, s));
  if (dn > 0)
    HIP_TRY(gemm(mk(N, Gkv * dn, rkv, ckv, kv_out, true, w->Wuk, rkv, true, knope, (int64_t)Gkv * dn, d.t, d.t), nullptr, 0, s));
  HIP_TRY(gemm(mk(N, Gkv * dv, rkv, ckv, kv_out, true, w->Wuv, rkv, true, v, (int64_t)Gkv * dv, d.t, d.t), nullptr, 0, s));
  // decoupled RoPE on q^rope (rope group i / (H/G_r)) and on k^PE
  HIP_TRY(rope_apply(q, d.t, N, T, H, (int64_t)H * dqk, dqk, dn, dr / 2, H / Gr, cs, sn, s));
  HIP_TRY(rope_apply(ckv, d.t, N, T, Gr, kv_out, dr, rkv, dr / 2, 1, cs, sn, s));
  // Eq. 2-4 with q = [q^nope; R q^rope], k = [k^nope_{g(i)}; R k^PE_{r(i)}]
  Attn a;
  a.B = (int)d.B; a.T = T; a.H = H; a.dqk = dqk; a.dnope = dn; a.dv = dv;
  a.Q = HeadView{q, (int64_t)H * dqk, dqk, 1};
  a.Ka = HeadView{knope, (int64_t)Gkv * dn, dn, H / Gkv};
  a.Kb = HeadView{ckv + (size_t)rkv * ts, kv_out, dr, H / Gr};
  a.V = HeadView{v, (int64_t)Gkv * dv, dv, H / Gkv};
  a.O = o; a.o_tok = (int64_t)H * dv; a.lse = lse; a.scale = cfg->softmax_scale; a.t = d.t;
  a.o_ref = o_ref; a.o_diff = o_diff;
  HIP_TRY(attn_fwd(a, s));
  // the teacher's frozen W_O
  if (A_s)
    HIP_TRY(gemm(mk(N, D, H * dv, o, (int64_t)H * dv, true, Wo, (int64_t)H * dv, true, A_s, D, d.t, DT_F32), nullptr, 0, s));
  return MLA_OK;
}

int mla_recon_student_fwd(const mla_recon_cfg* cfg, const void* h, const mla_student_w* w,
                          const void* Wo, float* A_s, void* ws, size_t ws_bytes,
                          void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!h || !Wo || !A_s || !student_w_ok(cfg, w))
    return fail(MLA_ERR_INVALID_ARG, "student_fwd: NULL pointer argument");
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  return student_impl(cfg, L, h, w, Wo, A_s, nullptr, nullptr, ws, (hipStream_t)hip_stream);
}

int mla_recon_loss(const mla_recon_cfg* cfg, const float* A_s, const float* A_t,
                   const uint8_t* mask, float* loss, void* dA, void* ws, size_t ws_bytes,
                   void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!A_s || !A_t || !loss) return fail(MLA_ERR_INVALID_ARG, "loss: NULL pointer argument");
  if (((uintptr_t)A_s | (uintptr_t)A_t) % 16 || (dA && (uintptr_t)dA % 16))
    return fail(MLA_ERR_INVALID_ARG, "loss: A_s, A_t and dA must be 16-byte aligned");
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  const Dims d = dims_of(cfg);
  HIP_TRY(recon_loss(A_s, A_t, mask, d.N, (int)d.D, loss, dA, d.t, at(ws, L.l_scr),
                     (hipStream_t)hip_stream));
  return MLA_OK;
}

static int check_grads(const mla_recon_cfg* cfg, const mla_student_grads* gr, const char* who) {
  if (cfg->q_rank == 0 && gr->dWdq)
    return fail(MLA_ERR_INVALID_ARG, "%s: dWdq given but q_rank == 0 (no W_DQ)", who);
  if (cfg->nope_dim == 0 && gr->dWuk)
    return fail(MLA_ERR_INVALID_ARG, "%s: dWuk given but nope_dim == 0 (no W_UK)", who);
  return MLA_OK;
}

static int bwd_impl(const mla_recon_cfg* cfg, const Layout& L, const void* h,
                    const mla_student_w* w, const void* Wo, const void* dA,
                    const mla_student_grads* gr, void* ws, hipStream_t s,
                    const void* loss_ref = nullptr, double* loss_part = nullptr) {
  const bool need_q = gr->dWuq || gr->dWdq;
  const bool need_kv = gr->dWuk || gr->dWuv || gr->dWdkv_kr;
  if (!need_q && !need_kv) return MLA_OK;
  const Dims d = dims_of(cfg);
  const int N = (int)d.N, D = (int)d.D, H = (int)d.H, T = (int)d.T;
  const int rq = (int)d.rq, rkv = (int)d.rkv, dn = (int)d.dn, dr = (int)d.dr, dqk = (int)d.dqk;
  const int dv = (int)d.dv, Gkv = (int)d.Gkv, Gr = (int)d.Gr, kv_out = (int)d.kv_out;
  const size_t ts = d.ts;
  const DType t = d.t;
  float* cs = (float*)at(ws, L.s_cos);
  float* sn = (float*)at(ws, L.s_sin);
  char* cq = at(ws, L.s_cq);
  char* q = at(ws, L.s_q);
  char* ckv = at(ws, L.s_ckv);
  char* knope = at(ws, L.s_knope);
  char* v = at(ws, L.s_v);
  char* o = at(ws, L.s_o);
  float* lse = (float*)at(ws, L.s_lse);
  char* dO = at(ws, L.b_do);
  float* delta = (float*)at(ws, L.b_delta);
  float* dqacc = (float*)at(ws, L.b_dqacc);
  char* dq = at(ws, L.b_dq);
  char* dkv = at(ws, L.b_dkv);
  float* dkpe = (float*)at(ws, L.b_dkpe);
  char* dckv = at(ws, L.b_dckv);
  char* dcq = at(ws, L.b_dcq);
  float* split = (float*)at(ws, L.b_split);
  const size_t se = L.b_split_elems;
  const int64_t ld_dkv = (int64_t)Gkv * (dn + dv);

  // dO = dA W_O  (W_O frozen: no dW_O); without dA, dO is already in place
  if (dA)
    HIP_TRY(gemm(mk(N, H * dv, D, dA, D, true, Wo, (int64_t)H * dv, false, dO, (int64_t)H * dv, t, t), nullptr, 0, s));
  // softmax-attention backward -> dq (rotary block rotated back), dk^nope, dv, dk^PE partials
  AttnBwd ab;
  Attn& a = ab.f;
  a.B = (int)d.B; a.T = T; a.H = H; a.dqk = dqk; a.dnope = dn; a.dv = dv;
  a.Q = HeadView{q, (int64_t)H * dqk, dqk, 1};
  a.Ka = HeadView{knope, (int64_t)Gkv * dn, dn, H / Gkv};
  a.Kb = HeadView{ckv + (size_t)rkv * ts, kv_out, dr, H / Gr};
  a.V = HeadView{v, (int64_t)Gkv * dv, dv, H / Gkv};
  a.O = o; a.o_tok = (int64_t)H * dv; a.lse = lse; a.scale = cfg->softmax_scale; a.t = t;
  ab.dO = dO; ab.delta = delta; ab.dq_acc = dqacc;
  ab.dq = dq; ab.rdiv = H / Gr; ab.cos_t = cs; ab.sin_t = sn;
  ab.dKa = dkv; ab.dka_tok = ld_dkv;
  ab.dV = dkv + (size_t)Gkv * dn * ts; ab.dv_tok = ld_dkv;
  ab.dkb_part = dkpe; ab.n_ka_groups = Gkv;
  ab.dsT = L.b_ds_bytes ? at(ws, L.b_ds) : nullptr;
  ab.kcat = L.b_ds_bytes ? at(ws, L.b_kcat) : nullptr;
  ab.statT = L.b_ds_bytes ? (float*)at(ws, L.b_statT) : nullptr;
  ab.chunk_seqs = L.chunk;
  ab.loss_ref = loss_ref;
  ab.loss_part = loss_part;
  HIP_TRY(attn_bwd(ab, s));

  if (need_q) {
    const void* qin = rq > 0 ? (const void*)cq : h;
    const int qk = rq > 0 ? rq : D;
    // dW_UQ = dq^T c^Q
    if (gr->dWuq)
      HIP_TRY(gemm(mk(H * dqk, qk, N, dq, (int64_t)H * dqk, false, qin, qk, false, gr->dWuq, qk, t, DT_F32), split, se, s));
    if (gr->dWdq) {
      // dc^Q = dq W_UQ, dW_DQ = dc^Q^T h
      HIP_TRY(gemm(mk(N, rq, H * dqk, dq, (int64_t)H * dqk, true, w->Wuq, rq, false, dcq, rq, t, t), nullptr, 0, s));
      HIP_TRY(gemm(mk(rq, D, N, dcq, rq, false, h, D, false, gr->dWdq, D, t, DT_F32), split, se, s));
    }
  }
  if (need_kv) {
    // Eq. 5 backward: dW_UK = dk^nope^T c^KV, dW_UV = dv^T c^KV.  In bf16 both are one
    // product over the adjacent [dk^nope | dv] columns of dkv, its split-K sum written to the
    // two outputs (one launch pair instead of two for these short, wide-K products)
    Gemm both = mk(Gkv * (dn + dv), rkv, N, dkv, ld_dkv, false, ckv, kv_out, false, gr->dWuk, rkv, t, DT_F32);
    both.C2 = gr->dWuv;
    both.m2 = Gkv * dn;
    if (t == DT_BF16 && gr->dWuk && gr->dWuv && dn > 0 && rkv % 4 == 0 &&
        (uintptr_t)gr->dWuk % 16 == 0 && (uintptr_t)gr->dWuv % 16 == 0 &&
        gemm_scratch_elems(both) <= se) {
      HIP_TRY(gemm(both, split, se, s));
    } else {
      if (gr->dWuk && dn > 0)
        HIP_TRY(gemm(mk(Gkv * dn, rkv, N, dkv, ld_dkv, false, ckv, kv_out, false, gr->dWuk, rkv, t, DT_F32), split, se, s));
      if (gr->dWuv)
        HIP_TRY(gemm(mk(Gkv * dv, rkv, N, dkv + (size_t)Gkv * dn * ts, ld_dkv, false, ckv, kv_out, false, gr->dWuv, rkv, t, DT_F32), split, se, s));
    }
    if (gr->dWdkv_kr) {
      // dc^KV = dk^nope W_UK + dv W_UV; dk^PE = R^T sum of the head partials
      if (dn > 0)
        HIP_TRY(gemm(mk(N, rkv, Gkv * dn, dkv, ld_dkv, true, w->Wuk, rkv, false, dckv, kv_out, t, t), nullptr, 0, s));
      HIP_TRY(gemm(mk(N, rkv, Gkv * dv, dkv + (size_t)Gkv * dn * ts, ld_dkv, true, w->Wuv, rkv, false, dckv, kv_out, t, t, dn > 0 ? 1.f : 0.f), nullptr, 0, s));
      HIP_TRY(dkpe_finish(dkpe, dckv + (size_t)rkv * ts, t, kv_out, N, T, Gr, Gkv / Gr, dr, cs, sn, s));
      // d[W_DKV; W_KR] = [dc^KV | dk^PE]^T h
      HIP_TRY(gemm(mk(kv_out, D, N, dckv, kv_out, false, h, D, false, gr->dWdkv_kr, D, t, DT_F32), split, se, s));
    }
  }
  return MLA_OK;
}

int mla_recon_bwd(const mla_recon_cfg* cfg, const void* h, const mla_student_w* w,
                  const void* Wo, const void* dA, const mla_student_grads* gr, void* ws,
                  size_t ws_bytes, void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!h || !Wo || !dA || !gr || !student_w_ok(cfg, w))
    return fail(MLA_ERR_INVALID_ARG, "bwd: NULL pointer argument");
  if ((rc = check_grads(cfg, gr, "bwd"))) return rc;
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  return bwd_impl(cfg, L, h, w, Wo, dA, gr, ws, (hipStream_t)hip_stream);
}

// W_O^T W_O (bf16, ws region l_gram) for the step without dA
static int gram_impl(const Dims& d, const Layout& L, const void* Wo, void* ws, hipStream_t s) {
  const int D = (int)d.D, HV = (int)(d.H * d.dv);
  HIP_TRY(gemm(mk(HV, HV, D, Wo, HV, false, Wo, HV, false, at(ws, L.l_gram), HV, d.t, d.t), nullptr, 0, s));
  return MLA_OK;
}

// Everything of the single-call step after the teacher: o_t is in ws (t_o) and, for the
// bf16 step without dA, W_O^T W_O in ws (l_gram).
static int student_step_impl(const mla_recon_cfg* cfg, const Layout& L, const void* h,
                             const mla_student_w* sw, const void* Wo, const uint8_t* mask,
                             float* loss, void* dA, const mla_student_grads* gr, void* ws,
                             hipStream_t s) {
  const Dims d = dims_of(cfg);
  int rc;
  // o_s (kept for the backward) and o_s - o_t, the latter into the teacher's q/k/v region,
  // which is free once the teacher's attention has run
  void* odiff = at(ws, L.t_qkv);
  if ((rc = student_impl(cfg, L, h, sw, Wo, nullptr, at(ws, L.t_o), odiff, ws, s))) return rc;
  // A_s - A_t = (o_s - o_t) W_O^T: both blocks end in the same frozen W_O
  const int N = (int)d.N, D = (int)d.D, HV = (int)(d.H * d.dv);
  if (d.t == DT_BF16 && !dA) {
    // dA not requested: with Y = (o_s - o_t) W_O^T W_O, the backward's dO = dA W_O is
    // 2 M Y / (D sum M) and each token's squared error is its row of Y dotted with its row
    // of o_s - o_t
    void* scr = at(ws, L.l_scr);
    double* parts = (double*)at(ws, L.l_diff);
    void* dO = at(ws, L.b_do);
    int nparts = 0;
    HIP_TRY(loss_prepare(mask, d.N, D, scr, s));
    const bool any_grad = gr->dWdq || gr->dWuq || gr->dWdkv_kr || gr->dWuk || gr->dWuv;
    if (any_grad && d.dv % 8 == 0) {
      // the product writes dO only; the backward's delta pass, which streams dO anyway,
      // sums dO . (o_s - o_t) = 2 L (so the product's epilogue does not read o_s - o_t)
      HIP_TRY(gemm_masked_scale(mk(N, HV, HV, odiff, HV, true, at(ws, L.l_gram), HV, true, dO, HV, d.t, d.t),
                                loss_scale(scr), mask, parts, s));
      double* dot = (double*)at(ws, L.l_dot);
      int rc = bwd_impl(cfg, L, h, sw, Wo, nullptr, gr, ws, s, odiff, dot);
      if (rc) return rc;
      HIP_TRY(loss_from_dot(dot, attn_delta_parts((int64_t)d.N * d.H), D, loss, scr, s));
      return MLA_OK;
    }
    HIP_TRY(gemm_masked_sse(mk(N, HV, HV, odiff, HV, true, at(ws, L.l_gram), HV, true, dO, HV, d.t, d.t),
                            loss_scale(scr), mask, odiff, HV, parts, &nparts, s));
    HIP_TRY(loss_from_parts(parts, nparts, D, loss, scr, s));
    return bwd_impl(cfg, L, h, sw, Wo, nullptr, gr, ws, s);
  }
  if (!dA) dA = at(ws, L.l_da);
  if (d.t == DT_BF16) {
    // Eq. 11 in the product's epilogue: dA = 2 M (A_s - A_t) / (D sum M) written directly,
    // the squared masked differences summed per output tile
    void* scr = at(ws, L.l_scr);
    double* parts = (double*)at(ws, L.l_diff);
    int nparts = 0;
    HIP_TRY(loss_prepare(mask, d.N, D, scr, s));
    HIP_TRY(gemm_masked_sse(mk(N, D, HV, odiff, HV, true, Wo, HV, true, dA, D, d.t, d.t),
                            loss_scale(scr), mask, nullptr, 0, parts, &nparts, s));
    HIP_TRY(loss_from_parts(parts, nparts, D, loss, scr, s));
  } else {
    float* diff = (float*)at(ws, L.l_diff);
    HIP_TRY(gemm(mk(N, D, HV, odiff, HV, true, Wo, HV, true, diff, D, d.t, DT_F32), nullptr, 0, s));
    HIP_TRY(recon_loss(diff, nullptr, mask, d.N, D, loss, dA, d.t, at(ws, L.l_scr), s));
  }
  return bwd_impl(cfg, L, h, sw, Wo, dA, gr, ws, s);
}

static bool teacher_w_ok(const mla_teacher_w* tw) {
  return tw && tw->Wq && tw->Wk && tw->Wv && tw->Wo && tw->inv_freq;
}

static int check_step_args(const mla_recon_cfg* cfg, const void* h, const mla_student_w* sw,
                           float* loss, void* dA, const mla_student_grads* gr, const char* who) {
  if (!h || !student_w_ok(cfg, sw) || !loss || !gr)
    return fail(MLA_ERR_INVALID_ARG, "%s: NULL pointer argument", who);
  if ((uintptr_t)dA % 16) return fail(MLA_ERR_INVALID_ARG, "%s: dA must be 16-byte aligned", who);
  return check_grads(cfg, gr, who);
}

int mla_recon_step(const mla_recon_cfg* cfg, const void* h, const mla_teacher_w* tw,
                   const mla_student_w* sw, const uint8_t* mask, float* loss, void* dA,
                   const mla_student_grads* gr, void* ws, size_t ws_bytes, void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!teacher_w_ok(tw)) return fail(MLA_ERR_INVALID_ARG, "step: NULL pointer argument");
  if ((rc = check_step_args(cfg, h, sw, loss, dA, gr, "step"))) return rc;
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  hipStream_t s = (hipStream_t)hip_stream;
  if ((rc = teacher_impl(cfg, L, h, tw, nullptr, ws, s))) return rc;
  if (cfg->dtype == MLA_BF16 && !dA && (rc = gram_impl(dims_of(cfg), L, tw->Wo, ws, s))) return rc;
  return student_step_impl(cfg, L, h, sw, tw->Wo, mask, loss, dA, gr, ws, s);
}

int mla_recon_teacher_cache(const mla_recon_cfg* cfg, const void* h, const mla_teacher_w* tw,
                            void* ws, size_t ws_bytes, void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!h || !teacher_w_ok(tw)) return fail(MLA_ERR_INVALID_ARG, "teacher_cache: NULL pointer argument");
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  hipStream_t s = (hipStream_t)hip_stream;
  if ((rc = teacher_impl(cfg, L, h, tw, nullptr, ws, s))) return rc;
  if (cfg->dtype == MLA_BF16) return gram_impl(dims_of(cfg), L, tw->Wo, ws, s);
  return MLA_OK;
}

int mla_recon_student_step(const mla_recon_cfg* cfg, const void* h, const mla_student_w* sw,
                           const void* Wo, const uint8_t* mask, float* loss, void* dA,
                           const mla_student_grads* gr, void* ws, size_t ws_bytes,
                           void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!Wo) return fail(MLA_ERR_INVALID_ARG, "student_step: NULL pointer argument");
  if ((rc = check_step_args(cfg, h, sw, loss, dA, gr, "student_step"))) return rc;
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  return student_step_impl(cfg, L, h, sw, Wo, mask, loss, dA, gr, ws, (hipStream_t)hip_stream);
}

int mla_recon_rel_error(const mla_recon_cfg* cfg, const void* Wo, const uint8_t* mask,
                        float* loss, void* ws, size_t ws_bytes, void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!Wo || !loss) return fail(MLA_ERR_INVALID_ARG, "rel_error: NULL pointer argument");
  Layout L;
  if ((rc = check_ws(cfg, ws, ws_bytes, &L))) return rc;
  hipStream_t s = (hipStream_t)hip_stream;
  const Dims d = dims_of(cfg);
  const int N = (int)d.N, D = (int)d.D, HV = (int)(d.H * d.dv);
  void* scr = at(ws, L.l_scr);
  const void* o_t = at(ws, L.t_o);  // the teacher's attention output, kept by the step
  if (d.t == DT_BF16) {
    // sum M A_t^2 with A_t = o_t W_O^T, per output tile of the product (A_t not stored)
    double* parts = (double*)at(ws, L.l_diff);
    int nparts = 0;
    HIP_TRY(loss_prepare(mask, d.N, D, scr, s));
    HIP_TRY(gemm_masked_sse(mk(N, D, HV, o_t, HV, true, Wo, HV, true, nullptr, D, d.t, d.t),
                            loss_scale(scr), mask, nullptr, 0, parts, &nparts, s));
    HIP_TRY(loss_rel_from_parts(parts, nparts, 1, loss, scr, s));
    return MLA_OK;
  }
  // fp32 check mode: A_t formed in ws (l_diff, free after the step)
  float* A_t = (float*)at(ws, L.l_diff);
  HIP_TRY(gemm(mk(N, D, HV, o_t, HV, true, Wo, HV, true, A_t, D, d.t, DT_F32), nullptr, 0, s));
  HIP_TRY(loss_rel_fp32(A_t, mask, d.N, D, loss, scr, s));
  return MLA_OK;
}

int mla_recon_adamw(const mla_adamw_tensor* tensors, int32_t count, int32_t dtype, int32_t step,
                    float lr, float beta1, float beta2, float eps, float weight_decay,
                    void* hip_stream) {
  g_err[0] = 0;
  if (!tensors || count < 1 || count > ADAMW_MAX)
    return fail(MLA_ERR_INVALID_ARG, "adamw: between 1 and %d tensors", ADAMW_MAX);
  if (dtype != MLA_BF16 && dtype != MLA_FP32)
    return fail(MLA_ERR_INVALID_ARG, "adamw: unknown dtype %d", dtype);
  if (step < 1) return fail(MLA_ERR_INVALID_ARG, "adamw: step counts from 1");
  if (!(lr >= 0.f && lr < 1e30f) || !(beta1 >= 0.f && beta1 < 1.f) ||
      !(beta2 >= 0.f && beta2 < 1.f) || !(eps > 0.f && eps < 1e30f) ||
      !(weight_decay >= 0.f && weight_decay < 1e30f))
    return fail(MLA_ERR_INVALID_ARG, "adamw: hyperparameters out of range");
  AdamwTensor t[ADAMW_MAX];
  for (int i = 0; i < count; ++i) {
    const mla_adamw_tensor& x = tensors[i];
    if (x.n < 0) return fail(MLA_ERR_INVALID_ARG, "adamw: tensor %d has negative size", i);
    if (x.n > 0 && (!x.master || !x.m || !x.v || !x.w || !x.grad))
      return fail(MLA_ERR_INVALID_ARG, "adamw: tensor %d: NULL pointer", i);
    if (((uintptr_t)x.master | (uintptr_t)x.m | (uintptr_t)x.v | (uintptr_t)x.w |
         (uintptr_t)x.grad) % 16)
      return fail(MLA_ERR_INVALID_ARG, "adamw: tensor %d: arrays must be 16-byte aligned", i);
    t[i] = AdamwTensor{x.master, x.m, x.v, x.w, x.grad, x.n};
  }
  HIP_TRY(adamw_step(t, count, dtype == MLA_FP32 ? DT_F32 : DT_BF16, lr, beta1, beta2, eps,
                     weight_decay, step, (hipStream_t)hip_stream));
  return MLA_OK;
}

int mla_recon_residual_rmsnorm(float* x, const float* A, void* h, int64_t rows, int32_t hidden,
                               int32_t dtype, float eps, void* hip_stream) {
  g_err[0] = 0;
  if (rows < 0 || hidden < 1 || rows > (int64_t)0x7fffffff)
    return fail(MLA_ERR_INVALID_ARG, "residual_rmsnorm: bad shape");
  if (dtype != MLA_BF16 && dtype != MLA_FP32)
    return fail(MLA_ERR_INVALID_ARG, "residual_rmsnorm: unknown dtype %d", dtype);
  if (!(eps >= 0.f && eps < 1e30f)) return fail(MLA_ERR_INVALID_ARG, "residual_rmsnorm: bad eps");
  if (rows > 0 && (!x || !h)) return fail(MLA_ERR_INVALID_ARG, "residual_rmsnorm: NULL pointer");
  HIP_TRY(residual_rmsnorm(x, A, h, rows, hidden, dtype == MLA_FP32 ? DT_F32 : DT_BF16, eps,
                           (hipStream_t)hip_stream));
  return MLA_OK;
}

static int decode_check(const mla_recon_cfg* cfg, int32_t max_len) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (max_len < 1) return fail(MLA_ERR_INVALID_ARG, "decode: max_len must be positive");
  if (cfg->dtype != MLA_BF16) return fail(MLA_ERR_UNSUPPORTED, "decode: bf16 only");
  if (cfg->s_rope_groups != 1)
    return fail(MLA_ERR_UNSUPPORTED, "decode: one shared positional key (s_rope_groups == 1) only");
  if (!decode_supported(cfg->kv_rank + cfg->rope_dim, cfg->kv_rank))
    return fail(MLA_ERR_UNSUPPORTED, "decode: kv_rank %d with rope_dim %d not supported",
                cfg->kv_rank, cfg->rope_dim);
  if (cfg->head_dim != 128 && cfg->head_dim != 64)
    return fail(MLA_ERR_UNSUPPORTED, "decode: d_k must be 64 or 128");
  if (cfg->batch > 65535) return fail(MLA_ERR_UNSUPPORTED, "decode: at most 65535 sequences per call");
  return MLA_OK;
}

size_t mla_recon_decode_workspace_size(const mla_recon_cfg* cfg, int32_t max_len) {
  g_err[0] = 0;
  if (decode_check(cfg, max_len)) return 0;
  return decode_ws_bytes(cfg->batch, cfg->n_heads, cfg->kv_rank + cfg->rope_dim, cfg->kv_rank,
                         max_len);
}

static int decode_args(const mla_recon_cfg* cfg, const void* q, const void* cache,
                       const int32_t* lengths, const void* Wuk, const void* Wuv, void* o,
                       const char* who) {
  if (!q || !cache || !lengths || !Wuk || !Wuv || !o)
    return fail(MLA_ERR_INVALID_ARG, "%s: NULL pointer argument", who);
  if (((uintptr_t)q | (uintptr_t)cache | (uintptr_t)Wuv) % 16)
    return fail(MLA_ERR_INVALID_ARG, "%s: q, cache and Wuv must be 16-byte aligned", who);
  return MLA_OK;
}

static Decode decode_of(const mla_recon_cfg* cfg, const void* q, const void* cache, int32_t max_len,
                        const int32_t* lengths, const void* Wuk, const void* Wuv, void* o, void* ws) {
  Decode d;
  d.B = cfg->batch; d.H = cfg->n_heads; d.dn = cfg->nope_dim; d.dr = cfg->rope_dim;
  d.rkv = cfg->kv_rank; d.dv = cfg->head_dim; d.hpg = cfg->n_heads / cfg->s_kv_groups;
  d.q = q; d.cache = cache; d.Lmax = max_len; d.ldc = cfg->kv_rank + cfg->rope_dim;
  d.len = lengths; d.Wuk = Wuk; d.Wuv = Wuv; d.scale = cfg->softmax_scale; d.o = o; d.ws = ws;
  return d;
}

int mla_recon_decode(const mla_recon_cfg* cfg, const void* q, const void* cache, int32_t max_len,
                     const int32_t* lengths, const void* Wuk, const void* Wuv, void* o, void* ws,
                     size_t ws_bytes, void* hip_stream) {
  g_err[0] = 0;
  int rc = decode_check(cfg, max_len);
  if (rc) return rc;
  if ((rc = decode_args(cfg, q, cache, lengths, Wuk, Wuv, o, "decode"))) return rc;
  if (!ws) return fail(MLA_ERR_INVALID_ARG, "decode: NULL workspace");
  if ((uintptr_t)ws % 16) return fail(MLA_ERR_INVALID_ARG, "decode: ws must be 16-byte aligned");
  const size_t need = decode_ws_bytes(cfg->batch, cfg->n_heads, cfg->kv_rank + cfg->rope_dim,
                                      cfg->kv_rank, max_len);
  if (ws_bytes < need)
    return fail(MLA_ERR_WORKSPACE, "decode: workspace too small: %zu < %zu bytes", ws_bytes, need);
  HIP_TRY(decode_attention(decode_of(cfg, q, cache, max_len, lengths, Wuk, Wuv, o, ws),
                           (hipStream_t)hip_stream));
  return MLA_OK;
}

int mla_recon_decode_noalloc(const mla_recon_cfg* cfg, const void* q, const void* cache,
                             int32_t max_len, const int32_t* lengths, const void* Wuk,
                             const void* Wuv, void* o, void* hip_stream) {
  g_err[0] = 0;
  int rc = decode_check(cfg, max_len);
  if (rc) return rc;
  if ((rc = decode_args(cfg, q, cache, lengths, Wuk, Wuv, o, "decode_noalloc"))) return rc;
  const size_t need = decode_ws_bytes(cfg->batch, cfg->n_heads, cfg->kv_rank + cfg->rope_dim,
                                      cfg->kv_rank, max_len);
  if (need > decode_scratch_bytes())
    return fail(MLA_ERR_UNSUPPORTED,
                "decode_noalloc: %d sequences over %d rows need %zu bytes of scratch, above the "
                "%zu-byte static buffer (use mla_recon_decode with a workspace)",
                cfg->batch, max_len, need, decode_scratch_bytes());
  void* ws = nullptr;
  HIP_TRY(decode_scratch(&ws));
  HIP_TRY(decode_attention(decode_of(cfg, q, cache, max_len, lengths, Wuk, Wuv, o, ws),
                           (hipStream_t)hip_stream));
  return MLA_OK;
}

// ---- absorbed-form prefill and the W_UV fold -------------------------------------------
static size_t prefill_layout(const mla_recon_cfg* cfg, size_t* off_o, size_t* off_lat) {
  const int64_t rows = (int64_t)cfg->batch * cfg->seq;
  const int DK = cfg->kv_rank + cfg->rope_dim, DVL = cfg->kv_rank;
  size_t o = al(decode_ws_bytes((int)rows, cfg->n_heads, DK, DVL, cfg->seq));
  *off_o = o;
  o += al((size_t)rows * cfg->n_heads * cfg->head_dim * 2);
  *off_lat = o;
  o += al((size_t)rows * cfg->n_heads * DVL * 2);
  return o;
}

static int prefill_check(const mla_recon_cfg* cfg) {
  int rc = decode_check(cfg, cfg ? cfg->seq : 0);
  if (rc) return rc;
  if ((int64_t)cfg->batch * cfg->seq > 65535)
    return fail(MLA_ERR_UNSUPPORTED, "prefill: at most 65535 tokens per call");
  return MLA_OK;
}

size_t mla_recon_prefill_workspace_size(const mla_recon_cfg* cfg) {
  g_err[0] = 0;
  if (prefill_check(cfg)) return 0;
  size_t a, b;
  return prefill_layout(cfg, &a, &b);
}

int mla_recon_prefill(const mla_recon_cfg* cfg, const void* q, const void* cache, const void* Wuk,
                      const void* Wuv, const void* Wo, const void* Wo_folded, void* o, float* A,
                      void* ws, size_t ws_bytes, void* hip_stream) {
  g_err[0] = 0;
  int rc = prefill_check(cfg);
  if (rc) return rc;
  if (!q || !cache || !Wuk || !ws) return fail(MLA_ERR_INVALID_ARG, "prefill: NULL pointer argument");
  if (!o && !A) return fail(MLA_ERR_INVALID_ARG, "prefill: neither o nor A requested");
  if (o && !Wuv) return fail(MLA_ERR_INVALID_ARG, "prefill: o needs Wuv");
  if (A && !Wo_folded && !(Wo && Wuv))
    return fail(MLA_ERR_INVALID_ARG, "prefill: A needs Wo_folded, or Wo and Wuv");
  if (((uintptr_t)q | (uintptr_t)cache | (uintptr_t)ws | (uintptr_t)(Wuv ? Wuv : q)) % 16)
    return fail(MLA_ERR_INVALID_ARG, "prefill: q, cache, Wuv and ws must be 16-byte aligned");
  size_t off_o, off_lat;
  const size_t need = prefill_layout(cfg, &off_o, &off_lat);
  if (ws_bytes < need)
    return fail(MLA_ERR_WORKSPACE, "prefill: workspace too small: %zu < %zu bytes", ws_bytes, need);
  hipStream_t s = (hipStream_t)hip_stream;
  const int rows = cfg->batch * cfg->seq, H = cfg->n_heads, D = cfg->hidden;
  const int dv = cfg->head_dim, rkv = cfg->kv_rank;
  const bool folded = A && Wo_folded;
  // rows b T + t: token t of sequence b, against the first t + 1 rows of its cache
  Decode d = decode_of(cfg, q, cache, cfg->seq, nullptr, Wuk, Wuv, nullptr, ws);
  d.B = rows;
  d.tps = cfg->seq;
  void* obuf = o ? o : (A && !folded ? (void*)at(ws, off_o) : nullptr);
  d.o = obuf;
  if (folded) d.lat_out = at(ws, off_lat);
  HIP_TRY(decode_attention(d, s));
  if (A) {
    // A = o W_O^T, or with the folded weights A = latent W_O'^T (K = H r_kv)
    const int K = folded ? H * rkv : H * dv;
    HIP_TRY(gemm(mk(rows, D, K, folded ? d.lat_out : obuf, K, true, folded ? Wo_folded : Wo, K, true,
                    A, D, DT_BF16, DT_F32), nullptr, 0, s));
  }
  return MLA_OK;
}

int mla_recon_fold_uv_into_o(const mla_recon_cfg* cfg, const void* Wo, const void* Wuv,
                             void* Wo_folded, void* hip_stream) {
  g_err[0] = 0;
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (cfg->dtype != MLA_BF16) return fail(MLA_ERR_UNSUPPORTED, "fold_uv_into_o: bf16 only");
  if (!Wo || !Wuv || !Wo_folded) return fail(MLA_ERR_INVALID_ARG, "fold_uv_into_o: NULL pointer argument");
  const int H = cfg->n_heads, D = cfg->hidden, dv = cfg->head_dim, rkv = cfg->kv_rank;
  const int hpg = H / cfg->s_kv_groups;
  hipStream_t s = (hipStream_t)hip_stream;
  // head i: W_O'[:, i r_kv + c] = sum_e W_O[:, i d_k + e] W_UV[g(i) d_k + e][c]
  for (int i = 0; i < H; ++i)
    HIP_TRY(gemm(mk(D, rkv, dv, (const uint16_t*)Wo + (size_t)i * dv, (int64_t)H * dv, true,
                    (const uint16_t*)Wuv + (size_t)(i / hpg) * dv * rkv, rkv, false,
                    (uint16_t*)Wo_folded + (size_t)i * rkv, (int64_t)H * rkv, DT_BF16, DT_BF16),
                 nullptr, 0, s));
  return MLA_OK;
}

int mla_recon_prof_enable(int k, int on) {
  if (k < 0 || k >= KC_COUNT) return fail(MLA_ERR_INVALID_ARG, "bad kernel class %d", k);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  ProfClass& p = g_prof[k];
  if (on && p.ev.empty()) {
    p.ev.resize(2 * PROF_MAX);
    for (auto& e : p.ev) HIP_TRY(hipEventCreate(&e));
    p.kernel.assign(PROF_MAX, nullptr);
    p.kflops.assign(PROF_MAX, 0.0);
    p.kbytes.assign(PROF_MAX, 0.0);
  }
  p.on = on != 0;
  p.used = 0;
  p.flops = p.bytes = 0.0;
  return MLA_OK;
}

int mla_recon_prof_kernels(int k, mla_prof_kernel* out, int cap) {
  if (k < 0 || k >= KC_COUNT) return fail(MLA_ERR_INVALID_ARG, "bad kernel class %d", k);
  if (cap < 0 || (cap > 0 && !out)) return fail(MLA_ERR_INVALID_ARG, "prof_kernels: bad output array");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  ProfClass& p = g_prof[k];
  std::vector<mla_prof_kernel> acc;
  for (int i = 0; i < p.used; ++i) {
    HIP_TRY(hipEventSynchronize(p.ev[2 * i + 1]));
    float e = 0.f;
    HIP_TRY(hipEventElapsedTime(&e, p.ev[2 * i], p.ev[2 * i + 1]));
    size_t j = 0;
    while (j < acc.size() && strcmp(acc[j].kernel, p.kernel[i]) != 0) ++j;
    if (j == acc.size()) acc.push_back(mla_prof_kernel{p.kernel[i], 0.0, 0, 0.0, 0.0});
    acc[j].ms += e;
    acc[j].launches += 1;
    acc[j].alg_flops += p.kflops[i];
    acc[j].alg_bytes += p.kbytes[i];
  }
  for (size_t j = 0; j < acc.size() && (int)j < cap; ++j) out[j] = acc[j];
  return (int)acc.size();
}

int mla_recon_prof_read(int k, double* total_ms, int64_t* launches, double* alg_flops,
                        double* alg_bytes) {
  if (k < 0 || k >= KC_COUNT) return fail(MLA_ERR_INVALID_ARG, "bad kernel class %d", k);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  ProfClass& p = g_prof[k];
  double ms = 0.0;
  for (int i = 0; i < p.used; ++i) {
    HIP_TRY(hipEventSynchronize(p.ev[2 * i + 1]));
    float e = 0.f;
    HIP_TRY(hipEventElapsedTime(&e, p.ev[2 * i], p.ev[2 * i + 1]));
    ms += e;
  }
  if (total_ms) *total_ms = ms;
  if (launches) *launches = p.used;
  if (alg_flops) *alg_flops = p.flops;
  if (alg_bytes) *alg_bytes = p.bytes;
  p.used = 0;
  p.flops = p.bytes = 0.0;
  return MLA_OK;
}

}  // extern "C"
