// Causal softmax attention (Eq. 2-4) on gfx950 matrix cores, bf16 operands, fp32 softmax.
//
// Forward.  A workgroup (4 wavefronts) owns 128 queries of one (sequence, head); each
// wavefront owns 32 of them.  Keys/values stream through LDS 64 at a time (double
// buffered, the next tile's global loads in flight during the current tile's math).
// The logits are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: the
// query is the MFMA column, so every lane owns one query and the online-softmax state
// (running max m, running sum l, the output row O^T) of that query lives in that lane.
// The accumulator layout of S^T is then reused directly as the B operand of
// O^T = V^T P^T (the key order inside one MFMA K-step is permuted identically on the
// V^T side), so P never leaves registers.  V is transposed to [d_v][key] while it is
// staged in LDS.  Softmax runs in base 2 with the logit scale folded into one FMA.
// Tiles entirely above the causal diagonal are skipped per wavefront; only diagonal tiles
// are masked.  The key of head i is [Ka_{i/div_a} ; Kb_{i/div_b}] (non-positional part
// from one buffer, rotary part from another), which serves both the teacher
// (Ka = full key) and the MLA student (k^nope of the KV group, k^PE of the rope group).
#include "common.h"
#include "kernels.h"
#include "mfma.h"
#include "simt.h"

namespace mla {

namespace {

constexpr int BQ = 128;   // queries per workgroup
constexpr int BKV = 64;   // keys per tile
constexpr int KPAD = 8;
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

struct AttnDev {
  int B, T, H, dnope;
  float sl2;  // softmax scale * log2(e)
  const bf16_t* Q; int64_t q_tok; int q_head;
  const bf16_t* Ka; int64_t ka_tok; int ka_head; int ka_div;
  const bf16_t* Kb; int64_t kb_tok; int kb_head; int kb_div;
  const bf16_t* V; int64_t v_tok; int v_head; int v_div;
  bf16_t* O; int64_t o_tok;
  float* lse;
  int nqb;
};

AttnDev to_dev(const Attn& a) {
  AttnDev d;
  d.B = a.B; d.T = a.T; d.H = a.H; d.dnope = a.dnope;
  d.sl2 = a.scale * LOG2E;
  d.Q = (const bf16_t*)a.Q.p; d.q_tok = a.Q.tok; d.q_head = (int)a.Q.head;
  d.Ka = (const bf16_t*)a.Ka.p; d.ka_tok = a.Ka.tok; d.ka_head = (int)a.Ka.head; d.ka_div = a.Ka.div;
  d.Kb = (const bf16_t*)a.Kb.p; d.kb_tok = a.Kb.tok; d.kb_head = (int)a.Kb.head; d.kb_div = a.Kb.div;
  d.V = (const bf16_t*)a.V.p; d.v_tok = a.V.tok; d.v_head = (int)a.V.head; d.v_div = a.V.div;
  d.O = (bf16_t*)a.O; d.o_tok = a.o_tok; d.lse = a.lse;
  d.nqb = (a.T + BQ - 1) / BQ;
  return d;
}

// 8 (rows) x 8 (cols) bf16 block held as 8 rows of u32x4 -> transposed row mm
__device__ __forceinline__ u32x4 transpose_row(const u32x4 (&r)[8], int mm) {
  const int w = mm >> 1, sh = (mm & 1) * 16;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t lo = (r[2 * q][w] >> sh) & 0xffffu;
    uint32_t hi = (r[2 * q + 1][w] >> sh) & 0xffffu;
    o[q] = lo | (hi << 16);
  }
  return o;
}

template <int DQK, int DV>
struct KVStage {
  static constexpr int KCH = BKV * (DQK / 8);            // 16-byte chunks of the K tile
  static constexpr int KPER = (KCH + 255) / 256;
  static constexpr int VBLK = (BKV / 8) * (DV / 8);      // 8x8 blocks of the V tile
  static constexpr int VPER = (VBLK + 255) / 256;
  u32x4 k[KPER];
  u32x4 v[VPER][8];

  // keys j0 .. j0+63 of sequence b for head i
  __device__ __forceinline__ void load(const AttnDev& a, int b, int i, int j0) {
    const int ga = i / a.ka_div, gb = i / a.kb_div, gv = i / a.v_div;
#pragma unroll
    for (int it = 0; it < KPER; ++it) {
      const int c = threadIdx.x + it * 256;
      const int key = c / (DQK / 8), dc = (c % (DQK / 8)) * 8;
      const int j = j0 + key;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (c < KCH && j < a.T) {
        const int64_t n = (int64_t)b * a.T + j;
        const bf16_t* src = dc < a.dnope
                                ? a.Ka + n * a.ka_tok + (int64_t)ga * a.ka_head + dc
                                : a.Kb + n * a.kb_tok + (int64_t)gb * a.kb_head + (dc - a.dnope);
        val = *(const u32x4*)src;
      }
      k[it] = val;
    }
#pragma unroll
    for (int it = 0; it < VPER; ++it) {
      const int blk = threadIdx.x + it * 256;
      const int kb8 = (blk % (BKV / 8)) * 8, db8 = (blk / (BKV / 8)) * 8;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int j = j0 + kb8 + r;
        u32x4 val = {0u, 0u, 0u, 0u};
        if (blk < VBLK && j < a.T)
          val = *(const u32x4*)(a.V + ((int64_t)b * a.T + j) * a.v_tok + (int64_t)gv * a.v_head + db8);
        v[it][r] = val;
      }
    }
  }

  __device__ __forceinline__ void store(bf16_t* ks, bf16_t* vt) const {
#pragma unroll
    for (int it = 0; it < KPER; ++it) {
      const int c = threadIdx.x + it * 256;
      if (c < KCH) {
        const int key = c / (DQK / 8), dc = (c % (DQK / 8)) * 8;
        *(u32x4*)(ks + key * (DQK + KPAD) + dc) = k[it];
      }
    }
#pragma unroll
    for (int it = 0; it < VPER; ++it) {
      const int blk = threadIdx.x + it * 256;
      if (blk < VBLK) {
        const int kb8 = (blk % (BKV / 8)) * 8, db8 = (blk / (BKV / 8)) * 8;
#pragma unroll
        for (int mm = 0; mm < 8; ++mm)
          *(u32x4*)(vt + (db8 + mm) * (BKV + KPAD) + kb8) = transpose_row(v[it], mm);
      }
    }
  }
};

template <int DQK, int DV, bool LSE>
__global__ __launch_bounds__(256) void attn_fwd_mfma_kernel(AttnDev a) {
  constexpr int KS = BKV * (DQK + KPAD);
  constexpr int VS = DV * (BKV + KPAD);
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (KS + VS)];
  constexpr int NKK = DQK / 16;  // MFMA K-steps of the logits
  constexpr int NC = DV / 32;    // 32-row tiles of O^T

  // work item: XCD-aware remap so that the query blocks of neighbouring heads (which share
  // K/V) run on one XCD; heavy (late) query blocks first inside each head
  const int nwork = a.B * a.H * a.nqb;
  const int pid = xcd_remap(blockIdx.x, nwork);
  const int bh = pid / a.nqb;
  const int qb = a.nqb - 1 - pid % a.nqb;
  const int b = bh / a.H, i = bh % a.H;
  const int q0 = qb * BQ;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int qw0 = q0 + wave * 32;
  const int my_q = qw0 + col;
  const int64_t nq = (int64_t)b * a.T + min(my_q, a.T - 1);

  // this lane's query, as MFMA B operand fragments (d = 16 kk + 8 half + 0..7)
  bf16x8 qf[NKK];
  {
    const bf16_t* qp = a.Q + nq * a.q_tok + (int64_t)i * a.q_head + 8 * half;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[kk] = *(const bf16x8*)(qp + 16 * kk);
  }

  f32x16 acc_o[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[c][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int kend = min(a.T, q0 + BQ);
  const int nkb = (kend + BKV - 1) / BKV;
  KVStage<DQK, DV> st;
  st.load(a, b, i, 0);
  st.store(smem, smem + KS);
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const int j0 = kb * BKV;
    if (kb + 1 < nkb) st.load(a, b, i, j0 + BKV);
    const bf16_t* ks = smem + cur * (KS + VS);
    const bf16_t* vt = ks + KS;
    if (j0 <= qw0 + 31) {  // wave-uniform: some key of this tile is visible to the wave
      f32x16 s[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int e = 0; e < 16; ++e) s[t][e] = 0.f;
        const bf16_t* kp = ks + (32 * t + col) * (DQK + KPAD) + 8 * half;
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
          s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(kp + 16 * kk), qf[kk],
                                                         s[t], 0, 0, 0);
      }
      // scale to base-2 units, causal mask on diagonal tiles, tile max of this query
      float mx = -INFINITY;
      const bool diag = j0 + BKV - 1 > qw0;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float x = s[t][e] * a.sl2;
          if (diag) {
            const int key = j0 + 32 * t + 8 * (e >> 2) + 4 * half + (e & 3);
            if (key > my_q) x = -INFINITY;
          }
          s[t][e] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float corr = __builtin_amdgcn_exp2f(m_run - m_use);
      m_run = m_new;
      l_run *= corr;
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc_o[c][e] *= corr;
      // P = 2^(x - m), packed to bf16 as the B operand of O^T = V^T P^T
      bf16x8 pf[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        u32x4 w;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float p0 = __builtin_amdgcn_exp2f(s[u >> 1][8 * (u & 1) + 2 * q] - m_use);
          const float p1 = __builtin_amdgcn_exp2f(s[u >> 1][8 * (u & 1) + 2 * q + 1] - m_use);
          l_run += p0 + p1;
          w[q] = pack2bf(p0, p1);
        }
        pf[u] = __builtin_bit_cast(bf16x8, w);
      }
      // O^T += V^T P^T; the K-step u covers keys 32(u/2) + 16(u%2) + {4h..4h+3, 8+4h..8+4h+3}
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const bf16_t* vp = vt + (32 * c + col) * (BKV + KPAD) + 4 * half;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int kofs = 32 * (u >> 1) + 16 * (u & 1);
          u32x2 lo = *(const u32x2*)(vp + kofs);
          u32x2 hi = *(const u32x2*)(vp + kofs + 8);
          u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
          acc_o[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w), pf[u],
                                                             acc_o[c], 0, 0, 0);
        }
      }
    }
    if (kb + 1 < nkb) {
      bf16_t* nxt = smem + (cur ^ 1) * (KS + VS);
      st.store(nxt, nxt + KS);
    }
    __syncthreads();
  }

  // normalise and store: lane holds query my_q, d = 32c + 8(e/4) + 4 half + e%4
  const float l = l_run + __shfl_xor(l_run, 32, 64);
  if (my_q >= a.T) return;
  const float inv = 1.f / l;
  bf16_t* op = a.O + ((int64_t)b * a.T + my_q) * a.o_tok + (int64_t)i * DV + 4 * half;
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      u32x2 w = {pack2bf(acc_o[c][4 * g] * inv, acc_o[c][4 * g + 1] * inv),
                 pack2bf(acc_o[c][4 * g + 2] * inv, acc_o[c][4 * g + 3] * inv)};
      *(u32x2*)(op + 32 * c + 8 * g) = w;
    }
  if (LSE && half == 0) a.lse[((int64_t)b * a.T + my_q) * a.H + i] = (m_run + __log2f(l)) * LN2;
}

template <int DQK, int DV>
hipError_t fwd_launch(const Attn& at, hipStream_t s) {
  AttnDev d = to_dev(at);
  const int nwork = d.B * d.H * d.nqb;
  if (at.lse)
    attn_fwd_mfma_kernel<DQK, DV, true><<<nwork, 256, 0, s>>>(d);
  else
    attn_fwd_mfma_kernel<DQK, DV, false><<<nwork, 256, 0, s>>>(d);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------------------
// Backward.  A workgroup owns 128 keys of one (sequence, Ka group) and walks every head of
// the group and every query block of 64 at or after its keys.  Each wavefront owns 32
// keys: S = Q K^T and dP = dO V^T are computed with the key as the MFMA column, so the
// accumulator layout of P and dS is directly the B operand of dV^T += dO^T P and
// dK^T += Q^T dS (gradients of keys/values accumulate in registers over all heads and
// query blocks).  dO^T and Q^T operands are read from the natural [query][dim] LDS tiles
// with gfx950's transposing LDS read.  dS goes through LDS once ([key][query]) so that
// dQ = dS K for the 64 x d_qk query tile can be split across the four wavefronts; the
// per-workgroup partial dQ is added to an fp32 accumulator with hardware float atomics.
// P = 2^(S log2e scale - lse log2e) reuses the forward's log-sum-exp.
// ---------------------------------------------------------------------------------------
constexpr int BKB = 128;  // keys per workgroup
constexpr int BQB = 64;   // queries per iteration

struct BwdDev {
  AttnDev f;
  const bf16_t* dO;      // [N][H*dv]
  const float* delta;    // [N][H]
  float* dq_acc;         // [N][H][dqk]
  bf16_t* dKa; int64_t dka_tok;
  bf16_t* dV; int64_t dv_tok;
  float* dkb_part;       // [G][N][dqk - dnope]
  int G;                 // Ka groups
  float scale;
};

template <int DQK, int DV>
struct BwdStage {
  static constexpr int QCH = BQB * (DQK / 8);
  static constexpr int QPER = (QCH + 255) / 256;
  static constexpr int OCH = BQB * (DV / 8);
  static constexpr int OPER = (OCH + 255) / 256;
  u32x4 q[QPER];
  u32x4 o[OPER];
  float stat;

  __device__ __forceinline__ void load(const BwdDev& w, int b, int i, int q0) {
    const AttnDev& a = w.f;
#pragma unroll
    for (int it = 0; it < QPER; ++it) {
      const int c = threadIdx.x + it * 256;
      const int r = c / (DQK / 8), dc = (c % (DQK / 8)) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (c < QCH && q0 + r < a.T)
        v = *(const u32x4*)(a.Q + ((int64_t)b * a.T + q0 + r) * a.q_tok + (int64_t)i * a.q_head + dc);
      q[it] = v;
    }
#pragma unroll
    for (int it = 0; it < OPER; ++it) {
      const int c = threadIdx.x + it * 256;
      const int r = c / (DV / 8), dc = (c % (DV / 8)) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (c < OCH && q0 + r < a.T)
        v = *(const u32x4*)(w.dO + ((int64_t)b * a.T + q0 + r) * ((int64_t)a.H * DV) + (int64_t)i * DV + dc);
      o[it] = v;
    }
    const int t = threadIdx.x & 63;
    const int q = q0 + t;
    if (threadIdx.x < 64)
      stat = q < a.T ? a.lse[((int64_t)b * a.T + q) * a.H + i] * LOG2E : INFINITY;
    else if (threadIdx.x < 128)
      stat = q < a.T ? w.delta[((int64_t)b * a.T + q) * a.H + i] : 0.f;
  }

  __device__ __forceinline__ void store(bf16_t* Qs, bf16_t* dOs, float* st) const {
#pragma unroll
    for (int it = 0; it < QPER; ++it) {
      const int c = threadIdx.x + it * 256;
      if (c < QCH) *(u32x4*)(Qs + (c / (DQK / 8)) * (DQK + KPAD) + (c % (DQK / 8)) * 8) = q[it];
    }
#pragma unroll
    for (int it = 0; it < OPER; ++it) {
      const int c = threadIdx.x + it * 256;
      if (c < OCH) *(u32x4*)(dOs + (c / (DV / 8)) * (DV + KPAD) + (c % (DV / 8)) * 8) = o[it];
    }
    if (threadIdx.x < 128) st[threadIdx.x] = stat;
  }
};

template <int DQK, int DV>
__global__ __launch_bounds__(256) void attn_bwd_mfma_kernel(BwdDev w) {
  const AttnDev& a = w.f;
  constexpr int LDK = DQK + KPAD, LDO = DV + KPAD, LDT = BQB + 16;
  constexpr int NKK = DQK / 16, NVK = DV / 16;
  constexpr int NCK = DQK / 32, NCV = DV / 32;
  constexpr int SM = BKB * LDK + BQB * LDK + BQB * LDO + BKB * LDT;
  __shared__ __attribute__((aligned(16))) bf16_t smem[SM + 2 * BQB * 2];
  bf16_t* Ks = smem;
  bf16_t* Qs = Ks + BKB * LDK;
  bf16_t* dOs = Qs + BQB * LDK;
  bf16_t* dSt = dOs + BQB * LDO;
  float* st_lse = (float*)(dSt + BKB * LDT);
  float* st_dl = st_lse + BQB;

  const int nbg = a.B * w.G;
  const int kb = blockIdx.x / nbg;  // early key blocks (the most query blocks) first
  const int bg = blockIdx.x % nbg;
  const int b = bg / w.G, g = bg % w.G;
  const int hpg = a.H / w.G;
  const int k0 = kb * BKB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int kw0 = k0 + 32 * wave;
  const int my_key = kw0 + col;
  const int i0 = g * hpg;

  // keys of this block into LDS ([key][d]); this wave's values as B operand fragments
  {
    constexpr int KCH = BKB * (DQK / 8);
    const int ga = i0 / a.ka_div, gb = i0 / a.kb_div;
    for (int c = threadIdx.x; c < KCH; c += 256) {
      const int key = c / (DQK / 8), dc = (c % (DQK / 8)) * 8;
      const int j = k0 + key;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (j < a.T) {
        const int64_t n = (int64_t)b * a.T + j;
        const bf16_t* src = dc < a.dnope
                                ? a.Ka + n * a.ka_tok + (int64_t)ga * a.ka_head + dc
                                : a.Kb + n * a.kb_tok + (int64_t)gb * a.kb_head + (dc - a.dnope);
        val = *(const u32x4*)src;
      }
      *(u32x4*)(Ks + key * LDK + dc) = val;
    }
  }
  bf16x8 vf[NVK];
  {
    const int gv = i0 / a.v_div;
    const int jj = min(my_key, a.T - 1);
    const bf16_t* vp = a.V + ((int64_t)b * a.T + jj) * a.v_tok + (int64_t)gv * a.v_head + 8 * half;
#pragma unroll
    for (int kk = 0; kk < NVK; ++kk) {
      u32x4 v = *(const u32x4*)(vp + 16 * kk);
      if (my_key >= a.T) v = u32x4{0u, 0u, 0u, 0u};
      vf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x16 dk[NCK], dv[NCV];
#pragma unroll
  for (int c = 0; c < NCK; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) dk[c][e] = 0.f;
#pragma unroll
  for (int c = 0; c < NCV; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) dv[c][e] = 0.f;

  const int qb0 = k0 / BQB;
  const int nqb = (a.T + BQB - 1) / BQB;
  const int nper = nqb - qb0;
  const int niter = hpg * nper;
  BwdStage<DQK, DV> stg;
  if (niter > 0) {
    stg.load(w, b, i0, qb0 * BQB);
    stg.store(Qs, dOs, st_lse);
  }
  __syncthreads();

  for (int it = 0; it < niter; ++it) {
    const int i = i0 + it / nper;
    const int q0 = (qb0 + it % nper) * BQB;
    if (it + 1 < niter) stg.load(w, b, i0 + (it + 1) / nper, (qb0 + (it + 1) % nper) * BQB);

    const bool active = kw0 <= min(q0 + BQB - 1, a.T - 1);
    bf16_t* dst_row = dSt + (32 * wave + col) * LDT + 4 * half;
    if (active) {
      f32x16 sp[2], dp[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
#pragma unroll
        for (int e = 0; e < 16; ++e) { sp[qt][e] = 0.f; dp[qt][e] = 0.f; }
        const bf16_t* qrow = Qs + (32 * qt + col) * LDK + 8 * half;
        const bf16_t* krow = Ks + (32 * wave + col) * LDK + 8 * half;
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
          sp[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(qrow + 16 * kk),
                                                          *(const bf16x8*)(krow + 16 * kk), sp[qt], 0, 0, 0);
        const bf16_t* orow = dOs + (32 * qt + col) * LDO + 8 * half;
#pragma unroll
        for (int kk = 0; kk < NVK; ++kk)
          dp[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(orow + 16 * kk), vf[kk],
                                                          dp[qt], 0, 0, 0);
      }
      // P = 2^(S sl2 - lse2), dS = P (dP - delta); rows q = q0 + 32 qt + 8(e/4) + 4 half + e%4
      const bool diag = kw0 + 31 > q0;
      bf16x8 pf[4], sf[4];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int qr = 32 * qt + 8 * e4 + 4 * half;
          const f32x4 l2 = *(const f32x4*)(st_lse + qr);
          const f32x4 dl = *(const f32x4*)(st_dl + qr);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int e = 4 * e4 + r;
            float p = __builtin_amdgcn_exp2f(sp[qt][e] * a.sl2 - l2[r]);
            if (diag && my_key > q0 + qr + r) p = 0.f;
            sp[qt][e] = p;
            dp[qt][e] = p * (dp[qt][e] - dl[r]);
          }
          // dS^T to LDS: row = this lane's key, 4 consecutive queries
          u32x2 wv = {pack2bf(dp[qt][4 * e4], dp[qt][4 * e4 + 1]),
                      pack2bf(dp[qt][4 * e4 + 2], dp[qt][4 * e4 + 3])};
          *(u32x2*)(dst_row + 32 * qt + 8 * e4) = wv;
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        u32x4 wp, wd;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          wp[q] = pack2bf(sp[u >> 1][8 * (u & 1) + 2 * q], sp[u >> 1][8 * (u & 1) + 2 * q + 1]);
          wd[q] = pack2bf(dp[u >> 1][8 * (u & 1) + 2 * q], dp[u >> 1][8 * (u & 1) + 2 * q + 1]);
        }
        pf[u] = __builtin_bit_cast(bf16x8, wp);
        sf[u] = __builtin_bit_cast(bf16x8, wd);
      }
      // dV^T += dO^T P,  dK^T += Q^T dS   (K-step u: queries 32(u/2) + 16(u%2) + {4h.., 8+4h..})
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int klo = 32 * (u >> 1) + 16 * (u & 1) + 4 * half;
#pragma unroll
        for (int c = 0; c < NCV; ++c)
          dv[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_operand_tr(dOs, LDO, 32 * c, klo, klo + 8),
                                                         pf[u], dv[c], 0, 0, 0);
#pragma unroll
        for (int c = 0; c < NCK; ++c)
          dk[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_operand_tr(Qs, LDK, 32 * c, klo, klo + 8),
                                                         sf[u], dk[c], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) *(u32x2*)(dst_row + 32 * qt + 8 * e4) = u32x2{0u, 0u};
    }
    __syncthreads();
    if (it + 1 < niter) stg.store(Qs, dOs, st_lse);

    // dQ (64 x DQK) = dS (64 x 128 keys) K (128 x DQK): 2 * DQK/32 tiles over 4 wavefronts
    constexpr int NT = 2 * NCK;
    for (int tau = wave; tau < NT; tau += 4) {
      const int qt = tau / NCK, dt = tau % NCK;
      f32x16 acc;
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < BKB / 16; ++ks) {
        const int klo = 16 * ks + 8 * half;
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_operand_tr(dSt, LDT, 32 * qt, klo, klo + 4),
                                                      lds_operand_tr(Ks, LDK, 32 * dt, klo, klo + 4),
                                                      acc, 0, 0, 0);
      }
      float* dqp = w.dq_acc + (int64_t)i * DQK + 32 * dt + col;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int q = q0 + 32 * qt + 8 * (e >> 2) + 4 * half + (e & 3);
        if (q < a.T) unsafeAtomicAdd(dqp + ((int64_t)b * a.T + q) * ((int64_t)a.H * DQK), acc[e] * w.scale);
      }
    }
    __syncthreads();
  }

  // epilogue: this lane's key; rows d = 32c + 8(e/4) + 4 half + e%4
  if (my_key >= a.T) return;
  const int64_t n = (int64_t)b * a.T + my_key;
  const int dr = DQK - a.dnope;
#pragma unroll
  for (int c = 0; c < NCV; ++c)
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const int d = 32 * c + 8 * e4 + 4 * half;
      u32x2 wv = {pack2bf(dv[c][4 * e4], dv[c][4 * e4 + 1]), pack2bf(dv[c][4 * e4 + 2], dv[c][4 * e4 + 3])};
      *(u32x2*)(w.dV + n * w.dv_tok + (int64_t)g * DV + d) = wv;
    }
#pragma unroll
  for (int c = 0; c < NCK; ++c)
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const int d = 32 * c + 8 * e4 + 4 * half;
      const float s = w.scale;
      if (d < a.dnope) {
        u32x2 wv = {pack2bf(s * dk[c][4 * e4], s * dk[c][4 * e4 + 1]),
                    pack2bf(s * dk[c][4 * e4 + 2], s * dk[c][4 * e4 + 3])};
        *(u32x2*)(w.dKa + n * w.dka_tok + (int64_t)g * a.dnope + d) = wv;
      } else {
        f32x4 v = {s * dk[c][4 * e4], s * dk[c][4 * e4 + 1], s * dk[c][4 * e4 + 2], s * dk[c][4 * e4 + 3]};
        *(f32x4*)(w.dkb_part + ((int64_t)g * ((int64_t)a.B * a.T) + n) * dr + (d - a.dnope)) = v;
      }
    }
}

__global__ void zero_f32_kernel(float* __restrict__ p, int64_t n4) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n4) ((f32x4*)p)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
}

template <int DQK, int DV>
hipError_t bwd_launch(const AttnBwd& wb, hipStream_t s) {
  const Attn& at = wb.f;
  BwdDev w;
  w.f = to_dev(at);
  w.dO = (const bf16_t*)wb.dO; w.delta = wb.delta; w.dq_acc = wb.dq_acc;
  w.dKa = (bf16_t*)wb.dKa; w.dka_tok = wb.dka_tok;
  w.dV = (bf16_t*)wb.dV; w.dv_tok = wb.dv_tok;
  w.dkb_part = wb.dkb_part; w.G = wb.n_ka_groups; w.scale = at.scale;
  const int64_t n4 = (int64_t)at.B * at.T * at.H * DQK / 4;
  zero_f32_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, s>>>(wb.dq_acc, n4);
  const int nkb = (at.T + BKB - 1) / BKB;
  attn_bwd_mfma_kernel<DQK, DV><<<nkb * at.B * w.G, 256, 0, s>>>(w);
  return hipGetLastError();
}

}  // namespace

#define MLA_MFMA_SHAPES(X) X(64, 64) X(128, 128) X(96, 64) X(128, 64) X(192, 128)

bool attn_mfma_supported(int dqk, int dv) {
#define X(a_, b_) if (dqk == a_ && dv == b_) return true;
  MLA_MFMA_SHAPES(X)
#undef X
  return false;
}

hipError_t attn_bwd_mfma(const AttnBwd& w, hipStream_t s) {
  hipError_t e = attn_delta(w, s);
  if (e != hipSuccess) return e;
#define X(a_, b_) if (w.f.dqk == a_ && w.f.dv == b_) return bwd_launch<a_, b_>(w, s);
  MLA_MFMA_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

hipError_t attn_fwd_mfma(const Attn& a, hipStream_t s) {
#define X(a_, b_) if (a.dqk == a_ && a.dv == b_) return fwd_launch<a_, b_>(a, s);
  MLA_MFMA_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace mla
