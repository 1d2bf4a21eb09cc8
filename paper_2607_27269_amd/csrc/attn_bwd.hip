// Causal softmax attention backward (gradients of Eq. 2-4) on gfx950 matrix cores.
#include "attn_common.h"
#include "mfma.h"
#include "simt.h"

namespace mla {
namespace attn {
namespace {

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

hipError_t bwd_dispatch(const AttnBwd& w, hipStream_t s) {
#define X(a_, b_) if (w.f.dqk == a_ && w.f.dv == b_) return bwd_launch<a_, b_>(w, s);
  MLA_MFMA_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace attn

hipError_t attn_bwd_mfma(const AttnBwd& w, hipStream_t s) {
  hipError_t e = attn_delta(w, s);
  if (e != hipSuccess) return e;
  return attn::bwd_dispatch(w, s);
}

}  // namespace mla
