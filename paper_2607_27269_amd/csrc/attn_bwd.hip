// Causal softmax attention backward (gradients of Eq. 2-4) on gfx950 matrix cores.
//
//   P = exp(S - lse) (recomputed from the forward's log-sum-exp), dV = P^T dO,
//   dP = dO V^T, dS = P (dP - delta) with delta = rowsum(dO . O),
//   dQ = scale dS K, dK = scale dS^T Q.
//
// Two kernels, each sized so that its accumulators stay in registers:
//
// * dK/dV: a workgroup owns 128 keys of one (sequence, KV group); each of its 4
//   wavefronts owns 32 keys (K staged once in LDS, V held as MFMA B-operand fragments) and walks
//   every 64-query block at or after its keys (last block first) and every head of the group.  S = Q K^T and
//   dP = dO V^T put the key in the MFMA column, so the accumulators of P and dS are
//   directly the B operands of dV^T += dO^T P and dK^T += Q^T dS; dO^T and Q^T come from
//   the natural [query][dim] LDS tiles through gfx950's transposing LDS read.  The rotary
//   part of dK is summed over the group's heads and left as an fp32 partial per group
//   (the positional key may be shared by several groups).
// * dV and dS^T, preferred when a dS^T buffer fits: the same walk (256 keys per
//   workgroup) computes only dV and stores dS^T in bf16, transposed through LDS so that
//   the stores run along key rows, zeros included wherever the dQ product below reads a
//   masked pair; dK = scale dS^T Q is then a GEMM as well.
// * dQ, preferred: dQ = scale dS K as a batched causal GEMM (one batch entry per
//   (sequence, head)) over the stored dS^T and the keys gathered per group into one
//   [token][group][dqk] tensor; no recomputation of S or dP.
// * dQ, when no dS^T buffer fits: a kernel laid out like the forward (a lane owns one
//   query; 4 wavefronts x 32 queries): S^T = K Q^T, dP^T = V dO^T, and dQ^T += K^T dS^T
//   with K^T read transposed from the [key][dim] tile, written once in bf16.
// Either way the rotary block of dQ is then rotated back with R^T.
#include "attn_common.h"
#include "mfma.h"
#include "simt.h"

namespace mla {
namespace attn {
namespace {

constexpr int BKB = 128;  // keys per dK/dV workgroup
constexpr int BQB = 64;   // queries per dK/dV step
constexpr int DQ_BQ = 128;  // queries per dQ workgroup

struct BwdDev {
  AttnDev f;
  const bf16_t* dO;      // [N][H*dv]
  const float* delta;    // [N][H]
  bf16_t* dq;            // [N][H*dqk]
  int rdiv;
  const float* cos_t;
  const float* sin_t;
  bf16_t* dKa; int64_t dka_tok;
  bf16_t* dV; int64_t dv_tok;
  float* dkb_part;       // [G][N][dqk - dnope]
  int G;                 // Ka groups
  float scale;
  bf16_t* dsT;           // [B*H][T][ds_ld] when ds_on
  int64_t ds_ld;
  int ds_on;
  bf16_t* ds_dummy;      // scratch rows for stores of lanes past the sequence end
  const float* statT;    // [2][H][B][tpad]: log2-scaled lse, delta (dV kernel)
  int tpad;
  int off32;             // one sequence's Q / dO rows and the statistics span < 2^31 bytes
};

// dS^T tile rows a dQ GEMM row tile reads: queries from the start of the 256-query tile
// that holds the key (the GEMM's row tile) to the end
constexpr int DQ_TILE = 256;

// ---------------------------------------------------------------------------------------
// dK / dV
// ---------------------------------------------------------------------------------------
template <int DQK, int DV, int BQ = BQB>
struct QStage {
  static constexpr int LDQ = ld_of(DQK);
  static constexpr int LDO = ld_of(DV);
  using QT = DmaTile<BQ, DQK, LDQ, 4>;
  using OT = DmaTile<BQ, DV, LDO, 4>;
  static constexpr int QS = QT::ALLOC, OS = OT::ALLOC;
  static constexpr int BUF = QS + OS + 2 * BQ * 2;  // bf16 elements incl. lse2, delta
  QT qt;
  OT ot;
  float stat;

  __device__ __forceinline__ void init() {
    qt.init();
    ot.init();
  }

  // queries q0 .. q0+BQ-1 of head i into buf (rows past the end load the last valid row;
  // their lse is +inf so they carry zero probability)
  __device__ __forceinline__ void issue(const BwdDev& w, int b, int i, int q0, bf16_t* buf) {
    const AttnDev& a = w.f;
    const int last = a.T - 1;
    const int64_t n0 = (int64_t)b * a.T;
    const bf16_t* qb = a.Q + n0 * a.q_tok + (int64_t)i * a.q_head;
    const bf16_t* ob = w.dO + n0 * ((int64_t)a.H * DV) + (int64_t)i * DV;
    qt.issue(buf, [&](int r, int c) { return qb + (int64_t)min(q0 + r, last) * a.q_tok + c; });
    ot.issue(buf + QS, [&](int r, int c) {
      return ob + (int64_t)min(q0 + r, last) * ((int64_t)a.H * DV) + c;
    });
    const int q = q0 + (int)(threadIdx.x % BQ);
    if (threadIdx.x < BQ)
      stat = q < a.T ? a.lse[(n0 + q) * a.H + i] * LOG2E : INFINITY;
    else if (threadIdx.x < 2 * BQ)
      stat = q < a.T ? w.delta[(n0 + q) * a.H + i] : 0.f;
  }

  __device__ __forceinline__ void store_stats(bf16_t* buf) const {
    float* st = (float*)(buf + QS + OS);
    if (threadIdx.x < 2 * BQ) st[threadIdx.x] = stat;
  }
};

// WITH_DK = false: dK is left to the GEMM over the stored dS^T (no dK accumulators here)
template <int DQK, int DV, bool WITH_DK>
__global__ __launch_bounds__(256) void attn_dkdv_mfma_kernel(BwdDev w) {
  using Stage = QStage<DQK, DV>;
  constexpr int LDQ = Stage::LDQ, LDO = Stage::LDO;
  constexpr int NKK = DQK / 16, NVK = DV / 16;
  constexpr int NCK = DQK / 32, NCV = DV / 32;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[2 * Stage::BUF + BKB * ld_of(DQK)];
  const AttnDev& a = w.f;

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

  // keys of this workgroup in LDS ([key][d], read as B operand fragments each step); this
  // lane's value as B operand fragments in registers (col = key, k = 16 kk + 8 half + 0..7)
  bf16_t* Ks = smem + 2 * Stage::BUF;
  {
    constexpr int KCH = BKB * (DQK / 8);
    const int ga = i0 / a.ka_div, gb = i0 / a.kb_div;
    for (int c = threadIdx.x; c < KCH; c += 256) {
      const int key = c / (DQK / 8), dc = (c % (DQK / 8)) * 8;
      const int j = k0 + key;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (j < a.T) {
        const int64_t n = (int64_t)b * a.T + j;
        const bf16_t* src = dc < a.dnope ? a.Ka + n * a.ka_tok + (int64_t)ga * a.ka_head + dc
                                         : a.Kb + n * a.kb_tok + (int64_t)gb * a.kb_head + (dc - a.dnope);
        val = *(const u32x4*)src;
      }
      *(u32x4*)(Ks + key * LDQ + dc) = val;
    }
  }
  // dS^T rows of this workgroup's keys: the queries in [tile start, k0) precede every key
  // here, so their entries are zeros that no step below writes
  const int zq0 = k0 / DQ_TILE * DQ_TILE;
  if (w.ds_on && zq0 < k0) {
    const int nz = k0 - zq0;                       // multiple of 128
    const int cpr = nz / 8;                        // 16-byte chunks per key row
    const int kr = min(BKB, a.T - k0);
    for (int h = 0; h < hpg; ++h) {
      bf16_t* plane = w.dsT + ((int64_t)b * a.H + i0 + h) * a.T * w.ds_ld;
      for (int c = threadIdx.x; c < kr * cpr; c += 256) {
        const int r = c / cpr, q = zq0 + (c % cpr) * 8;
        *(u32x4*)(plane + (int64_t)(k0 + r) * w.ds_ld + q) = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }
  const bf16_t* krow = Ks + (32 * wave + col) * LDQ + 8 * half;
  bf16x8 vf[NVK];
  {
    const int jj = min(my_key, a.T - 1);
    const int64_t n = (int64_t)b * a.T + jj;
    const int gv = i0 / a.v_div;
    const bf16_t* vp = a.V + n * a.v_tok + (int64_t)gv * a.v_head + 8 * half;
#pragma unroll
    for (int kk = 0; kk < NVK; ++kk) {
      u32x4 v = *(const u32x4*)(vp + 16 * kk);
      if (my_key >= a.T) v = u32x4{0u, 0u, 0u, 0u};
      vf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  constexpr int NCKA = WITH_DK ? NCK : 1;
  f32x16 dk[NCKA], dv[NCV];
#pragma unroll
  for (int c = 0; c < NCKA; ++c)
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
  Stage stg;
  stg.init();
  // step it -> (query block, head): query blocks in descending order with the group's heads
  // innermost, so that all key blocks of a (sequence, group) stream the same Q/dO tile at
  // the same time and share it through L2
  auto q_of = [&](int it) { return (nqb - 1 - it / hpg) * BQB; };
  auto h_of = [&](int it) { return i0 + it % hpg; };
  if (niter > 0) {
    stg.issue(w, b, h_of(0), q_of(0), smem);
    stg.store_stats(smem);
  }
  wait_all();
  __syncthreads();

  for (int it = 0; it < niter; ++it) {
    const int q0 = q_of(it);
    const bf16_t* Qs = smem + (it & 1) * Stage::BUF;
    const bf16_t* dOs = Qs + Stage::QS;
    const float* st_lse = (const float*)(dOs + Stage::OS);
    const float* st_dl = st_lse + BQB;
    if (it + 1 < niter)
      stg.issue(w, b, h_of(it + 1), q_of(it + 1), smem + ((it + 1) & 1) * Stage::BUF);

    // this lane's dS^T row segment for the block: queries q0 + 4 half + {0..3, 8..11, ...}
    // (a wave-uniform plane base and a 32-bit lane offset)
    bf16_t* dsplane = w.ds_on ? w.dsT + ((int64_t)b * a.H + h_of(it)) * a.T * w.ds_ld : nullptr;
    const uint32_t dsoff = (uint32_t)my_key * (uint32_t)w.ds_ld + (uint32_t)(q0 + 4 * half);
    const bool dsrow = dsplane != nullptr && my_key < a.T;
    if (kw0 <= min(q0 + BQB - 1, a.T - 1)) {  // wave-uniform: some pair is visible
      f32x16 sp[2], dp[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int e = 0; e < 16; ++e) { sp[qt][e] = 0.f; dp[qt][e] = 0.f; }
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        const bf16x8 kf = *(const bf16x8*)(krow + 16 * kk);
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
          sp[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              *(const bf16x8*)(Qs + (32 * qt + col) * LDQ + 16 * kk + 8 * half), kf, sp[qt], 0, 0, 0);
      }
#pragma unroll
      for (int kk = 0; kk < NVK; ++kk)
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
          dp[qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              *(const bf16x8*)(dOs + (32 * qt + col) * LDO + 16 * kk + 8 * half), vf[kk], dp[qt], 0, 0, 0);
      // P = 2^(S sl2 - lse2), dS = P (dP - delta); rows q = q0 + 32 qt + 8(e/4) + 4 half + e%4
      const bool diag = kw0 + 31 > q0;
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int qr = 32 * qt + 8 * e4 + 4 * half;
          const f32x4 l2 = *(const f32x4*)(st_lse + qr);
          const f32x4 dl = *(const f32x4*)(st_dl + qr);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int e = 4 * e4 + r;
            float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sp[qt][e], a.sl2, -l2[r]));
            if (diag && my_key > q0 + qr + r) p = 0.f;
            sp[qt][e] = p;
            dp[qt][e] = p * (dp[qt][e] - dl[r]);
          }
        }
      // dS^T in bf16: element e of tile qt is query 32 qt + 8 (e/4) + 4 half + e%4
      if (dsrow) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt)
#pragma unroll
          for (int e4 = 0; e4 < 4; ++e4)
            st_global8(dsplane + dsoff + (32 * qt + 8 * e4),
                       u32x2{pack2bf(dp[qt][4 * e4], dp[qt][4 * e4 + 1]),
                             pack2bf(dp[qt][4 * e4 + 2], dp[qt][4 * e4 + 3])});
      }
      // dV^T += dO^T P,  dK^T += Q^T dS   (K-step u: queries 32(u/2) + 16(u%2) + {4h.., 8+4h..})
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        u32x4 wp, wd;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          wp[q] = pack2bf(sp[u >> 1][8 * (u & 1) + 2 * q], sp[u >> 1][8 * (u & 1) + 2 * q + 1]);
          wd[q] = pack2bf(dp[u >> 1][8 * (u & 1) + 2 * q], dp[u >> 1][8 * (u & 1) + 2 * q + 1]);
        }
        const bf16x8 pf = __builtin_bit_cast(bf16x8, wp), sf = __builtin_bit_cast(bf16x8, wd);
        const int klo = 32 * (u >> 1) + 16 * (u & 1) + 4 * half;
#pragma unroll
        for (int c = 0; c < NCV; ++c)
          dv[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_operand_tr(dOs, LDO, 32 * c, klo, klo + 8),
                                                         pf, dv[c], 0, 0, 0);
        if constexpr (WITH_DK) {
#pragma unroll
          for (int c = 0; c < NCK; ++c)
            dk[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                lds_operand_tr(Qs, LDQ, 32 * c, klo, klo + 8), sf, dk[c], 0, 0, 0);
        }
      }
    } else if (dsrow) {
      // every key of this wavefront follows every query of the block: zeros
#pragma unroll
      for (int o = 0; o < BQB; o += 8) st_global8(dsplane + dsoff + o, u32x2{0u, 0u});
    }
    if (it + 1 < niter) stg.store_stats(smem + ((it + 1) & 1) * Stage::BUF);
    wait_all();
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
  if constexpr (!WITH_DK) return;
  const float sc = w.scale;
#pragma unroll
  for (int c = 0; c < NCKA; ++c)
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const int d = 32 * c + 8 * e4 + 4 * half;
      if (d < a.dnope) {
        u32x2 wv = {pack2bf(sc * dk[c][4 * e4], sc * dk[c][4 * e4 + 1]),
                    pack2bf(sc * dk[c][4 * e4 + 2], sc * dk[c][4 * e4 + 3])};
        *(u32x2*)(w.dKa + n * w.dka_tok + (int64_t)g * a.dnope + d) = wv;
      } else {
        f32x4 v = {sc * dk[c][4 * e4], sc * dk[c][4 * e4 + 1], sc * dk[c][4 * e4 + 2], sc * dk[c][4 * e4 + 3]};
        *(f32x4*)(w.dkb_part + ((int64_t)g * ((int64_t)a.B * a.T) + n) * dr + (d - a.dnope)) = v;
      }
    }
}

// ---------------------------------------------------------------------------------------
// dV and dS^T (the path where dK and dQ are GEMMs over the stored dS^T)
// ---------------------------------------------------------------------------------------
// A workgroup owns 256 keys of one (sequence, KV group), 32 per wavefront (8 wavefronts,
// one workgroup per CU), and walks the group's heads and 32-query blocks.  K and V of the
// lane's key are B-operand fragments held in registers; only the 32-query Q / dO tiles
// and their softmax statistics pass through LDS, in a ring of two stages, each block's
// copy issued one step before its use; the more keys share a copied tile, the fewer
// copies per key.  Every wavefront issues the same number of copies per stage (the block
// count is padded) and of dS^T stores per step, so one counter wait names exactly the
// copies that must have landed.
constexpr int DV_BQ = 32;
// dS^T stores per lane per step: a wavefront's 32 x 32 block is transposed through a
// private LDS tile so that each 16-byte store continues its neighbours' along a key row
// (4 lanes write a row's 64 bytes)
constexpr int DS_STORES = DV_BQ * 32 * 2 / (64 * 16);
constexpr int DV_NST = 2;  // LDS stages: a step's copies are issued one step ahead
#ifndef DV_WAVES_OVERRIDE
constexpr int DV_WAVES = 8;
#else
constexpr int DV_WAVES = DV_WAVES_OVERRIDE;
#endif
constexpr int DV_BKB = 32 * DV_WAVES;  // keys per workgroup

// [2][H][B][Tpad] fp32: log2-scaled lse (+inf past the sequence end) and delta (0 there)
__global__ void attn_stats_t_kernel(const float* __restrict__ lse, const float* __restrict__ delta,
                                    int B, int T, int H, int Tpad, float* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = 2LL * H * B * Tpad;
  if (idx >= total) return;
  const int q = (int)(idx % Tpad);
  const int64_t r = idx / Tpad;
  const int b = (int)(r % B);
  const int h = (int)((r / B) % H);
  const int part = (int)(r / ((int64_t)B * H));
  float v;
  if (q < T) {
    const int64_t src = ((int64_t)b * T + q) * H + h;
    v = part == 0 ? lse[src] * LOG2E : delta[src];
  } else {
    v = part == 0 ? INFINITY : 0.f;
  }
  out[idx] = v;
}

template <int DQK, int DV>
struct DvStage {
  static constexpr int LDQ = ld_of(DQK);
  static constexpr int LDO = ld_of(DV);
  static constexpr int NQB = (DV_BQ * LDQ * 2 + 1023) / 1024;  // 1 KB blocks of the Q tile
  static constexpr int NOB = (DV_BQ * LDO * 2 + 1023) / 1024;  // ... of the dO tile
  static constexpr int NB = (NQB + NOB + 1 + DV_WAVES - 1) / DV_WAVES * DV_WAVES;  // + stats, padded
  static constexpr int PER = NB / DV_WAVES;                   // copies per wavefront
  static constexpr int OFF_O = NQB * 512, OFF_S = (NQB + NOB) * 512;  // bf16 elements
  static constexpr int ELEMS = NB * 512;

  // block blk = wave + DV_WAVES p: its kind is wave-uniform (blk < NQB: Q, < NQB + NOB: dO, then
  // the statistics block, then padding that re-copies Q row 0 into unused LDS).  A full
  // block (all 32 queries inside the sequence) is copied from wave-uniform row bases with
  // loop-invariant lane offsets, computed once (init); the last, partial block clamps rows
  // to the sequence end.
  uint32_t voff[PER];  // byte offset of this lane's chunk from its block's row base
  // with 32-bit row offsets (off32): each copy's base is fixed for the kernel (Q or dO of
  // the sequence, or the statistics of the sequence) and a step adds a uniform 32-bit row
  // offset, instead of 64-bit row addresses per step
  const void* pbase[PER];
  int pkind[PER];  // 0: Q (and padding), 1: dO, 2: statistics
  __device__ __forceinline__ void init(const BwdDev& w, int b) {
    const AttnDev& a = w.f;
    const int wave = wave_id(), lane = threadIdx.x & 63;
    const int64_t n0 = (int64_t)b * a.T;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int blk = wave + DV_WAVES * p;
      pkind[p] = blk < NQB ? 0 : blk < NQB + NOB ? 1 : blk == NQB + NOB ? 2 : 0;
      pbase[p] = pkind[p] == 0   ? (const void*)(a.Q + n0 * a.q_tok)
                 : pkind[p] == 1 ? (const void*)(w.dO + n0 * (int64_t)a.H * DV)
                                 : (const void*)(w.statT + (int64_t)b * w.tpad);
    }
    const int64_t o_tok = (int64_t)a.H * DV;
    const uint32_t s_part = (uint32_t)a.H * a.B * w.tpad * 4;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int blk = wave + DV_WAVES * p;
      uint32_t off = 0u;
      if (blk < NQB) {
        const int e = (blk * 1024 + 16 * lane) / 2;
        const int r = min(e / LDQ, DV_BQ - 1), c0 = e % LDQ, c = c0 < DQK ? c0 : 0;
        off = 2u * (uint32_t)(r * (int)a.q_tok + c);
      } else if (blk < NQB + NOB) {
        const int e = ((blk - NQB) * 1024 + 16 * lane) / 2;
        const int r = min(e / LDO, DV_BQ - 1), c0 = e % LDO, c = c0 < DV ? c0 : 0;
        off = 2u * (uint32_t)(r * (int)o_tok + c);
      } else if (blk == NQB + NOB) {
        off = ((lane >> 3) & 1) * s_part + 16u * (lane & 7);
      }
      voff[p] = off;
    }
  }
  __device__ __forceinline__ void issue(const BwdDev& w, int b, int h, int q0, bf16_t* stage) const {
    const AttnDev& a = w.f;
    const int wave = wave_id();
    // opaque copy of the lane id: the clamped path below recomputes its lane offsets at
    // every issue instead of keeping them live across the loop
    int lane = threadIdx.x & 63;
    asm volatile("" : "+v"(lane));
    const int last = a.T - 1;
    const int64_t n0 = (int64_t)b * a.T;
    const int64_t o_tok = (int64_t)a.H * DV;
    const float* sbase = w.statT + ((int64_t)h * a.B + b) * w.tpad + q0;  // lse2 row
    const uint32_t s_part = (uint32_t)a.H * a.B * w.tpad * 4;          // lse2 -> delta bytes
    if (w.off32 && q0 + DV_BQ - 1 <= last) {
      const uint32_t qo = 2u * ((uint32_t)q0 * (uint32_t)a.q_tok + (uint32_t)(h * a.q_head));
      const uint32_t oo = 2u * ((uint32_t)q0 * (uint32_t)(a.H * DV) + (uint32_t)(h * DV));
      const uint32_t so = 4u * ((uint32_t)(h * a.B) * (uint32_t)w.tpad + (uint32_t)q0);
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int blk = wave + DV_WAVES * p;
        const uint32_t ro = pkind[p] == 0 ? qo : pkind[p] == 1 ? oo : so;
        dma16_s(pbase[p], voff[p] + ro, stage + blk * 512);
      }
      return;
    }
    if (q0 + DV_BQ - 1 <= last) {
      const bf16_t* qrow = a.Q + (n0 + q0) * a.q_tok + (int64_t)h * a.q_head;
      const bf16_t* orow = w.dO + (n0 + q0) * o_tok + (int64_t)h * DV;
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int blk = wave + DV_WAVES * p;
        // statistics block: lanes 0-7 lse2 of queries q0 + 4 l .. + 3, lanes 8-15 delta, the
        // rest repeat; padding blocks re-copy Q row 0 (offset 0)
        const void* base = blk < NQB ? (const void*)qrow
                           : blk < NQB + NOB ? (const void*)orow
                           : blk == NQB + NOB ? (const void*)sbase : (const void*)qrow;
        dma16_s(base, voff[p], stage + blk * 512);
      }
      return;
    }
    const bf16_t* qb = a.Q + n0 * a.q_tok + (int64_t)h * a.q_head;
    const bf16_t* ob = w.dO + n0 * o_tok + (int64_t)h * DV;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int blk = wave + DV_WAVES * p;
      const bf16_t* src;
      if (blk < NQB) {
        const int e = (blk * 1024 + 16 * lane) / 2;
        const int r = min(e / LDQ, DV_BQ - 1), c0 = e % LDQ, c = c0 < DQK ? c0 : 0;
        src = qb + (int64_t)min(q0 + r, last) * a.q_tok + c;
      } else if (blk < NQB + NOB) {
        const int e = ((blk - NQB) * 1024 + 16 * lane) / 2;
        const int r = min(e / LDO, DV_BQ - 1), c0 = e % LDO, c = c0 < DV ? c0 : 0;
        src = ob + (int64_t)min(q0 + r, last) * o_tok + c;
      } else if (blk == NQB + NOB) {
        const int part = (lane >> 3) & 1, c = 4 * (lane & 7);
        src = (const bf16_t*)(sbase + (int64_t)part * a.H * a.B * w.tpad + c);
      } else {
        src = qb + (int64_t)min(q0, last) * a.q_tok;
      }
      dma16(src, stage + blk * 512);
    }
  }
};

template <int DQK, int DV>
__global__ __launch_bounds__(64 * DV_WAVES, 8 / DV_WAVES) void attn_dv_mfma_kernel(BwdDev w) {
  using Stage = DvStage<DQK, DV>;
  constexpr int LDQ = Stage::LDQ, LDO = Stage::LDO;
  constexpr int NKK = DQK / 16, NVK = DV / 16, NCV = DV / 32;
  constexpr int D = Stage::PER;
  static_assert(DS_STORES < 64, "counter range");
  // the Q / dO ring, then one 32 x 32 dS^T transpose tile per wavefront
  __shared__ __attribute__((aligned(1024))) bf16_t smem[DV_NST * Stage::ELEMS + DV_WAVES * 32 * DV_BQ];
  const AttnDev& a = w.f;

  const int nbg = a.B * w.G;
  const int kb = blockIdx.x / nbg;  // early key blocks (the most query blocks) first
  const int bg = blockIdx.x % nbg;
  const int b = bg / w.G, g = bg % w.G;
  const int hpg = a.H / w.G;
  const int k0 = kb * DV_BKB;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5, col = lane & 31;
  const int kw0 = k0 + 32 * wave;
  const int my_key = kw0 + col;
  const int i0 = g * hpg;

  // dS^T rows of this workgroup's keys: the queries in [tile start, k0) precede every key
  // here, so their entries are zeros that no step below writes
  const int zq0 = k0 / DQ_TILE * DQ_TILE;
  if (zq0 < k0) {
    const int nz = k0 - zq0;                       // multiple of the key block
    const int cpr = nz / 8;                        // 16-byte chunks per key row
    const int kr = min(DV_BKB, a.T - k0);
    for (int h = 0; h < hpg; ++h) {
      bf16_t* plane = w.dsT + ((int64_t)b * a.H + i0 + h) * a.T * w.ds_ld;
      for (int c = threadIdx.x; c < kr * cpr; c += 64 * DV_WAVES) {
        const int r = c / cpr, q = zq0 + (c % cpr) * 8;
        *(u32x4*)(plane + (int64_t)(k0 + r) * w.ds_ld + q) = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }

  // this lane's key and value as B operand fragments (col = key, k = 16 kk + 8 half + 0..7)
  bf16x8 kf[NKK], vf[NVK];
  {
    const int jj = min(my_key, a.T - 1);
    const int64_t n = (int64_t)b * a.T + jj;
    const int ga = i0 / a.ka_div, gb = i0 / a.kb_div, gv = i0 / a.v_div;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const int d = 16 * kk + 8 * half;
      const bf16_t* src = d < a.dnope ? a.Ka + n * a.ka_tok + (int64_t)ga * a.ka_head + d
                                      : a.Kb + n * a.kb_tok + (int64_t)gb * a.kb_head + (d - a.dnope);
      kf[kk] = *(const bf16x8*)src;
    }
    const bf16_t* vp = a.V + n * a.v_tok + (int64_t)gv * a.v_head + 8 * half;
#pragma unroll
    for (int kk = 0; kk < NVK; ++kk) vf[kk] = *(const bf16x8*)(vp + 16 * kk);
  }

  f32x16 dv[NCV];
#pragma unroll
  for (int c = 0; c < NCV; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) dv[c][e] = 0.f;

  const int qb0 = k0 / DV_BQ;
  const int nqb = (a.T + DV_BQ - 1) / DV_BQ;
  const int nper = nqb - qb0;
  const int niter = hpg * nper;  // >= 1
  Stage stg;
  stg.init(w, b);
  // steps walk (query block, head): query blocks in descending order with the group's heads
  // innermost, so that all key blocks of a (sequence, group) stream the same Q/dO tile at
  // the same time and share it through L2.  (qc, hc) is this step's pair, (qn, hn) the
  // next one (the last step's "next" re-copies the last pair into the free stage).
  int qc = (nqb - 1) * DV_BQ, hc = i0;
  int qn = qc, hn = hc;
  auto advance = [&](int& q, int& h) {
    if (++h == i0 + hpg) { h = i0; q -= DV_BQ; }
  };
  if (niter > 1) advance(qn, hn);
  auto stage_of = [&](int it) { return smem + (it & 1) * Stage::ELEMS; };
  bf16_t* scratch = w.ds_dummy + 64 * lane;
  // transpose tile: key row r holds 64 bytes (32 queries) as four 16-byte segments, segment
  // s stored at position s ^ ((r / 4) % 4) (the packed writes of 32 rows at one segment
  // spread over the banks; the 16-byte reads of 4 consecutive rows are conflict-free)
  bf16_t* tr = smem + DV_NST * Stage::ELEMS + wave * 32 * DV_BQ;
  static_assert(DV_BQ == 32 && DS_STORES == 2, "transpose tile layout");
  // reader side: lane handles rows rr + 16 j (j < 2), queries 8 sg .. 8 sg + 7
  const int rr = lane >> 2, sg = lane & 3;
  stg.issue(w, b, hc, qc, stage_of(0));
  wait_vm<0>();
  lds_barrier();

  for (int it = 0; it < niter; ++it) {
    const int q0 = qc;
    const bf16_t* Qs = stage_of(it);
    const bf16_t* dOs = Qs + Stage::OFF_O;
    const float* st_lse = (const float*)(Qs + Stage::OFF_S);
    const float* st_dl = st_lse + DV_BQ;
    // the stage of step it - 1 is free: every wave passed the barrier after reading it
    stg.issue(w, b, hn, qn, stage_of(it + 1));

    // this lane's dS^T store targets for the block: key rows kw0 + rr + 16 j, queries
    // q0 + 8 sg .. + 7; rows past the sequence end go to a scratch row instead, so that every
    // wavefront issues exactly DS_STORES stores per step
    // (computed where the stores are issued: short-lived registers)
    auto dst = [&](int j) {
      const int key = kw0 + rr + 16 * j;
      return key < a.T ? w.dsT + ((int64_t)b * a.H + hc) * a.T * w.ds_ld + (int64_t)key * w.ds_ld +
                             q0 + 8 * sg
                       : scratch + 8 * sg;
    };
    if (kw0 <= min(q0 + DV_BQ - 1, a.T - 1)) {  // wave-uniform: some pair is visible
      f32x16 sp, dp;
#pragma unroll
      for (int e = 0; e < 16; ++e) { sp[e] = 0.f; dp[e] = 0.f; }
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk)
        sp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            *(const bf16x8*)(Qs + col * LDQ + 16 * kk + 8 * half), kf[kk], sp, 0, 0, 0);
#pragma unroll
      for (int kk = 0; kk < NVK; ++kk)
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            *(const bf16x8*)(dOs + col * LDO + 16 * kk + 8 * half), vf[kk], dp, 0, 0, 0);
      // P = 2^(S sl2 - lse2), dS = P (dP - delta); rows q = q0 + 8(e/4) + 4 half + e%4
      // (lse2 = +inf past the sequence end)
      const bool diag = kw0 + 31 > q0;
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int qr = 8 * e4 + 4 * half;
        const f32x4 l2 = *(const f32x4*)(st_lse + qr);
        const f32x4 dl = *(const f32x4*)(st_dl + qr);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * e4 + r;
          float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sp[e], a.sl2, -l2[r]));
          if (diag && my_key > q0 + qr + r) p = 0.f;
          sp[e] = p;
          dp[e] = p * (dp[e] - dl[r]);
        }
      }
      // dS^T in bf16: element e is query 8 (e/4) + 4 half + e%4 of key row col, i.e. half
      // h of 16-byte segment e/4; through the transpose tile to row-contiguous stores
      // (LDS operations of one wavefront complete in order: the reads see the writes, and
      // the next step's writes follow these reads)
      asm volatile("" ::: "memory");
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4)
        *(u32x2*)(tr + col * DV_BQ + 8 * (e4 ^ ((col >> 2) & 3)) + 4 * half) =
            u32x2{pack2bf(dp[4 * e4], dp[4 * e4 + 1]), pack2bf(dp[4 * e4 + 2], dp[4 * e4 + 3])};
      asm volatile("" ::: "memory");
      // dV^T += dO^T P   (K-step u: queries 16 u + {4h.., 8+4h..})
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 wp;
#pragma unroll
        for (int q = 0; q < 4; ++q) wp[q] = pack2bf(sp[8 * u + 2 * q], sp[8 * u + 2 * q + 1]);
        const bf16x8 pf = __builtin_bit_cast(bf16x8, wp);
        const int klo = 16 * u + 4 * half;
#pragma unroll
        for (int c = 0; c < NCV; ++c)
          dv[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_operand_tr(dOs, LDO, 32 * c, klo, klo + 8),
                                                         pf, dv[c], 0, 0, 0);
      }
      asm volatile("" ::: "memory");
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int r = rr + 16 * j;
        st_global16(dst(j), *(const u32x4*)(tr + r * DV_BQ + 8 * (sg ^ ((r >> 2) & 3))));
      }
      asm volatile("" ::: "memory");
    } else {
      // every key of this wavefront follows every query of the block: zeros
#pragma unroll
      for (int j = 0; j < 2; ++j) st_global16(dst(j), u32x4{0u, 0u, 0u, 0u});
    }
    // step it + 1's copies have landed; younger are only this step's stores (counters
    // complete in issue order)
    wait_vm<DS_STORES>();
    lds_barrier();
    qc = qn;
    hc = hn;
    if (it + 2 < niter) advance(qn, hn);
  }

  // epilogue: this lane's key; rows d = 32c + 8(e/4) + 4 half + e%4
  if (my_key >= a.T) return;
  const int64_t n = (int64_t)b * a.T + my_key;
#pragma unroll
  for (int c = 0; c < NCV; ++c)
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const int d = 32 * c + 8 * e4 + 4 * half;
      u32x2 wv = {pack2bf(dv[c][4 * e4], dv[c][4 * e4 + 1]), pack2bf(dv[c][4 * e4 + 2], dv[c][4 * e4 + 3])};
      *(u32x2*)(w.dV + n * w.dv_tok + (int64_t)g * DV + d) = wv;
    }
}

// ---------------------------------------------------------------------------------------
// dQ
// ---------------------------------------------------------------------------------------
template <int DQK, int DV>
__global__ __launch_bounds__(256) void attn_dq_mfma_kernel(BwdDev w) {
  using Stage = KVStage<DQK, DV, 4>;
  constexpr int LDK = Stage::LDK, LDV = Stage::LDV;
  constexpr int KS = Stage::KS, VS = Stage::VS;
  constexpr int NKK = DQK / 16, NVK = DV / 16, NCK = DQK / 32;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[2 * (KS + VS)];
  const AttnDev& a = w.f;

  const int nqb = (a.T + DQ_BQ - 1) / DQ_BQ;
  const int nwork = a.B * a.H * nqb;
  const int pid = xcd_remap(blockIdx.x, nwork);
  const int bh = pid / nqb;
  const int qb = nqb - 1 - pid % nqb;
  const int b = bh / a.H, i = bh % a.H;
  const int q0 = qb * DQ_BQ;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5, col = lane & 31;
  const int qw0 = q0 + 32 * wave;
  const int my_q = qw0 + col;
  const bool qvalid = my_q < a.T;
  const int64_t nq = (int64_t)b * a.T + min(my_q, a.T - 1);

  // this lane's query and output gradient as B operand fragments (col = query)
  bf16x8 qf[NKK], of[NVK];
  {
    const bf16_t* qp = a.Q + nq * a.q_tok + (int64_t)i * a.q_head + 8 * half;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[kk] = *(const bf16x8*)(qp + 16 * kk);
    const bf16_t* op = w.dO + nq * ((int64_t)a.H * DV) + (int64_t)i * DV + 8 * half;
#pragma unroll
    for (int kk = 0; kk < NVK; ++kk) of[kk] = *(const bf16x8*)(op + 16 * kk);
  }
  const float lse2 = qvalid ? a.lse[nq * a.H + i] * LOG2E : INFINITY;
  const float dlt = qvalid ? w.delta[nq * a.H + i] : 0.f;

  f32x16 dq[NCK];
#pragma unroll
  for (int c = 0; c < NCK; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) dq[c][e] = 0.f;

  const int kend = min(a.T, q0 + DQ_BQ);
  const int nkb = (kend + BKV - 1) / BKV;
  Stage st;
  st.init(a, b, i);
  st.issue(0, smem, smem + KS);
  wait_all();
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const int j0 = kb * BKV;
    if (kb + 1 < nkb) {
      bf16_t* nxt = smem + (cur ^ 1) * (KS + VS);
      st.issue(j0 + BKV, nxt, nxt + KS);
    }
    const bf16_t* ks = smem + cur * (KS + VS);
    const bf16_t* vs = ks + KS;
    if (j0 <= qw0 + 31) {
      f32x16 s[2], dp[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) { s[t][e] = 0.f; dp[t][e] = 0.f; }
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
        for (int t = 0; t < 2; ++t)
          s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              *(const bf16x8*)(ks + (32 * t + col) * LDK + 16 * kk + 8 * half), qf[kk], s[t], 0, 0, 0);
#pragma unroll
      for (int kk = 0; kk < NVK; ++kk)
#pragma unroll
        for (int t = 0; t < 2; ++t)
          dp[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              *(const bf16x8*)(vs + (32 * t + col) * LDV + 16 * kk + 8 * half), of[kk], dp[t], 0, 0, 0);
      const bool diag = j0 + BKV - 1 > qw0;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[t][e], a.sl2, -lse2));
          if (diag && j0 + 32 * t + 8 * (e >> 2) + 4 * half + (e & 3) > my_q) p = 0.f;
          dp[t][e] = p * (dp[t][e] - dlt);
        }
      // dQ^T += K^T dS^T; K-step u covers keys 32(u/2) + 16(u%2) + {4h.., 8+4h..}
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        u32x4 wd;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          wd[q] = pack2bf(dp[u >> 1][8 * (u & 1) + 2 * q], dp[u >> 1][8 * (u & 1) + 2 * q + 1]);
        const bf16x8 sf = __builtin_bit_cast(bf16x8, wd);
        const int klo = 32 * (u >> 1) + 16 * (u & 1) + 4 * half;
#pragma unroll
        for (int c = 0; c < NCK; ++c)
          dq[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_operand_tr(ks, LDK, 32 * c, klo, klo + 8),
                                                         sf, dq[c], 0, 0, 0);
      }
    }
    wait_all();
    __syncthreads();
  }

  // epilogue: rows d = 32c + 8(e/4) + 4 half + e%4 of this lane's query (the rotary block is
  // rotated back by the caller's R^T pass)
  if (!qvalid) return;
  const float sc = w.scale;
  bf16_t* dst = w.dq + nq * ((int64_t)a.H * DQK) + (int64_t)i * DQK + 4 * half;
#pragma unroll
  for (int c = 0; c < NCK; ++c)
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      u32x2 wv = {pack2bf(sc * dq[c][4 * e4], sc * dq[c][4 * e4 + 1]),
                  pack2bf(sc * dq[c][4 * e4 + 2], sc * dq[c][4 * e4 + 3])};
      *(u32x2*)(dst + 32 * c + 8 * e4) = wv;
    }
}

// kcat[n][g][d] = the logit key of Ka group g at token n: d < dnope from Ka, the rest from
// Kb (rope group of the group's first head); 8 elements per thread
__global__ void kcat_kernel(AttnDev a, int G, int DQK, bf16_t* __restrict__ out) {
  const int cpr = DQK / 8;
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)a.B * a.T * G * cpr;
  if (c >= total) return;
  const int d = (int)(c % cpr) * 8;
  const int64_t ng = c / cpr;
  const int g = (int)(ng % G);
  const int64_t n = ng / G;
  const int i = g * (a.H / G);
  const bf16_t* src = d < a.dnope
                          ? a.Ka + n * a.ka_tok + (int64_t)(i / a.ka_div) * a.ka_head + d
                          : a.Kb + n * a.kb_tok + (int64_t)(i / a.kb_div) * a.kb_head + (d - a.dnope);
  *(u32x4*)(out + ng * DQK + d) = *(const u32x4*)src;
}

// dK of the GEMM ([N][G][DQK] fp32) split into the layouts the caller expects: the first
// dnope dims in bf16 at dKa[n*dka_tok + g*dnope + d], the rest as the per-group fp32
// partials dkb_part[g][n][d - dnope]; 4 elements per thread
__global__ void dk_split_kernel(const float* __restrict__ dk, int64_t N, int G, int DQK,
                                int dnope, bf16_t* __restrict__ dKa, int64_t dka_tok,
                                float* __restrict__ dkb_part) {
  const int cpr = DQK / 4;
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= N * G * cpr) return;
  const int d = (int)(c % cpr) * 4;
  const int64_t ng = c / cpr;
  const int g = (int)(ng % G);
  const int64_t n = ng / G;
  const f32x4 v = *(const f32x4*)(dk + ng * DQK + d);
  if (d < dnope) {
    *(u32x2*)(dKa + n * dka_tok + (int64_t)g * dnope + d) = u32x2{pack2bf(v[0], v[1]), pack2bf(v[2], v[3])};
  } else {
    *(f32x4*)(dkb_part + ((int64_t)g * N + n) * (DQK - dnope) + (d - dnope)) = v;
  }
}

template <int DQK, int DV>
hipError_t bwd_launch(const AttnBwd& wb, hipStream_t s) {
  const Attn& at = wb.f;
  BwdDev w;
  w.f = to_dev(at);
  w.dO = (const bf16_t*)wb.dO; w.delta = wb.delta;
  w.dq = (bf16_t*)wb.dq; w.rdiv = wb.rdiv; w.cos_t = wb.cos_t; w.sin_t = wb.sin_t;
  w.dKa = (bf16_t*)wb.dKa; w.dka_tok = wb.dka_tok;
  w.dV = (bf16_t*)wb.dV; w.dv_tok = wb.dv_tok;
  w.dkb_part = wb.dkb_part; w.G = wb.n_ka_groups; w.scale = at.scale;
  const bool ds_path = wb.dsT != nullptr && wb.kcat != nullptr && wb.dk_tmp != nullptr &&
                       wb.statT != nullptr;
  w.dsT = (bf16_t*)wb.dsT;
  w.ds_on = ds_path ? 1 : 0;
  w.ds_ld = attn_ds_ld(at.T);
  w.ds_dummy = w.dsT + (ds_path ? (int64_t)at.B * at.H * at.T * w.ds_ld : 0);
  w.statT = wb.statT;
  w.tpad = attn_stats_tpad(at.T);
  w.off32 = (int64_t)at.T * at.Q.tok * 2 < (1ll << 31) &&
            (int64_t)at.T * at.H * at.dv * 2 < (1ll << 31) &&
            (int64_t)at.H * at.B * w.tpad * 4 * 2 < (1ll << 31);
  const double pairs = attn_causal_pairs(at);
  const double N = (double)at.B * at.T;
  // delta = rowsum(dO . O), then the dK/dV kernel: algorithmic dV = P^T dO, dP = dO V^T,
  // dK = dS^T Q; reads Q, dO, K, V, lse, delta once, writes dK, dV
  prof_begin(KC_ELEM, s);
  hipError_t e = attn_delta(wb, s);
  prof_end(KC_ELEM, s, 0.0, N * at.H * (2.0 * DV * 2.0 + 4.0));
  if (e != hipSuccess) return e;
  const int nkb = (at.T + BKB - 1) / BKB;
  const int hpg = at.H / w.G;
  if (ds_path) {
    // statistics per (head, sequence) in query order, then dV (and dS^T) from the fused
    // kernel: algorithmic dV = P^T dO, dP = dO V^T
    prof_begin(KC_ELEM, s);
    const int64_t nst = 2LL * at.H * at.B * w.tpad;
    attn_stats_t_kernel<<<(unsigned)((nst + 255) / 256), 256, 0, s>>>(at.lse, wb.delta, at.B, at.T, at.H,
                                                                      w.tpad, wb.statT);
    prof_end(KC_ELEM, s, 0.0, nst * 4.0 * 2.0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    prof_begin(KC_ATTN_DKDV, s);
    const int nkb_dv = (at.T + DV_BKB - 1) / DV_BKB;
    attn_dv_mfma_kernel<DQK, DV><<<nkb_dv * at.B * w.G, 64 * DV_WAVES, 0, s>>>(w);
    prof_end(KC_ATTN_DKDV, s, 2.0 * pairs * (2.0 * DV),
             N * at.H * (DQK + DV) * 2.0 + N * w.G * (DQK + DV) * 2.0 + N * at.H * 8.0 +
                 pairs * 2.0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // dK = scale dS^T Q per (sequence, group), the group's heads stacked along K:
    // algorithmic dS read once, Q read once, dK written once (fp32)
    {
      Gemm g;
      g.M = at.T; g.N = DQK; g.K = at.T;
      g.A = wb.dsT; g.lda = w.ds_ld; g.a_kmajor = true;
      g.B = at.Q.p; g.ldb = at.Q.tok; g.b_kmajor = false;
      g.C = wb.dk_tmp; g.ldc = (int64_t)w.G * DQK;
      g.in_t = DT_BF16; g.c_t = DT_F32; g.alpha = at.scale; g.beta = 0.f;
      GemmBatch bt;
      bt.nbatch = at.B * w.G; bt.zdiv = w.G; bt.bdiv = 1; bt.mstore = at.T;
      bt.rev = 1; bt.kgroups = hpg;
      bt.sA = (int64_t)hpg * at.T * w.ds_ld; bt.sAk = (int64_t)at.T * w.ds_ld;
      bt.sB1 = (int64_t)at.T * at.Q.tok; bt.sB2 = (int64_t)hpg * at.Q.head; bt.sBk = at.Q.head;
      bt.sC1 = (int64_t)at.T * w.G * DQK; bt.sC2 = DQK;
      prof_begin(KC_ATTN_DK, s);
      e = gemm_mfma_causal(g, bt, s);
      prof_end(KC_ATTN_DK, s, 2.0 * pairs * DQK, pairs * 2.0 + N * at.H * DQK * 2.0 + N * w.G * DQK * 4.0);
      if (e != hipSuccess) return e;
      prof_begin(KC_ELEM, s);
      const int64_t chunks = (int64_t)at.B * at.T * w.G * (DQK / 4);
      dk_split_kernel<<<(unsigned)((chunks + 255) / 256), 256, 0, s>>>(
          wb.dk_tmp, (int64_t)at.B * at.T, w.G, DQK, at.dnope, w.dKa, w.dka_tok, w.dkb_part);
      prof_end(KC_ELEM, s, 0.0, N * w.G * DQK * 4.0 * 2.0);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    // keys of each group gathered into one operand, then dQ = scale dS K per (sequence,
    // head): algorithmic dS read once, K read once per head, dQ written once
    prof_begin(KC_ELEM, s);
    const int64_t chunks = (int64_t)at.B * at.T * w.G * (DQK / 8);
    kcat_kernel<<<(unsigned)((chunks + 255) / 256), 256, 0, s>>>(w.f, w.G, DQK, (bf16_t*)wb.kcat);
    prof_end(KC_ELEM, s, 0.0, N * w.G * DQK * 2.0 * 2.0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    Gemm g;
    g.M = (int)w.ds_ld; g.N = DQK; g.K = at.T;
    g.A = wb.dsT; g.lda = w.ds_ld; g.a_kmajor = false;
    g.B = wb.kcat; g.ldb = (int64_t)w.G * DQK; g.b_kmajor = false;
    g.C = wb.dq; g.ldc = (int64_t)at.H * DQK;
    g.in_t = DT_BF16; g.c_t = DT_BF16; g.alpha = at.scale; g.beta = 0.f;
    GemmBatch bt;
    bt.nbatch = at.B * at.H; bt.zdiv = at.H; bt.bdiv = at.H / w.G; bt.mstore = at.T;
    bt.sA = (int64_t)at.T * w.ds_ld;
    bt.sB1 = (int64_t)at.T * w.G * DQK; bt.sB2 = DQK;
    bt.sC1 = (int64_t)at.T * at.H * DQK; bt.sC2 = DQK;
    bt.rev = 0; bt.kgroups = 1; bt.sAk = bt.sBk = 0;
    prof_begin(KC_ATTN_DQ, s);
    e = gemm_mfma_causal(g, bt, s);
    prof_end(KC_ATTN_DQ, s, 2.0 * pairs * DQK,
             pairs * 2.0 + N * at.H * DQK * 2.0 * 2.0);
  } else {
    prof_begin(KC_ATTN_DKDV, s);
    attn_dkdv_mfma_kernel<DQK, DV, true><<<nkb * at.B * w.G, 256, 0, s>>>(w);
    prof_end(KC_ATTN_DKDV, s, 2.0 * pairs * (2.0 * DV + DQK),
             N * at.H * (DQK + DV) * 2.0 + N * w.G * (DQK + DV) * 4.0 + N * at.H * 8.0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // dQ kernel: algorithmic dQ = dS K
    prof_begin(KC_ATTN_DQ, s);
    const int nqb = (at.T + DQ_BQ - 1) / DQ_BQ;
    attn_dq_mfma_kernel<DQK, DV><<<nqb * at.B * at.H, 256, 0, s>>>(w);
    prof_end(KC_ATTN_DQ, s, 2.0 * pairs * DQK,
             N * at.H * (2.0 * DQK + DV) * 2.0 + N * w.G * (DQK + DV) * 2.0 + N * at.H * 8.0);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  // rotary block of dQ back to the pre-rotation basis: R^T
  const int np = (DQK - at.dnope) / 2;
  return rope_apply(wb.dq, DT_BF16, at.B * at.T, at.T, at.H, (int64_t)at.H * DQK, DQK, at.dnope,
                    np, wb.rdiv, wb.cos_t, wb.sin_t, s, true);
}

}  // namespace

hipError_t bwd_dispatch(const AttnBwd& w, hipStream_t s) {
#define X(a_, b_) if (w.f.dqk == a_ && w.f.dv == b_) return bwd_launch<a_, b_>(w, s);
  MLA_MFMA_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace attn

hipError_t attn_bwd_mfma(const AttnBwd& w, hipStream_t s) { return attn::bwd_dispatch(w, s); }

int64_t attn_ds_ld(int T) { return ((int64_t)T + 63) / 64 * 64; }
int attn_stats_tpad(int T) { return (T + 31) / 32 * 32; }
size_t attn_stats_bytes(int B, int H, int T) { return 2ull * H * B * attn_stats_tpad(T) * 4; }
size_t attn_ds_bytes(int B, int H, int T) {
  // + scratch rows: 64 lanes x 64 elements
  return (size_t)B * H * (size_t)T * (size_t)attn_ds_ld(T) * 2 + 64 * 64 * 2;
}

}  // namespace mla
