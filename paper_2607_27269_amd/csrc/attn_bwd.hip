// Causal softmax attention backward (gradients of Eq. 2-4) on gfx950 matrix cores.
//
//   P = exp(S - lse) (recomputed from the forward's log-sum-exp), dV = P^T dO,
//   dP = dO V^T, dS = P (dP - delta) with delta = rowsum(dO . O),
//   dQ = scale dS K, dK = scale dS^T Q.
//
// * dV and dS^T: a workgroup owns 256 keys of one (sequence, KV group) and walks the
//   group's heads and 32-query blocks; it accumulates dV in registers and stores dS^T in
//   bf16 as 32 x 32 tiles ([32 keys][32 queries], 2 KB each; each wavefront writes whole
//   tiles), zeros included wherever the products below read a masked pair.
// * dK = scale dS^T Q: a batched causal GEMM per (sequence, group), the group's heads
//   stacked along K.
// * dQ = scale dS K: a batched causal GEMM per (sequence, head) over the stored dS^T and
//   the keys gathered per group into one [token][group][dqk] tensor; no recomputation of
//   S or dP.
// The dS^T buffer holds at most 16 GiB: larger batches run in chunks of whole sequences.
// The rotary block of dQ is then rotated back with R^T.
#include <algorithm>

#include "attn_common.h"
#include "mfma.h"
#include "simt.h"

namespace mla {
namespace attn {
namespace {

struct BwdDev {
  AttnDev f;
  const bf16_t* dO;      // [N][H*dv]
  bf16_t* dV; int64_t dv_tok;
  int G;                 // Ka groups
  bf16_t* dsT;           // [B*H] planes of ds_ld x ds_ld in 32 x 32 tiles (ds_at)
  int64_t ds_ld;
  bf16_t* ds_dummy;      // scratch rows for stores of lanes past the sequence end
  const float* statT;    // [2][H][B][tpad]: log2-scaled lse, delta
  int tpad;
  int off32;             // one sequence's Q / dO rows and the statistics span < 2^31 bytes
};

// dS^T tile rows a dQ GEMM row tile reads: queries from the start of the 256-query tile
// that holds the key (the GEMM's row tile) to the end
constexpr int DQ_TILE = 256;

// element (key, query) of a dS^T plane: 32 x 32 tiles of [32 keys][32 queries], the tiles
// of a key block in query order (ld / 32 per row of tiles), key blocks in order.  A
// wavefront's 32 x 32 block is then 2 KB of whole lines, and the products' slices are
// runs of consecutive tiles.
__device__ __forceinline__ int64_t ds_at(int64_t key, int64_t q, int64_t ld) {
  return ((key >> 5) * (ld >> 5) + (q >> 5)) * 1024 + (key & 31) * 32 + (q & 31);
}

// ---------------------------------------------------------------------------------------
// dV and dS^T (the path where dK and dQ are GEMMs over the stored dS^T)
// ---------------------------------------------------------------------------------------
// A workgroup owns 256 keys of one (sequence, KV group), 32 per wavefront (8 wavefronts,
// one workgroup per CU), and walks the group's heads and 32-query blocks.  K and V of the
// lane's key are B-operand fragments held in registers; only the 32-query Q / dO tiles
// and their softmax statistics pass through LDS, in a ring of three stages, each block's
// copy issued two steps before its use; the more keys share a copied tile, the fewer
// copies per key.  Every wavefront issues the same number of copies per stage (the block
// count is padded) and of dS^T stores per step, so one counter wait names exactly the
// copies that must have landed.
constexpr int DV_BQ = 32;
// dS^T stores per lane per step: a wavefront's 32 x 32 block is transposed through a
// private LDS tile into the [key][query] order of its 2 KB dS^T tile, which two 16-byte
// stores per lane write whole (1 KB per store instruction)
constexpr int DS_STORES = DV_BQ * 32 * 2 / (64 * 16);
constexpr int DV_NST = 3;  // LDS stages: a step's copies are issued two steps ahead
constexpr int DV_WAVES = 8;
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
      bf16_t* plane = w.dsT + ((int64_t)b * a.H + i0 + h) * w.ds_ld * w.ds_ld;
      for (int c = threadIdx.x; c < kr * cpr; c += 64 * DV_WAVES) {
        const int r = c / cpr, q = zq0 + (c % cpr) * 8;
        *(u32x4*)(plane + ds_at(k0 + r, q, w.ds_ld)) = u32x4{0u, 0u, 0u, 0u};
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
  // the same time and share it through L2.  (qc, hc) is this step's pair, (q1, h1) the next
  // one, (qn, hn) the one whose copies this step issues (step sn = this step + 2, capped at
  // the last step: past the end the last pair is copied again into the free stage, so that
  // every step issues the same number of copies).
  int qc = (nqb - 1) * DV_BQ, hc = i0;
  auto advance = [&](int& q, int& h) {
    if (++h == i0 + hpg) { h = i0; q -= DV_BQ; }
  };
  int q1 = qc, h1 = hc;
  if (niter > 1) advance(q1, h1);
  int qn = q1, hn = h1, sn = niter > 1 ? 1 : 0;
  if (sn < niter - 1) { advance(qn, hn); ++sn; }
  // (stage offsets through readfirstlane: uniform, added to one per-lane address)
  auto stage_of = [&](int it) {
    return smem + __builtin_amdgcn_readfirstlane((it % DV_NST) * Stage::ELEMS);
  };
  bf16_t* scratch = w.ds_dummy + 64 * lane;
  // transpose tile: key row r holds 64 bytes (32 queries) as four 16-byte segments, segment
  // s stored at position s ^ ((r / 4) % 4) (the packed writes of 32 rows at one segment
  // spread over the banks; the 16-byte reads of 4 consecutive rows are conflict-free)
  bf16_t* tr = smem + DV_NST * Stage::ELEMS + wave * 32 * DV_BQ;
  static_assert(DV_BQ == 32 && DS_STORES == 2, "transpose tile layout");
  // reader side: lane handles rows rr + 16 j (j < 2), queries 8 sg .. 8 sg + 7
  const int rr = lane >> 2, sg = lane & 3;
  stg.issue(w, b, hc, qc, stage_of(0));
  stg.issue(w, b, h1, q1, stage_of(1));
  wait_vm<D>();
  lds_barrier();

  for (int it = 0; it < niter; ++it) {
    const int q0 = qc;
    const bf16_t* Qs = stage_of(it);
    const bf16_t* dOs = Qs + Stage::OFF_O;
    const float* st_lse = (const float*)(Qs + Stage::OFF_S);
    const float* st_dl = st_lse + DV_BQ;
    // the stage of step it - 1 is free: every wave passed the barrier after reading it
    stg.issue(w, b, hn, qn, stage_of(it + 2));

    // this lane's dS^T store targets for the block: key rows kw0 + rr + 16 j, queries
    // q0 + 8 sg .. + 7, i.e. 16 bytes at 8 lane + 512 j of the block's tile (kw0 and q0
    // are multiples of 32): a store instruction writes 1 KB of the tile; rows past the
    // sequence end go to a scratch row instead, so that every wavefront issues exactly
    // DS_STORES stores per step (computed where the stores are issued: short-lived
    // registers)
    auto dst = [&](int j) {
      const int key = kw0 + rr + 16 * j;
      return key < a.T ? w.dsT + ((int64_t)b * a.H + hc) * w.ds_ld * w.ds_ld +
                             ds_at(kw0, q0, w.ds_ld) + 512 * j + 8 * lane
                       : scratch + 8 * sg;
    };
    // every step runs the products: a step whose pairs are all masked (keys past every
    // query of the block) gets zeros from the mask branch below.  (A branch around the
    // whole step made dV's accumulators live in two register sets, copied every step.)
    {
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
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int qr = 8 * e4 + 4 * half;
        const f32x4 l2 = *(const f32x4*)(st_lse + qr);
        const f32x4 dl = *(const f32x4*)(st_dl + qr);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * e4 + r;
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sp[e], a.sl2, -l2[r]));
          sp[e] = p;
          dp[e] = p * (dp[e] - dl[r]);
        }
      }
      // causal mask, on the diagonal (and fully masked) steps only (a real branch: the
      // empty asm keeps the compiler from selecting per element on every step)
      if (kw0 + 31 > q0) {
        asm volatile("");
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (my_key > q0 + 8 * (e >> 2) + 4 * half + (e & 3)) {
            sp[e] = 0.f;
            dp[e] = 0.f;
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
        st_global16_nt(dst(j), *(const u32x4*)(tr + r * DV_BQ + 8 * (sg ^ ((r >> 2) & 3))));
      }
      asm volatile("" ::: "memory");
    }
    // step it + 1's copies have landed; younger are this step's stores, step it + 2's copies
    // and (from step 1 on) the previous step's stores (counters complete in issue order)
    if (it == 0) wait_vm<D + DS_STORES>(); else wait_vm<D + 2 * DS_STORES>();
    lds_barrier();
    advance(qc, hc);
    if (sn < niter - 1) { advance(qn, hn); ++sn; }
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

// The attention of sequences b0 .. b0 + nb - 1 as a problem of its own (token-major views
// shifted by b0 T tokens)
static Attn seq_slice(const Attn& a, int b0, int nb) {
  Attn c = a;
  const int64_t n0 = (int64_t)b0 * a.T;
  auto shift = [&](HeadView& v) {
    if (v.p) v.p = (const bf16_t*)v.p + n0 * v.tok;
  };
  shift(c.Q); shift(c.Ka); shift(c.Kb); shift(c.V);
  c.O = (bf16_t*)a.O + n0 * a.o_tok;
  c.lse = a.lse + n0 * a.H;
  c.B = nb;
  return c;
}

// dV, dK and dQ of sequences b0 .. b0 + nb - 1 (their dS^T fits the buffer)
template <int DQK, int DV>
hipError_t bwd_chunk(const AttnBwd& wb, int b0, int nb, hipStream_t s) {
  const Attn at = seq_slice(wb.f, b0, nb);
  const int64_t n0 = (int64_t)b0 * at.T;
  const int64_t Ntot = (int64_t)wb.f.B * at.T;
  const int dr = DQK - at.dnope;
  const bf16_t* dO = (const bf16_t*)wb.dO + n0 * at.H * DV;
  const float* delta = wb.delta + n0 * at.H;
  bf16_t* dq = (bf16_t*)wb.dq + n0 * at.H * DQK;
  bf16_t* dKa = (bf16_t*)wb.dKa + n0 * wb.dka_tok;
  float* dkb = wb.dkb_part + n0 * dr;
  BwdDev w;
  w.f = to_dev(at);
  w.dO = dO;
  w.dV = (bf16_t*)wb.dV + n0 * wb.dv_tok; w.dv_tok = wb.dv_tok;
  w.G = wb.n_ka_groups;
  w.dsT = (bf16_t*)wb.dsT;
  w.ds_ld = attn_ds_ld(at.T);
  w.ds_dummy = w.dsT + (int64_t)at.B * at.H * w.ds_ld * w.ds_ld;
  w.statT = wb.statT;
  w.tpad = attn_stats_tpad(at.T);
  w.off32 = (int64_t)at.T * at.Q.tok * 2 < (1ll << 31) &&
            (int64_t)at.T * at.H * at.dv * 2 < (1ll << 31) &&
            (int64_t)at.H * at.B * w.tpad * 4 * 2 < (1ll << 31);
  const double pairs = attn_causal_pairs(at);
  const double N = (double)at.B * at.T;
  const int hpg = at.H / w.G;
  // statistics per (head, sequence) in query order, then dV and dS^T: algorithmic
  // dV = P^T dO, dP = dO V^T
  prof_begin(KC_ELEM, s);
  const int64_t nst = 2LL * at.H * at.B * w.tpad;
  attn_stats_t_kernel<<<(unsigned)((nst + 255) / 256), 256, 0, s>>>(at.lse, delta, at.B, at.T, at.H,
                                                                    w.tpad, wb.statT);
  prof_end(KC_ELEM, s, 0.0, nst * 4.0 * 2.0, KLABEL("attn_stats_t_kernel"));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  prof_begin(KC_ATTN_DKDV, s);
  const int nkb_dv = (at.T + DV_BKB - 1) / DV_BKB;
  attn_dv_mfma_kernel<DQK, DV><<<nkb_dv * at.B * w.G, 64 * DV_WAVES, 0, s>>>(w);
  prof_end(KC_ATTN_DKDV, s, 2.0 * pairs * (2.0 * DV),
           N * at.H * (DQK + DV) * 2.0 + N * w.G * (DQK + DV) * 2.0 + N * at.H * 8.0 +
               pairs * 2.0,
           KLABEL("attn_dv_mfma_kernel<%d,%d>", DQK, DV));
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // dK = scale dS^T Q per (sequence, group), the group's heads stacked along K:
  // algorithmic dS read once, Q read once, dK written once (fp32)
  {
    Gemm g;
    g.M = at.T; g.N = DQK; g.K = at.T;
    g.A = wb.dsT; g.lda = w.ds_ld; g.a_kmajor = true;
    g.B = at.Q.p; g.ldb = at.Q.tok; g.b_kmajor = false;
    // written split: dk^nope in bf16 into dKa, the dk^PE partials (fp32) into dkb
    g.C = dkb; g.ldc = dr;
    g.in_t = DT_BF16; g.c_t = DT_F32; g.alpha = at.scale; g.beta = 0.f;
    GemmBatch bt;
    bt.nbatch = at.B * w.G; bt.zdiv = w.G; bt.bdiv = 1; bt.mstore = at.T;
    bt.rev = 1; bt.kgroups = hpg;
    bt.sA = (int64_t)hpg * w.ds_ld * w.ds_ld; bt.sAk = w.ds_ld * w.ds_ld;
    bt.sB1 = (int64_t)at.T * at.Q.tok; bt.sB2 = (int64_t)hpg * at.Q.head; bt.sBk = at.Q.head;
    bt.sC1 = (int64_t)at.T * dr; bt.sC2 = Ntot * dr;
    bt.split_n = at.dnope; bt.c_lo = dKa;
    bt.ldc_lo = wb.dka_tok; bt.sC1_lo = (int64_t)at.T * wb.dka_tok; bt.sC2_lo = at.dnope;
    prof_begin(KC_ATTN_DK, s);
    e = gemm_mfma_causal(g, bt, s);
    prof_end(KC_ATTN_DK, s, 2.0 * pairs * DQK,
             pairs * 2.0 + N * at.H * DQK * 2.0 + N * w.G * (at.dnope * 2.0 + dr * 4.0),
             KLABEL("attn_ds_gemm_persist_kernel<256,%d,dK,fp32>", DQK));
    if (e != hipSuccess) return e;
  }
  // keys of each group gathered into one operand, then dQ = scale dS K per (sequence,
  // head): algorithmic dS read once, K read once per head, dQ written once
  prof_begin(KC_ELEM, s);
  const int64_t chunks = (int64_t)at.B * at.T * w.G * (DQK / 8);
  kcat_kernel<<<(unsigned)((chunks + 255) / 256), 256, 0, s>>>(w.f, w.G, DQK, (bf16_t*)wb.kcat);
  prof_end(KC_ELEM, s, 0.0, N * w.G * DQK * 2.0 * 2.0, KLABEL("kcat_kernel"));
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  Gemm g;
  g.M = (int)w.ds_ld; g.N = DQK; g.K = at.T;
  g.A = wb.dsT; g.lda = w.ds_ld; g.a_kmajor = false;
  g.B = wb.kcat; g.ldb = (int64_t)w.G * DQK; g.b_kmajor = false;
  g.C = dq; g.ldc = (int64_t)at.H * DQK;
  g.in_t = DT_BF16; g.c_t = DT_BF16; g.alpha = at.scale; g.beta = 0.f;
  GemmBatch bt;
  bt.nbatch = at.B * at.H; bt.zdiv = at.H; bt.bdiv = at.H / w.G; bt.mstore = at.T;
  bt.sA = w.ds_ld * w.ds_ld;
  bt.sB1 = (int64_t)at.T * w.G * DQK; bt.sB2 = DQK;
  bt.sC1 = (int64_t)at.T * at.H * DQK; bt.sC2 = DQK;
  bt.rev = 0; bt.kgroups = 1; bt.sAk = bt.sBk = 0;
  prof_begin(KC_ATTN_DQ, s);
  e = gemm_mfma_causal(g, bt, s);
  prof_end(KC_ATTN_DQ, s, 2.0 * pairs * DQK, pairs * 2.0 + N * at.H * DQK * 2.0 * 2.0,
           KLABEL("attn_ds_gemm_kernel<256,%d,dQ,bf16>", DQK));
  return e;
}

template <int DQK, int DV>
hipError_t bwd_launch(const AttnBwd& wb, hipStream_t s) {
  const Attn& at = wb.f;
  const int chunk = wb.chunk_seqs;
  if (chunk < 1 || chunk > attn_bwd_chunk_seqs(at.B, at.H, at.T, at.dqk, at.dv, at.t) || !wb.dsT || !wb.kcat || !wb.statT) return hipErrorInvalidValue;
  // delta = rowsum(dO . O) of every token
  prof_begin(KC_ELEM, s);
  hipError_t e = attn_delta(wb, s);
  // reads dO and O (and o_s - o_t when it also sums Eq. 11), writes delta
  prof_end(KC_ELEM, s, 0.0, (double)at.B * at.T * at.H * ((wb.loss_ref ? 3.0 : 2.0) * DV * 2.0 + 4.0),
           KLABEL("attn_delta_bf16x8_kernel"));
  if (e != hipSuccess) return e;
  for (int b0 = 0; b0 < at.B; b0 += chunk) {
    e = bwd_chunk<DQK, DV>(wb, b0, std::min(chunk, at.B - b0), s);
    if (e != hipSuccess) return e;
  }
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
  // square ds_ld x ds_ld planes (whole 32 x 32 tiles in both directions) + scratch rows:
  // 64 lanes x 64 elements
  return (size_t)B * H * (size_t)attn_ds_ld(T) * (size_t)attn_ds_ld(T) * 2 + 64 * 64 * 2;
}

}  // namespace mla
