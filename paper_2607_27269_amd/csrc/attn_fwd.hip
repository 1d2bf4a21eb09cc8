// Causal softmax attention (Eq. 2-4) on gfx950 matrix cores, bf16 operands, fp32 softmax.
//
// Forward.  A workgroup (8 wavefronts) owns 256 queries of one (sequence, head); each
// wavefront owns 32 of them.  Keys/values stream through a ring of three LDS stages, 64
// keys at a time, copied straight from HBM into LDS.  The loop is software-pipelined in
// blocks of 32 keys: while the vector ALUs exponentiate the logits of one block, the matrix
// cores already compute the logits of the next (the second half of the tile, or the first
// half of tile kb + 1, whose keys are resident), then O is updated with the block's values;
// tile kb + 2 is in flight meanwhile.
// The logits are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: the
// query is the MFMA column, so every lane owns one query and the online-softmax state
// (running max m, running sum l, the output row O^T) of that query lives in that lane.
// The accumulator layout of S^T is then reused directly as the B operand of
// O^T = V^T P^T (the key order inside one MFMA K-step is permuted identically on the
// V^T side), so P never leaves registers.  V stays [key][d_v] in LDS and its transposed
// operand comes from gfx950's transposing LDS read.  Softmax runs in base 2 with the
// logit scale folded into one FMA, and the output is only rescaled when the running
// maximum grows by more than 2^8 (P stays <= 2^8 otherwise).
// Tiles entirely above the causal diagonal are skipped per wavefront; only diagonal tiles
// are masked.  The key of head i is [Ka_{i/div_a} ; Kb_{i/div_b}] (non-positional part
// from one buffer, rotary part from another), which serves both the teacher
// (Ka = full key) and the MLA student (k^nope of the KV group, k^PE of the rope group).
#include "attn_common.h"
#include "mfma.h"

namespace mla {
namespace attn {
namespace {

constexpr int FWD_WAVES = 8;
constexpr int FWD_BQ = 32 * FWD_WAVES;   // queries per workgroup
constexpr float RESCALE_SLACK = 8.f;     // log2 units the running reference max may lag

// HG heads that share their keys and values (a KV group) per workgroup: wavefront w works
// on head i0 + w % HG and queries 32 (w / HG) .. of the workgroup's 256 / HG per head, so
// that one K/V tile in LDS serves all HG heads (HG = 1: 256 queries of one head)
template <int DQK, int DV, bool LSE, int HG>
__device__ __forceinline__ void fwd_tile(const AttnDev& a, int pid, bf16_t* smem) {
  using Stage = KVStage<DQK, DV, FWD_WAVES>;
  constexpr int LDK = Stage::LDK, LDV = Stage::LDV;
  constexpr int KS = Stage::KS, VS = Stage::VS;
  constexpr int NST = 3;  // K/V ring: tile kb (V in use), kb + 1 (K in use), kb + 2 (landing)
  constexpr int NKK = DQK / 16;  // MFMA K-steps of the logits
  constexpr int NC = DV / 32;    // 32-row tiles of O^T

  // work item pid (XCD-aware order: the query blocks of neighbouring head groups, which
  // share K/V, run on one XCD); heavy (late) query blocks first inside each head group
  constexpr int BQH = FWD_BQ / HG;  // queries per head
  const int ngr = a.H / HG;
  const int bh = pid / a.nqb;
  const int qb = a.nqb - 1 - pid % a.nqb;
  const int b = bh / ngr, i0 = (bh % ngr) * HG;
  const int q0 = qb * BQH;

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5, col = lane & 31;
  const int i = i0 + wave % HG;  // this wavefront's head
  const int qw0 = q0 + (wave / HG) * 32;
  // this lane's part of a transposing V read (lds_operand_tr's addressing): key row
  // 4 (lane half) + (lane % 16) / 4, column 16 ((lane / 16) % 2) + 4 (lane % 4)
  const int vlane = (4 * half + ((lane & 15) >> 2)) * LDV + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int my_q = qw0 + col;
  const int64_t nq = (int64_t)b * a.T + min(my_q, a.T - 1);

  // this lane's query, as MFMA B operand fragments (d = 16 kk + 8 half + 0..7)
  bf16x8 qf[NKK];
  {
    const bf16_t* qp = a.Q + nq * a.q_tok + (int64_t)i * a.q_head + 8 * half;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[kk] = *(const bf16x8*)(qp + 16 * kk);
    // optional R_t on the whole query (rotate-half pairs (p, p + DQK / 2)): the lane holds
    // both dims of each pair (fragments kk and kk + NKK / 2; compile-time indices keep the
    // fragments in registers)
    if (a.qcos) {  // uniform
      const int t = min(my_q, a.T - 1);
      constexpr int kn = NKK / 2;
#pragma unroll
      for (int kk = 0; kk < kn; ++kk) {
        const int p = 16 * kk + 8 * half;
        const float* cp = a.qcos + (int64_t)t * a.qnp + p;
        const float* sp = a.qsin + (int64_t)t * a.qnp + p;
        const f32x4 c0 = *(const f32x4*)cp, c1 = *(const f32x4*)(cp + 4);
        const f32x4 s0 = *(const f32x4*)sp, s1 = *(const f32x4*)(sp + 4);
        const u32x4 w1 = __builtin_bit_cast(u32x4, qf[kk]);
        const u32x4 w2 = __builtin_bit_cast(u32x4, qf[kk + kn]);
        u32x4 o1, o2;
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const float ca = e2 < 2 ? c0[2 * e2] : c1[2 * e2 - 4];
          const float cb = e2 < 2 ? c0[2 * e2 + 1] : c1[2 * e2 - 3];
          const float sa = e2 < 2 ? s0[2 * e2] : s1[2 * e2 - 4];
          const float sb = e2 < 2 ? s0[2 * e2 + 1] : s1[2 * e2 - 3];
          const float x1a = __uint_as_float(w1[e2] << 16), x1b = __uint_as_float(w1[e2] & 0xffff0000u);
          const float x2a = __uint_as_float(w2[e2] << 16), x2b = __uint_as_float(w2[e2] & 0xffff0000u);
          o1[e2] = pack2bf(x1a * ca - x2a * sa, x1b * cb - x2b * sb);
          o2[e2] = pack2bf(x1a * sa + x2a * ca, x1b * sb + x2b * cb);
        }
        qf[kk] = __builtin_bit_cast(bf16x8, o1);
        qf[kk + kn] = __builtin_bit_cast(bf16x8, o2);
      }
    }
  }

  f32x16 acc_o[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[c][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int kend = min(a.T, q0 + BQH);
  const int nkb = (kend + BKV - 1) / BKV;
  // tiles this wavefront sees (a prefix: the causal diagonal cuts its queries last)
  const int nvis = min(nkb, (qw0 + 31) / BKV + 1);
  Stage st;
  st.init(a, b, i0);  // the group's keys and values
  st.issue(0, smem, smem + KS);
  if (nkb > 1) st.issue(BKV, smem + (KS + VS), smem + (KS + VS) + KS);
  wait_all();
  __syncthreads();
  // the query fragments are in registers from here on: otherwise the compiler keeps
  // waiting for their loads inside the loop, and its counter waits there would also wait
  // for the K/V copies in flight
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) asm volatile("" : "+v"(qf[kk]));

  // S^T of 32 keys (rows of ks) against this lane's query
  auto logits = [&](const bf16_t* ks, f32x16& s) {
#pragma unroll
    for (int e = 0; e < 16; ++e) s[e] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          *(const bf16x8*)(ks + col * LDK + 16 * kk + 8 * half), qf[kk], s, 0, 0, 0);
  };

  // Half h (32 keys) of tile kb, its logits in sc: the softmax of this half runs while the
  // matrix cores compute the logits of the next half (into sn: the other half of this
  // tile, or the first half of tile kb + 1, whose keys are resident; past the last tile
  // they come from a stale but finite stage and are not used), then O^T += V^T P^T.
  auto step = [&](int kb, int h, f32x16& sc, f32x16& sn) {
    const int j0 = kb * BKV + 32 * h;
    // stage offsets pass through readfirstlane: opaque to the loop optimiser, which would
    // otherwise keep one induction variable per LDS read and add the stage in per read
    const int cur = __builtin_amdgcn_readfirstlane((kb % NST) * (KS + VS));
    const int nxt = __builtin_amdgcn_readfirstlane(((kb + 1) % NST) * (KS + VS));
    const bf16_t* ksn = h == 0 ? smem + cur + 32 * LDK : smem + nxt;
    const bf16_t* vs = smem + cur + KS;
    // causal mask on diagonal halves; max of this lane's query (raw logits)
    // (the empty asm keeps this a branch: the compiler would otherwise select per element
    // on every half)
    if (j0 + 31 > qw0) {
      asm volatile("");
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (j0 + 8 * (e >> 2) + 4 * half + (e & 3) > my_q) sc[e] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[e]);
    mx = pair_max32(mx) * a.sl2;
    // lazy rescale: the reference max moves only when a block max exceeds it by more
    // than RESCALE_SLACK (so P <= 2^RESCALE_SLACK); wave-uniform branch
    if (__ballot(mx > m_run + RESCALE_SLACK) != 0) {
      const float m_new = fmaxf(m_run, mx);
      const float corr = __builtin_amdgcn_exp2f(m_run - (m_new == -INFINITY ? 0.f : m_new));
      m_run = m_new;
      l_run *= corr;
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc_o[c][e] *= corr;
    }
    const float m_use = m_run == -INFINITY ? 0.f : m_run;
    logits(ksn, sn);
    // P = 2^(s sl2 - m), packed to bf16 as the B operand of O^T = V^T P^T
    bf16x8 pf[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 w;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[8 * u + 2 * q], a.sl2, -m_use));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[8 * u + 2 * q + 1], a.sl2, -m_use));
        l_run += p0 + p1;
        w[q] = pack2bf(p0, p1);
      }
      pf[u] = __builtin_bit_cast(bf16x8, w);
    }
    // O^T += V^T P^T; K-step u covers keys 32 h + 16 u + {4h'..4h'+3, 8+4h'..8+4h'+3}
    // (h' = the lane half): transposing reads at the lane's offset plus constants
    const bf16_t* vp = vs + vlane + 32 * h * LDV;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const u32x2 lo = lds_read_tr4(vp + 16 * u * LDV + 32 * c);
        const u32x2 hi = lds_read_tr4(vp + (16 * u + 8) * LDV + 32 * c);
        const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
        acc_o[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w), pf[u],
                                                           acc_o[c], 0, 0, 0);
      }
    }
  };

  f32x16 sa, sb;
  if (nvis > 0) logits(smem, sa);
  for (int kb = 0; kb < nkb; ++kb) {
    if (kb + 2 < nkb) {
      bf16_t* nxt = smem + ((kb + 2) % NST) * (KS + VS);
      st.issue((kb + 2) * BKV, nxt, nxt + KS);
    }
    if (kb < nvis) {  // wave-uniform; a second half entirely above the diagonal is skipped
      step(kb, 0, sa, sb);
      if (kb * BKV + 32 <= qw0) step(kb, 1, sb, sa);
    }
    // tile kb + 2 has landed and nobody reads tile kb's stage any more
    wait_all();
    __syncthreads();
  }

  // normalise and store: lane holds query my_q, d = 32c + 8(e/4) + 4 half + e%4
  const float l = pair_sum32(l_run);
  if (my_q >= a.T) return;
  const float inv = 1.f / l;
  const int64_t ooff = ((int64_t)b * a.T + my_q) * a.o_tok + (int64_t)i * DV + 4 * half;
  bf16_t* op = a.O + ooff;
  // the reference rows first, all loads before any store: interleaved, each load would
  // wait (one in-order memory counter) for every store issued before it
  u32x2 rf[NC][4];
  if (a.Odiff) {  // uniform
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) rf[c][g] = *(const u32x2*)(a.Oref + ooff + 32 * c + 8 * g);
  }
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      u32x2 w = {pack2bf(acc_o[c][4 * g] * inv, acc_o[c][4 * g + 1] * inv),
                 pack2bf(acc_o[c][4 * g + 2] * inv, acc_o[c][4 * g + 3] * inv)};
      *(u32x2*)(op + 32 * c + 8 * g) = w;
      if (a.Odiff) {  // uniform
        const u32x2 r = rf[c][g];
        auto lo = [](uint32_t x) { return __uint_as_float(x << 16); };
        auto hi = [](uint32_t x) { return __uint_as_float(x & 0xffff0000u); };
        *(u32x2*)(a.Odiff + ooff + 32 * c + 8 * g) =
            u32x2{pack2bf(lo(w[0]) - lo(r[0]), hi(w[0]) - hi(r[0])),
                  pack2bf(lo(w[1]) - lo(r[1]), hi(w[1]) - hi(r[1]))};
      }
    }
  if (LSE && half == 0) a.lse[((int64_t)b * a.T + my_q) * a.H + i] = (m_run + __log2f(l)) * LN2;
}

// one work item per workgroup
template <int DQK, int DV, bool LSE, int HG>
__global__ __launch_bounds__(64 * FWD_WAVES) void attn_fwd_mfma_kernel(AttnDev a) {
  using Stage = KVStage<DQK, DV, FWD_WAVES>;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[3 * (Stage::KS + Stage::VS)];
  const int nwork = a.B * (a.H / HG) * a.nqb;
  fwd_tile<DQK, DV, LSE, HG>(a, xcd_remap(blockIdx.x, nwork), smem);
}

// persistent: FWD_PCU workgroups per XCD (one per CU) walk that XCD's share of the work
// items in the same order (rounds of FWD_PCU items), in snake order (forward in even rounds,
// backward in odd ones), so that heavy and light query blocks of a head pair up on a CU
constexpr int FWD_PCU = 32;
template <int DQK, int DV, bool LSE, int HG>
__global__ __launch_bounds__(64 * FWD_WAVES) void attn_fwd_persist_kernel(AttnDev a) {
  using Stage = KVStage<DQK, DV, FWD_WAVES>;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[3 * (Stage::KS + Stage::VS)];
  const int per = a.B * (a.H / HG) * a.nqb / 8;  // items of one XCD
  const int x = blockIdx.x % 8, j = blockIdx.x / 8;
  for (int r = 0;; ++r) {
    const int local = r * FWD_PCU + ((r & 1) ? FWD_PCU - 1 - j : j);
    if (local >= per) break;
    if (r > 0) __syncthreads();  // every wavefront is done with the previous item's LDS
    fwd_tile<DQK, DV, LSE, HG>(a, x * per + local, smem);
  }
}

template <int DQK, int DV, int HG>
hipError_t fwd_launch_hg(const Attn& at, hipStream_t s, const char** kernel) {
  AttnDev d = to_dev(at);
  constexpr int BQH = FWD_BQ / HG;
  d.nqb = (at.T + BQH - 1) / BQH;
  const int nwork = d.B * (d.H / HG) * d.nqb;
  // the persistent walk needs whole XCD shares of several rounds
  if (nwork % 8 == 0 && nwork / 8 >= 2 * FWD_PCU) {
    if (at.lse) {
      attn_fwd_persist_kernel<DQK, DV, true, HG><<<8 * FWD_PCU, 64 * FWD_WAVES, 0, s>>>(d);
      *kernel = KLABEL("attn_fwd_persist_kernel<%d,%d,lse>", DQK, DV);
    } else {
      attn_fwd_persist_kernel<DQK, DV, false, HG><<<8 * FWD_PCU, 64 * FWD_WAVES, 0, s>>>(d);
      *kernel = KLABEL("attn_fwd_persist_kernel<%d,%d>", DQK, DV);
    }
    return hipGetLastError();
  }
  if (at.lse) {
    attn_fwd_mfma_kernel<DQK, DV, true, HG><<<nwork, 64 * FWD_WAVES, 0, s>>>(d);
    *kernel = KLABEL("attn_fwd_mfma_kernel<%d,%d,lse>", DQK, DV);
  } else {
    attn_fwd_mfma_kernel<DQK, DV, false, HG><<<nwork, 64 * FWD_WAVES, 0, s>>>(d);
    *kernel = KLABEL("attn_fwd_mfma_kernel<%d,%d>", DQK, DV);
  }
  return hipGetLastError();
}

// four heads per workgroup when they share every key / value source (the head -> group
// divisors are multiples of 4), else one
template <int DQK, int DV>
hipError_t fwd_launch(const Attn& at, hipStream_t s, const char** kernel) {
  const bool share4 = at.H % 4 == 0 && at.Ka.div % 4 == 0 && at.V.div % 4 == 0 &&
                      (at.dnope == DQK || at.Kb.div % 4 == 0);
  return share4 ? fwd_launch_hg<DQK, DV, 4>(at, s, kernel) : fwd_launch_hg<DQK, DV, 1>(at, s, kernel);
}


}  // namespace

bool supported(int dqk, int dv) {
#define X(a_, b_) if (dqk == a_ && dv == b_) return true;
  MLA_MFMA_SHAPES(X)
#undef X
  return false;
}

}  // namespace attn

bool attn_mfma_supported(int dqk, int dv) { return attn::supported(dqk, dv); }

hipError_t attn_fwd_mfma(const Attn& a, hipStream_t s, const char** kernel) {
#define X(a_, b_) if (a.dqk == a_ && a.dv == b_) return attn::fwd_launch<a_, b_>(a, s, kernel);
  MLA_MFMA_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace mla
