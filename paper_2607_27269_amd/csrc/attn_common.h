// Shared definitions of the bf16 MFMA attention kernels (forward and backward).
#pragma once
#include "common.h"
#include "kernels.h"

// (logit width, value width) pairs the MFMA attention kernels are built for
#define MLA_MFMA_SHAPES(X) X(64, 64) X(128, 128) X(96, 64) X(128, 64) X(192, 128)

namespace mla {
namespace attn {

constexpr int BKV = 64;   // keys per streamed K/V tile

// Row length (bf16 elements) of a [row][D] LDS tile.  The stride in 4-byte banks is made
// congruent to 12, 28, 36 or 52 modulo 64, so both access patterns used on these tiles are
// free of bank conflicts: 16-byte reads of 16 consecutive rows (MFMA operands in natural
// layout) and the transposing read (4 consecutive rows x 32 bytes).
constexpr int ld_of(int D) {
  for (int p = 8; p <= 64; p += 8) {
    const int r = ((D + p) / 2) % 64;
    if (r == 12 || r == 28 || r == 36 || r == 52) return D + p;
  }
  return D + 8;
}
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

inline AttnDev to_dev(const Attn& a) {
  AttnDev d;
  d.B = a.B; d.T = a.T; d.H = a.H; d.dnope = a.dnope;
  d.sl2 = a.scale * LOG2E;
  d.Q = (const bf16_t*)a.Q.p; d.q_tok = a.Q.tok; d.q_head = (int)a.Q.head;
  d.Ka = (const bf16_t*)a.Ka.p; d.ka_tok = a.Ka.tok; d.ka_head = (int)a.Ka.head; d.ka_div = a.Ka.div;
  d.Kb = (const bf16_t*)a.Kb.p; d.kb_tok = a.Kb.tok; d.kb_head = (int)a.Kb.head; d.kb_div = a.Kb.div;
  d.V = (const bf16_t*)a.V.p; d.v_tok = a.V.tok; d.v_head = (int)a.V.head; d.v_div = a.V.div;
  d.O = (bf16_t*)a.O; d.o_tok = a.o_tok; d.lse = a.lse;
  d.nqb = 0;
  return d;
}

// K and V tiles of BKV keys, staged global -> registers -> LDS in their natural
// [key][dim] layout (16-byte chunks).  Source addresses are formed once per workgroup and
// advanced by one tile per step; only the ragged last tile checks the sequence end.
template <int DQK, int DV, int NTHR>
struct KVStage {
  static constexpr int KCH = BKV * (DQK / 8);
  static constexpr int KPER = (KCH + NTHR - 1) / NTHR;
  static constexpr int VCH = BKV * (DV / 8);
  static constexpr int VPER = (VCH + NTHR - 1) / NTHR;
  static constexpr int LDK = ld_of(DQK);
  static constexpr int LDV = ld_of(DV);
  u32x4 k[KPER];
  u32x4 v[VPER];
  const bf16_t* ksrc[KPER];
  const bf16_t* vsrc[VPER];
  int64_t kstr[KPER];
  int krow[KPER], vrow[VPER];

  __device__ __forceinline__ void init(const AttnDev& a, int b, int i) {
    const int ga = i / a.ka_div, gb = i / a.kb_div, gv = i / a.v_div;
#pragma unroll
    for (int it = 0; it < KPER; ++it) {
      const int c = min((int)threadIdx.x + it * NTHR, KCH - 1);
      const int key = c / (DQK / 8), dc = (c % (DQK / 8)) * 8;
      const int64_t n = (int64_t)b * a.T + key;
      krow[it] = key;
      const bool nope = dc < a.dnope;
      kstr[it] = nope ? a.ka_tok : a.kb_tok;
      ksrc[it] = nope ? a.Ka + n * a.ka_tok + (int64_t)ga * a.ka_head + dc
                      : a.Kb + n * a.kb_tok + (int64_t)gb * a.kb_head + (dc - a.dnope);
    }
#pragma unroll
    for (int it = 0; it < VPER; ++it) {
      const int c = min((int)threadIdx.x + it * NTHR, VCH - 1);
      const int key = c / (DV / 8), dc = (c % (DV / 8)) * 8;
      vrow[it] = key;
      vsrc[it] = a.V + ((int64_t)b * a.T + key) * a.v_tok + (int64_t)gv * a.v_head + dc;
    }
  }

  // tile starting at key j0 (a multiple of BKV)
  __device__ __forceinline__ void load(const AttnDev& a, int j0) {
    const bool full = j0 + BKV <= a.T;
#pragma unroll
    for (int it = 0; it < KPER; ++it) {
      u32x4 val = {0u, 0u, 0u, 0u};
      const bool in = KCH % NTHR == 0 || (int)threadIdx.x + it * NTHR < KCH;
      if (in && (full || j0 + krow[it] < a.T)) val = *(const u32x4*)(ksrc[it] + (int64_t)j0 * kstr[it]);
      k[it] = val;
    }
#pragma unroll
    for (int it = 0; it < VPER; ++it) {
      u32x4 val = {0u, 0u, 0u, 0u};
      const bool in = VCH % NTHR == 0 || (int)threadIdx.x + it * NTHR < VCH;
      if (in && (full || j0 + vrow[it] < a.T)) val = *(const u32x4*)(vsrc[it] + (int64_t)j0 * a.v_tok);
      v[it] = val;
    }
  }

  __device__ __forceinline__ void store(bf16_t* ks, bf16_t* vs) const {
#pragma unroll
    for (int it = 0; it < KPER; ++it) {
      const int c = (int)threadIdx.x + it * NTHR;
      if (KCH % NTHR == 0 || c < KCH)
        *(u32x4*)(ks + (c / (DQK / 8)) * LDK + (c % (DQK / 8)) * 8) = k[it];
    }
#pragma unroll
    for (int it = 0; it < VPER; ++it) {
      const int c = (int)threadIdx.x + it * NTHR;
      if (VCH % NTHR == 0 || c < VCH)
        *(u32x4*)(vs + (c / (DV / 8)) * LDV + (c % (DV / 8)) * 8) = v[it];
    }
  }
};


}  // namespace attn
}  // namespace mla
