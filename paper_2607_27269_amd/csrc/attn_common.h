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
  const bf16_t* Oref; bf16_t* Odiff;  // optional: Odiff = O - Oref (rounded O), layout of O
  const float* qcos; const float* qsin; int qroff, qnp;  // optional: Q rotated on load
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
  d.Oref = (const bf16_t*)a.o_ref; d.Odiff = (bf16_t*)a.o_diff;
  d.qcos = a.q_cos; d.qsin = a.q_sin; d.qroff = a.q_roff; d.qnp = a.q_np;
  d.nqb = 0;
  return d;
}

// K and V tiles of BKV keys streamed straight into padded [key][dim] LDS tiles.  Keys at or
// past the sequence end load the last valid key (finite data; such keys are causally
// masked or carry zero probability).
template <int DQK, int DV, int NW>
struct KVStage {
  static constexpr int LDK = ld_of(DQK);
  static constexpr int LDV = ld_of(DV);
  using KT = DmaTile<BKV, DQK, LDK, NW>;
  using VT = DmaTile<BKV, DV, LDV, NW>;
  static constexpr int KS = KT::ALLOC;  // LDS elements of the K tile
  static constexpr int VS = VT::ALLOC;
  KT kt;
  VT vt;
  const bf16_t* ka;   // key rows of this (sequence, head): element (n, d) at ka + n*ka_tok + d
  const bf16_t* kb;
  const bf16_t* vb;
  int64_t ka_tok, kb_tok, v_tok;
  int dnope, T;

  __device__ __forceinline__ void init(const AttnDev& a, int b, int i) {
    kt.init();
    vt.init();
    const int64_t n0 = (int64_t)b * a.T;
    ka = a.Ka + n0 * a.ka_tok + (int64_t)(i / a.ka_div) * a.ka_head;
    kb = a.Kb + n0 * a.kb_tok + (int64_t)(i / a.kb_div) * a.kb_head - a.dnope;
    vb = a.V + n0 * a.v_tok + (int64_t)(i / a.v_div) * a.v_head;
    ka_tok = a.ka_tok; kb_tok = a.kb_tok; v_tok = a.v_tok;
    dnope = a.dnope; T = a.T;
  }

  // keys j0 .. j0+BKV-1 into (ks, vs)
  __device__ __forceinline__ void issue(int j0, bf16_t* ks, bf16_t* vs) const {
    const int last = T - 1;
    kt.issue(ks, [&](int r, int c) {
      const int64_t n = min(j0 + r, last);
      return c < dnope ? ka + n * ka_tok + c : kb + n * kb_tok + c;
    });
    vt.issue(vs, [&](int r, int c) {
      const int64_t n = min(j0 + r, last);
      return vb + n * v_tok + c;
    });
  }
};

}  // namespace attn
}  // namespace mla
