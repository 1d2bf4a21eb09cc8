// Shared definitions of the bf16 MFMA attention kernels (forward and backward).
#pragma once
#include "common.h"
#include "kernels.h"

// (logit width, value width) pairs the MFMA attention kernels are built for
#define MLA_MFMA_SHAPES(X) X(64, 64) X(128, 128) X(96, 64) X(128, 64) X(192, 128)

namespace mla {
namespace attn {

constexpr int BKV = 64;   // keys per forward tile
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

}  // namespace attn
}  // namespace mla
