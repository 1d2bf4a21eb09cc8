// fp32 check-mode kernels: the same GEMM and causal attention (forward and backward) as
// the bf16 MFMA path, written as plain vector-ALU code that accumulates in fp32.  They
// serve MLA_FP32 (the 1e-5 parity mode) and accept bf16 storage as well.
#include "common.h"
#include "kernels.h"
#include "simt.h"

#include <math.h>

namespace mla {

// ---------------------------------------------------------------------------------------
// GEMM: 64x64 output tile per 256-thread workgroup, 16-deep K slices staged in LDS,
// 4x4 outputs per thread.
// ---------------------------------------------------------------------------------------
template <typename TI, typename TC>
__global__ __launch_bounds__(256) void gemm_simt_kernel(Gemm g) {
  __shared__ float As[16][65];
  __shared__ float Bs[16][65];
  const TI* A = (const TI*)g.A;
  const TI* B = (const TI*)g.B;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < g.K; k0 += 16) {
    for (int e = threadIdx.x; e < 1024; e += 256) {
      int mm, kk;
      if (g.a_kmajor) { mm = e / 16; kk = e % 16; } else { kk = e / 64; mm = e % 64; }
      int m = m0 + mm;
      int64_t k = k0 + kk;
      float v = 0.f;
      if (m < g.M && k0 + kk < g.K)
        v = ld(A + (g.a_kmajor ? (int64_t)m * g.lda + k : k * g.lda + m));
      As[kk][mm] = v;
      int nn;
      if (g.b_kmajor) { nn = e / 16; kk = e % 16; } else { kk = e / 64; nn = e % 64; }
      int n = n0 + nn;
      k = k0 + kk;
      v = 0.f;
      if (n < g.N && k0 + kk < g.K)
        v = ld(B + (g.b_kmajor ? (int64_t)n * g.ldb + k : k * g.ldb + n));
      Bs[kk][nn] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
  TC* C = (TC*)g.C;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int m = m0 + ty + 16 * i;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int n = n0 + tx + 16 * j;
      if (n >= g.N) continue;
      TC* c = C + (int64_t)m * g.ldc + n;
      float v = g.alpha * acc[i][j];
      if (g.beta != 0.f) v += g.beta * ld(c);
      st(c, v);
    }
  }
}

hipError_t gemm_simt(const Gemm& g, hipStream_t s) {
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, 1);
  if (g.in_t == DT_F32 && g.c_t == DT_F32) gemm_simt_kernel<float, float><<<grid, 256, 0, s>>>(g);
  else if (g.in_t == DT_F32) gemm_simt_kernel<float, bf16_t><<<grid, 256, 0, s>>>(g);
  else if (g.c_t == DT_F32) gemm_simt_kernel<bf16_t, float><<<grid, 256, 0, s>>>(g);
  else gemm_simt_kernel<bf16_t, bf16_t><<<grid, 256, 0, s>>>(g);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Attention forward: one thread per query, keys streamed through LDS 32 at a time,
// online softmax (running max m, running sum l) in fp32.
// ---------------------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ float key_elem(const Attn& a, int64_t n, int i, int d) {
  if (d < a.dnope) {
    const T* p = (const T*)a.Ka.p;
    return ld(p + n * a.Ka.tok + (int64_t)(i / a.Ka.div) * a.Ka.head + d);
  }
  const T* p = (const T*)a.Kb.p;
  return ld(p + n * a.Kb.tok + (int64_t)(i / a.Kb.div) * a.Kb.head + (d - a.dnope));
}

template <typename T>
__device__ __forceinline__ float head_elem(const HeadView& v, int64_t n, int i, int d) {
  const T* p = (const T*)v.p;
  return ld(p + n * v.tok + (int64_t)(i / v.div) * v.head + d);
}

template <typename T, int DQK, int DV>
__global__ __launch_bounds__(64) void attn_fwd_simt_kernel(Attn a) {
  __shared__ float Ks[32][DQK];
  __shared__ float Vs[32][DV];
  const int b = blockIdx.z, i = blockIdx.y;
  const int t = blockIdx.x * 64 + threadIdx.x;
  const int tq = t < a.T ? t : a.T - 1;
  const int64_t nq = (int64_t)b * a.T + tq;
  float q[DQK], o[DV];
#pragma unroll
  for (int d = 0; d < DQK; ++d) q[d] = head_elem<T>(a.Q, nq, i, d);
#pragma unroll
  for (int d = 0; d < DV; ++d) o[d] = 0.f;
  float m = -INFINITY, l = 0.f;
  const int kend = min(a.T, (int)blockIdx.x * 64 + 64);
  for (int j0 = 0; j0 < kend; j0 += 32) {
    __syncthreads();
    for (int e = threadIdx.x; e < 32 * DQK; e += 64) {
      int jj = e / DQK, d = e % DQK;
      int j = min(j0 + jj, a.T - 1);
      Ks[jj][d] = key_elem<T>(a, (int64_t)b * a.T + j, i, d);
    }
    for (int e = threadIdx.x; e < 32 * DV; e += 64) {
      int jj = e / DV, d = e % DV;
      int j = min(j0 + jj, a.T - 1);
      Vs[jj][d] = head_elem<T>(a.V, (int64_t)b * a.T + j, i, d);
    }
    __syncthreads();
    for (int jj = 0; jj < 32; ++jj) {
      int j = j0 + jj;
      if (j > t || j >= a.T) break;
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < DQK; ++d) s += q[d] * Ks[jj][d];
      s *= a.scale;
      if (s > m) {
        float corr = expf(m - s);
        l *= corr;
#pragma unroll
        for (int d = 0; d < DV; ++d) o[d] *= corr;
        m = s;
      }
      float p = expf(s - m);
      l += p;
#pragma unroll
      for (int d = 0; d < DV; ++d) o[d] += p * Vs[jj][d];
    }
  }
  if (t >= a.T) return;
  float inv = 1.f / l;
  T* O = (T*)a.O + nq * a.o_tok + (int64_t)i * DV;
#pragma unroll
  for (int d = 0; d < DV; ++d) st(O + d, o[d] * inv);
  if (a.lse) a.lse[nq * a.H + i] = m + logf(l);
}

// ---------------------------------------------------------------------------------------
// Attention backward
//   delta[n, i] = sum_d dO . O                              (softmax-backward row term)
//   dQ (one thread per query):  dq = scale * sum_j P (dP - delta) k_j
//   dK, dV (one thread per key of a Ka group, summing over the group's heads):
//     dv_j = sum P dO_t,  dk_j = scale * sum (P (dP - delta)) q_t
// ---------------------------------------------------------------------------------------
template <typename T>
__global__ void attn_delta_kernel(const void* dO_, const void* O_, int64_t o_tok, int64_t N,
                                  int H, int dv, float* __restrict__ delta) {
  // 16 lanes per (n, i) row, each lane a strided set of elements; reduce within 16 lanes
  int64_t row = (int64_t)blockIdx.x * (blockDim.x / 16) + threadIdx.x / 16;
  int sub = threadIdx.x % 16;
  bool ok = row < N * H;
  int64_t n = ok ? row / H : 0;
  int i = ok ? (int)(row % H) : 0;
  const T* dO = (const T*)dO_ + n * (int64_t)H * dv + (int64_t)i * dv;
  const T* O = (const T*)O_ + n * o_tok + (int64_t)i * dv;
  float s = 0.f;
  if (ok)
    for (int d = sub; d < dv; d += 16) s += ld(dO + d) * ld(O + d);
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if (ok && sub == 0) delta[row] = s;
}

template <typename T, int DQK, int DV>
__global__ __launch_bounds__(64) void attn_dq_simt_kernel(AttnBwd w) {
  const Attn& a = w.f;
  __shared__ float Ks[32][DQK];
  __shared__ float Vs[32][DV];
  const int b = blockIdx.z, i = blockIdx.y;
  const int t = blockIdx.x * 64 + threadIdx.x;
  const int tq = t < a.T ? t : a.T - 1;
  const int64_t nq = (int64_t)b * a.T + tq;
  float q[DQK], dq[DQK], go[DV];
#pragma unroll
  for (int d = 0; d < DQK; ++d) { q[d] = head_elem<T>(a.Q, nq, i, d); dq[d] = 0.f; }
  const T* dOp = (const T*)w.dO + nq * (int64_t)a.H * DV + (int64_t)i * DV;
#pragma unroll
  for (int d = 0; d < DV; ++d) go[d] = ld(dOp + d);
  const float lse = a.lse[nq * a.H + i];
  const float dl = w.delta[nq * a.H + i];
  const int kend = min(a.T, (int)blockIdx.x * 64 + 64);
  for (int j0 = 0; j0 < kend; j0 += 32) {
    __syncthreads();
    for (int e = threadIdx.x; e < 32 * DQK; e += 64) {
      int jj = e / DQK, d = e % DQK;
      int j = min(j0 + jj, a.T - 1);
      Ks[jj][d] = key_elem<T>(a, (int64_t)b * a.T + j, i, d);
    }
    for (int e = threadIdx.x; e < 32 * DV; e += 64) {
      int jj = e / DV, d = e % DV;
      int j = min(j0 + jj, a.T - 1);
      Vs[jj][d] = head_elem<T>(a.V, (int64_t)b * a.T + j, i, d);
    }
    __syncthreads();
    for (int jj = 0; jj < 32; ++jj) {
      int j = j0 + jj;
      if (j > t || j >= a.T) break;
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int d = 0; d < DQK; ++d) s += q[d] * Ks[jj][d];
#pragma unroll
      for (int d = 0; d < DV; ++d) dp += go[d] * Vs[jj][d];
      float p = expf(s * a.scale - lse);
      float ds = p * (dp - dl);
#pragma unroll
      for (int d = 0; d < DQK; ++d) dq[d] += ds * Ks[jj][d];
    }
  }
  if (t >= a.T) return;
  float* out = w.dq_acc + (nq * a.H + i) * DQK;
#pragma unroll
  for (int d = 0; d < DQK; ++d) out[d] = a.scale * dq[d];
}

template <typename T, int DQK, int DV>
__global__ __launch_bounds__(64) void attn_dkv_simt_kernel(AttnBwd w) {
  const Attn& a = w.f;
  __shared__ float Qs[32][DQK];
  __shared__ float Gs[32][DV];
  __shared__ float Ls[32], Ds[32];
  const int b = blockIdx.z, g = blockIdx.y;
  const int j = blockIdx.x * 64 + threadIdx.x;
  const int jq = j < a.T ? j : a.T - 1;
  const int64_t nk = (int64_t)b * a.T + jq;
  const int hpg = a.Ka.div;                  // heads per Ka group
  const int i0 = g * hpg;
  float k[DQK], v[DV], dk[DQK], dv[DV];
#pragma unroll
  for (int d = 0; d < DQK; ++d) { k[d] = key_elem<T>(a, nk, i0, d); dk[d] = 0.f; }
#pragma unroll
  for (int d = 0; d < DV; ++d) { v[d] = head_elem<T>(a.V, nk, i0, d); dv[d] = 0.f; }
  const int tstart = blockIdx.x * 64;
  for (int i = i0; i < i0 + hpg; ++i) {
    for (int t0 = tstart; t0 < a.T; t0 += 32) {
      __syncthreads();
      for (int e = threadIdx.x; e < 32 * DQK; e += 64) {
        int tt = e / DQK, d = e % DQK;
        int t = min(t0 + tt, a.T - 1);
        Qs[tt][d] = head_elem<T>(a.Q, (int64_t)b * a.T + t, i, d);
      }
      for (int e = threadIdx.x; e < 32 * DV; e += 64) {
        int tt = e / DV, d = e % DV;
        int t = min(t0 + tt, a.T - 1);
        Gs[tt][d] = ld((const T*)w.dO + ((int64_t)b * a.T + t) * a.H * DV + (int64_t)i * DV + d);
      }
      if (threadIdx.x < 32) {
        int t = min(t0 + (int)threadIdx.x, a.T - 1);
        Ls[threadIdx.x] = a.lse[((int64_t)b * a.T + t) * a.H + i];
        Ds[threadIdx.x] = w.delta[((int64_t)b * a.T + t) * a.H + i];
      }
      __syncthreads();
      for (int tt = 0; tt < 32; ++tt) {
        int t = t0 + tt;
        if (t >= a.T) break;
        if (t < j) continue;
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < DQK; ++d) s += Qs[tt][d] * k[d];
#pragma unroll
        for (int d = 0; d < DV; ++d) dp += Gs[tt][d] * v[d];
        float p = expf(s * a.scale - Ls[tt]);
        float ds = p * (dp - Ds[tt]);
#pragma unroll
        for (int d = 0; d < DV; ++d) dv[d] += p * Gs[tt][d];
#pragma unroll
        for (int d = 0; d < DQK; ++d) dk[d] += ds * Qs[tt][d];
      }
    }
  }
  if (j >= a.T) return;
  T* dKa = (T*)w.dKa + nk * w.dka_tok + (int64_t)g * a.dnope;
  for (int d = 0; d < a.dnope; ++d) st(dKa + d, a.scale * dk[d]);
  T* dV = (T*)w.dV + nk * w.dv_tok + (int64_t)g * DV;
#pragma unroll
  for (int d = 0; d < DV; ++d) st(dV + d, dv[d]);
  const int dr = DQK - a.dnope;
  if (dr > 0) {
    float* part = w.dkb_part + ((int64_t)g * ((int64_t)a.B * a.T) + nk) * dr;
    for (int e = 0; e < dr; ++e) part[e] = a.scale * dk[a.dnope + e];
  }
}

// bf16 rows of 8-element multiples: each of a row's 16 lanes loads 16-byte pieces (eight
// consecutive elements) of dO and O, so a row of 128 takes one load per tensor per lane.
// With R set, the workgroup also leaves part[blockIdx.x] = the sum over its 16 rows of
// dO . R (R laid out as dO), in a fixed order.
// (groups of 16 rows, walked by a fixed grid in a fixed order: block b takes groups b,
// b + grid, ...; with R its partial sums its groups in that order)
constexpr int DELTA_MAX_BLOCKS = 2048;
__global__ void attn_delta_bf16x8_kernel(const bf16_t* __restrict__ dO, const bf16_t* __restrict__ O,
                                         int64_t o_tok, int64_t N, int H, int dv,
                                         float* __restrict__ delta, const bf16_t* __restrict__ R,
                                         double* __restrict__ part) {
  __shared__ double red[16];
  const int sub = threadIdx.x % 16;
  auto dot8 = [](u32x4 a, u32x4 b) {
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      t += __uint_as_float(a[k] << 16) * __uint_as_float(b[k] << 16) +
           __uint_as_float(a[k] & 0xffff0000u) * __uint_as_float(b[k] & 0xffff0000u);
    return t;
  };
  const int64_t groups = (N * H + 15) / 16;
  double acc = 0.0;  // this lane's (sub == 0) rows of dO . R, in group order
  for (int64_t grp = blockIdx.x; grp < groups; grp += gridDim.x) {
    const int64_t row = grp * 16 + threadIdx.x / 16;
    const bool ok = row < N * H;
    const int64_t n = ok ? row / H : 0;
    const int i = ok ? (int)(row % H) : 0;
    const bf16_t* g = dO + n * (int64_t)H * dv + (int64_t)i * dv;
    const bf16_t* o = O + n * o_tok + (int64_t)i * dv;
    float s = 0.f, sr = 0.f;
    if (ok)
      for (int d = 8 * sub; d < dv; d += 128) {
        const u32x4 a = *(const u32x4*)(g + d);
        // O and o_s - o_t are not read again: non-temporal loads
        s += dot8(a, __builtin_nontemporal_load((const u32x4*)(o + d)));
        if (R) sr += dot8(a, __builtin_nontemporal_load((const u32x4*)(R + n * (int64_t)H * dv + (int64_t)i * dv + d)));
      }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (ok && sub == 0) delta[row] = s;
    if (R) {  // uniform
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) sr += __shfl_xor(sr, off, 64);
      acc += (double)sr;
    }
  }
  if (R) {
    if (sub == 0) red[threadIdx.x / 16] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
      double t = 0.0;
      for (int r = 0; r < (int)(blockDim.x / 16); ++r) t += red[r];
      part[blockIdx.x] = t;
    }
  }
}

static int64_t delta_grid(int64_t rows) {
  const int64_t g = (rows + 15) / 16;
  return g < DELTA_MAX_BLOCKS ? g : DELTA_MAX_BLOCKS;
}
int64_t attn_delta_parts(int64_t rows) { return delta_grid(rows); }

template <typename T>
hipError_t delta_launch(const AttnBwd& w, hipStream_t s) {
  const Attn& a = w.f;
  int64_t rows = (int64_t)a.B * a.T * a.H;
  if (a.t == DT_BF16 && a.dv % 8 == 0 && a.o_tok % 8 == 0 && (uintptr_t)w.dO % 16 == 0 &&
      (uintptr_t)a.O % 16 == 0) {
    attn_delta_bf16x8_kernel<<<(unsigned)delta_grid(rows), 256, 0, s>>>(
        (const bf16_t*)w.dO, (const bf16_t*)a.O, a.o_tok, (int64_t)a.B * a.T, a.H, a.dv, w.delta,
        (const bf16_t*)w.loss_ref, w.loss_part);
    return hipGetLastError();
  }
  if (w.loss_ref) return hipErrorInvalidValue;  // the dot needs the bf16 row path
  attn_delta_kernel<T><<<(unsigned)((rows + 15) / 16), 256, 0, s>>>(w.dO, a.O, a.o_tok,
                                                                  (int64_t)a.B * a.T, a.H, a.dv,
                                                                  w.delta);
  return hipGetLastError();
}

hipError_t attn_delta(const AttnBwd& w, hipStream_t s) {
  return w.f.t == DT_BF16 ? delta_launch<bf16_t>(w, s) : delta_launch<float>(w, s);
}

template <typename T, int DQK, int DV>
static hipError_t simt_fwd_launch(const Attn& a, hipStream_t s) {
  dim3 grid((a.T + 63) / 64, a.H, a.B);
  attn_fwd_simt_kernel<T, DQK, DV><<<grid, 64, 0, s>>>(a);
  return hipGetLastError();
}

template <typename T, int DQK, int DV>
static hipError_t simt_bwd_launch(const AttnBwd& w, hipStream_t s) {
  const Attn& a = w.f;
  hipError_t e = attn_delta(w, s);
  if (e != hipSuccess) return e;
  dim3 gq((a.T + 63) / 64, a.H, a.B);
  attn_dq_simt_kernel<T, DQK, DV><<<gq, 64, 0, s>>>(w);
  dim3 gk((a.T + 63) / 64, w.n_ka_groups, a.B);
  attn_dkv_simt_kernel<T, DQK, DV><<<gk, 64, 0, s>>>(w);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return dq_finish(w.dq_acc, w.dq, a.t, a.B * a.T, a.T, a.H, DQK, a.dnope, w.rdiv, w.cos_t,
                   w.sin_t, s);
}

#define MLA_SIMT_SHAPES(X) \
  X(64, 64) X(128, 128) X(96, 64) X(128, 64) X(192, 128) X(64, 32) X(32, 32) X(16, 16) X(12, 8) X(8, 8)

bool attn_simt_supported(int dqk, int dv) {
#define X(a_, b_) if (dqk == a_ && dv == b_) return true;
  MLA_SIMT_SHAPES(X)
#undef X
  return false;
}

hipError_t attn_fwd_simt(const Attn& a, hipStream_t s) {
#define X(a_, b_)                                                                      \
  if (a.dqk == a_ && a.dv == b_)                                                      \
    return a.t == DT_BF16 ? simt_fwd_launch<bf16_t, a_, b_>(a, s)                      \
                          : simt_fwd_launch<float, a_, b_>(a, s);
  MLA_SIMT_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

hipError_t attn_bwd_simt(const AttnBwd& w, hipStream_t s) {
  const Attn& a = w.f;
#define X(a_, b_)                                                                      \
  if (a.dqk == a_ && a.dv == b_)                                                      \
    return a.t == DT_BF16 ? simt_bwd_launch<bf16_t, a_, b_>(w, s)                      \
                          : simt_bwd_launch<float, a_, b_>(w, s);
  MLA_SIMT_SHAPES(X)
#undef X
  return hipErrorInvalidValue;
}

}  // namespace mla
