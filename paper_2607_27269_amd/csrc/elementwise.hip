// Bandwidth-bound kernels of the reconstruction step: RoPE tables and rotation, the
// fused Eq. 11 loss + gradient, and the finishing passes of the attention backward.
// Every kernel reads and writes HBM once, with consecutive lanes on consecutive
// addresses, and reduces inside a wavefront with cross-lane shuffles.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace mla {

// ---------------------------------------------------------------------------------------
// RoPE (Sec. 3.1): R_t rotates rotate-half pair p of a head by t * inv_freq[p].
// ---------------------------------------------------------------------------------------
__global__ void rope_table_kernel(const float* __restrict__ inv_freq, int G, int T, int np,
                                  float* __restrict__ cos_t, float* __restrict__ sin_t) {
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = (int64_t)G * T * np;
  if (idx >= total) return;
  int p = (int)(idx % np);
  int t = (int)((idx / np) % T);
  int g = (int)(idx / ((int64_t)np * T));
  double ang = (double)t * (double)inv_freq[g * np + p];
  cos_t[idx] = (float)cos(ang);
  sin_t[idx] = (float)sin(ang);
}

hipError_t rope_tables(const float* inv_freq, int G, int T, int npairs, float* cos_t,
                       float* sin_t, hipStream_t s) {
  int64_t total = (int64_t)G * T * npairs;
  if (total == 0) return hipSuccess;
  prof_begin(KC_ELEM, s);
  rope_table_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(inv_freq, G, T, npairs,
                                                                    cos_t, sin_t);
  prof_end(KC_ELEM, s, 0.0, (double)total * 8.0 + G * npairs * 4.0, KLABEL("rope_table_kernel"));
  return hipGetLastError();
}

template <typename T> struct Vec4;
template <> struct Vec4<float> {
  static __device__ __forceinline__ f32x4 load(const float* p) { return *(const f32x4*)p; }
  static __device__ __forceinline__ void store(float* p, f32x4 v) { *(f32x4*)p = v; }
};
template <> struct Vec4<bf16_t> {
  static __device__ __forceinline__ f32x4 load(const bf16_t* p) {
    u32x2 w = *(const u32x2*)p;
    return f32x4{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xffff0000u),
                 __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xffff0000u)};
  }
  static __device__ __forceinline__ void store(bf16_t* p, f32x4 v) {
    *(u32x2*)p = u32x2{pack2bf(v[0], v[1]), pack2bf(v[2], v[3])};
  }
};

// in-place rotation of pairs (p, p + np), 4 consecutive pairs per thread
template <typename T>
__global__ void rope_apply_kernel(T* __restrict__ x, int N, int Tseq, int nheads, int64_t tok,
                                  int64_t head, int off, int np, int div,
                                  const float* __restrict__ cos_t,
                                  const float* __restrict__ sin_t, float sgn) {
  const int nq = np / 4;
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = (int64_t)N * nheads * nq;
  if (idx >= total) return;
  int p = (int)(idx % nq) * 4;
  int h = (int)((idx / nq) % nheads);
  int64_t n = idx / ((int64_t)nq * nheads);
  int t = (int)(n % Tseq);
  int g = h / div;
  const int64_t ti = ((int64_t)g * Tseq + t) * np + p;
  f32x4 c = *(const f32x4*)(cos_t + ti), sn = *(const f32x4*)(sin_t + ti) * sgn;
  T* base = x + n * tok + (int64_t)h * head + off;
  f32x4 x1 = Vec4<T>::load(base + p), x2 = Vec4<T>::load(base + p + np);
  Vec4<T>::store(base + p, x1 * c - x2 * sn);
  Vec4<T>::store(base + p + np, x1 * sn + x2 * c);
}

// the same for bf16 with 8 consecutive pairs per thread (16-byte loads and stores)
__global__ void rope_apply8_kernel(bf16_t* __restrict__ x, int N, int Tseq, int nheads, int64_t tok,
                                   int64_t head, int off, int np, int div,
                                   const float* __restrict__ cos_t,
                                   const float* __restrict__ sin_t, float sgn) {
  const int nq = np / 8;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)N * nheads * nq) return;
  const int p = (int)(idx % nq) * 8;
  const int h = (int)((idx / nq) % nheads);
  const int64_t n = idx / ((int64_t)nq * nheads);
  const int t = (int)(n % Tseq), g = h / div;
  const float* cp = cos_t + ((int64_t)g * Tseq + t) * np + p;
  const float* sp = sin_t + ((int64_t)g * Tseq + t) * np + p;
  bf16_t* base = x + n * tok + (int64_t)h * head + off;
  const u32x4 a = *(const u32x4*)(base + p), b = *(const u32x4*)(base + p + np);
  u32x4 oa, ob;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const f32x4 c = *(const f32x4*)(cp + 4 * q), sn = *(const f32x4*)(sp + 4 * q) * sgn;
    const f32x4 x1 = {__uint_as_float(a[2 * q] << 16), __uint_as_float(a[2 * q] & 0xffff0000u),
                      __uint_as_float(a[2 * q + 1] << 16), __uint_as_float(a[2 * q + 1] & 0xffff0000u)};
    const f32x4 x2 = {__uint_as_float(b[2 * q] << 16), __uint_as_float(b[2 * q] & 0xffff0000u),
                      __uint_as_float(b[2 * q + 1] << 16), __uint_as_float(b[2 * q + 1] & 0xffff0000u)};
    const f32x4 r1 = x1 * c - x2 * sn, r2 = x1 * sn + x2 * c;
    oa[2 * q] = pack2bf(r1[0], r1[1]);
    oa[2 * q + 1] = pack2bf(r1[2], r1[3]);
    ob[2 * q] = pack2bf(r2[0], r2[1]);
    ob[2 * q + 1] = pack2bf(r2[2], r2[3]);
  }
  *(u32x4*)(base + p) = oa;
  *(u32x4*)(base + p + np) = ob;
}

hipError_t rope_apply(void* x, DType t, int N, int T, int nheads, int64_t tok, int64_t head,
                      int off, int npairs, int div, const float* cos_t, const float* sin_t,
                      hipStream_t s, bool inverse) {
  const float sgn = inverse ? -1.f : 1.f;
  int64_t total = (int64_t)N * nheads * (npairs / 4);
  if (total == 0) return hipSuccess;
  unsigned grid = (unsigned)((total + 255) / 256);
  prof_begin(KC_ELEM, s);
  const bool v8 = t == DT_BF16 && npairs % 8 == 0 && tok % 8 == 0 && head % 8 == 0 &&
                  off % 8 == 0 && (uintptr_t)x % 16 == 0;
  if (v8) {
    const int64_t total8 = (int64_t)N * nheads * (npairs / 8);
    rope_apply8_kernel<<<(unsigned)((total8 + 255) / 256), 256, 0, s>>>(
        (bf16_t*)x, N, T, nheads, tok, head, off, npairs, div, cos_t, sin_t, sgn);
  } else if (t == DT_BF16)
    rope_apply_kernel<bf16_t><<<grid, 256, 0, s>>>((bf16_t*)x, N, T, nheads, tok, head, off,
                                                   npairs, div, cos_t, sin_t, sgn);
  else
    rope_apply_kernel<float><<<grid, 256, 0, s>>>((float*)x, N, T, nheads, tok, head, off,
                                                  npairs, div, cos_t, sin_t, sgn);
  prof_end(KC_ELEM, s, 0.0, (double)N * nheads * npairs * 4.0 * dsize(t), 
           v8 ? KLABEL("rope_apply8_kernel") : KLABEL("rope_apply_kernel"));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Backward finishing: rotate the rotary gradients back with R^T and cast.
// ---------------------------------------------------------------------------------------
template <typename T>
__global__ void dq_finish_kernel(const float* __restrict__ acc, T* __restrict__ dq, int N,
                                 int Tseq, int H, int dqk, int dnope, int rdiv,
                                 const float* __restrict__ cos_t,
                                 const float* __restrict__ sin_t) {
  // one thread per 4 elements: chunks [0, dnope/4) copy, chunks [dnope/4, +np/4) rotate
  // 4 pairs (p .. p+3, p+np .. p+np+3) back with R^T
  const int np = (dqk - dnope) / 2;
  const int per_head = dnope / 4 + np / 4;
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = (int64_t)N * H * per_head;
  if (idx >= total) return;
  int e = (int)(idx % per_head);
  int i = (int)((idx / per_head) % H);
  int64_t n = idx / ((int64_t)per_head * H);
  const float* a = acc + (n * H + i) * dqk;
  T* o = dq + (n * H + i) * dqk;
  if (e < dnope / 4) {
    Vec4<T>::store(o + 4 * e, *(const f32x4*)(a + 4 * e));
    return;
  }
  int p = 4 * (e - dnope / 4);
  int t = (int)(n % Tseq);
  int g = i / rdiv;
  const int64_t ti = ((int64_t)g * Tseq + t) * np + p;
  f32x4 c = *(const f32x4*)(cos_t + ti), sn = *(const f32x4*)(sin_t + ti);
  f32x4 x1 = *(const f32x4*)(a + dnope + p), x2 = *(const f32x4*)(a + dnope + p + np);
  Vec4<T>::store(o + dnope + p, x1 * c + x2 * sn);
  Vec4<T>::store(o + dnope + p + np, x2 * c - x1 * sn);
}

hipError_t dq_finish(const float* dq_acc, void* dq, DType t, int N, int T, int H, int dqk,
                     int dnope, int rdiv, const float* cos_t, const float* sin_t,
                     hipStream_t s) {
  int64_t total = (int64_t)N * H * (dnope / 4 + (dqk - dnope) / 8);
  if (total == 0) return hipSuccess;
  unsigned grid = (unsigned)((total + 255) / 256);
  prof_begin(KC_ELEM, s);
  if (t == DT_BF16)
    dq_finish_kernel<bf16_t><<<grid, 256, 0, s>>>(dq_acc, (bf16_t*)dq, N, T, H, dqk, dnope,
                                                  rdiv, cos_t, sin_t);
  else
    dq_finish_kernel<float><<<grid, 256, 0, s>>>(dq_acc, (float*)dq, N, T, H, dqk, dnope, rdiv,
                                                 cos_t, sin_t);
  prof_end(KC_ELEM, s, 0.0, (double)N * H * dqk * (4.0 + dsize(t)), KLABEL("dq_finish_kernel"));
  return hipGetLastError();
}

template <typename T>
__global__ void dkpe_finish_kernel(const float* __restrict__ part, T* __restrict__ out,
                                   int64_t out_tok, int N, int Tseq, int Gr, int per, int dr,
                                   const float* __restrict__ cos_t,
                                   const float* __restrict__ sin_t) {
  int np = dr / 2;
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = (int64_t)N * Gr * np;
  if (idx >= total) return;
  int p = (int)(idx % np);
  int r = (int)((idx / np) % Gr);
  int64_t n = idx / ((int64_t)np * Gr);
  float x1 = 0.f, x2 = 0.f;
  for (int k = 0; k < per; ++k) {  // fixed order: deterministic
    const float* src = part + ((int64_t)(r * per + k) * N + n) * dr;
    x1 += src[p];
    x2 += src[p + np];
  }
  int t = (int)(n % Tseq);
  float c = cos_t[((int64_t)r * Tseq + t) * np + p];
  float sn = sin_t[((int64_t)r * Tseq + t) * np + p];
  T* o = out + n * out_tok + (int64_t)r * dr;
  st(o + p, x1 * c + x2 * sn);
  st(o + p + np, -x1 * sn + x2 * c);
}

hipError_t dkpe_finish(const float* part, void* out, DType t, int64_t out_tok, int N, int T,
                       int Gr, int per, int drope, const float* cos_t, const float* sin_t,
                       hipStream_t s) {
  int64_t total = (int64_t)N * Gr * (drope / 2);
  if (total == 0) return hipSuccess;
  unsigned grid = (unsigned)((total + 255) / 256);
  prof_begin(KC_ELEM, s);
  if (t == DT_BF16)
    dkpe_finish_kernel<bf16_t><<<grid, 256, 0, s>>>(part, (bf16_t*)out, out_tok, N, T, Gr, per,
                                                    drope, cos_t, sin_t);
  else
    dkpe_finish_kernel<float><<<grid, 256, 0, s>>>(part, (float*)out, out_tok, N, T, Gr, per,
                                                   drope, cos_t, sin_t);
  prof_end(KC_ELEM, s, 0.0, (double)N * Gr * drope * (4.0 * per + dsize(t)), KLABEL("dkpe_finish_kernel"));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Eq. 11: L = sum (M (A_s - A_t))^2 / (D sum M), dA = 2 M (A_s - A_t) / (D sum M).
// Pass 1 counts the valid tokens, pass 2 streams A_s and A_t once (float4 loads), writes
// dA and leaves one fp64 partial (sse, ref) per workgroup, pass 3 sums the partials in a
// fixed order.  A fixed grid makes the result bitwise reproducible.
// ---------------------------------------------------------------------------------------
static constexpr int LOSS_BLOCKS = 2048;
static constexpr int LOSS_THREADS = 256;

struct LossScratch {
  double count;
  float scale;  // 2 / (D count): dL/dA per unit of masked difference (0 if nothing is valid)
  float pad_f;
  double sse;   // the last loss's sum of squared masked differences
  double pad[29];
  double part[2 * LOSS_BLOCKS];
};

size_t loss_scratch_bytes() { return sizeof(LossScratch); }

__global__ void mask_count_kernel(const uint8_t* __restrict__ mask, int64_t N, int D,
                                  LossScratch* __restrict__ ws) {
  __shared__ double red[16];
  double c = 0.0;
  if (mask) {
    // 16 mask bytes per thread and step where the mask is 16-byte aligned, the tail byte-wise
    const int64_t nv = (uintptr_t)mask % 16 == 0 ? N / 16 : 0;
    int cnt = 0;
    for (int64_t v = threadIdx.x; v < nv; v += blockDim.x) {
      const u32x4 w = ((const u32x4*)mask)[v];
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int b = 0; b < 4; ++b) cnt += ((w[k] >> (8 * b)) & 0xffu) != 0u;
    }
    for (int64_t i = nv * 16 + threadIdx.x; i < N; i += blockDim.x) cnt += mask[i] ? 1 : 0;
    c = (double)cnt;
  } else if (threadIdx.x == 0) {
    c = (double)N;
  }
  c = warp_sum_d(c);
  int w = threadIdx.x / 64, l = threadIdx.x % 64;
  if (l == 0) red[w] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int i = 0; i < (int)(blockDim.x / 64); ++i) t += red[i];
    ws->count = t;
    ws->scale = t > 0.0 ? (float)(2.0 / ((double)D * t)) : 0.f;
  }
}

template <typename T>
__device__ __forceinline__ void store4(T* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  *(float4*)p = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
  *(u32x2*)p = u32x2{pack2bf(a, b), pack2bf(c, d)};
}

template <typename T>
__global__ __launch_bounds__(LOSS_THREADS) void loss_main_kernel(
    const float* __restrict__ As, const float* __restrict__ At,
    const uint8_t* __restrict__ mask, int64_t N, int D, T* __restrict__ dA,
    LossScratch* __restrict__ ws) {
  __shared__ double red[2][LOSS_THREADS / 64];
  const double cnt = ws->count;
  const float g = cnt > 0.0 ? (float)(2.0 / ((double)D * cnt)) : 0.f;
  const int64_t nvec = N * (int64_t)D / 4;
  const int dv = D / 4;
  float sse = 0.f, ref = 0.f;
  for (int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; v < nvec;
       v += (int64_t)gridDim.x * blockDim.x) {
    int64_t n = v / dv;
    float m = (mask == nullptr || mask[n]) ? 1.f : 0.f;
    float4 a = ((const float4*)As)[v];
    // (no reference: As already holds the difference A_s - A_t)
    float4 b = At ? ((const float4*)At)[v] : make_float4(0.f, 0.f, 0.f, 0.f);
    float e0 = m * (a.x - b.x), e1 = m * (a.y - b.y), e2 = m * (a.z - b.z), e3 = m * (a.w - b.w);
    sse += e0 * e0 + e1 * e1 + e2 * e2 + e3 * e3;
    float r0 = m * b.x, r1 = m * b.y, r2 = m * b.z, r3 = m * b.w;
    ref += r0 * r0 + r1 * r1 + r2 * r2 + r3 * r3;
    if (dA) store4<T>(dA + v * 4, g * e0, g * e1, g * e2, g * e3);
  }
  double s = warp_sum_d((double)sse), r = warp_sum_d((double)ref);
  int w = threadIdx.x / 64, l = threadIdx.x % 64;
  if (l == 0) {
    red[0][w] = s;
    red[1][w] = r;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double ts = 0.0, tr = 0.0;
    for (int i = 0; i < LOSS_THREADS / 64; ++i) {
      ts += red[0][i];
      tr += red[1][i];
    }
    ws->part[2 * blockIdx.x] = ts;
    ws->part[2 * blockIdx.x + 1] = tr;
  }
}

__global__ __launch_bounds__(256) void loss_final_kernel(LossScratch* __restrict__ ws,
                                                         int nblocks, int D, bool has_ref,
                                                         float* __restrict__ loss) {
  // thread t sums partials t, t+256, ... in order; then a fixed tree over the 256 threads
  __shared__ double red[2][256];
  double s = 0.0, r = 0.0;
  for (int i = threadIdx.x; i < nblocks; i += 256) {
    s += ws->part[2 * i];
    r += ws->part[2 * i + 1];
  }
  red[0][threadIdx.x] = s;
  red[1][threadIdx.x] = r;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      red[0][threadIdx.x] += red[0][threadIdx.x + w];
      red[1][threadIdx.x] += red[1][threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x != 0) return;
  s = red[0][0];
  r = red[1][0];
  ws->sse = s;
  double den = (double)D * ws->count;
  if (den == 0.0) {
    loss[0] = 0.f;
    loss[1] = 0.f;
    return;
  }
  loss[0] = (float)(s / den);
  // (a zero reference is the only degenerate denominator: a NaN one propagates)
  loss[1] = !has_ref ? NAN : r == 0.0 ? (s == 0.0 ? 0.f : INFINITY) : (float)(s / r);
}

hipError_t recon_loss(const float* A_s, const float* A_t, const uint8_t* mask, int64_t N, int D,
                      float* loss, void* dA, DType t, void* scratch, hipStream_t s) {
  LossScratch* ws = (LossScratch*)scratch;
  int64_t nvec = N * (int64_t)D / 4;
  int blocks = (int)std::min<int64_t>(LOSS_BLOCKS, std::max<int64_t>(1, (nvec + LOSS_THREADS - 1) / LOSS_THREADS));
  prof_begin(KC_LOSS, s);
  mask_count_kernel<<<1, 1024, 0, s>>>(mask, N, D, ws);
  if (t == DT_BF16)
    loss_main_kernel<bf16_t><<<blocks, LOSS_THREADS, 0, s>>>(A_s, A_t, mask, N, D, (bf16_t*)dA, ws);
  else
    loss_main_kernel<float><<<blocks, LOSS_THREADS, 0, s>>>(A_s, A_t, mask, N, D, (float*)dA, ws);
  loss_final_kernel<<<1, 256, 0, s>>>(ws, blocks, D, A_t != nullptr, loss);
  double bytes = (double)N * D * ((A_t ? 8.0 : 4.0) + (dA ? dsize(t) : 0)) + (mask ? N : 0);
  prof_end(KC_LOSS, s, 0.0, bytes, KLABEL("mask_count_kernel + loss_main_kernel + loss_final_kernel"));
  return hipGetLastError();
}

// Eq. 11 from per-tile sums of squared masked differences ------------------------------
hipError_t loss_prepare(const uint8_t* mask, int64_t N, int D, void* scratch, hipStream_t s) {
  prof_begin(KC_LOSS, s);
  mask_count_kernel<<<1, 1024, 0, s>>>(mask, N, D, (LossScratch*)scratch);
  prof_end(KC_LOSS, s, 0.0, mask ? (double)N : 0.0, KLABEL("mask_count_kernel"));
  return hipGetLastError();
}

const float* loss_scale(const void* scratch) { return &((const LossScratch*)scratch)->scale; }

// the fixed-order sum of part[i * stride], i < n, for a 256-thread block: thread t sums
// i = t, t+256, ... in order, then a fixed tree over the threads; the total is valid in
// thread 0
__device__ double sum_parts_ordered(const double* __restrict__ part, int n, int stride) {
  __shared__ double red[256];
  double v = 0.0;
  for (int i = threadIdx.x; i < n; i += 256) v += part[(int64_t)i * stride];
  red[threadIdx.x] = v;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  return red[0];
}

__global__ __launch_bounds__(256) void loss_parts_kernel(const double* __restrict__ part,
                                                         int nparts, int D,
                                                         LossScratch* __restrict__ ws,
                                                         float* __restrict__ loss) {
  const double v = sum_parts_ordered(part, nparts, 1);
  if (threadIdx.x != 0) return;
  ws->sse = v;
  const double den = (double)D * ws->count;
  loss[0] = den > 0.0 ? (float)(v / den) : 0.f;
  loss[1] = NAN;
}

hipError_t loss_from_parts(const double* part, int nparts, int D, float* loss,
                           void* scratch, hipStream_t s) {
  prof_begin(KC_LOSS, s);
  loss_parts_kernel<<<1, 256, 0, s>>>(part, nparts, D, (LossScratch*)scratch, loss);
  prof_end(KC_LOSS, s, 0.0, 8.0 * nparts, KLABEL("loss_parts_kernel"));
  return hipGetLastError();
}

// Eq. 11 from the partials of sum dO . (o_s - o_t): with dO = 2 M Y / (D sum M), the
// squared-error sum is sum M Y . (o_s - o_t) = dot D count / 2 and L = dot / 2
// (tens of thousands of partials: thread t sums the contiguous run t * per .. in order,
// with independent loads, then a fixed tree over the 1024 threads)
__global__ __launch_bounds__(1024) void loss_dot_kernel(const double* __restrict__ part,
                                                        int nparts, int D,
                                                        LossScratch* __restrict__ ws,
                                                        float* __restrict__ loss) {
  __shared__ double red[1024];
  const int per = (nparts + 1023) / 1024;
  const int b0 = (int)threadIdx.x * per, b1 = min(nparts, b0 + per);
  double v = 0.0;
  for (int i = b0; i < b1; ++i) v += part[i];
  red[threadIdx.x] = v;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  v = red[0];
  if (threadIdx.x != 0) return;
  const double cnt = ws->count;
  ws->sse = cnt > 0.0 ? v * (double)D * cnt / 2.0 : 0.0;
  loss[0] = cnt > 0.0 ? (float)(v / 2.0) : 0.f;
  loss[1] = NAN;
}

hipError_t loss_from_dot(const double* part, int64_t nparts, int D, float* loss, void* scratch,
                         hipStream_t s) {
  prof_begin(KC_LOSS, s);
  loss_dot_kernel<<<1, 1024, 0, s>>>(part, (int)nparts, D, (LossScratch*)scratch, loss);
  prof_end(KC_LOSS, s, 0.0, 8.0 * nparts, KLABEL("loss_dot_kernel"));
  return hipGetLastError();
}

// relative error: the kept sum of squared masked differences over sum M A_t^2
__global__ __launch_bounds__(256) void loss_rel_kernel(const double* __restrict__ part,
                                                       int nparts, int stride,
                                                       const LossScratch* __restrict__ ws,
                                                       float* __restrict__ loss) {
  const double r = sum_parts_ordered(part, nparts, stride);
  if (threadIdx.x != 0) return;
  const double e = ws->sse;
  loss[1] = ws->count == 0.0 ? 0.f : r == 0.0 ? (e == 0.0 ? 0.f : INFINITY) : (float)(e / r);
}

hipError_t loss_rel_from_parts(const double* part, int nparts, int stride, float* loss,
                               const void* scratch, hipStream_t s) {
  prof_begin(KC_LOSS, s);
  loss_rel_kernel<<<1, 256, 0, s>>>(part, nparts, stride, (const LossScratch*)scratch, loss);
  prof_end(KC_LOSS, s, 0.0, 8.0 * nparts, KLABEL("loss_rel_kernel"));
  return hipGetLastError();
}

hipError_t loss_rel_fp32(const float* A_t, const uint8_t* mask, int64_t N, int D, float* loss,
                         void* scratch, hipStream_t s) {
  LossScratch* ws = (LossScratch*)scratch;
  const int64_t nvec = N * (int64_t)D / 4;
  const int blocks = (int)std::min<int64_t>(LOSS_BLOCKS, std::max<int64_t>(1, (nvec + LOSS_THREADS - 1) / LOSS_THREADS));
  prof_begin(KC_LOSS, s);
  mask_count_kernel<<<1, 1024, 0, s>>>(mask, N, D, ws);
  // with no reference, the first partial of each workgroup is its sum of M A_t^2
  loss_main_kernel<float><<<blocks, LOSS_THREADS, 0, s>>>(A_t, nullptr, mask, N, D, nullptr, ws);
  loss_rel_kernel<<<1, 256, 0, s>>>(ws->part, blocks, 2, ws, loss);
  prof_end(KC_LOSS, s, 0.0, (double)N * D * 4.0 + (mask ? N : 0),
           KLABEL("mask_count_kernel + loss_main_kernel + loss_rel_kernel"));
  return hipGetLastError();
}

// four consecutive elements (8- or 16-byte aligned) as fp32
__device__ __forceinline__ f32x4 load4(const float* p) { return *(const f32x4*)p; }
__device__ __forceinline__ f32x4 load4(const bf16_t* p) {
  const u32x2 w = *(const u32x2*)p;
  return f32x4{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xffff0000u),
               __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xffff0000u)};
}

// out = a - b elementwise (n elements of the storage dtype), computed in fp32
template <typename T>
__global__ void sub_kernel(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ out,
                           int64_t n) {
  const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i0 >= n) return;
  if (i0 + 4 <= n) {
    const f32x4 x = load4(a + i0), y = load4(b + i0);
    store4<T>(out + i0, x[0] - y[0], x[1] - y[1], x[2] - y[2], x[3] - y[3]);
  } else {
    for (int64_t i = i0; i < n; ++i) st<T>(out + i, ld(a + i) - ld(b + i));
  }
}

hipError_t sub_elementwise(const void* a, const void* b, void* out, int64_t n, DType t,
                           hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((n + 4 * 256 - 1) / (4 * 256));
  prof_begin(KC_ELEM, s);
  if (t == DT_BF16)
    sub_kernel<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)a, (const bf16_t*)b, (bf16_t*)out, n);
  else
    sub_kernel<float><<<grid, 256, 0, s>>>((const float*)a, (const float*)b, (float*)out, n);
  prof_end(KC_ELEM, s, 0.0, 3.0 * n * dsize(t), KLABEL("sub_kernel"));
  return hipGetLastError();
}

// AdamW over up to ADAMW_MAX tensors in one launch (blockIdx.y = tensor) ----------------
struct AdamwArgs {
  AdamwTensor t[ADAMW_MAX];
  float lr, b1, b2, eps, wd, bc1, bc2;  // bc = 1 / (1 - beta^step)
};

template <typename T>
__device__ __forceinline__ void adamw_one(const AdamwArgs& a, float& w, float& m, float& v, float g) {
  m = a.b1 * m + (1.f - a.b1) * g;
  v = a.b2 * v + (1.f - a.b2) * g * g;
  w = w - a.lr * ((m * a.bc1) / (sqrtf(v * a.bc2) + a.eps) + a.wd * w);
}

template <typename T>
__global__ __launch_bounds__(256) void adamw_kernel(AdamwArgs a) {
  const AdamwTensor& t = a.t[blockIdx.y];
  const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i0 >= t.n) return;
  T* w = (T*)t.w;
  if (i0 + 4 <= t.n) {
    f32x4 ws = *(const f32x4*)(t.master + i0), ms = *(const f32x4*)(t.m + i0);
    f32x4 vs = *(const f32x4*)(t.v + i0);
    const f32x4 gs = *(const f32x4*)(t.g + i0);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float wk = ws[k], mk = ms[k], vk = vs[k];
      adamw_one<T>(a, wk, mk, vk, gs[k]);
      ws[k] = wk;
      ms[k] = mk;
      vs[k] = vk;
    }
    *(f32x4*)(t.master + i0) = ws;
    *(f32x4*)(t.m + i0) = ms;
    *(f32x4*)(t.v + i0) = vs;
    store4<T>(w + i0, ws[0], ws[1], ws[2], ws[3]);
  } else {
    for (int64_t i = i0; i < t.n; ++i) {
      float wi = t.master[i], mi = t.m[i], vi = t.v[i];
      adamw_one<T>(a, wi, mi, vi, t.g[i]);
      t.master[i] = wi;
      t.m[i] = mi;
      t.v[i] = vi;
      st<T>(w + i, wi);
    }
  }
}

hipError_t adamw_step(const AdamwTensor* t, int count, DType wt, float lr, float beta1,
                      float beta2, float eps, float weight_decay, int step, hipStream_t s) {
  if (count < 1 || count > ADAMW_MAX) return hipErrorInvalidValue;
  AdamwArgs a;
  int64_t nmax = 0;
  double bytes = 0.0;
  for (int i = 0; i < ADAMW_MAX; ++i) {
    a.t[i] = i < count ? t[i] : AdamwTensor{nullptr, nullptr, nullptr, nullptr, nullptr, 0};
    nmax = std::max(nmax, a.t[i].n);
    bytes += (double)a.t[i].n * (4.0 * 7 + dsize(wt));
  }
  a.lr = lr; a.b1 = beta1; a.b2 = beta2; a.eps = eps; a.wd = weight_decay;
  a.bc1 = (float)(1.0 / (1.0 - std::pow((double)beta1, step)));
  a.bc2 = (float)(1.0 / (1.0 - std::pow((double)beta2, step)));
  if (nmax == 0) return hipSuccess;
  const dim3 grid((unsigned)((nmax + 1023) / 1024), (unsigned)count);
  prof_begin(KC_ELEM, s);
  if (wt == DT_BF16) adamw_kernel<bf16_t><<<grid, 256, 0, s>>>(a);
  else adamw_kernel<float><<<grid, 256, 0, s>>>(a);
  prof_end(KC_ELEM, s, 0.0, bytes, KLABEL("adamw_kernel"));
  return hipGetLastError();
}

// Residual add and RMS normalisation of one row per workgroup -------------------------------
// x[n] += A[n] (A optional); h[n] = x[n] / sqrt(mean(x[n]^2) + eps) in h's dtype.  The row
// sum runs in a fixed order (per-thread strided partials, then a fixed tree).
template <typename T>
__global__ __launch_bounds__(256) void residual_rmsnorm_kernel(float* __restrict__ x,
                                                               const float* __restrict__ A,
                                                               T* __restrict__ h, int D,
                                                               float eps) {
  __shared__ float red[256];
  const int64_t row = blockIdx.x;
  float* xr = x + row * D;
  const float* ar = A ? A + row * D : nullptr;
  float ss = 0.f;
  for (int d = threadIdx.x; d < D; d += 256) {
    float v = xr[d];
    if (ar) {
      v += ar[d];
      xr[d] = v;
    }
    ss += v * v;
  }
  red[threadIdx.x] = ss;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const float inv = 1.f / sqrtf(red[0] / (float)D + eps);
  T* hr = h + row * D;
  for (int d = threadIdx.x; d < D; d += 256) st<T>(hr + d, xr[d] * inv);
}

hipError_t residual_rmsnorm(float* x, const float* A, void* h, int64_t N, int D, DType t, float eps,
                            hipStream_t s) {
  if (N <= 0 || D <= 0) return hipSuccess;
  prof_begin(KC_ELEM, s);
  if (t == DT_BF16)
    residual_rmsnorm_kernel<bf16_t><<<(unsigned)N, 256, 0, s>>>(x, A, (bf16_t*)h, D, eps);
  else
    residual_rmsnorm_kernel<float><<<(unsigned)N, 256, 0, s>>>(x, A, (float*)h, D, eps);
  prof_end(KC_ELEM, s, 0.0, (double)N * D * ((A ? 12.0 : 4.0) + dsize(t)), KLABEL("residual_rmsnorm_kernel"));
  return hipGetLastError();
}

}  // namespace mla
