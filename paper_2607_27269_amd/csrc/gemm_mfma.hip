// bf16 GEMM on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation.
//
//   C[m, n] = alpha * sum_k A(m, k) B(n, k) + beta * C[m, n]
//
// Either operand may be K-contiguous ("k-major": rows of a weight or of activations) or
// M/N-contiguous (the transposed operand of the weight-gradient and data-gradient
// products).  A workgroup owns a BM x BN output tile and walks K in BK = 64 slices staged
// in LDS in the operand's natural layout: k-major tiles as [row][k] (16-byte operand reads,
// 8 consecutive k per lane) and m-major tiles as [k][row], whose operands come from
// gfx950's transposing LDS read.  Both give the same k order inside an MFMA step, so the
// two kinds mix freely.  LDS is double buffered: full K slices are copied straight from
// HBM into LDS (global_load_lds) while the current slice feeds the matrix cores; a ragged
// last slice goes through registers with zero fill.  Operand fragments are double buffered
// in registers as well: the LDS reads of the next 16-wide k step are in flight while the
// matrix cores work on the current one, and the first step of the next slice is read
// right after the barrier that publishes it.  The epilogue stages each 32-row strip of a
// wavefront's tile in LDS and writes it back with 16-byte (fp32) or 8-byte (bf16) stores.  Row strides are padded so that the
// operand reads of a wavefront hit distinct banks.  Large problems use 256 x 256 tiles on
// 8 wavefronts (128 x 64 each), which halves the LDS bytes per MFMA compared with
// 128 x 128 tiles on 4 wavefronts (64 x 64 each), used for small problems.  Workgroup
// ids are remapped so that neighbouring tiles (sharing A row panels or B column panels)
// run on one XCD and hit its L2.  Weight gradients reduce over all tokens (K up to 1e5)
// and have few output tiles: they are split along K into fp32 partials that a second
// kernel sums in a fixed order (deterministic).
#include "common.h"
#include "kernels.h"
#include "mfma.h"

#include <algorithm>

namespace mla {

namespace {

constexpr int BK = 64;

struct GemmDev {
  int M, N;
  const bf16_t* A; int64_t lda;
  const bf16_t* B; int64_t ldb;
  void* C; int64_t ldc;
  float* part;        // split-K partials [splits][M][N], or null
  float alpha, beta;
  int kchunk;         // K elements per split (multiple of BK)
  int ktotal;
};

// row stride (elements) of an m-major [k][ROWS] tile, read only through the transposing
// read (32 lanes cover 4 consecutive rows x 64 bytes): a stride of 16 or 48 banks modulo
// 64 puts the 4 rows on disjoint banks
constexpr int mm_ld(int rows) {
  for (int p = 8; p <= 64; p += 8) {
    const int r = ((rows + p) / 2) % 64;
    if (r == 16 || r == 48) return rows + p;
  }
  return rows + 32;
}
constexpr int KM_LD = BK + 8;  // k-major [row][k] tile: 144-byte rows

// ---- global -> register staging -------------------------------------------------------
template <bool KMAJOR, int ROWS, int NTHR>
struct Loader;

// k-major tile: ROWS x BK, chunk c -> row c / 8, k-chunk c % 8
template <int ROWS, int NTHR>
struct Loader<true, ROWS, NTHR> {
  static constexpr int CHUNKS = ROWS * (BK / 8);
  static constexpr int PER = CHUNKS / NTHR;
  static constexpr int ELEMS = ((ROWS * KM_LD * 2 + 1023) / 1024) * 512;  // whole 1 KB blocks
  static_assert(CHUNKS % NTHR == 0, "tile / thread mismatch");
  u32x4 r[PER];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int row = c / (BK / 8), kc = (c % (BK / 8)) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row < rows_valid && k0 + kc < kend)
        v = *(const u32x4*)(p + (int64_t)(row0 + row) * ld + k0 + kc);
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      *(u32x4*)(lds + (c / (BK / 8)) * KM_LD + (c % (BK / 8)) * 8) = r[i];
    }
  }
  // full k-slice straight from HBM into LDS (rows past the end repeat the last row;
  // their outputs are not stored)
  using Dma = DmaTile<ROWS, BK, KM_LD, NTHR / 64>;
  __device__ __forceinline__ void dma(const Dma& t, const bf16_t* __restrict__ p, int64_t ld,
                                      int row0, int rows_valid, int k0, bf16_t* lds) const {
    const bf16_t* base = p + (int64_t)row0 * ld + k0;
    const int rl = rows_valid - 1;
    t.issue(lds, [&](int r, int c) { return base + (int64_t)min(r, rl) * ld + c; });
  }
  // operand fragment: rows row0 + lane%32, k = 16 kk + 8 half + 0..7
  static __device__ __forceinline__ bf16x8 frag(const bf16_t* lds, int row0, int kk) {
    const int lane = threadIdx.x & 63;
    return *(const bf16x8*)(lds + (row0 + (lane & 31)) * KM_LD + 16 * kk + 8 * (lane >> 5));
  }
};

// m-major tile (global [k][row]): BK x ROWS, chunk c -> k-row c / (ROWS/8), row-chunk c % (ROWS/8)
template <int ROWS, int NTHR>
struct Loader<false, ROWS, NTHR> {
  static constexpr int LD = mm_ld(ROWS);
  static constexpr int CPR = ROWS / 8;
  static constexpr int CHUNKS = BK * CPR;
  static constexpr int PER = CHUNKS / NTHR;
  static constexpr int ELEMS = ((BK * LD * 2 + 1023) / 1024) * 512;  // whole 1 KB blocks
  static_assert(CHUNKS % NTHR == 0, "tile / thread mismatch");
  u32x4 r[PER];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int kr = c / CPR, rc = (c % CPR) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (rc < rows_valid && k0 + kr < kend)
        v = *(const u32x4*)(p + (int64_t)(k0 + kr) * ld + row0 + rc);
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      *(u32x4*)(lds + (c / CPR) * LD + (c % CPR) * 8) = r[i];
    }
  }
  using Dma = DmaTile<BK, ROWS, LD, NTHR / 64>;
  __device__ __forceinline__ void dma(const Dma& t, const bf16_t* __restrict__ p, int64_t ld,
                                      int row0, int rows_valid, int k0, bf16_t* lds) const {
    const bf16_t* base = p + (int64_t)k0 * ld + row0;
    const int cl = rows_valid - 8;
    t.issue(lds, [&](int r, int c) { return base + (int64_t)r * ld + min(c, cl); });
  }
  static __device__ __forceinline__ bf16x8 frag(const bf16_t* lds, int row0, int kk) {
    const int klo = 16 * kk + 8 * ((threadIdx.x & 63) >> 5);
    return lds_operand_tr(lds, LD, row0, klo, klo + 4);
  }
};

template <typename TC>
__device__ __forceinline__ void store_out(TC* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

// four consecutive outputs: alpha * v + beta * C
template <typename TC>
__device__ __forceinline__ void store4(TC* p, f32x4 v, float alpha, float beta);
template <>
__device__ __forceinline__ void store4<float>(float* p, f32x4 v, float alpha, float beta) {
  f32x4 o = v * alpha;
  if (beta != 0.f) o += beta * *(const f32x4*)p;
  *(f32x4*)p = o;
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, f32x4 v, float alpha, float beta) {
  f32x4 o = v * alpha;
  if (beta != 0.f) {
    const u32x2 c = *(const u32x2*)p;
    o[0] += beta * bf2f((bf16_t)(c[0] & 0xffff)); o[1] += beta * bf2f((bf16_t)(c[0] >> 16));
    o[2] += beta * bf2f((bf16_t)(c[1] & 0xffff)); o[3] += beta * bf2f((bf16_t)(c[1] >> 16));
  }
  u32x2 w;
  w[0] = (uint32_t)f2bf(o[0]) | ((uint32_t)f2bf(o[1]) << 16);
  w[1] = (uint32_t)f2bf(o[2]) | ((uint32_t)f2bf(o[3]) << 16);
  *(u32x2*)p = w;
}

// ---- the kernel --------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC>
__global__ __launch_bounds__(64 * WM * WN) void gemm_mfma_kernel(GemmDev g) {
  constexpr int NTHR = 64 * WM * WN;
  constexpr int TM = BM / WM / 32;  // 32x32 MFMA tiles per wave along M
  constexpr int TN = BN / WN / 32;
  using LA = Loader<AK, BM, NTHR>;
  using LB = Loader<BKM, BN, NTHR>;
  constexpr int STAGE = LA::ELEMS + LB::ELEMS;
  __shared__ __attribute__((aligned(1024))) bf16_t lds[2 * STAGE];

  const int ntm = (g.M + BM - 1) / BM, ntn = (g.N + BN - 1) / BN;
  const int ntiles = ntm * ntn;
  // XCD-aware remap, then group 8 row panels together for L2 reuse
  int pid = xcd_remap(blockIdx.x, ntiles);
  const int GROUP = 8;
  int group = pid / (GROUP * ntn);
  int first = group * GROUP;
  int gsz = min(ntm - first, GROUP);
  int tm = first + (pid % (GROUP * ntn)) % gsz;
  int tn = (pid % (GROUP * ntn)) / gsz;
  const int m0 = tm * BM, n0 = tn * BN;
  const int split = blockIdx.y;
  const int kbeg = split * g.kchunk;
  const int kend = min(g.ktotal, kbeg + g.kchunk);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int wrow0 = wm * (BM / WM), wcol0 = wn * (BN / WN);

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  LA la;
  LB lb;
  typename LA::Dma da;
  typename LB::Dma db;
  da.init();
  db.init();
  const int mvalid = g.M - m0, nvalid = g.N - n0;
  const int nk = (kend - kbeg + BK - 1) / BK;
  const int nfull = (kend - kbeg) / BK;  // slices copied straight to LDS; a ragged last
                                         // slice goes through registers with zero fill
  auto stage = [&](int kt, bf16_t* dst) {
    const int k0 = kbeg + kt * BK;
    if (kt < nfull) {
      la.dma(da, g.A, g.lda, m0, mvalid, k0, dst);
      lb.dma(db, g.B, g.ldb, n0, nvalid, k0, dst + LA::ELEMS);
    } else {
      la.load(g.A, g.lda, m0, mvalid, k0, kend);
      lb.load(g.B, g.ldb, n0, nvalid, k0, kend);
      la.store(dst);
      lb.store(dst + LA::ELEMS);
    }
  };
  if (nk > 0) stage(0, lds);
  wait_all();
  __syncthreads();
  // fragments of one 16-wide k step, double buffered in registers: the reads of step
  // kk + 1 are issued before the matrix ops of step kk
  bf16x8 af[2][TM], bfr[2][TN];
  auto load_frags = [&](const bf16_t* As, int kk, bf16x8* a, bf16x8* b) {
    const bf16_t* Bs = As + LA::ELEMS;
#pragma unroll
    for (int i = 0; i < TM; ++i) a[i] = LA::frag(As, wrow0 + i * 32, kk);
#pragma unroll
    for (int j = 0; j < TN; ++j) b[j] = LB::frag(Bs, wcol0 + j * 32, kk);
  };
  auto mma = [&](const bf16x8* a, const bf16x8* b) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  };
  if (nk > 0) load_frags(lds, 0, af[0], bfr[0]);
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) stage(kt + 1, lds + (cur ^ 1) * STAGE);
    const bf16_t* As = lds + cur * STAGE;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      if (kk + 1 < BK / 16) {
        load_frags(As, kk + 1, af[(kk + 1) & 1], bfr[(kk + 1) & 1]);
      } else {
        // next slice: its copy must have landed and every wave must be done with this one
        wait_all();
        __syncthreads();
        if (kt + 1 < nk) load_frags(lds + (cur ^ 1) * STAGE, 0, af[0], bfr[0]);
      }
      __builtin_amdgcn_sched_barrier(0);
      mma(af[kk & 1], bfr[kk & 1]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // epilogue: each wavefront stages one 32-row strip of its tile at a time in a private
  // LDS region (the main loop's last barrier has retired every operand read) and writes
  // it back row by row, 4 consecutive columns per lane.  In the MFMA result a lane holds
  // column lane % 32 and rows 8 (e / 4) + 4 (lane / 32) + e % 4 of each 32 x 32 block.
  constexpr int WTN = BN / WN;              // columns of the wave tile
  constexpr int SLD = WTN + 8;              // strip row stride (floats)
  static_assert(NTHR / 64 * 32 * SLD * 4 <= (int)sizeof(lds), "epilogue strip too large");
  float* strip = (float*)lds + wave * 32 * SLD;
  TC* C = (TC*)g.C;
  const bool vec = (g.ldc % 4) == 0;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        strip[((e >> 2) * 8 + (lane >> 5) * 4 + (e & 3)) * SLD + j * 32 + (lane & 31)] =
            acc[i][j][e];
    constexpr int CPR = WTN / 4;            // float4 chunks per strip row
#pragma unroll
    for (int it = 0; it < 32 * CPR / 64; ++it) {
      const int c = it * 64 + lane;
      const int r = c / CPR, col = (c % CPR) * 4;
      const int m = m0 + wrow0 + i * 32 + r, n = n0 + wcol0 + col;
      if (m >= g.M || n >= g.N) continue;
      const f32x4 v = *(const f32x4*)(strip + r * SLD + col);
      if (g.part) {
        float* p = g.part + ((int64_t)split * g.M + m) * g.N + n;
        if (n + 4 <= g.N && (g.N % 4) == 0) {
          *(f32x4*)p = v;
        } else {
          for (int q = 0; q < 4 && n + q < g.N; ++q) p[q] = v[q];
        }
        continue;
      }
      TC* p = C + (int64_t)m * g.ldc + n;
      if (vec && n + 4 <= g.N) {
        store4<TC>(p, v, g.alpha, g.beta);
      } else {
        for (int q = 0; q < 4 && n + q < g.N; ++q) {
          float x = g.alpha * v[q];
          if (g.beta != 0.f) x += g.beta * ld(p + q);
          store_out<TC>(p + q, x);
        }
      }
    }
  }
}

// C = alpha * sum_s part[s] + beta * C, summed in split order
template <typename TC>
__global__ void splitk_reduce_kernel(const float* __restrict__ part, int splits, int M, int N,
                                     TC* __restrict__ C, int64_t ldc, float alpha, float beta) {
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = (int64_t)M * N;
  if (idx >= total) return;
  int m = (int)(idx / N), n = (int)(idx % N);
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += part[(int64_t)z * total + idx];
  TC* c = C + (int64_t)m * ldc + n;
  float v = alpha * s;
  if (beta != 0.f) v += beta * ld(c);
  store_out<TC>(c, v);
}

// tile shape: 256 x 256 on 8 wavefronts when that still yields enough workgroups
struct Plan {
  bool big;
  int bm, bn, splits, kchunk;
};

Plan plan_of(const Gemm& g, bool allow_split) {
  Plan p;
  const int t256 = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  const int t128 = ((g.M + 127) / 128) * ((g.N + 127) / 128);
  // a 256-tile wastes work on ragged edges; use it when the padded area stays small
  const double waste = (double)((g.M + 255) / 256 * 256) * ((g.N + 255) / 256 * 256) /
                       ((double)((g.M + 127) / 128 * 128) * ((g.N + 127) / 128 * 128));
  const bool splittable = allow_split && g.K >= 8 * BK * 8;
  p.big = waste < 1.15 && (t256 >= 192 || splittable);
  p.bm = p.bn = p.big ? 256 : 128;
  const int tiles = p.big ? t256 : t128;
  p.splits = 1;
  if (splittable && tiles < 512) {
    const int want = (512 + tiles - 1) / tiles;
    const int maxs = g.K / (BK * 8);  // at least 512 k per split
    p.splits = std::max(1, std::min(want, maxs));
  }
  int kchunk = (g.K + p.splits - 1) / p.splits;
  kchunk = (kchunk + BK - 1) / BK * BK;
  p.kchunk = std::max(kchunk, BK);
  p.splits = (g.K + p.kchunk - 1) / p.kchunk;
  if (p.splits < 1) p.splits = 1;
  return p;
}

template <bool AK, bool BKM, typename TC>
void launch(const GemmDev& d, const Plan& p, hipStream_t s) {
  const int tiles = ((d.M + p.bm - 1) / p.bm) * ((d.N + p.bn - 1) / p.bn);
  dim3 grid(tiles, p.splits);
  if (p.big)
    gemm_mfma_kernel<256, 256, 2, 4, AK, BKM, TC><<<grid, 512, 0, s>>>(d);
  else
    gemm_mfma_kernel<128, 128, 2, 2, AK, BKM, TC><<<grid, 256, 0, s>>>(d);
}

}  // namespace

size_t gemm_mfma_scratch_elems(const Gemm& g) {
  Plan p = plan_of(g, true);
  return p.splits > 1 ? (size_t)p.splits * g.M * g.N : 0;
}

hipError_t gemm_mfma(const Gemm& g, float* scratch, size_t scratch_elems, hipStream_t s) {
  GemmDev d;
  d.M = g.M; d.N = g.N; d.ktotal = g.K;
  d.A = (const bf16_t*)g.A; d.lda = g.lda;
  d.B = (const bf16_t*)g.B; d.ldb = g.ldb;
  d.C = g.C; d.ldc = g.ldc; d.alpha = g.alpha; d.beta = g.beta;
  Plan p = plan_of(g, true);
  if (p.splits > 1 && (scratch == nullptr || scratch_elems < (size_t)p.splits * g.M * g.N))
    p = plan_of(g, false);
  d.kchunk = p.kchunk;
  d.part = p.splits > 1 ? scratch : nullptr;
  const bool f32 = g.c_t == DT_F32;
#define L_(AK, BK_)                                                                     \
  if (g.a_kmajor == AK && g.b_kmajor == BK_) {                                          \
    if (f32) launch<AK, BK_, float>(d, p, s);                                           \
    else launch<AK, BK_, bf16_t>(d, p, s);                                              \
  }
  L_(true, true) else L_(true, false) else L_(false, false) else L_(false, true)
#undef L_
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits == 1) return e;
  int64_t total = (int64_t)g.M * g.N;
  unsigned grid = (unsigned)((total + 255) / 256);
  if (f32)
    splitk_reduce_kernel<float><<<grid, 256, 0, s>>>(scratch, p.splits, g.M, g.N, (float*)g.C,
                                                     g.ldc, g.alpha, g.beta);
  else
    splitk_reduce_kernel<bf16_t><<<grid, 256, 0, s>>>(scratch, p.splits, g.M, g.N, (bf16_t*)g.C,
                                                      g.ldc, g.alpha, g.beta);
  return hipGetLastError();
}

}  // namespace mla
