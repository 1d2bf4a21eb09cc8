// bf16 GEMM on gfx950 matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation.
//
//   C[m, n] = alpha * sum_k A(m, k) B(n, k) + beta * C[m, n]
//
// Either operand may be K-contiguous ("k-major": a row of the weight / activation) or
// M/N-contiguous (the transposed operand of the weight-gradient and data-gradient
// products).  A workgroup of 4 wavefronts owns a BM x BN output tile and walks K in
// BK = 64 slices that are staged in LDS as [row][k] with k contiguous, the layout the MFMA
// operand registers want (8 consecutive k per lane).  M/N-contiguous operands are
// transposed on the way in: a thread loads an 8 (k) x 8 (m) block with eight 16-byte
// loads, transposes it in registers and writes eight 16-byte rows.  LDS is double
// buffered: the next slice's global loads are in flight while the current one feeds the
// matrix cores.  Rows are padded by 16 bytes so the 16-byte operand reads of a wavefront
// hit distinct banks.  Workgroup ids are remapped so that neighbouring tiles (which share
// A row panels or B column panels) run on the same XCD and hit its L2.  Weight gradients
// reduce over all tokens (K up to 1e5) and have few output tiles: they are split along K
// into fp32 partials that a second kernel sums in a fixed order (deterministic).
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace mla {

namespace {

constexpr int BK = 64;
constexpr int PADK = BK + 8;  // LDS row length in bf16 elements (144 bytes)
constexpr int NTHR = 256;

struct GemmDev {
  int M, N, K;        // K here is the K range of one split
  const bf16_t* A; int64_t lda;
  const bf16_t* B; int64_t ldb;
  void* C; int64_t ldc;
  float* part;        // split-K partials [splits][M][N], or null
  float alpha, beta;
  int kchunk;         // K elements per split (multiple of BK)
  int ktotal;
};

// ---- global -> register staging -------------------------------------------------------
// k-major tile: ROWS x BK, 16-byte chunks, chunk c -> row c / 8, k-chunk c % 8
template <int ROWS>
struct KMajorLoader {
  static constexpr int CHUNKS = ROWS * (BK / 8);
  static constexpr int PER = (CHUNKS + NTHR - 1) / NTHR;
  u32x4 r[PER];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int c = threadIdx.x + i * NTHR;
      int row = c / (BK / 8), kc = (c % (BK / 8)) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (c < CHUNKS && row < rows_valid && k0 + kc < kend)
        v = *(const u32x4*)(p + (int64_t)(row0 + row) * ld + k0 + kc);
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int c = threadIdx.x + i * NTHR;
      if (c < CHUNKS) {
        int row = c / (BK / 8), kc = (c % (BK / 8)) * 8;
        *(u32x4*)(lds + row * PADK + kc) = r[i];
      }
    }
  }
};

// m-major tile (global [k][m]): 8 x 8 blocks, block b -> m-block b % (ROWS/8), k-block b / (ROWS/8)
template <int ROWS>
struct MMajorLoader {
  static constexpr int MB = ROWS / 8;
  static constexpr int BLOCKS = MB * (BK / 8);
  static constexpr int PER = (BLOCKS + NTHR - 1) / NTHR;
  u32x4 r[PER][8];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int b = threadIdx.x + i * NTHR;
      int mb = (b % MB) * 8, kb = (b / MB) * 8;
      bool ok = b < BLOCKS && mb < rows_valid;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (ok && k0 + kb + j < kend)
          v = *(const u32x4*)(p + (int64_t)(k0 + kb + j) * ld + row0 + mb);
        r[i][j] = v;
      }
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      int b = threadIdx.x + i * NTHR;
      if (b >= BLOCKS) continue;
      int mb = (b % MB) * 8, kb = (b / MB) * 8;
      // transpose the 8 (k) x 8 (m) block: row mm of the output holds k = 0..7 of m = mm
#pragma unroll
      for (int mm = 0; mm < 8; ++mm) {
        const int w = mm >> 1, sh = (mm & 1) * 16;
        u32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t lo = (r[i][2 * q][w] >> sh) & 0xffffu;
          uint32_t hi = (r[i][2 * q + 1][w] >> sh) & 0xffffu;
          o[q] = lo | (hi << 16);
        }
        *(u32x4*)(lds + (mb + mm) * PADK + kb) = o;
      }
    }
  }
};

template <bool KMAJOR, int ROWS>
struct Loader;
template <int ROWS>
struct Loader<true, ROWS> : KMajorLoader<ROWS> {};
template <int ROWS>
struct Loader<false, ROWS> : MMajorLoader<ROWS> {};

template <typename TC>
__device__ __forceinline__ void store_out(TC* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

// ---- the kernel --------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC>
__global__ __launch_bounds__(NTHR) void gemm_mfma_kernel(GemmDev g) {
  static_assert(WM * WN == 4, "4 wavefronts");
  constexpr int TM = BM / WM / 32;  // 32x32 MFMA tiles per wave along M
  constexpr int TN = BN / WN / 32;
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][(BM + BN) * PADK];

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

  Loader<AK, BM> la;
  Loader<BKM, BN> lb;
  const int mvalid = g.M - m0, nvalid = g.N - n0;
  const int nk = (kend - kbeg + BK - 1) / BK;
  if (nk > 0) {
    la.load(g.A, g.lda, m0, mvalid, kbeg, kend);
    lb.load(g.B, g.ldb, n0, nvalid, kbeg, kend);
    la.store(lds[0]);
    lb.store(lds[0] + BM * PADK);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load(g.A, g.lda, m0, mvalid, kbeg + (kt + 1) * BK, kend);
      lb.load(g.B, g.ldb, n0, nvalid, kbeg + (kt + 1) * BK, kend);
    }
    const bf16_t* As = lds[cur];
    const bf16_t* Bs = lds[cur] + BM * PADK;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int koff = kk * 16 + (lane >> 5) * 8;
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *(const bf16x8*)(As + (wrow0 + i * 32 + (lane & 31)) * PADK + koff);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *(const bf16x8*)(Bs + (wcol0 + j * 32 + (lane & 31)) * PADK + koff);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      la.store(lds[cur ^ 1]);
      lb.store(lds[cur ^ 1] + BM * PADK);
    }
    __syncthreads();
  }

  // epilogue: lane holds column (lane % 32) and rows 8*(e/4) + 4*(lane/32) + e%4 of a tile
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wcol0 + j * 32 + (lane & 31);
      if (n >= g.N) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wrow0 + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
        if (m >= g.M) continue;
        if (g.part) {
          g.part[((int64_t)split * g.M + m) * g.N + n] = acc[i][j][e];
        } else {
          TC* c = (TC*)g.C + (int64_t)m * g.ldc + n;
          float v = g.alpha * acc[i][j][e];
          if (g.beta != 0.f) v += g.beta * ld(c);
          store_out<TC>(c, v);
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

constexpr int TILE_M = 128, TILE_N = 128;

int choose_splits(const Gemm& g) {
  const int tiles = ((g.M + TILE_M - 1) / TILE_M) * ((g.N + TILE_N - 1) / TILE_N);
  if (tiles >= 512 || g.K < 4 * BK * 8) return 1;
  int want = (768 + tiles - 1) / tiles;
  int maxs = g.K / (BK * 8);  // keep at least 512 k per split
  return std::max(1, std::min(want, maxs));
}

template <bool AK, bool BKM, typename TC>
void launch(const GemmDev& d, int splits, hipStream_t s) {
  const int tiles = ((d.M + TILE_M - 1) / TILE_M) * ((d.N + TILE_N - 1) / TILE_N);
  dim3 grid(tiles, splits);
  gemm_mfma_kernel<TILE_M, TILE_N, 2, 2, AK, BKM, TC><<<grid, NTHR, 0, s>>>(d);
}

}  // namespace

size_t gemm_mfma_scratch_elems(const Gemm& g) {
  int sp = choose_splits(g);
  return sp > 1 ? (size_t)sp * g.M * g.N : 0;
}

hipError_t gemm_mfma(const Gemm& g, float* scratch, size_t scratch_elems, hipStream_t s) {
  GemmDev d;
  d.M = g.M; d.N = g.N; d.ktotal = g.K;
  d.A = (const bf16_t*)g.A; d.lda = g.lda;
  d.B = (const bf16_t*)g.B; d.ldb = g.ldb;
  d.C = g.C; d.ldc = g.ldc; d.alpha = g.alpha; d.beta = g.beta;
  int splits = choose_splits(g);
  if (splits > 1 && (scratch == nullptr || scratch_elems < (size_t)splits * g.M * g.N))
    splits = 1;
  int kchunk = (g.K + splits - 1) / splits;
  kchunk = (kchunk + BK - 1) / BK * BK;
  splits = (g.K + kchunk - 1) / kchunk;
  d.kchunk = kchunk;
  d.K = kchunk;
  d.part = splits > 1 ? scratch : nullptr;
  const bool f32 = g.c_t == DT_F32;
#define L_(AK, BK_)                                                                     \
  if (g.a_kmajor == AK && g.b_kmajor == BK_) {                                          \
    if (f32) launch<AK, BK_, float>(d, splits, s);                                      \
    else launch<AK, BK_, bf16_t>(d, splits, s);                                         \
  }
  L_(true, true) else L_(true, false) else L_(false, false) else L_(false, true)
#undef L_
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  int64_t total = (int64_t)g.M * g.N;
  unsigned grid = (unsigned)((total + 255) / 256);
  if (f32)
    splitk_reduce_kernel<float><<<grid, 256, 0, s>>>(scratch, splits, g.M, g.N, (float*)g.C, g.ldc,
                                                     g.alpha, g.beta);
  else
    splitk_reduce_kernel<bf16_t><<<grid, 256, 0, s>>>(scratch, splits, g.M, g.N, (bf16_t*)g.C,
                                                      g.ldc, g.alpha, g.beta);
  return hipGetLastError();
}

}  // namespace mla
