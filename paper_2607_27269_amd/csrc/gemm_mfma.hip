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
// wavefront's tile in LDS and writes it back with 16-byte (fp32) or 8-byte (bf16) stores.
// Plain products run persistent: one workgroup per CU slot walks the tiles, and the next
// tile's first slice is copied while the current one finishes and writes its epilogue.
// The operand reads of a wavefront hit distinct banks: k-major rows are XOR-swizzled in
// 16-byte chunks, m-major row strides are padded.  Large problems use 256 x 256 tiles on
// 8 wavefronts (128 x 64 each), which halves the LDS bytes per MFMA compared with
// 128 x 128 tiles on 4 wavefronts (64 x 64 each), used for small problems.  Workgroup
// ids are remapped so that neighbouring tiles (sharing A row panels or B column panels)
// run on one XCD and hit its L2.  Weight gradients reduce over all tokens (K up to 1e5)
// and have few output tiles: they are split along K into fp32 partials that a second
// kernel sums in a fixed order (deterministic).  NT products of whole tiles run on a
// four-wavefront kernel whose k steps are scheduled by hand (below, gemm_nt4_persist_kernel).
#include <atomic>
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "mfma.h"

#include <algorithm>

namespace mla {

namespace {

constexpr int BK = 64;  // K granule of split-K chunks (and the slice of the small tiles)
// slice depth, LDS ring depth and wavefront grid of the 256 x 256 tiles (measured on the
// step's shapes: deeper rings of 32-deep slices and 4-wavefront grids of 128 x 128 were
// slower)
constexpr int GBK = 64, GNST = 2, GWM = 2, GWN = 4;

struct GemmDev {
  int M, N;
  const bf16_t* A; int64_t lda;
  const bf16_t* B; int64_t ldb;
  void* C; int64_t ldc;
  float* part;        // split-K partials [splits][M][N], or null
  // masked-loss epilogue (with lpart set): C = lscale[0] mask[m] acc (not stored when C is
  // NULL) and lpart[tile] = the sum over the tile of mask[m] acc^2, or of mask[m] acc
  // lref[m, n] when lref is set
  const float* lscale; const uint8_t* lmask; double* lpart;
  const bf16_t* lref; int64_t ldref;
  float alpha, beta;
  int kchunk;         // K elements per split (multiple of BK)
  int nsplit;         // split-K chunks (persistent launch)
  int ktotal;
  int mstore;         // rows of C written (M is the row count operand A may be read at)
  // batched causal mode (causal != 0): workgroup z of nbatch works on A + z sA,
  // B + (z / zdiv) sB1 + ((z % zdiv) / bdiv) sB2, C + (z / zdiv) sC1 + (z % zdiv) sC2; the
  // K range of an M tile ends at its last row (entries with k > m are zero) or, with rev,
  // starts at its first row (entries with k < m are zero); it is walked kgroups times, the
  // j-th time on A + j sAk and B + j sBk (a sum over stacked operands)
  int causal, rev, nbatch, zdiv, bdiv, kgroups;
  int64_t sA, sB1, sB2, sC1, sC2, sAk, sBk;
  // split output of the persistent causal k-major product (dK), when split_n > 0: columns
  // n < split_n in bf16 at c_lo + z1 sC1_lo + z2 sC2_lo + m ldc_lo + n, the rest (fp32) at C
  // with the strides above, column n - split_n
  int split_n;
  bf16_t* c_lo; int64_t ldc_lo, sC1_lo, sC2_lo;
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
// A operand of the batched causal products: dS^T stored in 32 x 32 tiles, element (key r,
// query c) at ((r / 32) tq + c / 32) 1024 + (r % 32) 32 + c % 32 (tq: tiles per row of
// tiles), so that each wavefront of the producer writes its 32 x 32 block as 2 KB of
// whole lines and a slice of 32 keys x 256 queries is 16 KB of consecutive tiles
__device__ __forceinline__ int64_t tile32_off(int64_t r, int64_t c, int64_t tq) {
  return ((r >> 5) * tq + (c >> 5)) * 1024 + (r & 31) * 32 + (c & 31);
}

// ---- global -> register staging -------------------------------------------------------
template <bool KMAJOR, int ROWS, int NTHR, int BK, bool TILED = false>
struct Loader;

// k-major tile: ROWS x BK, chunk c -> row c / (BK/8), k-chunk c % (BK/8).  Rows are not
// padded: the 16-byte chunk holding k-chunk c of row r sits at position c ^ swz(r) of its
// row, so that the 16 rows one operand read covers per LDS cycle (one k-chunk each) fall on
// 16 distinct 16-byte bank groups (a 256-byte bank window holds 128 / BK rows)
template <int ROWS, int NTHR, int BK>
struct Loader<true, ROWS, NTHR, BK, false> {
  static constexpr int KM_LD = BK;
  static constexpr int NCH = BK / 8;    // 16-byte chunks per row
  static constexpr int RPW = 128 / BK;  // rows per 256-byte bank window
  static_assert(BK == 32 || BK == 64, "k-major slice depth");
  static __device__ __forceinline__ int swz(int row) { return (row / RPW) % NCH; }
  static constexpr int CHUNKS = ROWS * NCH;
  static constexpr int PER = (CHUNKS + NTHR - 1) / NTHR;
  using Dma = DmaTile<ROWS, BK, KM_LD, NTHR / 64, true>;
  static constexpr int ELEMS = Dma::ALLOC;  // whole 1 KB blocks, a multiple per wavefront
  // the copy that fills LDS position (row, p) fetches k-chunk p ^ swz(row)
  static __device__ __forceinline__ void swizzle(Dma& t) {
#pragma unroll
    for (int p = 0; p < Dma::PER; ++p)
      t.col[p] = (short)(8 * ((t.col[p] / 8) ^ swz(t.row[p])));
  }
  u32x4 r[PER];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int row = c / NCH, kc = (c % NCH) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if ((CHUNKS % NTHR == 0 || c < CHUNKS) && row < rows_valid && k0 + kc < kend)
        v = *(const u32x4*)(p + (int64_t)(row0 + row) * ld + k0 + kc);
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int row = c / NCH;
      if (CHUNKS % NTHR == 0 || c < CHUNKS)
        *(u32x4*)(lds + row * KM_LD + 8 * ((c % NCH) ^ swz(row))) = r[i];
    }
  }
  // full k-slice of a full tile straight from HBM into LDS (uniform base + lane offset)
  __device__ __forceinline__ void dma(const Dma& t, const bf16_t* __restrict__ p, int64_t ld,
                                      int row0, int rows_valid, int k0, bf16_t* lds) const {
    t.issue_s(lds, p + (int64_t)row0 * ld + k0, [&](int r, int c) { return r * (int)ld + c; });
  }
  // operand fragment: rows row0 + lane%32, k = 16 kk + 8 half + 0..7 (row0 is a multiple of
  // 32, so the swizzle depends on the lane only)
  static __device__ __forceinline__ bf16x8 frag(const bf16_t* lds, int row0, int kk) {
    const int lane = threadIdx.x & 63, l = lane & 31;
    const int c = 2 * kk + (lane >> 5);
    return *(const bf16x8*)(lds + (row0 + l) * KM_LD + 8 * (c ^ swz(l)));
  }
};

// m-major tile (global [k][row]): BK x ROWS, chunk c -> k-row c / (ROWS/8), row-chunk c % (ROWS/8).
// Rows of a multiple of 64 elements are unpadded and XOR-swizzled in aligned groups of four
// 16-byte chunks (64 bytes, 16 banks), so that the 4 k-rows x 64 bytes one transposing read
// covers per half-wavefront fall on 4 distinct 16-bank groups: with rows a multiple of
// 256 bytes long every row starts on the same bank, and group G of k-row k sits at
// G ^ (k mod 4); with rows an odd multiple of 128 bytes, odd rows start half a bank
// window (two groups) later, and group G sits at G ^ ((k / 2) mod 2).  Other widths keep padded rows.
template <int ROWS, int NTHR, int BK>
struct Loader<false, ROWS, NTHR, BK, false> {
  static constexpr bool SWZ = ROWS % 64 == 0;
  static constexpr bool SWZ4 = ROWS % 128 == 0;  // else rows are an odd multiple of 128 B
  static constexpr int LD = SWZ ? ROWS : mm_ld(ROWS);
  static constexpr int CPR = ROWS / 8;
  static constexpr int CHUNKS = BK * CPR;
  static constexpr int PER = (CHUNKS + NTHR - 1) / NTHR;
  using Dma = DmaTile<BK, ROWS, LD, NTHR / 64, true>;
  static constexpr int ELEMS = Dma::ALLOC;  // whole 1 KB blocks, a multiple per wavefront
  static __device__ __forceinline__ int pos(int k, int c) {
    return !SWZ ? c : SWZ4 ? c ^ (4 * (k & 3)) : c ^ (4 * ((k >> 1) & 1));
  }
  // the copy that fills LDS position (k, p) fetches chunk pos(k, p) (an involution)
  static __device__ __forceinline__ void swizzle(Dma& t) {
    if constexpr (SWZ) {
#pragma unroll
      for (int p = 0; p < Dma::PER; ++p) t.col[p] = (short)(8 * pos(t.row[p], t.col[p] / 8));
    }
  }
  u32x4 r[PER];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int kr = c / CPR, rc = (c % CPR) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if ((CHUNKS % NTHR == 0 || c < CHUNKS) && rc < rows_valid && k0 + kr < kend)
        v = *(const u32x4*)(p + (int64_t)(k0 + kr) * ld + row0 + rc);
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int kr = c / CPR;
      if (CHUNKS % NTHR == 0 || c < CHUNKS)
        *(u32x4*)(lds + kr * LD + pos(kr, c % CPR) * 8) = r[i];
    }
  }
  __device__ __forceinline__ void dma(const Dma& t, const bf16_t* __restrict__ p, int64_t ld,
                                      int row0, int rows_valid, int k0, bf16_t* lds) const {
    t.issue_s(lds, p + (int64_t)k0 * ld + row0, [&](int r, int c) { return r * (int)ld + c; });
  }

  // operand fragment through the transposing read (lds_operand_tr's lane pattern: k-rows
  // klo + lane%16/4 and klo + 4 + lane%16/4, columns row0 + 16 ((lane/16) % 2) + 4 (lane % 4));
  // klo is a multiple of 4, so the swizzle's k mod 4 is the lane's lane%16/4
  static __device__ __forceinline__ bf16x8 frag(const bf16_t* lds, int row0, int kk) {
    const int lane = threadIdx.x & 63, g = lane >> 4, r = lane & 15;
    const int klo = 16 * kk + 8 * (lane >> 5), kq = r >> 2;
    const int m = row0 + 16 * (g & 1) + 4 * (r & 3);
    const int mc = SWZ ? pos(kq, m >> 3) * 8 + (m & 7) : m;
    const u32x2 lo = lds_read_tr4(lds + (klo + kq) * LD + mc);
    const u32x2 hi = lds_read_tr4(lds + (klo + 4 + kq) * LD + mc);
    const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
    return __builtin_bit_cast(bf16x8, w);
  }
};

// A of the batched causal products: dS^T in 32 x 32 tiles (tile32_off), ld = the plane's
// row length (a multiple of 32).  The LDS copy of a slice holds the slice's tiles whole and
// in order, so that each 1 KB copy instruction moves 1 KB of consecutive global memory.
//
// Rows = keys, k = queries (the dK product): the slice's tiles (key tile i, query tile j)
// at (i NQT + j) 1024 elements; inside a tile, key row r (64 bytes) holds its 16-byte chunk
// q at position q ^ ((r / 4) % 4), so that the 16 rows one operand read covers per LDS
// cycle fall on 16 distinct 16-byte bank groups.
template <int ROWS, int NTHR, int BK>
struct Loader<true, ROWS, NTHR, BK, true> {
  static_assert(ROWS % 32 == 0 && BK % 32 == 0, "whole tiles");
  static constexpr int NQT = BK / 32;   // query tiles per slice
  static constexpr int NCH = BK / 8;    // 16-byte chunks per row
  static constexpr int CHUNKS = ROWS * NCH;
  static constexpr int PER = (CHUNKS + NTHR - 1) / NTHR;
  using Dma = DmaTile<ROWS * BK / 64, 64, 64, NTHR / 64, true>;  // the slice as flat 1 KB blocks
  static constexpr int ELEMS = Dma::ALLOC;
  static __device__ __forceinline__ int sw(int r) { return (r >> 2) & 3; }
  // LDS element of (row, k) of the slice (k a multiple of 8)
  static __device__ __forceinline__ int lds_off(int row, int k) {
    return ((row >> 5) * NQT + (k >> 5)) * 1024 + (row & 31) * 32 + 8 * (((k & 31) >> 3) ^ sw(row & 31));
  }
  static __device__ __forceinline__ void swizzle(Dma&) {}
  u32x4 r[PER];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int row = c / NCH, kc = (c % NCH) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if ((CHUNKS % NTHR == 0 || c < CHUNKS) && row < rows_valid && k0 + kc < kend)
        v = *(const u32x4*)(p + tile32_off(row0 + row, k0 + kc, ld >> 5));
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      if (CHUNKS % NTHR == 0 || c < CHUNKS) *(u32x4*)(lds + lds_off(c / NCH, (c % NCH) * 8)) = r[i];
    }
  }
  // LDS element e = 64 r + c of the flat block layout holds tile e / 1024 (key tile i,
  // query tile j), row (e % 1024) / 32, chunk position (e % 32) / 8; it is copied from the
  // same row of global tile (i, j), chunk position ^ sw(row)
  __device__ __forceinline__ void dma(const Dma& t, const bf16_t* __restrict__ p, int64_t ld,
                                      int row0, int rows_valid, int k0, bf16_t* lds) const {
    const int tq = (int)(ld >> 5);
    // dS^T is streamed once per product: non-temporal, so that it displaces less of the
    // B operand (Q) the caches keep between the row tiles of a batch entry
    t.template issue_s<true>(lds, p + tile32_off(row0, k0, tq), [&](int r, int c) {
      const int e = 64 * r + c, tile = e >> 10, w = e & 1023, rr = w >> 5;
      return ((tile / NQT) * tq + tile % NQT) * 1024 + rr * 32 + 8 * (((w & 31) >> 3) ^ sw(rr));
    });
  }
  // operand fragment: rows row0 + lane%32 (row0 a multiple of 32: one key tile), k = 16 kk +
  // 8 half + 0..7
  static __device__ __forceinline__ bf16x8 frag(const bf16_t* lds, int row0, int kk) {
    const int lane = threadIdx.x & 63, l = lane & 31;
    const int c = 2 * kk + (lane >> 5);
    return *(const bf16x8*)(lds + ((row0 >> 5) * NQT + (c >> 2)) * 1024 + l * 32 + 8 * ((c & 3) ^ sw(l)));
  }
};

// k = keys, rows = queries (the dQ product, 32-deep slices: one key tile per slice): the
// slice's query tiles in order, each a copy of its global tile ([32 keys][32 queries]); the
// transposing read of 4 key rows x 32 queries is then 256 consecutive bytes
template <int ROWS, int NTHR, int BK>
struct Loader<false, ROWS, NTHR, BK, true> {
  static_assert(BK == 32 && ROWS % 32 == 0, "one key tile per slice");
  static constexpr int CPR = ROWS / 8;
  static constexpr int CHUNKS = BK * CPR;
  static constexpr int PER = (CHUNKS + NTHR - 1) / NTHR;
  using Dma = DmaTile<BK, ROWS, ROWS, NTHR / 64, true>;
  static constexpr int ELEMS = Dma::ALLOC;
  static __device__ __forceinline__ int lds_off(int k, int m) { return (m >> 5) * 1024 + k * 32 + (m & 31); }
  static __device__ __forceinline__ void swizzle(Dma&) {}
  u32x4 r[PER];
  __device__ __forceinline__ void load(const bf16_t* __restrict__ p, int64_t ld, int row0,
                                       int rows_valid, int k0, int kend) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      const int kr = c / CPR, rc = (c % CPR) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if ((CHUNKS % NTHR == 0 || c < CHUNKS) && rc < rows_valid && k0 + kr < kend)
        v = *(const u32x4*)(p + tile32_off(k0 + kr, row0 + rc, ld >> 5));
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * NTHR;
      if (CHUNKS % NTHR == 0 || c < CHUNKS) *(u32x4*)(lds + lds_off(c / CPR, (c % CPR) * 8)) = r[i];
    }
  }
  // LDS element e = ROWS r + c of the flat block layout is element e of the slice's tiles
  // in global memory (they are consecutive)
  __device__ __forceinline__ void dma(const Dma& t, const bf16_t* __restrict__ p, int64_t ld,
                                      int row0, int rows_valid, int k0, bf16_t* lds) const {
    // dS^T streamed once: non-temporal (the keys stay cached between row tiles)
    t.template issue_s<true>(lds, p + tile32_off(k0, row0, ld >> 5),
                             [&](int r, int c) { return ROWS * r + c; });
  }
  static __device__ __forceinline__ bf16x8 frag(const bf16_t* lds, int row0, int kk) {
    const int lane = threadIdx.x & 63, g = lane >> 4, r = lane & 15;
    const int klo = 16 * kk + 8 * (lane >> 5), kq = r >> 2;
    const int m = row0 + 16 * (g & 1) + 4 * (r & 3);
    const u32x2 lo = lds_read_tr4(lds + lds_off(klo + kq, m));
    const u32x2 hi = lds_read_tr4(lds + lds_off(klo + 4 + kq, m));
    const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
    return __builtin_bit_cast(bf16x8, w);
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
  *(u32x2*)p = u32x2{pack2bf(o[0], o[1]), pack2bf(o[2], o[3])};
}

// ---- the kernel --------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC, int BK, int NST,
          bool ATILE = false>
__device__ __forceinline__ void gemm_tile(const GemmDev& g) {
  constexpr int NTHR = 64 * WM * WN;
  constexpr int TM = BM / WM / 32;  // 32x32 MFMA tiles per wave along M
  constexpr int TN = BN / WN / 32;
  constexpr int KK = BK / 16;       // MFMA k-steps per slice
  using LA = Loader<AK, BM, NTHR, BK, ATILE>;
  using LB = Loader<BKM, BN, NTHR, BK>;
  constexpr int STAGE = LA::ELEMS + LB::ELEMS;
  constexpr int D = LA::Dma::PER + LB::Dma::PER;  // copies per wavefront per slice
  static_assert(NST >= 2 && NST <= 4 && (NST - 2) * D < 64, "stages / counter range");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[NST * STAGE];

  const int ntm = (g.M + BM - 1) / BM, ntn = (g.N + BN - 1) / BN;
  const int ntiles = ntm * ntn;
  int tm, tn;
  const bf16_t* gA = g.A;
  const bf16_t* gB = g.B;
  TC* C = (TC*)g.C;
  if (g.causal) {
    // the longest K ranges first (row tile by row tile); inside one row tile, batch entries
    // that share their B panel (bdiv consecutive entries) are dispatched to one XCD
    // (workgroup ids go round-robin over the 8 XCDs) so that they stream it through one L2
    const int pid = blockIdx.x;
    const int per = g.nbatch * ntn;
    tm = g.rev ? pid / per : ntm - 1 - pid / per;
    const int r = pid % per;
    tn = r / g.nbatch;
    int z = r % g.nbatch;
    if (g.bdiv > 1 && g.nbatch % (8 * g.bdiv) == 0) {
      const int x = z % 8, j = z / 8;
      z = (x + 8 * (j / g.bdiv)) * g.bdiv + j % g.bdiv;
    }
    const int z1 = z / g.zdiv, z2 = z % g.zdiv;
    gA += z * g.sA;
    gB += z1 * g.sB1 + (z2 / g.bdiv) * g.sB2;
    C += z1 * g.sC1 + z2 * g.sC2;
  } else {
    // XCD-aware remap, then group 8 row panels together for L2 reuse
    const int pid = xcd_remap(blockIdx.x, ntiles);
    const int GROUP = 8;
    const int group = pid / (GROUP * ntn);
    const int first = group * GROUP;
    const int gsz = min(ntm - first, GROUP);
    tm = first + (pid % (GROUP * ntn)) % gsz;
    tn = (pid % (GROUP * ntn)) / gsz;
  }
  const int m0 = tm * BM, n0 = tn * BN;
  const int split = blockIdx.y;
  int kbeg, kend;
  if (g.causal) {
    kbeg = g.rev ? m0 : 0;
    kend = g.rev ? g.ktotal : min(g.ktotal, m0 + BM);
  } else {
    kbeg = split * g.kchunk;
    kend = min(g.ktotal, kbeg + g.kchunk);
  }

  const int lane = threadIdx.x & 63, wave = wave_id();
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
  LA::swizzle(da);
  LB::swizzle(db);
  const int mvalid = g.M - m0, nvalid = g.N - n0;
  const int nkg = (kend - kbeg + BK - 1) / BK;  // slices per operand group
  const int nk = nkg * (g.causal ? g.kgroups : 1);
  // slices copied straight to LDS; a ragged last slice, and every slice of a tile that is
  // cut by the matrix edge or whose operand rows are too far apart for 32-bit offsets,
  // goes through registers with zero fill
  const bool dma_ok = mvalid >= BM && nvalid >= BN &&
                      (AK ? (int64_t)BM * g.lda : (int64_t)BK * g.lda) < (1ll << 30) &&
                      (BKM ? (int64_t)BN * g.ldb : (int64_t)BK * g.ldb) < (1ll << 30);
  const int nfull = dma_ok ? (kend - kbeg) / BK : 0;
  // rev: slices are walked from the top of the K range down, so that all row tiles of a
  // batch entry (whose ranges share their top) stream the same B rows at the same time
  auto stage = [&](int kt, bf16_t* dst) {
    const int grp = g.causal && g.kgroups > 1 ? kt / nkg : 0, ks0 = kt - grp * nkg;
    const int ks = g.causal && g.rev ? nkg - 1 - ks0 : ks0;
    const int k0 = kbeg + ks * BK;
    const bf16_t* pa = gA + grp * g.sAk;
    const bf16_t* pb = gB + grp * g.sBk;
    if (ks < nfull) {
      la.dma(da, pa, g.lda, m0, mvalid, k0, dst);
      lb.dma(db, pb, g.ldb, n0, nvalid, k0, dst + LA::ELEMS);
    } else {
      la.load(pa, g.lda, m0, mvalid, k0, kend);
      lb.load(pb, g.ldb, n0, nvalid, k0, kend);
      la.store(dst);
      lb.store(dst + LA::ELEMS);
    }
  };
  // slice s waits for its own copies while up to n later slices may still be in flight
  auto wait_slice = [&](int n) {
    if constexpr (NST >= 4) {
      if (n >= 2) { wait_vm<2 * D>(); return; }
    }
    if constexpr (NST >= 3) {
      if (n >= 1) { wait_vm<D>(); return; }
    }
    wait_vm<0>();
  };
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
  // ring of NST slices: slices kt + 1 .. kt + NST - 1 are in flight while slice kt feeds the
  // matrix cores
#pragma unroll
  for (int s0 = 0; s0 < NST - 1; ++s0)
    if (s0 < nk) stage(s0, lds + s0 * STAGE);
  wait_slice(min(NST - 2, nk - 1));
  lds_barrier();
  if (nk > 0) load_frags(lds, 0, af[0], bfr[0]);
  for (int kt = 0; kt < nk; ++kt) {
    const bf16_t* As = lds + (kt % NST) * STAGE;
    // the stage of slice kt - 1 is free: every wave passed the barrier after its last read
    if (kt + NST - 1 < nk) stage(kt + NST - 1, lds + ((kt + NST - 1) % NST) * STAGE);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (kk + 1 < KK) {
        load_frags(As, kk + 1, af[(kk + 1) & 1], bfr[(kk + 1) & 1]);
      } else {
        // next slice: its copies must have landed (later ones may still fly) and every
        // wave must be done reading this one
        wait_slice(min(NST - 2, nk - 2 - kt));
        lds_barrier();
        if (kt + 1 < nk) load_frags(lds + ((kt + 1) % NST) * STAGE, 0, af[0], bfr[0]);
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
  const bool vec = (g.ldc % 4) == 0;
  const bool lmode = g.lpart != nullptr;  // uniform
  const float lsc = lmode ? *g.lscale : 0.f;
  float sse = 0.f;
  // two copies, as in the persistent epilogue: with beta = 0 no C is read
  auto epilogue = [&](auto with_beta) {
    constexpr bool WB = decltype(with_beta)::value;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          strip[((e >> 2) * 8 + (lane >> 5) * 4 + (e & 3)) * SLD + j * 32 + (lane & 31)] =
              acc[i][j][e];
      constexpr int CPR = WTN / 4;            // float4 chunks per strip row
      constexpr int NIT = 32 * CPR / 64;
      // the strip's reads first (all inside the strip), then the stores
      f32x4 vv[NIT];
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int c = it * 64 + lane;
        vv[it] = *(const f32x4*)(strip + (c / CPR) * SLD + (c % CPR) * 4);
      }
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int c = it * 64 + lane;
        const int r = c / CPR, col = (c % CPR) * 4;
        const int m = m0 + wrow0 + i * 32 + r, n = n0 + wcol0 + col;
        if (m >= g.mstore || n >= g.N) continue;
        f32x4 v = vv[it];
        if (lmode) {
          if (n + 4 > g.N) v = f32x4{v[0], n + 1 < g.N ? v[1] : 0.f, n + 2 < g.N ? v[2] : 0.f, 0.f};
          if (g.lmask && !g.lmask[m]) v = f32x4{0.f, 0.f, 0.f, 0.f};
          f32x4 r = v;
          if (g.lref) {
            const bf16_t* rp = g.lref + (int64_t)m * g.ldref + n;
            if (n + 4 <= g.N && (g.ldref & 3) == 0) {
              const u32x2 w = *(const u32x2*)rp;
              r = f32x4{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xffff0000u),
                        __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xffff0000u)};
            } else {
              r = f32x4{bf2f(rp[0]), n + 1 < g.N ? bf2f(rp[1]) : 0.f,
                        n + 2 < g.N ? bf2f(rp[2]) : 0.f, n + 3 < g.N ? bf2f(rp[3]) : 0.f};
            }
          }
          sse += v[0] * r[0] + v[1] * r[1] + v[2] * r[2] + v[3] * r[3];
          if (C == nullptr) continue;  // tile sums only
          v *= lsc;
        }
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
          store4<TC>(p, v, g.alpha, WB ? g.beta : 0.f);
        } else {
          for (int q = 0; q < 4 && n + q < g.N; ++q) {
            float x = g.alpha * v[q];
            if (WB && g.beta != 0.f) x += g.beta * ld(p + q);
            store_out<TC>(p + q, x);
          }
        }
      }
    }
  };
  // (the dS^T products never accumulate into C: beta = 0 is checked at their launch)
  if constexpr (ATILE) epilogue(std::false_type{});
  else if (g.beta != 0.f) epilogue(std::true_type{}); else epilogue(std::false_type{});
  if (lmode) {
    // the tile's sum in a fixed order: lanes (fixed tree), then wavefronts in order
    // (the last bytes of the operand LDS, past every wavefront's strip)
    static_assert(NTHR / 64 * 32 * SLD * 4 + 8 * (NTHR / 64) <= (int)sizeof(lds), "LDS");
    double* lred = (double*)((char*)lds + sizeof(lds)) - NTHR / 64;
    const double ws = warp_sum_d((double)sse);
    if (lane == 0) lred[wave] = ws;
    __syncthreads();
    if (threadIdx.x == 0) {
      double t = 0.0;
      for (int w = 0; w < NTHR / 64; ++w) t += lred[w];
      g.lpart[blockIdx.x] = t;
    }
  }
}


// Persistent variant (no loss epilogue): a grid of one workgroup per CU slot walks the
// output tiles (x split-K chunks, or x batch entries of the causal products) in steps of the
// grid size, in the same tile order as the one-tile-per-workgroup launch.  The ring of two
// LDS stages runs on across tiles: the next tile's first slice is copied into the free
// stage while the last slice of this tile feeds the matrix cores, and while the epilogue
// stages its 16-row half strips in the stage the last slice occupied.  The causal tiles come
// longest K range first, and a workgroup takes them in snake order (forward in even rounds,
// backward in odd ones), so that long and short ranges pair up on every CU.
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC, int BK, int NST,
          bool CAUSAL>
__device__ __forceinline__ void gemm_persist(const GemmDev& g) {
  // the causal products read a 32 x 32-tiled A (tile32_off)
  constexpr bool ATILE = CAUSAL;
  static_assert(NST == 2, "the cross-tile copy assumes a two-stage ring");
  constexpr int NTHR = 64 * WM * WN;
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  constexpr int KK = BK / 16;
  using LA = Loader<AK, BM, NTHR, BK, ATILE>;
  using LB = Loader<BKM, BN, NTHR, BK>;
  constexpr int STAGE = LA::ELEMS + LB::ELEMS;
  __shared__ __attribute__((aligned(1024))) bf16_t lds[NST * STAGE];

  const int ntm = (g.M + BM - 1) / BM, ntn = (g.N + BN - 1) / BN;
  const int ntiles = ntm * ntn;
  const int nitems = ntiles * (CAUSAL ? g.nbatch : g.nsplit);
  const int G = (int)gridDim.x;
  int round = 0;
  int w = blockIdx.x;
  if (w >= nitems) return;

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int wm = wave / WN, wn = wave % WN;
  const int wrow0 = wm * (BM / WM), wcol0 = wn * (BN / WN);

  LA la;
  LB lb;
  typename LA::Dma da;
  typename LB::Dma db;
  da.init();
  db.init();
  LA::swizzle(da);
  LB::swizzle(db);

  // nkg: slices of one operand group (the causal products walk kgroups stacked operands)
  struct Item { int m0, n0, split, kbeg, kend, nk, nkg, nfull; int64_t aoff, boff, coff, coff_lo; };
  auto item = [&](int it) {
    Item t;
    int tm, tn;
    t.aoff = t.boff = t.coff = t.coff_lo = 0;
    if constexpr (CAUSAL) {
      // the one-tile launch's order: row tiles by K range, longest first; inside one, batch
      // entries that share their B panel on one XCD
      const int per = g.nbatch * ntn;
      tm = g.rev ? it / per : ntm - 1 - it / per;
      const int r = it % per;
      tn = r / g.nbatch;
      int z = r % g.nbatch;
      if (g.bdiv > 1 && g.nbatch % (8 * g.bdiv) == 0) {
        const int x = z % 8, j = z / 8;
        z = (x + 8 * (j / g.bdiv)) * g.bdiv + j % g.bdiv;
      }
      const int z1 = z / g.zdiv, z2 = z % g.zdiv;
      t.aoff = z * g.sA;
      t.boff = z1 * g.sB1 + (z2 / g.bdiv) * g.sB2;
      t.coff = z1 * g.sC1 + z2 * g.sC2;
      if constexpr (AK) t.coff_lo = z1 * g.sC1_lo + z2 * g.sC2_lo;
      t.split = 0;
    } else {
      const int x = it % ntiles;
      t.split = it / ntiles;
      const int pid = xcd_remap(x, ntiles);
      const int GROUP = 8;
      const int group = pid / (GROUP * ntn);
      const int first = group * GROUP;
      const int gsz = min(ntm - first, GROUP);
      tm = first + (pid % (GROUP * ntn)) % gsz;
      tn = (pid % (GROUP * ntn)) / gsz;
    }
    t.m0 = tm * BM;
    t.n0 = tn * BN;
    if constexpr (CAUSAL) {
      t.kbeg = g.rev ? t.m0 : 0;
      t.kend = g.rev ? g.ktotal : min(g.ktotal, t.m0 + BM);
      t.nkg = (t.kend - t.kbeg + BK - 1) / BK;
      t.nk = t.nkg * g.kgroups;
    } else {
      t.kbeg = t.split * g.kchunk;
      t.kend = min(g.ktotal, t.kbeg + g.kchunk);
      t.nk = t.nkg = (t.kend - t.kbeg + BK - 1) / BK;
    }
    const bool dma_ok = g.M - t.m0 >= BM && g.N - t.n0 >= BN &&
                        (AK ? (int64_t)BM * g.lda : (int64_t)BK * g.lda) < (1ll << 30) &&
                        (BKM ? (int64_t)BN * g.ldb : (int64_t)BK * g.ldb) < (1ll << 30);
    t.nfull = dma_ok ? (t.kend - t.kbeg) / BK : 0;
    // uniform by construction: keep every field in scalar registers
    t.m0 = __builtin_amdgcn_readfirstlane(t.m0);
    t.n0 = __builtin_amdgcn_readfirstlane(t.n0);
    t.split = __builtin_amdgcn_readfirstlane(t.split);
    t.kbeg = __builtin_amdgcn_readfirstlane(t.kbeg);
    t.kend = __builtin_amdgcn_readfirstlane(t.kend);
    t.nk = __builtin_amdgcn_readfirstlane(t.nk);
    t.nkg = __builtin_amdgcn_readfirstlane(t.nkg);
    t.nfull = __builtin_amdgcn_readfirstlane(t.nfull);
    return t;
  };
  // slice kt of a tile: operand group kt / nkg, walked from the top of its K range down
  // with rev (so that all row tiles of a batch entry stream the same B rows together)
  auto stage = [&](const Item& t, int kt, bf16_t* dst) {
    const bf16_t* pa = g.A + t.aoff;
    const bf16_t* pb = g.B + t.boff;
    int ks = kt;
    if constexpr (CAUSAL) {
      const int grp = g.kgroups > 1 ? kt / t.nkg : 0, ks0 = kt - grp * t.nkg;
      ks = g.rev ? t.nkg - 1 - ks0 : ks0;
      pa += grp * g.sAk;
      pb += grp * g.sBk;
    }
    const int k0 = t.kbeg + ks * BK;
    if (ks < t.nfull) {
      la.dma(da, pa, g.lda, t.m0, g.M - t.m0, k0, dst);
      lb.dma(db, pb, g.ldb, t.n0, g.N - t.n0, k0, dst + LA::ELEMS);
    } else {
      la.load(pa, g.lda, t.m0, g.M - t.m0, k0, t.kend);
      lb.load(pb, g.ldb, t.n0, g.N - t.n0, k0, t.kend);
      la.store(dst);
      lb.store(dst + LA::ELEMS);
    }
  };
  bf16x8 af[2][TM], bfr[2][TN];
  auto load_frags = [&](const bf16_t* As, int kk, bf16x8* a, bf16x8* b) {
    const bf16_t* Bs = As + LA::ELEMS;
#pragma unroll
    for (int i = 0; i < TM; ++i) a[i] = LA::frag(As, wrow0 + i * 32, kk);
#pragma unroll
    for (int j = 0; j < TN; ++j) b[j] = LB::frag(Bs, wcol0 + j * 32, kk);
  };
  f32x16 acc[TM][TN];
  auto mma = [&](const bf16x8* a, const bf16x8* b) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  };

  constexpr int WTN = BN / WN;
  constexpr int SLD = WTN + 8;
  static_assert(NTHR / 64 * 16 * SLD * 4 <= STAGE * 2, "epilogue half strip too large");
  const bool vec = (g.ldc % 4) == 0;
  TC* C = (TC*)g.C;

  Item cur = item(w);
  int rb = 0;          // stage of the current tile's first slice
  bool issued = false; // the current tile's first slice is already in flight
  for (;;) {
    const int wnext = CAUSAL ? (round + 1) * G + ((round & 1) ? (int)blockIdx.x : G - 1 - (int)blockIdx.x)
                             : w + G;
    const bool has_next = wnext < nitems;
    Item nxt{};
    if (has_next) nxt = item(wnext);
    if (!issued) {
      lds_barrier();  // every wavefront is past its previous epilogue
      if (cur.nk > 0) stage(cur, 0, lds + rb * STAGE);
    }
    bool pre = false;  // the next tile's first slice was issued during this tile
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    // the first slice (and the previous epilogue's stores) complete; every wavefront is done
    // with the previous epilogue's strips before the other stage is refilled
    wait_vm<0>();
    lds_barrier();
    if (cur.nk > 0) load_frags(lds + rb * STAGE, 0, af[0], bfr[0]);
    for (int kt = 0; kt < cur.nk; ++kt) {
      const bf16_t* As = lds + ((rb + kt) & 1) * STAGE;
      bf16_t* other = lds + ((rb + kt + 1) & 1) * STAGE;
      const bool last = kt + 1 == cur.nk;
      // the other stage is free: every wave passed the barrier after its last read
      if (!last) {
        stage(cur, kt + 1, other);
      } else if (has_next && nxt.nk > 0) {
        stage(nxt, 0, other);
        pre = true;
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        if (kk + 1 < KK) {
          load_frags(As, kk + 1, af[(kk + 1) & 1], bfr[(kk + 1) & 1]);
        } else if (!last) {
          wait_vm<0>();
          lds_barrier();
          load_frags(other, 0, af[0], bfr[0]);
        } else {
          // every wave is done reading this stage (the epilogue reuses it); the next
          // tile's copies stay in flight
          lds_barrier();
        }
        __builtin_amdgcn_sched_barrier(0);
        mma(af[kk & 1], bfr[kk & 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // epilogue in the stage of the last slice, 16 rows of a wavefront's strip at a time
    const int es = cur.nk > 0 ? (rb + cur.nk - 1) & 1 : rb;
    // the lane index made opaque here, so that the epilogue's per-lane addresses are formed
    // per tile instead of being hoisted out of the tile loop (and held through the main loop)
    int el = lane;
    asm volatile("" : "+v"(el));
    float* strip = (float*)(lds + es * STAGE) + wave * 16 * SLD;
    // two copies: with beta = 0 the epilogue reads no C, so the compiler has no loads to
    // wait for before each store (a wait that would also cover the next tile's copy and
    // every earlier store)
    auto epilogue = [&](auto with_beta) {
      constexpr bool WB = decltype(with_beta)::value;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 8 * h; e < 8 * h + 8; ++e)
              strip[(((e >> 2) & 1) * 8 + (el >> 5) * 4 + (e & 3)) * SLD + j * 32 + (el & 31)] =
                  acc[i][j][e];
          constexpr int CPR = WTN / 4;
          constexpr int NIT = 16 * CPR / 64;
          // the strip's reads first (all inside the strip), then the stores: the reads go
          // out together instead of one wait per store (not for the causal products, where
          // reading as it stores measured faster)
          constexpr bool BATCH = !CAUSAL;
          f32x4 vv[BATCH ? NIT : 1];
          if constexpr (BATCH) {
#pragma unroll
            for (int it = 0; it < NIT; ++it) {
              const int c = it * 64 + el;
              vv[it] = *(const f32x4*)(strip + (c / CPR) * SLD + (c % CPR) * 4);
            }
          }
#pragma unroll
          for (int it = 0; it < NIT; ++it) {
            const int c = it * 64 + el;
            const int r = c / CPR, col = (c % CPR) * 4;
            const int m = cur.m0 + wrow0 + i * 32 + 16 * h + r, n = cur.n0 + wcol0 + col;
            if (m >= g.mstore || n >= g.N) continue;
            f32x4 v;
            if constexpr (BATCH) v = vv[it];
            else v = *(const f32x4*)(strip + r * SLD + col);
            if (g.part) {
              float* p = g.part + ((int64_t)cur.split * g.M + m) * g.N + n;
              if (n + 4 <= g.N && (g.N % 4) == 0) {
                *(f32x4*)p = v;
              } else {
                for (int q = 0; q < 4 && n + q < g.N; ++q) p[q] = v[q];
              }
              continue;
            }
            if constexpr (CAUSAL && AK) {
              if (g.split_n > 0) {  // uniform; whole 4-column groups (split_n % 4 == 0)
                if (n < g.split_n) {
                  const f32x4 o = v * g.alpha;
                  *(u32x2*)(g.c_lo + cur.coff_lo + (int64_t)m * g.ldc_lo + n) =
                      u32x2{pack2bf(o[0], o[1]), pack2bf(o[2], o[3])};
                } else {
                  *(f32x4*)((float*)g.C + cur.coff + (int64_t)m * g.ldc + (n - g.split_n)) = v * g.alpha;
                }
                continue;
              }
            }
            TC* p = C + cur.coff + (int64_t)m * g.ldc + n;
            if (vec && n + 4 <= g.N) {
              store4<TC>(p, v, g.alpha, WB ? g.beta : 0.f);
            } else {
              for (int q = 0; q < 4 && n + q < g.N; ++q) {
                float x = g.alpha * v[q];
                if (WB && g.beta != 0.f) x += g.beta * ld(p + q);
                store_out<TC>(p + q, x);
              }
            }
          }
        }
      }
    };
    // (the causal products never accumulate into C: beta = 0 is checked at their launch)
    if constexpr (CAUSAL) epilogue(std::false_type{});
    else if (g.beta != 0.f) epilogue(std::true_type{}); else epilogue(std::false_type{});
    if (!has_next) break;
    rb = (rb + cur.nk) & 1;
    issued = pre;
    cur = nxt;
    w = wnext;
    ++round;
  }
}

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC, int BK, int NST>
__global__ __launch_bounds__(64 * WM * WN) void gemm_mfma_persist_kernel(GemmDev g) {
  gemm_persist<BM, BN, WM, WN, AK, BKM, TC, BK, NST, false>(g);
}
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC, int BK, int NST>
__global__ __launch_bounds__(64 * WM * WN) void attn_ds_gemm_persist_kernel(GemmDev g) {
  gemm_persist<BM, BN, WM, WN, AK, BKM, TC, BK, NST, true>(g);
}
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC, int BK, int NST>
__global__ __launch_bounds__(64 * WM * WN) void gemm_mfma_kernel(GemmDev g) {
  gemm_tile<BM, BN, WM, WN, AK, BKM, TC, BK, NST>(g);
}
// the same tile program for the dS products of attention's backward, on the 32 x 32-tiled
// dS^T (own name, so that profiles tell them apart)
template <int BM, int BN, int WM, int WN, bool AK, bool BKM, typename TC, int BK, int NST>
__global__ __launch_bounds__(64 * WM * WN) void attn_ds_gemm_kernel(GemmDev g) {
  gemm_tile<BM, BN, WM, WN, AK, BKM, TC, BK, NST, true>(g);
}

// ---- NT products on four wavefronts, k-steps scheduled by hand ------------------------
//
// Both operands K-contiguous, M a multiple of 256, N of the tile width (256 or 192), K a
// multiple of 128.  A workgroup of four wavefronts (one per SIMD) owns a 256 x 256 tile,
// 128 x 128 per wavefront (16 accumulators of 32 x 32 in AGPRs; 256 x 192 tiles: 128 x 96,
// 12 accumulators); per 16-wide k step each wavefront reads 8 KB of operands from LDS,
// a third fewer LDS bytes per MFMA than the 8-wavefront tiles.  With one wavefront per SIMD no other wavefront hides its waits, so
// each k step is one block of inline assembly in a fixed order: the 16 MFMAs of the step,
// one operand read for the step after next between every other pair of them (operands
// are read two k steps ahead into four register buffers), and on the two steps after
// each slice barrier the 8 LDS DMA copies of the next-but-one slice between the others.
// The compiler does not see the assembly's LDS and memory operations: every block starts
// with the wait for the reads of the step before last (at most 8 reads are younger), and
// each slice barrier waits for all copies.  A persistent grid walks the tiles; the next
// tile's first two slices are copied, and its first two k steps read, while the current
// tile finishes, and the epilogue stages 8-row strips in a 17 KB LDS region of its own.
// Measured on the 16384 x 4096 x 4096 product: 475 us against 532 us for the 8-wavefront
// tile, the matrix cores 81% busy instead of 62%.  (The other operand layouts read one
// operand with the transposing LDS read, 8 bytes of a fragment per instruction; inline
// assembly cannot name the halves of a 128-bit operand, so they stay compiler-scheduled.)
#define NT4_MF(c, a, b) "v_mfma_f32_32x32x16_bf16 %[" #c "], %[" #a "], %[" #b "], %[" #c "]\n"
#define NT4_RD(d, base, off) "ds_read_b128 %[" #d "], %[" #base "] offset:" #off "\n"
#define NT4_CP(o, src, m, off) \
  "s_add_u32 m0, %[" #m "], " #off "\ns_nop 0\nglobal_load_lds_dwordx4 %[" #o "], %[" #src "]\n"
// the 16 MFMAs of one k step with the 8 operand reads of the step after next after
// MFMAs 0, 2, .., 14 (read order = first use: A0, B0..B3, A1..A3)
#define NT4_STEP_BODY(X0, X1, X2, X3, X4, X5, X6, X7)                                       \
  "s_waitcnt lgkmcnt(8)\n"                                                                \
  NT4_MF(c00, a0, b0) NT4_RD(nA0, ra, 0) NT4_MF(c01, a0, b1) X0                             \
  NT4_MF(c02, a0, b2) NT4_RD(nB0, rb, 0) NT4_MF(c03, a0, b3) X1                             \
  NT4_MF(c10, a1, b0) NT4_RD(nB1, rb, 4096) NT4_MF(c11, a1, b1) X2                          \
  NT4_MF(c12, a1, b2) NT4_RD(nB2, rb, 8192) NT4_MF(c13, a1, b3) X3                          \
  NT4_MF(c20, a2, b0) NT4_RD(nB3, rb, 12288) NT4_MF(c21, a2, b1) X4                         \
  NT4_MF(c22, a2, b2) NT4_RD(nA1, ra, 4096) NT4_MF(c23, a2, b3) X5                          \
  NT4_MF(c30, a3, b0) NT4_RD(nA2, ra, 8192) NT4_MF(c31, a3, b1) X6                          \
  NT4_MF(c32, a3, b2) NT4_RD(nA3, ra, 12288) NT4_MF(c33, a3, b3) X7
#define NT4_OUTS                                                                            \
  [c00] "+a"(acc[0][0]), [c01] "+a"(acc[0][1]), [c02] "+a"(acc[0][2]), [c03] "+a"(acc[0][3]), \
  [c10] "+a"(acc[1][0]), [c11] "+a"(acc[1][1]), [c12] "+a"(acc[1][2]), [c13] "+a"(acc[1][3]), \
  [c20] "+a"(acc[2][0]), [c21] "+a"(acc[2][1]), [c22] "+a"(acc[2][2]), [c23] "+a"(acc[2][3]), \
  [c30] "+a"(acc[3][0]), [c31] "+a"(acc[3][1]), [c32] "+a"(acc[3][2]), [c33] "+a"(acc[3][3]), \
  [nA0] "=&v"(nx[0]), [nA1] "=&v"(nx[1]), [nA2] "=&v"(nx[2]), [nA3] "=&v"(nx[3]),          \
  [nB0] "=&v"(nx[4]), [nB1] "=&v"(nx[5]), [nB2] "=&v"(nx[6]), [nB3] "=&v"(nx[7])
#define NT4_INS                                                                             \
  [a0] "v"(cu[0]), [a1] "v"(cu[1]), [a2] "v"(cu[2]), [a3] "v"(cu[3]), [b0] "v"(cu[4]),      \
  [b1] "v"(cu[5]), [b2] "v"(cu[6]), [b3] "v"(cu[7]), [ra] "v"(ra), [rb] "v"(rb)
// the same for 256 x 192 tiles (128 x 96 per wavefront): 12 MFMAs, 7 reads (A0, B0..B2,
// A1..A3), up to 7 copies
#define NT4_STEP_BODY3(X0, X1, X2, X3, X4, X5, X6)                                          \
  "s_waitcnt lgkmcnt(7)\n"                                                                \
  NT4_MF(c00, a0, b0) NT4_RD(nA0, ra, 0) NT4_MF(c01, a0, b1) X0                             \
  NT4_MF(c02, a0, b2) NT4_RD(nB0, rb, 0) NT4_MF(c10, a1, b0) X1                             \
  NT4_MF(c11, a1, b1) NT4_RD(nB1, rb, 4096) NT4_MF(c12, a1, b2) X2                          \
  NT4_MF(c20, a2, b0) NT4_RD(nB2, rb, 8192) NT4_MF(c21, a2, b1) X3                          \
  NT4_MF(c22, a2, b2) NT4_RD(nA1, ra, 4096) NT4_MF(c30, a3, b0) X4                          \
  NT4_MF(c31, a3, b1) NT4_RD(nA2, ra, 8192) NT4_MF(c32, a3, b2) X5                          \
  NT4_RD(nA3, ra, 12288) X6
#define NT4_OUTS3                                                                           \
  [c00] "+a"(acc[0][0]), [c01] "+a"(acc[0][1]), [c02] "+a"(acc[0][2]), [c10] "+a"(acc[1][0]), \
  [c11] "+a"(acc[1][1]), [c12] "+a"(acc[1][2]), [c20] "+a"(acc[2][0]), [c21] "+a"(acc[2][1]), \
  [c22] "+a"(acc[2][2]), [c30] "+a"(acc[3][0]), [c31] "+a"(acc[3][1]), [c32] "+a"(acc[3][2]), \
  [nA0] "=&v"(nx[0]), [nA1] "=&v"(nx[1]), [nA2] "=&v"(nx[2]), [nA3] "=&v"(nx[3]),          \
  [nB0] "=&v"(nx[4]), [nB1] "=&v"(nx[5]), [nB2] "=&v"(nx[6])
#define NT4_INS3                                                                            \
  [a0] "v"(cu[0]), [a1] "v"(cu[1]), [a2] "v"(cu[2]), [a3] "v"(cu[3]), [b0] "v"(cu[4]),      \
  [b1] "v"(cu[5]), [b2] "v"(cu[6]), [ra] "v"(ra), [rb] "v"(rb)

template <int BN, typename TC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_nt4_persist_kernel(GemmDev g) {
  constexpr int BM = 256, BKK = 64, TM = 4, TN = BN / 64;  // 4 or 3 fragments of B
  constexpr int WTN = BN / 2;                              // columns per wavefront
  using LA = Loader<true, BM, 256, BKK>;  // operand tile layouts (swizzled rows)
  using LB = Loader<true, BN, 256, BKK>;
  constexpr int STAGE = LA::ELEMS + LB::ELEMS;  // elements: A [256][64], then B [BN][64]
  constexpr int SLD = WTN + 4;                  // epilogue strip row (floats)
  constexpr int EPI = 4 * 8 * SLD;              // floats: four wavefronts x 8 rows
  constexpr int PB = LB::Dma::PER;              // B copies per lane per slice: 8 or 6
  static_assert(BN == 256 || BN == 192, "tile widths");
  static_assert(LA::Dma::PER == 8 && PB == TN * 2, "copies per lane per operand slice");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[2 * STAGE + 2 * EPI];
  const int ntm = g.M / BM, ntn = g.N / BN, ntiles = ntm * ntn;
  const int G = (int)gridDim.x;
  int w = blockIdx.x;
  if (w >= ntiles) return;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int wrow0 = (wave >> 1) * 128, wcol0 = (wave & 1) * WTN;
  // the tile order of the one-tile launch: XCD-aware remap, 8 row panels per group
  auto tile_of = [&](int x, int& m0, int& n0) {
    const int pid = xcd_remap(x, ntiles);
    const int group = pid / (8 * ntn), first = group * 8, gsz = min(ntm - first, 8);
    m0 = __builtin_amdgcn_readfirstlane((first + (pid % (8 * ntn)) % gsz) * BM);
    n0 = __builtin_amdgcn_readfirstlane(((pid % (8 * ntn)) / gsz) * BN);
  };
  typename LA::Dma da;
  typename LB::Dma db;
  da.init();
  db.init();
  LA::swizzle(da);
  LB::swizzle(db);
  // copy p of a slice: this lane's byte offset from the slice's first element (A, B) and
  // LDS block wave + 4 p of the operand tile
  uint32_t oA[8], oB[8];
#pragma unroll
  for (int p = 0; p < 8; ++p) oA[p] = 2u * (uint32_t)(da.row[p] * (int)g.lda + da.col[p]);
#pragma unroll
  for (int p = 0; p < PB; ++p) oB[p] = 2u * (uint32_t)(db.row[p] * (int)g.ldb + db.col[p]);
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;  // LDS byte address
  // operand read addresses of stage st, k step kk (fragment i / j at + 4096 i bytes)
  const int l = lane & 31, h = lane >> 5;
  uint32_t adA[2][4], adB[2][4];
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint32_t sw = 16u * (uint32_t)((2 * kk + h) ^ LA::swz(l));
      adA[st][kk] = lds0 + st * STAGE * 2 + (wrow0 + l) * BKK * 2 + sw;
      adB[st][kk] = lds0 + st * STAGE * 2 + LA::ELEMS * 2 + (wcol0 + l) * BKK * 2 +
                    16u * (uint32_t)((2 * kk + h) ^ LB::swz(l));
    }
  const int nk = g.ktotal / BKK;  // even
  int m0, n0, nm0 = 0, nn0 = 0;
  tile_of(w, m0, n0);
  const bf16_t* baseA = g.A + (int64_t)m0 * g.lda;
  const bf16_t* baseB = g.B + (int64_t)n0 * g.ldb;
  int wnext = w + G;
  bool has_next = wnext < ntiles;
  const bf16_t* nbaseA = baseA;
  const bf16_t* nbaseB = baseB;
  if (has_next) {
    tile_of(wnext, nm0, nn0);
    nbaseA = g.A + (int64_t)nm0 * g.lda;
    nbaseB = g.B + (int64_t)nn0 * g.ldb;
  }
  f32x16 acc[TM][TN];
  bf16x8 F[4][8];  // operand buffers of four k steps: A 0..3, B 4..7
  // k step on buffer cur, reading step kk of stage st into buffer nxt
  auto step = [&](int cur, int nxt, int st, int kk) {
    const bf16x8* cu = F[cur];
    bf16x8* nx = F[nxt];
    const uint32_t ra = adA[st][kk], rb = adB[st][kk];
    if constexpr (TN == 4)
      asm volatile(NT4_STEP_BODY("", "", "", "", "", "", "", "") : NT4_OUTS : NT4_INS : "memory");
    else
      asm volatile(NT4_STEP_BODY3("", "", "", "", "", "", "") : NT4_OUTS3 : NT4_INS3 : "memory");
  };
  // the same with copies q (0: 0..3, 1: 4..7) of slice ks of this tile into stage ks % 2,
  // or of slice ks - nk of the next one (after the last tile: a repeat of this tile's last
  // slice into the stage nobody reads any more)
  auto step_copy = [&](int cur, int nxt, int st, int kk, int ks, int q) {
    const bf16x8* cu = F[cur];
    bf16x8* nx = F[nxt];
    const uint32_t ra = adA[st][kk], rb = adB[st][kk];
    const bool in_next = ks >= nk;
    const int kq = in_next ? (has_next ? ks - nk : nk - 1) : ks;
    const bf16_t* pa = (in_next && has_next ? nbaseA : baseA) + kq * BKK;
    const bf16_t* pb = (in_next && has_next ? nbaseB : baseB) + kq * BKK;
    // copies q of A: blocks wave + 4 p, p = 4 q .. 4 q + 3; of B: p = (PB / 2) q + u
    const uint32_t stg = lds0 + (ks & 1) * STAGE * 2 + wave * 1024;
    const uint32_t ma = (uint32_t)__builtin_amdgcn_readfirstlane((int)(stg + 16384 * q));
    const uint32_t mb = (uint32_t)__builtin_amdgcn_readfirstlane(
        (int)(stg + LA::ELEMS * 2 + 4096 * (PB / 2) * q));
    const uint64_t sa = uniform_ptr(pa), sb = uniform_ptr(pb);
    const uint32_t oa0 = oA[4 * q], oa1 = oA[4 * q + 1], oa2 = oA[4 * q + 2], oa3 = oA[4 * q + 3];
    const int qb = (PB / 2) * q;
    const uint32_t ob0 = oB[qb], ob1 = oB[qb + 1], ob2 = oB[qb + 2], ob3 = oB[PB == 8 ? qb + 3 : qb];
    uint32_t m0v;  // m0 (the copies' LDS destination) is written early by the block
    if constexpr (TN == 4)
      asm volatile(NT4_STEP_BODY(NT4_CP(oa0, sa, ma, 0), NT4_CP(oa1, sa, ma, 4096),
                                 NT4_CP(oa2, sa, ma, 8192), NT4_CP(oa3, sa, ma, 12288),
                                 NT4_CP(ob0, sb, mb, 0), NT4_CP(ob1, sb, mb, 4096),
                                 NT4_CP(ob2, sb, mb, 8192), NT4_CP(ob3, sb, mb, 12288))
                   : NT4_OUTS, [m0v] "=&{m0}"(m0v)
                   : NT4_INS, [oa0] "v"(oa0), [oa1] "v"(oa1), [oa2] "v"(oa2), [oa3] "v"(oa3),
                     [ob0] "v"(ob0), [ob1] "v"(ob1), [ob2] "v"(ob2), [ob3] "v"(ob3), [sa] "s"(sa),
                     [sb] "s"(sb), [ma] "s"(ma), [mb] "s"(mb)
                   : "memory");
    else
      asm volatile(NT4_STEP_BODY3(NT4_CP(oa0, sa, ma, 0), NT4_CP(oa1, sa, ma, 4096),
                                  NT4_CP(oa2, sa, ma, 8192), NT4_CP(oa3, sa, ma, 12288),
                                  NT4_CP(ob0, sb, mb, 0), NT4_CP(ob1, sb, mb, 4096),
                                  NT4_CP(ob2, sb, mb, 8192))
                   : NT4_OUTS3, [m0v] "=&{m0}"(m0v)
                   : NT4_INS3, [oa0] "v"(oa0), [oa1] "v"(oa1), [oa2] "v"(oa2), [oa3] "v"(oa3),
                     [ob0] "v"(ob0), [ob1] "v"(ob1), [ob2] "v"(ob2), [sa] "s"(sa), [sb] "s"(sb),
                     [ma] "s"(ma), [mb] "s"(mb)
                   : "memory");
  };
  // prologue: slices 0 and 1 of the first tile, steps 0 and 1 read
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    bf16_t* dst = lds + kt * STAGE;
#pragma unroll
    for (int p = 0; p < 8; ++p) dma16_s(baseA + kt * BKK, oA[p], dst + (wave + p * 4) * 512);
#pragma unroll
    for (int p = 0; p < PB; ++p) dma16_s(baseB + kt * BKK, oB[p], dst + LA::ELEMS + (wave + p * 4) * 512);
  }
  wait_vm<8 + PB>();
  lds_barrier();
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) F[kk][i] = LA::frag(lds, wrow0 + i * 32, kk);
#pragma unroll
    for (int j = 0; j < TN; ++j) F[kk][4 + j] = LB::frag(lds + LA::ELEMS, wcol0 + j * 32, kk);
  }
  // every read of the compiler's own has landed: its counter bookkeeping starts empty
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  // row-masked scale of the result, through a scalar load: a vector load would leave the
  // compiler counting it as outstanding in the tile loop, where its waits would also wait
  // for the copies in flight
  float lsc = 0.f;
  if (g.lscale) {  // uniform
    const uint64_t pl = uniform_ptr(g.lscale);
    uint32_t u;
    asm volatile("s_load_dword %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(u) : "s"(pl) : "memory");
    lsc = __uint_as_float(u);
  }
  float* strip = (float*)(lds + 2 * STAGE) + wave * 8 * SLD;
  for (;;) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    // two slices per pass: slice kt in stage 0, slice kt + 1 in stage 1
    for (int kt = 0; kt < nk; kt += 2) {
      step(0, 2, 0, 2);
      step(1, 3, 0, 3);
      wait_vm<0>();
      lds_barrier();  // slice kt + 1 has landed; nobody reads stage 0 any more
      step_copy(2, 0, 1, 0, kt + 2, 0);
      step_copy(3, 1, 1, 1, kt + 2, 1);
      step(0, 2, 1, 2);
      step(1, 3, 1, 3);
      wait_vm<0>();
      lds_barrier();  // slice kt + 2 (or the next tile's slice 0) has landed
      step_copy(2, 0, 0, 0, kt + 3, 0);
      step_copy(3, 1, 0, 1, kt + 3, 1);
    }
    // epilogue: rows 8 gq .. 8 gq + 7 of each 32-row block, staged in this wavefront's
    // region (a lane holds column l of rows 4 h .. 4 h + 3 of the group) and written back
    // 4 columns per lane.  Two copies: with beta = 0 (every product of the step) the
    // epilogue reads no C, so the compiler has no loads to wait for before each store (it
    // would otherwise wait for every memory operation in flight, the next tile's copies
    // included)
    TC* C = (TC*)g.C;
    // (beta and the masked scale are compile-time in each copy: with no branch inside, the
    // four strip reads of a row group are issued together, then converted and stored)
    auto epilogue = [&](auto with_beta, auto with_scale) {
      constexpr bool WB = decltype(with_beta)::value;
      constexpr bool LS = decltype(with_scale)::value;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        // the row mask of this 32-row block through one scalar load (the launcher checks its
        // 4-byte alignment): a vector load here would wait, in order, for the next tile's
        // copies already in flight
        u32x8 mk = {1u, 1u, 1u, 1u, 1u, 1u, 1u, 1u};
        if (LS && g.lmask) {  // uniform
          const uint64_t pa = uniform_ptr(g.lmask + m0 + wrow0 + i * 32);
          asm volatile("s_load_dwordx8 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(mk) : "s"(pa) : "memory");
        }
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) strip[(4 * h + q) * SLD + j * 32 + l] = acc[i][j][4 * gq + q];
          f32x4 v[TN];
#pragma unroll
          for (int it = 0; it < TN; ++it) {
            const int c = it * 64 + lane;
            v[it] = *(const f32x4*)(strip + (c / (WTN / 4)) * SLD + (c % (WTN / 4)) * 4);
          }
#pragma unroll
          for (int it = 0; it < TN; ++it) {
            const int c = it * 64 + lane;
            const int r = c / (WTN / 4), col = (c % (WTN / 4)) * 4;
            const int m = m0 + wrow0 + i * 32 + 8 * gq + r, n = n0 + wcol0 + col;
            f32x4 o = v[it];
            if constexpr (LS) {  // row r of the block's 8-row group gq: byte 8 gq + r of mk
              const uint32_t dw = r >= 4 ? mk[2 * gq + 1] : mk[2 * gq];
              const bool keep = ((dw >> (8 * (r & 3))) & 0xffu) != 0u;
              const f32x4 so = o * lsc;  // masked rows exactly 0 (also where o is not finite)
              o = f32x4{keep ? so[0] : 0.f, keep ? so[1] : 0.f, keep ? so[2] : 0.f, keep ? so[3] : 0.f};
            }
            store4<TC>(C + (int64_t)m * g.ldc + n, o, g.alpha, WB ? g.beta : 0.f);
          }
        }
      }
    };
    if (g.lscale) {  // the masked dO product (beta = 0)
      if (g.beta != 0.f) epilogue(std::true_type{}, std::true_type{});
      else epilogue(std::false_type{}, std::true_type{});
    } else {
      if (g.beta != 0.f) epilogue(std::true_type{}, std::false_type{});
      else epilogue(std::false_type{}, std::false_type{});
    }
    if (!has_next) break;
    w = wnext;
    m0 = nm0;
    n0 = nn0;
    baseA = nbaseA;
    baseB = nbaseB;
    wnext = w + G;
    has_next = wnext < ntiles;
    if (has_next) {
      tile_of(wnext, nm0, nn0);
      nbaseA = g.A + (int64_t)nm0 * g.lda;
      nbaseB = g.B + (int64_t)nn0 * g.ldb;
    }
  }
}

// C = alpha * sum_s part[s] + beta * C, summed in split order (split s of the M x N block at
// part + s * sstride)
template <typename TC>
__global__ void splitk_reduce_kernel(const float* __restrict__ part, int splits, int64_t sstride,
                                     int M, int N, TC* __restrict__ C, int64_t ldc, float alpha,
                                     float beta) {
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t total = (int64_t)M * N;
  if (idx >= total) return;
  int m = (int)(idx / N), n = (int)(idx % N);
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += part[(int64_t)z * sstride + idx];
  TC* c = C + (int64_t)m * ldc + n;
  float v = alpha * s;
  if (beta != 0.f) v += beta * ld(c);
  store_out<TC>(c, v);
}

// the same, four consecutive outputs per thread (N and ldc multiples of 4)
template <typename TC>
__global__ void splitk_reduce4_kernel(const float* __restrict__ part, int splits, int64_t sstride,
                                      int M, int N, TC* __restrict__ C, int64_t ldc, float alpha,
                                      float beta) {
  const int64_t idx = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
  const int64_t total = (int64_t)M * N;
  if (idx >= total) return;
  const int m = (int)(idx / N), n = (int)(idx % N);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int z = 0; z < splits; ++z) acc += *(const f32x4*)(part + (int64_t)z * sstride + idx);
  store4<TC>(C + (int64_t)m * ldc + n, acc, alpha, beta);
}

// Tile shape and split-K factor.  Candidates: 256 x 256 and 256 x 192 tiles on 8
// wavefronts (one workgroup per CU) and 128 x 128 tiles on 4 (two per CU).  Workgroups run
// in rounds of one per CU slot, so a grid of 1.5 rounds costs two: the plan minimises
// rounds x (work of one workgroup) / (relative matrix-core rate of its tile), plus the
// split-K partials' traffic, over tile shapes and split factors.
struct Plan {
  int kind;  // 0: 256 x 256, 1: 256 x 192, 2: 128 x 128, 3: 192 x 256 (weight gradients)
  int bm, bn, splits, kchunk;
};

constexpr int NUM_CU = 256;

Plan plan_of(const Gemm& g, bool allow_split) {
  struct Cand { int kind, bm, bn, per_cu; double rate; };
  // relative per-CU rates (fitted to timings of the step's shapes): the narrower tile reads
  // more LDS bytes per matrix op (much more so with an M-contiguous A); two 4-wavefront
  // workgroups share one CU
  // 192-row tiles for the weight gradients whose rows are a multiple of 192 (the 576 rows
  // of [W_DKV; W_KR] without a ragged row tile; fewer rounds or splits for others)
  const bool tn192 = !g.a_kmajor && !g.b_kmajor && g.M % 192 == 0;
  const Cand cands[] = {{0, 256, 256, 1, 1.0}, {1, 256, 192, 1, g.a_kmajor ? 0.93 : 0.7},
                        {2, 128, 128, 2, 0.62}, {3, 192, 256, 1, 0.8}};
  Plan best{2, 128, 128, 1, 0};
  double best_t = 1e300;
  const int kslices = (g.K + BK - 1) / BK;
  for (const Cand& c : cands) {
    if (c.kind == 3 && !tn192) continue;
    const int64_t tiles = (int64_t)((g.M + c.bm - 1) / c.bm) * ((g.N + c.bn - 1) / c.bn);
    const int max_s = allow_split && g.K >= 8 * BK * 8 ? std::max(1, kslices / 8) : 1;
    for (int sp = 1; sp <= std::min(max_s, 64); ++sp) {
      const int kc_sl = (kslices + sp - 1) / sp;  // K slices per split
      const int splits = (kslices + kc_sl - 1) / kc_sl;
      if (splits != sp) continue;
      const int64_t wgs = tiles * splits;
      const int64_t slots = (int64_t)NUM_CU * c.per_cu;
      const int64_t rounds = (wgs + slots - 1) / slots;
      // time units: one 64-deep slice of a 256 x 256 tile at full rate on one CU
      double t = (double)rounds * kc_sl * ((double)c.bm * c.bn / 65536.0) * c.per_cu / c.rate;
      // partials written and read back (fp32): fitted to the same timings, about 3 MB per
      // unit of time (one 64-deep slice of a 256 x 256 tile)
      if (splits > 1) t += (double)(splits + 1) * g.M * g.N * 4 / 3.0e6;
      if (t < best_t * 0.999) {
        best_t = t;
        best = Plan{c.kind, c.bm, c.bn, splits, kc_sl * BK};
      }
    }
  }
  return best;
}

// Tile width of the four-wavefront NT kernel for this product: 256 or 192, or 0 where it
// does not apply (it needs whole tiles, K a multiple of 128, no split-K, operand rows
// within 32-bit offsets, 16-byte aligned operands and 4-element output rows).  Of the two
// widths, the one with fewer rounds x tile width (rounds of one tile per CU).
int nt4_bn(const GemmDev& d, const Plan& p) {
  const bool ok = p.splits == 1 && !d.part && !d.lpart && !d.causal && d.M % 256 == 0 &&
                  d.ktotal % 128 == 0 && d.ktotal >= 128 && d.lda % 8 == 0 && d.ldb % 8 == 0 &&
                  d.ldc % 4 == 0 && (uintptr_t)d.A % 16 == 0 && (uintptr_t)d.B % 16 == 0 &&
                  (uintptr_t)d.C % 16 == 0 && (int64_t)256 * d.lda * 2 < (1ll << 31) &&
                  (int64_t)256 * d.ldb * 2 < (1ll << 31);
  if (!ok) return 0;
  auto cost = [&](int bn) {
    const int64_t tiles = (int64_t)(d.M / 256) * (d.N / bn);
    return (double)((tiles + NUM_CU - 1) / NUM_CU) * bn;
  };
  const bool w256 = d.N % 256 == 0, w192 = d.N % 192 == 0;
  if (w256 && (!w192 || cost(256) <= cost(192))) return 256;
  return w192 ? 192 : 0;
}

template <bool AK, bool BKM, typename TC>
const char* launch(const GemmDev& d, const Plan& p, hipStream_t s) {
  if constexpr (AK && BKM) {
    const int bn = nt4_bn(d, p);
    if (bn == 256) {
      const int tiles = (d.M / 256) * (d.N / 256);
      gemm_nt4_persist_kernel<256, TC><<<std::min(tiles, NUM_CU), 256, 0, s>>>(d);
      return KLABEL("gemm_nt4_persist_kernel<256,256,NT,%s>", sizeof(TC) == 4 ? "fp32" : "bf16");
    }
    if (bn == 192) {
      const int tiles = (d.M / 256) * (d.N / 192);
      gemm_nt4_persist_kernel<192, TC><<<std::min(tiles, NUM_CU), 256, 0, s>>>(d);
      return KLABEL("gemm_nt4_persist_kernel<256,192,NT,%s>", sizeof(TC) == 4 ? "fp32" : "bf16");
    }
  }
  const int tiles = ((d.M + p.bm - 1) / p.bm) * ((d.N + p.bn - 1) / p.bn);
  const bool persist = d.lpart == nullptr;
#define GL_(name, bm, bn) KLABEL(name "<%d,%d,%s,%s>", bm, bn, AK ? (BKM ? "NT" : "NN") : (BKM ? "TT" : "TN"), \
                                 sizeof(TC) == 4 ? "fp32" : "bf16")
  if (persist) {
    GemmDev e = d;
    e.nsplit = p.splits;
    const int per_cu = p.kind == 2 ? 2 : 1;
    const int grid = std::min(tiles * p.splits, NUM_CU * per_cu);
    if (p.kind == 0) {
      gemm_mfma_persist_kernel<256, 256, GWM, GWN, AK, BKM, TC, GBK, GNST><<<grid, 64 * GWM * GWN, 0, s>>>(e);
      return GL_("gemm_mfma_persist_kernel", 256, 256);
    } else if (p.kind == 1) {
      gemm_mfma_persist_kernel<256, 192, 4, 2, AK, BKM, TC, GBK, GNST><<<grid, 512, 0, s>>>(e);
      return GL_("gemm_mfma_persist_kernel", 256, 192);
    } else if (p.kind == 3) {
      if constexpr (!AK && !BKM) {
        gemm_mfma_persist_kernel<192, 256, 2, 4, AK, BKM, TC, GBK, GNST><<<grid, 512, 0, s>>>(e);
        return GL_("gemm_mfma_persist_kernel", 192, 256);
      }
    }
    gemm_mfma_persist_kernel<128, 128, 2, 2, AK, BKM, TC, 64, 2><<<grid, 256, 0, s>>>(e);
    return GL_("gemm_mfma_persist_kernel", 128, 128);
  }
  // the masked-loss epilogue
  dim3 grid(tiles, p.splits);
  if (p.kind == 0) {
    gemm_mfma_kernel<256, 256, GWM, GWN, AK, BKM, TC, GBK, GNST><<<grid, 64 * GWM * GWN, 0, s>>>(d);
    return GL_("gemm_mfma_kernel(masked loss)", 256, 256);
  } else if (p.kind == 1) {
    gemm_mfma_kernel<256, 192, 4, 2, AK, BKM, TC, GBK, GNST><<<grid, 512, 0, s>>>(d);
    return GL_("gemm_mfma_kernel(masked loss)", 256, 192);
  }
  gemm_mfma_kernel<128, 128, 2, 2, AK, BKM, TC, 64, 2><<<grid, 256, 0, s>>>(d);
  return GL_("gemm_mfma_kernel(masked loss)", 128, 128);
#undef GL_
}


}  // namespace

size_t gemm_mfma_scratch_elems(const Gemm& g) {
  Plan p = plan_of(g, true);
  return p.splits > 1 || g.C2 ? (size_t)p.splits * g.M * g.N : 0;
}

hipError_t gemm_mfma(const Gemm& g, float* scratch, size_t scratch_elems, hipStream_t s, int kc,
                     double flops, double bytes) {
  GemmDev d;
  d.M = g.M; d.N = g.N; d.ktotal = g.K; d.nsplit = 1;
  d.A = (const bf16_t*)g.A; d.lda = g.lda;
  d.B = (const bf16_t*)g.B; d.ldb = g.ldb;
  d.C = g.C; d.ldc = g.ldc; d.alpha = g.alpha; d.beta = g.beta;
  d.mstore = g.M;
  d.lscale = nullptr; d.lmask = nullptr; d.lpart = nullptr; d.lref = nullptr; d.ldref = 0;
  d.causal = 0; d.rev = 0; d.nbatch = 1; d.zdiv = 1; d.bdiv = 1; d.kgroups = 1;
  d.sA = d.sB1 = d.sB2 = d.sC1 = d.sC2 = d.sAk = d.sBk = 0;
  d.split_n = 0; d.c_lo = nullptr; d.ldc_lo = d.sC1_lo = d.sC2_lo = 0;
  Plan p = plan_of(g, true);
  // two outputs: always through the partials (also unsplit), summed into C and C2
  const bool two = g.C2 != nullptr;
  if (two && (g.beta != 0.f || g.m2 <= 0 || g.m2 >= g.M || g.N % 4 || g.ldc % 4 ||
              (uintptr_t)g.C % 16 || (uintptr_t)g.C2 % 16 || g.c_t != DT_F32))
    return hipErrorInvalidValue;
  if ((p.splits > 1 || two) && (scratch == nullptr || scratch_elems < (size_t)p.splits * g.M * g.N)) {
    if (two) return hipErrorInvalidValue;
    p = plan_of(g, false);
  }
  d.kchunk = p.kchunk;
  d.part = p.splits > 1 || two ? scratch : nullptr;
  const bool f32 = g.c_t == DT_F32;
  const char* kname = nullptr;
  prof_begin(kc, s);
#define L_(AK, BK_)                                                                     \
  if (g.a_kmajor == AK && g.b_kmajor == BK_) {                                          \
    if (f32) kname = launch<AK, BK_, float>(d, p, s);                                   \
    else kname = launch<AK, BK_, bf16_t>(d, p, s);                                      \
  }
  L_(true, true) else L_(true, false) else L_(false, false) else L_(false, true)
#undef L_
  prof_end(kc, s, flops, bytes, kname);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || (p.splits == 1 && !two)) return e;
  // the split-K partials summed in a fixed order (an elementwise launch of its own)
  int64_t total = (int64_t)g.M * g.N;
  unsigned grid = (unsigned)((total + 255) / 256);
  const double rbytes = (double)total * (4.0 * p.splits + (f32 ? 4.0 : 2.0) * (g.beta != 0.f ? 2.0 : 1.0));
  prof_begin(KC_ELEM, s);
  if (two) {  // rows [0, m2) into C, [m2, M) into C2 (f32, 4-aligned: checked above)
    const int64_t t1 = (int64_t)g.m2 * g.N, t2 = total - t1;
    splitk_reduce4_kernel<float><<<(unsigned)((t1 / 4 + 255) / 256), 256, 0, s>>>(
        scratch, p.splits, total, g.m2, g.N, (float*)g.C, g.ldc, g.alpha, 0.f);
    splitk_reduce4_kernel<float><<<(unsigned)((t2 / 4 + 255) / 256), 256, 0, s>>>(
        scratch + t1, p.splits, total, g.M - g.m2, g.N, (float*)g.C2, g.ldc, g.alpha, 0.f);
    prof_end(KC_ELEM, s, 0.0, rbytes, KLABEL("splitk_reduce4_kernel"));
    return hipGetLastError();
  }
  if (g.N % 4 == 0 && g.ldc % 4 == 0 && (uintptr_t)g.C % (f32 ? 16 : 8) == 0) {
    const unsigned grid4 = (unsigned)((total / 4 + 255) / 256);
    if (f32)
      splitk_reduce4_kernel<float><<<grid4, 256, 0, s>>>(scratch, p.splits, total, g.M, g.N,
                                                         (float*)g.C, g.ldc, g.alpha, g.beta);
    else
      splitk_reduce4_kernel<bf16_t><<<grid4, 256, 0, s>>>(scratch, p.splits, total, g.M, g.N,
                                                          (bf16_t*)g.C, g.ldc, g.alpha, g.beta);
    prof_end(KC_ELEM, s, 0.0, rbytes, KLABEL("splitk_reduce4_kernel"));
    return hipGetLastError();
  }
  if (f32)
    splitk_reduce_kernel<float><<<grid, 256, 0, s>>>(scratch, p.splits, total, g.M, g.N,
                                                     (float*)g.C, g.ldc, g.alpha, g.beta);
  else
    splitk_reduce_kernel<bf16_t><<<grid, 256, 0, s>>>(scratch, p.splits, total, g.M, g.N,
                                                      (bf16_t*)g.C, g.ldc, g.alpha, g.beta);
  prof_end(KC_ELEM, s, 0.0, rbytes, KLABEL("splitk_reduce_kernel"));
  return hipGetLastError();
}

size_t gemm_mfma_masked_sse_parts(const Gemm& g) {
  return (size_t)((g.M + 127) / 128) * ((g.N + 127) / 128);
}

hipError_t gemm_mfma_masked_scale(const Gemm& g, const float* scale, const uint8_t* mask,
                                  double* part, hipStream_t s, const char** kernel) {
  if (g.beta != 0.f || g.alpha != 1.f || g.in_t != DT_BF16 || !scale || !g.C ||
      !g.a_kmajor || !g.b_kmajor)
    return hipErrorInvalidValue;
  GemmDev d;
  d.M = g.M; d.N = g.N; d.ktotal = g.K; d.nsplit = 1;
  d.A = (const bf16_t*)g.A; d.lda = g.lda;
  d.B = (const bf16_t*)g.B; d.ldb = g.ldb;
  d.C = g.C; d.ldc = g.ldc; d.alpha = 1.f; d.beta = 0.f;
  d.mstore = g.M;
  d.lscale = scale; d.lmask = mask; d.lpart = nullptr; d.lref = nullptr; d.ldref = 0;
  d.causal = 0; d.rev = 0; d.nbatch = 1; d.zdiv = 1; d.bdiv = 1; d.kgroups = 1;
  d.sA = d.sB1 = d.sB2 = d.sC1 = d.sC2 = d.sAk = d.sBk = 0;
  d.split_n = 0; d.c_lo = nullptr; d.ldc_lo = d.sC1_lo = d.sC2_lo = 0;
  const Plan p = plan_of(g, false);
  d.kchunk = p.kchunk;
  d.part = nullptr;
  // (the four-wavefront kernel reads the row mask with 32-byte scalar loads: 4-byte aligned)
  if (nt4_bn(d, p) && (uintptr_t)mask % 4 == 0) {
    *kernel = g.c_t == DT_F32 ? launch<true, true, float>(d, p, s) : launch<true, true, bf16_t>(d, p, s);
    return hipGetLastError();
  }
  // elsewhere the masked-loss kernel, its tile sums left unused
  int nparts = 0;
  return gemm_mfma_masked_sse(g, scale, mask, nullptr, 0, part, &nparts, s, kernel);
}

hipError_t gemm_mfma_masked_sse(const Gemm& g, const float* scale, const uint8_t* mask,
                                const void* ref, int64_t ldref, double* part, int* nparts,
                                hipStream_t s, const char** kernel) {
  if (g.beta != 0.f || g.alpha != 1.f || g.in_t != DT_BF16) return hipErrorInvalidValue;
  GemmDev d;
  d.M = g.M; d.N = g.N; d.ktotal = g.K; d.nsplit = 1;
  d.A = (const bf16_t*)g.A; d.lda = g.lda;
  d.B = (const bf16_t*)g.B; d.ldb = g.ldb;
  d.C = g.C; d.ldc = g.ldc; d.alpha = 1.f; d.beta = 0.f;
  d.mstore = g.M;
  d.lscale = scale; d.lmask = mask; d.lpart = part;
  d.lref = (const bf16_t*)ref; d.ldref = ldref;
  d.causal = 0; d.rev = 0; d.nbatch = 1; d.zdiv = 1; d.bdiv = 1; d.kgroups = 1;
  d.sA = d.sB1 = d.sB2 = d.sC1 = d.sC2 = d.sAk = d.sBk = 0;
  d.split_n = 0; d.c_lo = nullptr; d.ldc_lo = d.sC1_lo = d.sC2_lo = 0;
  const Plan p = plan_of(g, false);
  d.kchunk = p.kchunk;
  d.part = nullptr;
  *nparts = ((g.M + p.bm - 1) / p.bm) * ((g.N + p.bn - 1) / p.bn);
  const bool f32 = g.c_t == DT_F32;
  if (!g.a_kmajor || !g.b_kmajor) return hipErrorInvalidValue;
  *kernel = f32 ? launch<true, true, float>(d, p, s) : launch<true, true, bf16_t>(d, p, s);
  return hipGetLastError();
}

// Batched causal products of attention's backward: dQ = dS K (A = dS^T stored [key][query],
// M/N-contiguous, bf16 result) and dK = dS^T Q summed over a group's heads (A k-major, fp32
// result).  BN is the output width rounded up to the supported tile widths.
template <int BN, int WM, int WN, bool AK, typename TC>
static void launch_causal(const GemmDev& d, int nbatch, hipStream_t s) {
  const int ntm = (d.M + 255) / 256, ntn = (d.N + BN - 1) / BN;
  const int items = ntm * ntn * nbatch;
  if constexpr (!AK) {
    // dQ (M-contiguous A; K ranges end at the diagonal): one tile per workgroup, dispatched
    // longest range first, in 32-deep slices through a ring of four LDS stages.  The
    // product waits on its copies (the dS^T stream): three slices in flight (84 KB per CU)
    // instead of one 64-deep slice (56 KB) measured 3-6% faster (five stages, and a
    // persistent grid of the two-stage ring, were slower)
    attn_ds_gemm_kernel<256, BN, WM, WN, AK, false, TC, 32, 4>
        <<<dim3(items, 1), 64 * WM * WN, 0, s>>>(d);
  } else {
    // dK (K ranges start at the diagonal): persistent, 2.6% faster; as many workgroups as
    // fit on the CUs at once (the narrow tiles leave room for two per CU)
    // resident workgroups per CU, queried once per device
    constexpr int MAXDEV = 64;
    static std::atomic<int> occ[MAXDEV];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAXDEV) dev = 0;
    int per_cu = occ[dev].load(std::memory_order_relaxed);
    if (per_cu == 0) {
      int n = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
              &n, attn_ds_gemm_persist_kernel<256, BN, WM, WN, AK, false, TC, 64, 2>,
              64 * WM * WN, 0) != hipSuccess || n < 1)
        n = 1;
      per_cu = n;
      occ[dev].store(n, std::memory_order_relaxed);
    }
    attn_ds_gemm_persist_kernel<256, BN, WM, WN, AK, false, TC, 64, 2>
        <<<dim3(std::min(items, NUM_CU * per_cu), 1), 64 * WM * WN, 0, s>>>(d);
  }
}

template <bool AK, typename TC>
static hipError_t dispatch_causal(const GemmDev& d, int nbatch, hipStream_t s) {
  if (d.N <= 64) launch_causal<64, 4, 2, AK, TC>(d, nbatch, s);
  else if (d.N <= 96) launch_causal<96, 4, 1, AK, TC>(d, nbatch, s);
  else if (d.N <= 128) launch_causal<128, 4, 2, AK, TC>(d, nbatch, s);
  else if (d.N <= 192) launch_causal<192, 4, 2, AK, TC>(d, nbatch, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t gemm_mfma_causal(const Gemm& g, const GemmBatch& bt, hipStream_t s) {
  // (an M-contiguous A is read in 8-row chunks)
  const bool ok = !g.b_kmajor && g.in_t == DT_BF16 && g.beta == 0.f &&
                  (g.a_kmajor || g.M % 8 == 0) &&
                  g.N % 32 == 0 && g.lda % 8 == 0 && g.ldb % 8 == 0 && bt.mstore <= g.M &&
                  bt.kgroups >= 1 && (g.a_kmajor ? (bt.rev && g.c_t == DT_F32)
                                                 : (!bt.rev && g.c_t == DT_BF16)) &&
                  (bt.split_n == 0 || (g.a_kmajor && bt.split_n % 4 == 0 && bt.split_n <= g.N &&
                                       bt.c_lo && bt.ldc_lo % 4 == 0 && bt.sC1_lo % 4 == 0 &&
                                       bt.sC2_lo % 4 == 0 && (uintptr_t)bt.c_lo % 8 == 0 &&
                                       g.ldc % 4 == 0 && bt.sC1 % 4 == 0 && bt.sC2 % 4 == 0 &&
                                       (uintptr_t)g.C % 16 == 0));
  if (!ok) return hipErrorInvalidValue;
  GemmDev d;
  d.M = g.M; d.N = g.N; d.ktotal = g.K; d.nsplit = 1;
  d.A = (const bf16_t*)g.A; d.lda = g.lda;
  d.B = (const bf16_t*)g.B; d.ldb = g.ldb;
  d.C = g.C; d.ldc = g.ldc; d.alpha = g.alpha; d.beta = 0.f;
  d.part = nullptr;
  d.lscale = nullptr; d.lmask = nullptr; d.lpart = nullptr; d.lref = nullptr; d.ldref = 0;
  d.kchunk = (g.K + BK - 1) / BK * BK;
  d.mstore = bt.mstore;
  d.causal = 1; d.rev = bt.rev; d.nbatch = bt.nbatch; d.zdiv = bt.zdiv; d.bdiv = bt.bdiv;
  d.kgroups = bt.kgroups;
  d.sA = bt.sA; d.sB1 = bt.sB1; d.sB2 = bt.sB2; d.sC1 = bt.sC1; d.sC2 = bt.sC2;
  d.sAk = bt.sAk; d.sBk = bt.sBk;
  d.split_n = bt.split_n; d.c_lo = (bf16_t*)bt.c_lo;
  d.ldc_lo = bt.ldc_lo; d.sC1_lo = bt.sC1_lo; d.sC2_lo = bt.sC2_lo;
  return g.a_kmajor ? dispatch_causal<true, float>(d, bt.nbatch, s)
                    : dispatch_causal<false, bf16_t>(d, bt.nbatch, s);
}

}  // namespace mla
