// Shared device/host helpers of the gfx950 reconstruction library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mla {

typedef uint16_t bf16_t;  // raw bf16 bit pattern (storage)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// ---- scalar conversions ---------------------------------------------------------------
__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// float -> bf16, round to nearest even (NaN stays NaN)
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// two floats -> packed bf16 pair (lo in bits 0..15), round to nearest even
// (gfx950's v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  f32x2 v = {lo, hi};
  bf16x2_t b = __builtin_convertvector(v, bf16x2_t);
  return __builtin_bit_cast(uint32_t, b);
}

// max / sum of x over the lane pair (l, l ^ 32), from gfx950's v_permlane32_swap (swaps
// the upper half of one register with the lower half of another: with x in both, each lane
// then holds its own value and its partner's) - no LDS round trip
__device__ __forceinline__ float pair_max32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <typename T> __device__ __forceinline__ float ld(const T* p);
template <> __device__ __forceinline__ float ld<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t* p) { return bf2f(*p); }

template <typename T> __device__ __forceinline__ void st(T* p, float v);
template <> __device__ __forceinline__ void st<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void st<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ double warp_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Remap a linear workgroup id so that consecutive logical tiles land on the same XCD.
// Index of the calling wavefront in its workgroup, in an SGPR: the compiler does not treat
// threadIdx.x / 64 as uniform by itself, and branches on it would be lowered as divergent
// (exec-mask) code.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

// Workgroups are dispatched round-robin over the 8 XCDs (id % 8); the remap gives XCD x
// the contiguous logical range [x*per, (x+1)*per), keeping neighbouring tiles (which
// share A rows or B columns) in one XCD's L2.
__device__ __forceinline__ int xcd_remap(int pid, int nwg) {
  const int nx = 8;
  int per = nwg / nx;
  int full = per * nx;
  if (pid >= full) return pid;  // the tail keeps its id
  return (pid % nx) * per + pid / nx;
}

}  // namespace mla

namespace mla {

// gfx950 LDS transpose read (ds_read_b64_tr_b16).  Inside each group of 16 lanes, lane r
// supplies the address of 4 consecutive 16-bit elements; lane j of the group receives
// element (j % 4) of the rows supplied by lanes j/4, j/4 + 4, j/4 + 8, j/4 + 12.  With
// lane r pointing at row k0 + r/4, columns n0 + 4(r%4) of a [k][n] (n-contiguous) LDS
// matrix, lane j receives column n0 + j, rows k0 .. k0+3: a transposed 4 x 16 block.
__device__ __forceinline__ u32x2 lds_read_tr4(const bf16_t* p) {
  typedef short i16x4 __attribute__((ext_vector_type(4)));
  i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}

// MFMA 32x32x16 operand (lane: row/column m0 + lane%32, 8 k-values) read from an LDS
// matrix stored [k][m] with row stride ld.  The lane's k-slots 0..3 are rows klo..klo+3,
// slots 4..7 rows khi..khi+3, where klo / khi may differ between the two lane halves.
__device__ __forceinline__ bf16x8 lds_operand_tr(const bf16_t* base, int ld, int m0, int klo,
                                                 int khi) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const int n0 = m0 + 16 * (g & 1) + 4 * (r & 3);
  u32x2 lo = lds_read_tr4(base + (klo + (r >> 2)) * ld + n0);
  u32x2 hi = lds_read_tr4(base + (khi + (r >> 2)) * ld + n0);
  u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
  return __builtin_bit_cast(bf16x8, w);
}

// Direct global -> LDS copy (gfx950 global_load_lds_dwordx4) of a [ROWS][D] bf16 tile into
// a padded LDS tile with row stride LD.  The tile's LDS bytes are cut into 1 KB blocks; a
// wavefront fills one block per instruction (lane l writes 16 bytes at block + 16 l) and
// chooses each lane's global source so that the block matches the padded layout.  Lanes
// that land on row padding, or past the last row inside the final block, load a valid
// chunk of the tile that is never read.  Nothing passes through registers; completion is
// awaited with a counter wait before the workgroup barrier that publishes the tile.
//
// The copy is issued from inline assembly: with a global_load_lds in flight the compiler's
// counter bookkeeping cannot tell which LDS results are ready and waits for all of them
// (lgkmcnt(0)) before each use, which serialises the operand reads of the next MFMA step
// with the current one.  Out of its sight, the copies are awaited explicitly (wait_all,
// itself inline assembly so that it is never relaxed) before the barrier that publishes
// the tile.  m0 holds the wavefront's LDS destination; lane l writes 16 bytes at m0 + 16 l.
// (The low 32 bits of a generic pointer into LDS are the LDS byte address.)
__device__ __forceinline__ void dma16(const bf16_t* gsrc, bf16_t* lds_dst) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_dst);
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(gsrc), "{m0}"(l) : "memory");
}

// With EXACT, every wavefront issues the same number (PER) of copies: the block count is
// padded to a multiple of the wavefront count (the extra blocks land in reserved LDS), so
// that a counter wait can name how many copies of later tiles may still be in flight.
// Same copy with the global address split into a wave-uniform base (SGPRs) and a per-lane
// 32-bit byte offset: the per-lane part is usually loop-invariant, so a copy costs no
// 64-bit address arithmetic.  sbase must be the same in every lane.
// NT: the non-temporal cache policy, for data streamed once (it then displaces less of what
// the caches hold for other operands).
template <bool NT = false>
__device__ __forceinline__ void dma16_s(const void* sbase, uint32_t voff_bytes, bf16_t* lds_dst) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds_dst);
  // the base is uniform by contract; reading it from the first lane puts it in SGPRs (the
  // builtin returns a signed int: each half is zero-extended explicitly)
  const uint64_t a = (uint64_t)(uintptr_t)sbase;
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  const uint64_t su = ((uint64_t)hi << 32) | (uint64_t)lo;
  // s_nop 4: five wait states between a VALU write of the base SGPRs (the readfirstlane
  // above) and their read by the memory instruction, which the compiler cannot see inside
  // the asm; this also covers the m0 write before the LDS copy
  if constexpr (NT)
    asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1 nt" : : "v"(voff_bytes), "s"(su), "{m0}"(l)
                 : "memory");
  else
    asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(voff_bytes), "s"(su), "{m0}"(l)
                 : "memory");
}

// A pointer that is the same in every lane, as a 64-bit value in scalar registers (for an
// "s" operand of inline assembly)
__device__ __forceinline__ uint64_t uniform_ptr(const void* p) {
  const uint64_t a = (uint64_t)(uintptr_t)p;
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  return ((uint64_t)hi << 32) | (uint64_t)lo;
}

template <int ROWS, int D, int LD, int NW, bool EXACT = false>
struct DmaTile {
  static constexpr int BYTES = ROWS * LD * 2;
  static constexpr int NBLK0 = (BYTES + 1023) / 1024;
  static constexpr int PER = (NBLK0 + NW - 1) / NW;
  static constexpr int NBLK = EXACT ? PER * NW : NBLK0;
  static constexpr int ALLOC = NBLK * 512;  // bf16 elements reserved in LDS
  short row[PER], col[PER];

  __device__ __forceinline__ void init() {
    const int lane = threadIdx.x & 63, wave = wave_id();
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int b = wave + p * NW;
      const int e = (b * 1024 + 16 * lane) / 2;
      int r = e / LD, c = e % LD;
      if (c >= D) c = 0;
      if (r >= ROWS) r = ROWS - 1;
      row[p] = (short)r;
      col[p] = (short)c;
    }
  }
  // src(row, col) -> global address of the 16-byte chunk at (row, col) of this tile
  template <class F>
  __device__ __forceinline__ void issue(bf16_t* lds, F src) const {
    const int wave = wave_id();
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int b = wave + p * NW;
      if (NBLK % NW == 0 || b < NBLK)
        dma16(src(row[p], col[p]), lds + b * 512);
    }
  }
  // off(row, col) -> element offset of the chunk from sbase (uniform), below 2^31 bytes
  template <bool NT = false, class F>
  __device__ __forceinline__ void issue_s(bf16_t* lds, const bf16_t* sbase, F off) const {
    const int wave = wave_id();
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int b = wave + p * NW;
      if (NBLK % NW == 0 || b < NBLK)
        dma16_s<NT>(sbase, 2u * (uint32_t)off(row[p], col[p]), lds + b * 512);
    }
  }
};

// 8-byte store through an explicitly global pointer (no generic-address handling)
__device__ __forceinline__ void st_global8(bf16_t* p, u32x2 v) {
  *(__attribute__((address_space(1))) u32x2*)p = v;
}

// 16-byte store through an explicitly global pointer
__device__ __forceinline__ void st_global16(bf16_t* p, u32x4 v) {
  *(__attribute__((address_space(1))) u32x4*)p = v;
}

// the same with the non-temporal cache policy (data read back once, by a later launch)
__device__ __forceinline__ void st_global16_nt(bf16_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, (__attribute__((address_space(1))) u32x4*)p);
}

// at most N vector-memory operations of this wavefront (e.g. LDS DMA copies of later
// tiles) still in flight
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}
// LDS operations of this wavefront complete, then a workgroup barrier (no memory fence:
// global copies are awaited with wait_vm)
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory");
}

// all outstanding memory operations of this wavefront (incl. LDS DMA) complete
__device__ __forceinline__ void wait_all() {
  asm volatile("s_waitcnt vmcnt(0) expcnt(0) lgkmcnt(0)" : : : "memory");
}

}  // namespace mla
