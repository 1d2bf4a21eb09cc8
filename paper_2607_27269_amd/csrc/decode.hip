// Decoding with the reconstructed MLA block in absorbed form (one query token per sequence).
//
// The cache keeps, per token, the latent c^KV_j and the rotated positional key k^PE_j
// (Eq. 5; the [c^KV | k^PE] rows the student forward produces).  With a single positional
// key (G_r = 1) every head attends against the same cache row [c_j ; k^PE_j]: head i uses
// the absorbed query [W_UK[g]^T q^nope_i ; q^rope_i] and its output is W_UV[g] applied to
// the attention-weighted latent (g = i / (H / G_kv)).  So decoding is multi-query attention
// with key width r_kv + d_rope, value width r_kv (the latent itself) and all H heads in one
// MFMA column block, followed by a per-group projection.
//
// Kernels:
// * group_gemm_kernel (+ absorb_rest_kernel): the absorbed queries [B][HP][DK] bf16 (heads
//   padded to HP = 32k), the latent part as one product per KV group.
// * decode_attn_kernel: split-K over the cache (flash-decoding).  A workgroup (4 waves)
//   owns one (sequence, key chunk, block of 32 heads).  Key tiles of 32 rows are copied
//   straight into LDS in a ring of three stages (two tiles in flight).  The
//   tile's S^T = K Q^T (key in the MFMA row, head in the column, so each lane owns one
//   head's online-softmax state) is split over the 4 waves along the key width: each wave
//   multiplies a quarter of the 16-wide K steps (its absorbed-query fragments held in
//   registers) and the partial products are summed through
//   LDS in wave order, so every wave holds the same S^T (the same values in every wave).
//   Each wave then updates O^T += V^T P^T for its quarter of the latent width; V^T is the
//   tile's latent columns read with the transposing LDS read.  Partial (max, sum,
//   unnormalised output) per split.
// * decode_combine_kernel: merges the splits of a (sequence, head) in split order.
// * uv_proj_kernel: o = W_UV[g] (latent), one thread per output.
#include <mutex>

#include "attn_common.h"
#include "kernels.h"
#include "mfma.h"
#include "mla_recon.h"

namespace mla {

// Scratch of the allocation-free decoding entry point (mla_recon_decode_noalloc): a
// file-scope device array, one copy per GPU, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in symbol): it uses
// the per-device address hipGetSymbolAddress returns, obtained once per device with that
// device current.
constexpr size_t DECODE_SCRATCH_BYTES = MLA_DECODE_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[DECODE_SCRATCH_BYTES];

constexpr int SCRATCH_MAX_DEVICES = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[SCRATCH_MAX_DEVICES];

size_t decode_scratch_bytes() { return DECODE_SCRATCH_BYTES; }

hipError_t decode_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

namespace {

constexpr int DEC_KT = 32;     // keys per tile
constexpr int DEC_WAVES = 4;
constexpr float DEC_SLACK = 8.f;  // log2 units the running reference max may lag

struct DecodeDev {
  const bf16_t* qabs;   // [B][HP][DK]
  const bf16_t* cache;  // [B][Lmax][ldc]
  int64_t seq_stride;   // Lmax * ldc
  int ldc;              // row stride of the cache (elements)
  const int32_t* len;   // [B]
  int tps;              // prefill: query row b is token b % tps of sequence b / tps and
                        // attends to that sequence's first b % tps + 1 rows (0: decoding)
  int Lmax, HP, nsplit, chunk;
  float sl2;            // softmax scale * log2(e)
  float* part_o;        // [B][nsplit][HP][DVL]
  float* part_ml;       // [B][nsplit][HP][2]
};

// The query absorption as one product per KV group, C[r][n] = sum_k A[r][k] W_g[k][n] for
// the H / G_kv heads of group g = blockIdx.z and sequences b: row r = (b, j) is head
// i = g hpg + j of sequence b (A row at A + (b H + i) lda, C row at C + (b HC + i) ldc),
// W_g = W + g K N (W_UK[g] = Wuk[g K + k][n]).  32 x 32 output tiles (enough workgroups for these small products), K
// in chunks of 32 staged in LDS as fp32; each of the 256 threads owns 2 x 2 outputs.  fp32
// accumulation in k order, bf16 output.
template <typename TA>
__global__ __launch_bounds__(256) void group_gemm_kernel(const TA* __restrict__ A, int64_t lda,
                                                         const bf16_t* __restrict__ W,
                                                         bf16_t* __restrict__ C, int64_t ldc,
                                                         int HC, int B, int H, int hpg, int K,
                                                         int N) {
  constexpr int TR = 32, TN = 32, TK = 32;
  __shared__ float As[TK][TR + 1];
  __shared__ float Ws[TK][TN + 1];
  const int g = blockIdx.z, n0 = blockIdx.x * TN, r0 = blockIdx.y * TR;
  const int rows = B * hpg;
  const int tid = threadIdx.x, tr = tid / 16, tn = tid % 16;
  const bf16_t* Wg = W + (int64_t)g * K * N;
  float acc[2][2] = {};
  for (int k0 = 0; k0 < K; k0 += TK) {
    // A tile: 32 rows x 32 k, transposed into As[k][r]
    for (int e = tid; e < TR * TK; e += 256) {
      const int r = e / TK, k = e % TK, rr = r0 + r, kk = k0 + k;
      float v = 0.f;
      if (rr < rows && kk < K) {
        const int b = rr / hpg, i = g * hpg + rr % hpg;
        v = ld(A + ((int64_t)b * H + i) * lda + kk);
      }
      As[k][r] = v;
    }
    // W tile: 32 k x 32 n
    for (int e = tid; e < TK * TN; e += 256) {
      const int k = e / TN, n = e % TN, kk = k0 + k, nn = n0 + n;
      Ws[k][n] = kk < K && nn < N ? bf2f(Wg[(int64_t)kk * N + nn]) : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < TK; ++k) {
      const float a0 = As[k][tr], a1 = As[k][tr + 16], w0 = Ws[k][tn], w1 = Ws[k][tn + 16];
      acc[0][0] += a0 * w0;
      acc[0][1] += a0 * w1;
      acc[1][0] += a1 * w0;
      acc[1][1] += a1 * w1;
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int rr = r0 + tr + 16 * u;
    if (rr >= rows) continue;
    const int b = rr / hpg, i = g * hpg + rr % hpg;
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int nn = n0 + tn + 16 * v;
      if (nn < N) C[((int64_t)b * HC + i) * ldc + nn] = f2bf(acc[u][v]);
    }
  }
}

// The rest of the absorbed queries [B][HP][DK]: the rotary part copied from q, and zero
// rows for the padding heads i >= H (the latent part of heads < H comes from the group
// product).
__global__ void absorb_rest_kernel(const bf16_t* __restrict__ q, bf16_t* __restrict__ qabs, int B,
                                   int H, int HP, int dn, int dr, int rkv) {
  const int DK = rkv + dr;
  const int64_t n_rope = (int64_t)B * H * dr;
  const int64_t n_pad = (int64_t)B * (HP - H) * DK;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < n_rope) {
    const int c = (int)(idx % dr);
    const int64_t bi = idx / dr;  // b * H + i
    const int b = (int)(bi / H), i = (int)(bi % H);
    qabs[((int64_t)b * HP + i) * DK + rkv + c] = q[bi * (dn + dr) + dn + c];
  } else if (idx < n_rope + n_pad) {
    const int64_t e = idx - n_rope;
    const int c = (int)(e % DK);
    const int64_t bp = e / DK;
    const int b = (int)(bp / (HP - H)), i = H + (int)(bp % (HP - H));
    qabs[((int64_t)b * HP + i) * DK + c] = (bf16_t)0;
  }
}

template <int DK, int DVL>
__global__ __launch_bounds__(64 * DEC_WAVES) void decode_attn_kernel(DecodeDev a) {
  constexpr int LDK = attn::ld_of(DK);        // padded rows: conflict-free operand reads
  constexpr int NKK = DK / 16;
  constexpr int QMAX = (NKK + DEC_WAVES - 1) / DEC_WAVES;  // K steps per wave, at most
  constexpr int WV = DVL / DEC_WAVES;         // latent rows per wave
  constexpr int NCV = WV / 32;
  constexpr int NST = 3;                      // key-tile ring: two tiles in flight
  static_assert(DK % 16 == 0 && WV % 32 == 0, "decode shape");
  using KT = DmaTile<DEC_KT, DK, LDK, DEC_WAVES, true>;
  constexpr int D = KT::PER;                  // copies per wave per tile
  __shared__ __attribute__((aligned(1024))) bf16_t Ks[NST][KT::ALLOC];
  // partial S^T of each wave: [wave][e / 4][lane][4] (16-byte accesses, conflict-free)
  __shared__ __attribute__((aligned(16))) float Sp[DEC_WAVES][4][64][4];

  const int split = blockIdx.x, b = blockIdx.y, h0 = 32 * blockIdx.z;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5, col = lane & 31;
  const int len = a.tps ? b % a.tps + 1 : min(max(a.len[b], 0), a.Lmax);
  const int kbeg = split * a.chunk;
  const int kend = min(len, kbeg + a.chunk);
  const int64_t pbase = ((int64_t)b * a.nsplit + split) * a.HP + h0;
  // this wave's share of the K steps
  const int kk0 = wave * NKK / DEC_WAVES, kk1 = (wave + 1) * NKK / DEC_WAVES;

  const bf16_t* cs = a.cache + (int64_t)(a.tps ? b / a.tps : b) * a.seq_stride;
  KT kt_copy;
  kt_copy.init();
  // key tile t into stage t % NST; rows past the chunk end repeat its last row (finite,
  // and given no weight below)
  auto issue = [&](int t) {
    const int k0 = kbeg + t * DEC_KT;
    if (k0 + DEC_KT <= kend) {  // full tile: uniform row base plus 32-bit lane offsets
      kt_copy.issue_s(Ks[t % NST], cs + (int64_t)k0 * a.ldc,
                      [&](int r, int c) { return r * a.ldc + c; });
    } else {
      kt_copy.issue(Ks[t % NST], [&](int r, int c) {
        return cs + (int64_t)min(k0 + r, kend - 1) * a.ldc + c;
      });
    }
  };
  const int ntile = kend > kbeg ? (kend - kbeg + DEC_KT - 1) / DEC_KT : 0;
  if (ntile > 0) issue(0);
  if (ntile > 1) issue(1);
  // this lane's head as B-operand fragments for the wave's K steps (head h0 + col,
  // k = 16 kk + 8 half + 0..7)
  bf16x8 qf[QMAX];
  {
    const bf16_t* qsrc = a.qabs + ((int64_t)b * a.HP + h0 + col) * DK + 8 * half;
#pragma unroll
    for (int j = 0; j < QMAX; ++j)
      qf[j] = kk0 + j < kk1 ? *(const bf16x8*)(qsrc + 16 * (kk0 + j)) : bf16x8{};
  }
  wait_vm<0>();
#pragma unroll
  for (int j = 0; j < QMAX; ++j) asm volatile("" : "+v"(qf[j]));
  __syncthreads();

  f32x16 acc[NCV];
#pragma unroll
  for (int c = 0; c < NCV; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  for (int t = 0; t < ntile; ++t) {
    const bf16_t* kt = Ks[t % NST];
    const int k0 = kbeg + t * DEC_KT;
    // the stage of tile t - 1 is free: every wave passed the barrier that ended it
    if (t + 2 < ntile) issue(t + 2);
    // S^T (32 keys x 32 heads): key = MFMA row, head = column (this lane's head: col);
    // this wave's K steps, then the four partial products summed in wave order
    f32x16 s;
#pragma unroll
    for (int e = 0; e < 16; ++e) s[e] = 0.f;
#pragma unroll
    for (int j = 0; j < QMAX; ++j)
      if (kk0 + j < kk1)
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            *(const bf16x8*)(kt + col * LDK + 16 * (kk0 + j) + 8 * half), qf[j], s, 0, 0, 0);
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4)
      *(f32x4*)Sp[wave][e4][lane] = f32x4{s[4 * e4], s[4 * e4 + 1], s[4 * e4 + 2], s[4 * e4 + 3]};
    lds_barrier();
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      f32x4 u = *(const f32x4*)Sp[0][e4][lane];
#pragma unroll
      for (int w2 = 1; w2 < DEC_WAVES; ++w2) u += *(const f32x4*)Sp[w2][e4][lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) s[4 * e4 + r] = u[r];
    }
    // keys past the chunk end (last tile only; a real branch): no weight
    if (k0 + DEC_KT > kend) {
      asm volatile("");
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (k0 + 8 * (e >> 2) + 4 * half + (e & 3) >= kend) s[e] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[e]);
    mx = pair_max32(mx) * a.sl2;
    // lazy rescale: the reference max moves only when a block max exceeds it by more than
    // DEC_SLACK (so P <= 2^DEC_SLACK); wave-uniform, and the same in every wave (same S^T)
    if (__ballot(mx > m_run + DEC_SLACK) != 0) {
      const float m_new = fmaxf(m_run, mx);
      const float corr = __builtin_amdgcn_exp2f(m_run - (m_new == -INFINITY ? 0.f : m_new));
      m_run = m_new;
      l_run *= corr;
#pragma unroll
      for (int c = 0; c < NCV; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[c][e] *= corr;
    }
    const float m_use = m_run == -INFINITY ? 0.f : m_run;
    // P^T as the B operand of O^T = V^T P^T (K-step u: keys 16u + {4h'..4h'+3, 8+4h'..})
    bf16x8 pf[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 w;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[8 * u + 2 * q], a.sl2, -m_use));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[8 * u + 2 * q + 1], a.sl2, -m_use));
        l_run += p0 + p1;
        w[q] = pack2bf(p0, p1);
      }
      pf[u] = __builtin_bit_cast(bf16x8, w);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int klo = 16 * u + 4 * half;
#pragma unroll
      for (int c = 0; c < NCV; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            lds_operand_tr(kt, LDK, wave * WV + 32 * c, klo, klo + 8), pf[u], acc[c], 0, 0, 0);
    }
    // tile t + 1 has landed (tile t + 2's copies may still fly) and every wave is done with
    // tile t and the partial sums
    if (t + 2 < ntile) wait_vm<D>();
    else wait_vm<0>();
    lds_barrier();
  }

  // partial state of this split: lane (head col, half) holds rows
  // wave WV + 32 c + 8 (e / 4) + 4 half + e % 4 of the unnormalised latent output
  const float l = pair_sum32(l_run);
  const int64_t hrow = pbase + col;
  if (wave == 0 && half == 0) {
    a.part_ml[2 * hrow] = m_run;
    a.part_ml[2 * hrow + 1] = l;
  }
  float* po = a.part_o + hrow * DVL + wave * WV + 4 * half;
#pragma unroll
  for (int c = 0; c < NCV; ++c)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *(f32x4*)(po + 32 * c + 8 * g) =
          f32x4{acc[c][4 * g], acc[c][4 * g + 1], acc[c][4 * g + 2], acc[c][4 * g + 3]};
}

// lat[b][i][d] = sum_s o_s[d] 2^(m_s - M) / sum_s l_s 2^(m_s - M), splits in order (bf16:
// the operand of the W_UV product)
__global__ void decode_combine_kernel(const float* __restrict__ part_o,
                                      const float* __restrict__ part_ml, bf16_t* __restrict__ lat,
                                      int H, int HP, int nsplit, int DVL) {
  const int b = blockIdx.y, i = blockIdx.x;
  float M = -INFINITY;
  for (int sp = 0; sp < nsplit; ++sp) M = fmaxf(M, part_ml[2 * (((int64_t)b * nsplit + sp) * HP + i)]);
  float L = 0.f;
  for (int sp = 0; sp < nsplit; ++sp) {
    const int64_t r = ((int64_t)b * nsplit + sp) * HP + i;
    const float m = part_ml[2 * r];
    if (m != -INFINITY) L += part_ml[2 * r + 1] * __builtin_amdgcn_exp2f(m - M);
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  for (int d = threadIdx.x; d < DVL; d += blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < nsplit; ++sp) {
      const int64_t r = ((int64_t)b * nsplit + sp) * HP + i;
      const float m = part_ml[2 * r];
      if (m != -INFINITY) v += part_o[r * DVL + d] * __builtin_amdgcn_exp2f(m - M);
    }
    lat[((int64_t)b * H + i) * DVL + d] = f2bf(v * inv);
  }
}

// o[r][i][e] = sum_c W_UV[g dv + e][c] lat[r][i][c] (g = i / hpg) on the matrix cores: a
// workgroup owns 32 rows of one head, each of its DV / 32 wavefronts 32 of the head's dv
// outputs; both operands are K-contiguous rows read straight from memory (16 bytes per
// lane per K step; the workgroup's wavefronts share the latent rows through L1), fp32
// accumulation over the r_kv latent dims.  bf16 output.
template <int DV>
__global__ __launch_bounds__(64 * (DV / 32)) void uv_mfma_kernel(const bf16_t* __restrict__ lat,
                                                                  const bf16_t* __restrict__ Wuv,
                                                                  bf16_t* __restrict__ o, int rows,
                                                                  int H, int rkv, int hpg) {
  const int i = blockIdx.y, r0 = 32 * blockIdx.x;
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5, col = lane & 31;
  const int r = min(r0 + col, rows - 1);
  const bf16_t* ap = lat + ((int64_t)r * H + i) * rkv + 8 * half;
  const bf16_t* bp = Wuv + ((int64_t)(i / hpg) * DV + 32 * wave + col) * rkv + 8 * half;
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
  for (int k = 0; k < rkv; k += 16)
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(ap + k), *(const bf16x8*)(bp + k),
                                                  acc, 0, 0, 0);
  // acc: row r0 + 8 (e / 4) + 4 half + e % 4, output column 32 wave + col
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int rr = r0 + 8 * (e >> 2) + 4 * half + (e & 3);
    if (rr < rows) o[((int64_t)rr * H + i) * DV + 32 * wave + col] = f2bf(acc[e]);
  }
}

#define MLA_DECODE_SHAPES(X) X(576, 512) X(288, 256) X(160, 128)

int decode_chunk(int Lmax, int B) {
  // at least 4 tiles per workgroup, and no more workgroups than one round on the CUs (one
  // workgroup per CU): long streams per workgroup keep its copy ring full
  int chunk = DEC_KT * 4;
  while ((int64_t)B * ((Lmax + chunk - 1) / chunk) > 256 && chunk < (1 << 20)) chunk *= 2;
  return chunk;
}

}  // namespace

bool decode_supported(int DK, int DVL) {
#define X(a_, b_) if (DK == a_ && DVL == b_) return true;
  MLA_DECODE_SHAPES(X)
#undef X
  return false;
}

size_t decode_ws_bytes(int B, int H, int DK, int DVL, int Lmax) {
  const int HP = (H + 31) / 32 * 32;
  const int nsplit = (Lmax + decode_chunk(Lmax, B) - 1) / decode_chunk(Lmax, B);
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  return al((size_t)B * HP * DK * 2) + al((size_t)B * nsplit * HP * DVL * 4) +
         al((size_t)B * nsplit * HP * 2 * 4) + al((size_t)B * H * DVL * 2);
}

hipError_t decode_attention(const Decode& d, hipStream_t s) {
  const int DK = d.rkv + d.dr, DVL = d.rkv;
  if (!decode_supported(DK, DVL)) return hipErrorInvalidValue;
  const int HP = (d.H + 31) / 32 * 32;
  const int chunk = decode_chunk(d.Lmax, d.B);
  const int nsplit = (d.Lmax + chunk - 1) / chunk;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  char* w = (char*)d.ws;
  bf16_t* qabs = (bf16_t*)w;
  w += al((size_t)d.B * HP * DK * 2);
  float* part_o = (float*)w;
  w += al((size_t)d.B * nsplit * HP * DVL * 4);
  float* part_ml = (float*)w;
  w += al((size_t)d.B * nsplit * HP * 2 * 4);
  bf16_t* lat = d.lat_out ? (bf16_t*)d.lat_out : (bf16_t*)w;

  prof_begin(KC_ELEM, s);
  const int64_t nq = (int64_t)d.B * HP * DK;
  const int G = d.H / d.hpg;
  const int grow = (d.B * d.hpg + 31) / 32;
  // latent part: q_abs[b][i][:rkv] = q^nope[b][i] W_UK[g]
  if (d.tps == 0 || d.dn % 8 || d.rkv % 32) {
    group_gemm_kernel<bf16_t><<<dim3((d.rkv + 31) / 32, grow, G), 256, 0, s>>>(
        (const bf16_t*)d.q, d.dn + d.dr, (const bf16_t*)d.Wuk, qabs, DK, HP, d.B, d.H, d.hpg, d.dn,
        d.rkv);
  } else {
    // many query rows (prefill): one matrix-core product per head, [rows, d_nope] x
    // W_UK[g] ([d_nope, r_kv], N-contiguous)
    for (int i = 0; i < d.H; ++i) {
      Gemm g;
      g.M = d.B; g.N = d.rkv; g.K = d.dn;
      g.A = (const bf16_t*)d.q + (int64_t)i * (d.dn + d.dr); g.lda = (int64_t)d.H * (d.dn + d.dr);
      g.a_kmajor = true;
      g.B = (const bf16_t*)d.Wuk + (int64_t)(i / d.hpg) * d.dn * d.rkv; g.ldb = d.rkv; g.b_kmajor = false;
      g.C = qabs + (int64_t)i * DK; g.ldc = (int64_t)HP * DK;
      g.in_t = DT_BF16; g.c_t = DT_BF16; g.alpha = 1.f; g.beta = 0.f;
      hipError_t e = gemm(g, nullptr, 0, s);
      if (e != hipSuccess) return e;
    }
  }
  {
    const int64_t nrest = (int64_t)d.B * d.H * d.dr + (int64_t)d.B * (HP - d.H) * DK;
    absorb_rest_kernel<<<(unsigned)((nrest + 255) / 256), 256, 0, s>>>(
        (const bf16_t*)d.q, qabs, d.B, d.H, HP, d.dn, d.dr, d.rkv);
  }
  prof_end(KC_ELEM, s, 2.0 * d.B * d.H * d.dn * d.rkv, (double)nq * 2, KLABEL("group_gemm_kernel + absorb_rest_kernel"));

  DecodeDev a;
  a.qabs = qabs; a.cache = (const bf16_t*)d.cache; a.ldc = d.ldc;
  a.seq_stride = (int64_t)d.Lmax * d.ldc; a.len = d.len; a.tps = d.tps; a.Lmax = d.Lmax; a.HP = HP;
  a.nsplit = nsplit; a.chunk = chunk; a.sl2 = d.scale * attn::LOG2E;
  a.part_o = part_o; a.part_ml = part_ml;
  const dim3 grid(nsplit, d.B, HP / 32);
  // algorithmic work at full cache lengths: the cache rows once, 2 (DK + DVL) flops per
  // (head, key)
  prof_begin(KC_ATTN_FWD, s);
#define X(a_, b_) \
  if (DK == a_ && DVL == b_) decode_attn_kernel<a_, b_><<<grid, 64 * DEC_WAVES, 0, s>>>(a);
  MLA_DECODE_SHAPES(X)
#undef X
  prof_end(KC_ATTN_FWD, s, 2.0 * d.B * d.H * (double)d.Lmax * (DK + DVL),
           (double)d.B * d.Lmax * DK * 2, KLABEL("decode_attn_kernel"));
  prof_begin(KC_ELEM, s);
  decode_combine_kernel<<<dim3(d.H, d.B), 256, 0, s>>>(part_o, part_ml, lat, d.H, HP, nsplit, DVL);
  prof_end(KC_ELEM, s, 0.0, (double)d.B * nsplit * HP * (DVL + 2) * 4 + (double)d.B * d.H * DVL * 2,
           KLABEL("decode_combine_kernel"));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || d.o == nullptr) return e;
  // o = W_UV[g] lat per head (matrix cores)
  prof_begin(KC_ELEM, s);
  if (d.dv == 128)
    uv_mfma_kernel<128><<<dim3((d.B + 31) / 32, d.H), 256, 0, s>>>(lat, (const bf16_t*)d.Wuv,
                                                                   (bf16_t*)d.o, d.B, d.H, d.rkv, d.hpg);
  else if (d.dv == 64)
    uv_mfma_kernel<64><<<dim3((d.B + 31) / 32, d.H), 128, 0, s>>>(lat, (const bf16_t*)d.Wuv,
                                                                  (bf16_t*)d.o, d.B, d.H, d.rkv, d.hpg);
  else
    return hipErrorInvalidValue;
  prof_end(KC_ELEM, s, 2.0 * d.B * d.H * d.dv * d.rkv,
           (double)d.B * d.H * (d.dv + DVL) * 2 + (double)d.H / d.hpg * d.dv * d.rkv * 2,
           KLABEL("uv_mfma_kernel"));
  return hipGetLastError();
}

}  // namespace mla
