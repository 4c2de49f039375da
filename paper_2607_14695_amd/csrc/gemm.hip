// MFMA GEMMs for the dense projections of the action expert: packed QKV with
// the RoPE epilogue, output projection, packed gate|up with the gated-GELU
// epilogue, down projection, the conditioning MLPs and the frame K/V
// projection (Section 3.4 "Operator Fusion": packed W_QKV and packed gate/up).
//
// C[M][N] = A[M][K] * B[N][K]^T, both operands K-contiguous, fp32 accumulate.
//
// Paired strips.  Two epilogues combine two output columns that are far apart
// in N: the gated GELU needs gate column c and up column N + c, rotate-half
// RoPE needs columns d and d + head_dim/2 of the same head.  A workgroup
// therefore owns a strip of "first" columns together with the strip they pair
// with, so both values of every pair end up in the same lane of the same wave
// and the epilogue works in registers.  For QKV this lets the projection write
// RoPE-rotated bf16 q rows, dynamic keys and transposed dynamic values straight
// into the layouts the attention kernel reads.
//
// Two regimes:
//  * gemm_skinny (M <= 64): weight streaming.  At one environment the
//    activations are 51 rows while every weight byte is read once per Euler
//    step, so the kernel is bound by HBM bandwidth on the weights.  A workgroup
//    owns a 32-column strip (or a 16 + 16 paired strip) and a K range; its four
//    waves interleave k-steps so that, per weight row, the wave group reads 256
//    contiguous bytes per round; fragments go straight from global memory into
//    MFMA operands (every weight byte is used by all rows in one instruction).
//    The waves' partial tiles are summed through LDS.  K may be split across
//    workgroups for the plain fp32 epilogue; the consumer (the residual/norm
//    kernel) sums the split partials, so no atomics and no extra launch.
//  * gemm_tiled (M > 64): 128x128 workgroup tiles, 2x2 waves of 64x64, two
//    k-steps (128 bytes of K per row) per LDS stage, double-buffered LDS with
//    the next stage's global loads in flight during the MFMAs.
#include "common.h"
#include "kernels.h"

namespace reflex {

enum Pair : int { PAIR_NONE = 0, PAIR_N = 1, PAIR_HEAD = 2 };

template <int EPI>
struct EpiPair {
  static constexpr int value =
      EPI == EPI_GELU ? PAIR_N : ((EPI == EPI_ROPE || EPI == EPI_KV) ? PAIR_HEAD : PAIR_NONE);
};

// Store one output (plain epilogues) or one column pair (paired epilogues).
// For paired epilogues `col` is the first column, v its value, u the value of
// the paired column.
template <int EPI, typename T>
RFX_DEV void epilogue_store(const GemmArgs& p, int z, int split, int row, int col, float v, float u) {
  if constexpr (EPI == EPI_F32 || EPI == EPI_MOD) {
    if (EPI == EPI_MOD && p.mod_width > 0 && col >= p.mod_width) v = (col < 2 * p.mod_width) ? 0.f : 1.f;
    float* o = reinterpret_cast<float*>(p.out) + (int64_t)z * p.o_bstride +
               (int64_t)split * p.o_split_stride + (int64_t)row * p.ldo + col;
    *o = v;
  } else if constexpr (EPI == EPI_SILU) {
    T* o = reinterpret_cast<T*>(p.out) + (int64_t)z * p.o_bstride + (int64_t)row * p.ldo + col;
    *o = from_f<T>(silu(v));
  } else if constexpr (EPI == EPI_GELU) {
    T* o = reinterpret_cast<T*>(p.out) + (int64_t)z * p.o_bstride + (int64_t)row * p.ldo + col;
    *o = from_f<T>(gelu_tanh(v) * u);
  } else if constexpr (EPI == EPI_KV) {
    const KvOut& q = p.kv;
    const int dh = p.qkv.head_dim, half = dh >> 1;
    const int blk = col / dh, d = col - blk * dh;  // d < half
    const int l = blk >> 1;
    const int b = row / q.F, j = row - b * q.F;
    const int64_t bl = (int64_t)b * q.L + l;
    if ((blk & 1) == 0) {
      const float2 cs = q.rope[j * half + d];
      T* dst = reinterpret_cast<T*>(q.cache_k) + (bl * q.R + q.row0 + j) * dh;
      dst[d] = from_f<T>(v * cs.x - u * cs.y);
      dst[d + half] = from_f<T>(u * cs.x + v * cs.y);
    } else {
      T* dst = reinterpret_cast<T*>(q.cache_vt) + bl * dh * q.R + q.row0 + j;
      dst[(int64_t)d * q.R] = from_f<T>(v);
      dst[(int64_t)(d + half) * q.R] = from_f<T>(u);
    }
  } else {  // EPI_ROPE
    const QkvOut& q = p.qkv;
    const int dh = q.head_dim, half = dh >> 1;
    const int head = col / dh, d = col - head * dh;  // d < half
    const int b = row / q.T, i = row - b * q.T;
    if (head <= q.Hq) {
      const float2 cs = q.rope[i * half + d];
      const float lo = v * cs.x - u * cs.y;
      const float hi = u * cs.x + v * cs.y;
      T* dst = head < q.Hq
                   ? reinterpret_cast<T*>(q.q) + ((int64_t)b * q.rows_pad + i * q.Hq + head) * dh
                   : reinterpret_cast<T*>(q.k) + ((int64_t)b * q.T + i) * dh;
      dst[d] = from_f<T>(lo);
      dst[d + half] = from_f<T>(hi);
    } else {
      T* dst = reinterpret_cast<T*>(q.vt) + (int64_t)b * dh * q.tpad;
      dst[(int64_t)d * q.tpad + i] = from_f<T>(v);
      dst[(int64_t)(d + half) * q.tpad + i] = from_f<T>(u);
    }
  }
}

// Store four consecutive outputs (columns col .. col+3, col a multiple of 4)
// of one row; for paired epilogues u holds the four paired values.  Used by
// the tiled kernel, whose transposed MFMA layout gives each lane four
// consecutive columns of a row: 8- and 16-byte stores instead of scalars.
template <int EPI>
RFX_DEV void epilogue_store4(const GemmArgs& p, int z, int split, int row, int col, const float* v, const float* u) {
  using T = bf16_t;
  if constexpr (EPI == EPI_F32 || EPI == EPI_MOD) {
    float w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      w[e] = v[e];
      if (EPI == EPI_MOD && p.mod_width > 0 && col + e >= p.mod_width) w[e] = (col + e < 2 * p.mod_width) ? 0.f : 1.f;
    }
    float* o = reinterpret_cast<float*>(p.out) + (int64_t)z * p.o_bstride + (int64_t)split * p.o_split_stride +
               (int64_t)row * p.ldo + col;
    *reinterpret_cast<float4*>(o) = make_float4(w[0], w[1], w[2], w[3]);
  } else if constexpr (EPI == EPI_SILU || EPI == EPI_GELU) {
    float w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = EPI == EPI_SILU ? silu(v[e]) : gelu_tanh(v[e]) * u[e];
    T* o = reinterpret_cast<T*>(p.out) + (int64_t)z * p.o_bstride + (int64_t)row * p.ldo + col;
    *reinterpret_cast<uint2*>(o) = make_uint2((uint32_t)f2bf(w[0]) | ((uint32_t)f2bf(w[1]) << 16),
                                              (uint32_t)f2bf(w[2]) | ((uint32_t)f2bf(w[3]) << 16));
  } else if constexpr (EPI == EPI_KV) {
    const KvOut& q = p.kv;
    const int dh = p.qkv.head_dim, half = dh >> 1;
    const int blk = col / dh, d = col - blk * dh;  // d .. d+3 < half
    const int l = blk >> 1;
    const int b = row / q.F, j = row - b * q.F;
    const int64_t bl = (int64_t)b * q.L + l;
    if ((blk & 1) == 0) {
      const float4 c01 = *reinterpret_cast<const float4*>(q.rope + j * half + d);      // (cos, sin) of d, d+1
      const float4 c23 = *reinterpret_cast<const float4*>(q.rope + j * half + d + 2);  // of d+2, d+3
      const float cs[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
      float lo[4], hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = v[e] * cs[e] - u[e] * sn[e];
        hi[e] = u[e] * cs[e] + v[e] * sn[e];
      }
      T* dst = reinterpret_cast<T*>(q.cache_k) + (bl * q.R + q.row0 + j) * dh;
      *reinterpret_cast<uint2*>(dst + d) = make_uint2((uint32_t)f2bf(lo[0]) | ((uint32_t)f2bf(lo[1]) << 16),
                                                      (uint32_t)f2bf(lo[2]) | ((uint32_t)f2bf(lo[3]) << 16));
      *reinterpret_cast<uint2*>(dst + d + half) = make_uint2((uint32_t)f2bf(hi[0]) | ((uint32_t)f2bf(hi[1]) << 16),
                                                             (uint32_t)f2bf(hi[2]) | ((uint32_t)f2bf(hi[3]) << 16));
    } else {
      T* dst = reinterpret_cast<T*>(q.cache_vt) + bl * dh * q.R + q.row0 + j;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        dst[(int64_t)(d + e) * q.R] = f2bf(v[e]);
        dst[(int64_t)(d + e + half) * q.R] = f2bf(u[e]);
      }
    }
  } else {  // EPI_ROPE
    const QkvOut& q = p.qkv;
    const int dh = q.head_dim, half = dh >> 1;
    const int head = col / dh, d = col - head * dh;  // d .. d+3 < half
    const int b = row / q.T, i = row - b * q.T;
    if (head <= q.Hq) {
      const float4 c01 = *reinterpret_cast<const float4*>(q.rope + i * half + d);      // (cos, sin) of d, d+1
      const float4 c23 = *reinterpret_cast<const float4*>(q.rope + i * half + d + 2);  // of d+2, d+3
      const float cs[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
      float lo[4], hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = v[e] * cs[e] - u[e] * sn[e];
        hi[e] = u[e] * cs[e] + v[e] * sn[e];
      }
      T* dst = head < q.Hq ? reinterpret_cast<T*>(q.q) + ((int64_t)b * q.rows_pad + i * q.Hq + head) * dh
                           : reinterpret_cast<T*>(q.k) + ((int64_t)b * q.T + i) * dh;
      *reinterpret_cast<uint2*>(dst + d) = make_uint2((uint32_t)f2bf(lo[0]) | ((uint32_t)f2bf(lo[1]) << 16),
                                                      (uint32_t)f2bf(lo[2]) | ((uint32_t)f2bf(lo[3]) << 16));
      *reinterpret_cast<uint2*>(dst + d + half) = make_uint2((uint32_t)f2bf(hi[0]) | ((uint32_t)f2bf(hi[1]) << 16),
                                                             (uint32_t)f2bf(hi[2]) | ((uint32_t)f2bf(hi[3]) << 16));
    } else {
      T* dst = reinterpret_cast<T*>(q.vt) + (int64_t)b * dh * q.tpad;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        dst[(int64_t)(d + e) * q.tpad + i] = f2bf(v[e]);
        dst[(int64_t)(d + e + half) * q.tpad + i] = f2bf(u[e]);
      }
    }
  }
}

// --------------------------------------------------------------------------
// skinny: 16*MB rows per workgroup chunk, NB 16-col blocks per strip
// --------------------------------------------------------------------------
template <typename T, int MB, int NB, int EPI, int NW>
__global__ __launch_bounds__(64 * NW) void gemm_skinny(GemmArgs p) {
  constexpr int PAIR = EpiPair<EPI>::value;
  constexpr int KPF = ElemT<T>::kPerFrag;
  constexpr int KS = 4 * KPF;                      // elements per k-step
  constexpr int NBT = PAIR ? 2 * NB : NB;          // B fragments per k-step
  constexpr int COLS = 16 * NB;                    // first columns per workgroup
  constexpr int RCOLS = 16 * NBT + 1;              // LDS reduction row (padded)
  __shared__ float red[NW][MB * 16][RCOLS];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int z = blockIdx.z;
  const int mchunk = blockIdx.y / p.splits, split = blockIdx.y % p.splits;
  const int m0 = mchunk * (16 * MB);
  int n0, pair_off;
  if constexpr (PAIR == PAIR_HEAD) {
    const int half = p.qkv.head_dim >> 1, per_head = half / COLS;
    const int h = blockIdx.x / per_head;
    n0 = h * p.qkv.head_dim + (blockIdx.x - h * per_head) * COLS;
    pair_off = half;
  } else {
    n0 = blockIdx.x * COLS;
    pair_off = p.N;  // PAIR_N: up rows follow the gate rows
  }
  const int kbeg = split * p.k_per_split;
  const int kend = min(p.K, kbeg + p.k_per_split);

  const T* A = reinterpret_cast<const T*>(p.A) + (int64_t)z * p.a_bstride;
  const T* B = reinterpret_cast<const T*>(p.B) + (int64_t)z * p.b_bstride;
  const T* arow[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int r = min(m0 + mb * 16 + r16, p.M - 1);
    arow[mb] = A + (int64_t)r * p.lda + g * KPF;
  }
  const T* brow[NBT];
#pragma unroll
  for (int nb = 0; nb < NBT; ++nb) {
    int brw;
    if (PAIR == PAIR_NONE) {
      brw = min(n0 + nb * 16 + r16, p.N - 1);
    } else {
      const int c = n0 + (nb % NB) * 16 + r16;
      brw = nb >= NB ? c + pair_off : c;
    }
    brow[nb] = B + (int64_t)brw * p.ldb + g * KPF;
  }

  f32x4_v acc[MB][NBT];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb) acc[mb][nb] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  const int nsteps = (kend - kbeg + KS - 1) / KS;
  constexpr int U = 4;
  for (int s0 = wave; s0 < nsteps; s0 += NW * U) {
    uint4 bf[U][NBT], af[U][MB];
    // unconditional loads (clamped to k = kbeg when past the end), masked to
    // zero afterwards: no branch joins that would serialise the loads
    bool okv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kbeg + (s0 + NW * u) * KS;
      okv[u] = (s0 + NW * u < nsteps) && (k + g * KPF < kend);
      const int kc = okv[u] ? k : kbeg;
#pragma unroll
      for (int nb = 0; nb < NBT; ++nb) bf[u][nb] = ld16(brow[nb] + kc);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) af[u][mb] = ld16(arow[mb] + kc);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int nb = 0; nb < NBT; ++nb) bf[u][nb] = okv[u] ? bf[u][nb] : zero16();
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb) mfma_step(acc[mb][nb], af[u][mb], bf[u][nb], T());
    }
  }

#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][mb * 16 + 4 * g + i][nb * 16 + r16] = acc[mb][nb][i];
  __syncthreads();

  for (int e = threadIdx.x; e < MB * 16 * COLS; e += 64 * NW) {
    const int row = e / COLS, col = e % COLS;
    const int grow = m0 + row;
    const int gcol = n0 + col;
    if (grow >= p.M || (PAIR == PAIR_NONE && gcol >= p.N)) continue;
    float v = 0.f, u = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      v += red[w][row][col];
      if (PAIR) u += red[w][row][col + COLS];
    }
    epilogue_store<EPI, T>(p, z, split, grow, gcol, v, u);
  }
}

// --------------------------------------------------------------------------
// skinny, bf16, activations staged in LDS.  The activation rows of the
// workgroup's K range are copied to LDS with global_load_lds_dwordx4, each
// instruction moving 1 KB of consecutive bytes of one row, instead of being
// fetched as MFMA fragments (16 rows x 64 bytes per instruction) straight
// from global memory by every wave.  16-byte chunks are XOR-swizzled by
// (row mod 8) so the fragment reads are conflict-free.  Weights are still
// streamed as fragments into registers; the activation copy is issued first,
// so the wait for it leaves the weight loads in flight.  After the MFMAs the
// same LDS holds the cross-wave reduction.
// --------------------------------------------------------------------------
RFX_DEV void wg_barrier_lds() {
  // all of this wave's LDS reads are complete; then a plain barrier (the
  // memory clobber keeps the compiler from moving LDS accesses across it)
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int MB, int NB, int EPI, int NW>
__global__ __launch_bounds__(64 * NW) void gemm_skinny_lds(GemmArgs p) {
  using T = bf16_t;
  constexpr int PAIR = EpiPair<EPI>::value;
  constexpr int KS = 32;                           // elements per k-step
  constexpr int NBT = PAIR ? 2 * NB : NB;          // B fragments per k-step
  constexpr int COLS = 16 * NB;                    // first columns per workgroup
  constexpr int RCOLS = 16 * NBT + 1;              // reduction row (padded)
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int z = blockIdx.z;
  const int mchunk = blockIdx.y / p.splits, split = blockIdx.y % p.splits;
  const int m0 = mchunk * (16 * MB);
  int n0, pair_off;
  if constexpr (PAIR == PAIR_HEAD) {
    const int half = p.qkv.head_dim >> 1, per_head = half / COLS;
    const int h = blockIdx.x / per_head;
    n0 = h * p.qkv.head_dim + (blockIdx.x - h * per_head) * COLS;
    pair_off = half;
  } else {
    n0 = blockIdx.x * COLS;
    pair_off = p.N;
  }
  const int kbeg = split * p.k_per_split;
  const int kend = min(p.K, kbeg + p.k_per_split);
  const int nsteps = (kend - kbeg) / KS;  // K and k_per_split are multiples of 32
  // LDS bytes per activation row: this split's K range, rounded up to whole
  // groups of 8 chunks so the chunk swizzle (an XOR of the low 3 bits) stays
  // inside the row
  const int rs = (((kend - kbeg) * 2) + 127) & ~127;
  const int cpr = rs >> 4;  // 16-byte chunks per row

  const T* A = reinterpret_cast<const T*>(p.A) + (int64_t)z * p.a_bstride;
  const T* B = reinterpret_cast<const T*>(p.B) + (int64_t)z * p.b_bstride;

  // 1. activation rows m0 .. min(M, m0+16*MB)-1, chunks kbeg/8 .. ; chunk
  //    position q of row r holds logical chunk q ^ (r & 7).  Rows past M are
  //    not copied: an MFMA output row depends only on its own A row, and those
  //    rows are never stored.
  {
    const int rows = min(16 * MB, p.M - m0);
    const int total = rows * cpr;  // chunks
    const int kchunks = (kend - kbeg) >> 3;
    for (int i0 = wave * 64; i0 < total; i0 += NW * 64) {
      const int q = i0 + lane;
      const int r = q / cpr, pos = q - r * cpr;
      int lc = pos ^ (r & 7);
      lc = lc < kchunks ? lc : 0;  // a K range that is not a multiple of 64: any valid chunk
      const T* src = A + (int64_t)min(m0 + r, p.M - 1) * p.lda + kbeg + lc * 8;
      if (q < total) __builtin_amdgcn_global_load_lds(src, smem + i0 * 16, 16, 0, 0);
    }
  }

  // 2. weight fragments of this wave's k-steps (s = wave, wave + NW, ...)
  const T* brow[NBT];
#pragma unroll
  for (int nb = 0; nb < NBT; ++nb) {
    int brw;
    if (PAIR == PAIR_NONE) {
      brw = min(n0 + nb * 16 + r16, p.N - 1);
    } else {
      const int c = n0 + (nb % NB) * 16 + r16;
      brw = nb >= NB ? c + pair_off : c;
    }
    brow[nb] = B + (int64_t)brw * p.ldb + kbeg + g * 8;
  }

  f32x4_v acc[MB][NBT];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb) acc[mb][nb] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  // per-lane activation fragment offset: row 16mb + r16, chunk 4s + g at
  // position (4s + g) ^ (r16 & 7) = 8*(s >> 1) + ((4*(s & 1) + g) ^ (r16 & 7))
  const int aoff0 = r16 * rs + ((g) ^ (r16 & 7)) * 16;
  const int aoff1 = r16 * rs + ((4 + g) ^ (r16 & 7)) * 16;

  constexpr int U = 4;
  bool first = true;
  for (int s0 = wave; s0 < nsteps; s0 += NW * U) {
    uint4 bf[U][NBT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + NW * u;
      const int sc = s < nsteps ? s : s0;  // clamped: a valid address, result unused
#pragma unroll
      for (int nb = 0; nb < NBT; ++nb) bf[u][nb] = ld16(brow[nb] + sc * KS);
    }
    if (first) {
      // the activation copy was issued before these weight loads and loads
      // complete in order: wait for it, leave the weight loads in flight
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8) | ((U * NBT) & 15) | (((U * NBT) >> 4) << 14));
      wg_barrier_lds();
      first = false;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + NW * u;
      if (s >= nsteps) break;
      const unsigned char* ab = smem + (s >> 1) * 128 + ((s & 1) ? aoff1 : aoff0);
      uint4 af[MB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) af[mb] = *reinterpret_cast<const uint4*>(ab + mb * 16 * rs);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb) mfma_step(acc[mb][nb], af[mb], bf[u][nb], T());
    }
  }
  if (first) {  // waves without k-steps still take part in the barrier
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
    wg_barrier_lds();
  }

  // 3. cross-wave reduction through the (now free) activation LDS
  wg_barrier_lds();
  float* red = reinterpret_cast<float*>(smem);  // [NW][MB*16][RCOLS]
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[(wave * MB * 16 + mb * 16 + 4 * g + i) * RCOLS + nb * 16 + r16] = acc[mb][nb][i];
  __syncthreads();
  for (int e = threadIdx.x; e < MB * 16 * COLS; e += 64 * NW) {
    const int row = e / COLS, col = e % COLS;
    const int grow = m0 + row;
    const int gcol = n0 + col;
    if (grow >= p.M || (PAIR == PAIR_NONE && gcol >= p.N)) continue;
    float v = 0.f, u = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      v += red[(w * MB * 16 + row) * RCOLS + col];
      if (PAIR) u += red[(w * MB * 16 + row) * RCOLS + col + COLS];
    }
    epilogue_store<EPI, bf16_t>(p, z, split, grow, gcol, v, u);
  }
}

// launch helper for the LDS-staged skinny kernel (bf16, M <= 64)
template <int MB, int EPI>
static void launch_skinny_lds_cfg(const GemmArgs& a, hipStream_t s, int nw) {
  constexpr int PAIR = EpiPair<EPI>::value;
  constexpr int NB = PAIR ? 1 : 2;
  constexpr int NBT = PAIR ? 2 * NB : NB;
  int nx;
  if (PAIR == PAIR_HEAD)
    nx = a.N / 32;
  else if (PAIR == PAIR_N)
    nx = a.N / 16;
  else
    nx = (a.N + 16 * NB - 1) / (16 * NB);
  const int mch = (a.M + 16 * MB - 1) / (16 * MB);
  dim3 grid(nx, mch * a.splits, a.batch);
  const size_t klen = (size_t)(a.k_per_split < a.K ? a.k_per_split : a.K);
  const size_t tile = (size_t)16 * MB * ((klen * 2 + 127) & ~(size_t)127);
  const size_t red = (size_t)nw * MB * 16 * (16 * NBT + 1) * 4;
  const size_t shm = tile > red ? tile : red;
  if (nw == 8)
    RFX_LAUNCH((gemm_skinny_lds<MB, NB, EPI, 8>), grid, dim3(512), shm, s, a);
  else
    RFX_LAUNCH((gemm_skinny_lds<MB, NB, EPI, 4>), grid, dim3(256), shm, s, a);
}

// --------------------------------------------------------------------------
// tiled: 128 x 128 workgroup tile (paired: 128 rows x 64 first + 64 paired cols)
// --------------------------------------------------------------------------
constexpr int TBM = 128, TBN = 128, TROWB = 128, TPAD = 16;  // TROWB: bytes of K per stage row

template <typename T, int EPI>
__global__ __launch_bounds__(256) void gemm_tiled(GemmArgs p) {
  constexpr int PAIR = EpiPair<EPI>::value;
  constexpr int KPF = ElemT<T>::kPerFrag;
  constexpr int KSTAGE = TROWB / (int)sizeof(T);  // elements of K per stage
  constexpr int LROW = TROWB + TPAD;              // LDS row stride, bytes
  __shared__ __attribute__((aligned(16))) unsigned char As[2][TBM * LROW];
  __shared__ __attribute__((aligned(16))) unsigned char Bs[2][TBN * LROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int z = blockIdx.z / p.splits, split = blockIdx.z % p.splits;
  const int m0 = blockIdx.y * TBM;
  int n0, pair_off;
  if constexpr (PAIR == PAIR_HEAD) {
    const int half = p.qkv.head_dim >> 1, per_head = half / 64;
    const int h = blockIdx.x / per_head;
    n0 = h * p.qkv.head_dim + (blockIdx.x - h * per_head) * 64;
    pair_off = half;
  } else if constexpr (PAIR == PAIR_N) {
    n0 = blockIdx.x * 64;
    pair_off = p.N;
  } else {
    n0 = blockIdx.x * TBN;
    pair_off = 0;
  }
  const int kbeg = split * p.k_per_split;
  const int kend = min(p.K, kbeg + p.k_per_split);
  const int nstage = (kend - kbeg + KSTAGE - 1) / KSTAGE;

  const T* A = reinterpret_cast<const T*>(p.A) + (int64_t)z * p.a_bstride;
  const T* B = reinterpret_cast<const T*>(p.B) + (int64_t)z * p.b_bstride;

  // global -> register staging: thread loads rows (tid/8 + 32*i), chunk tid%8
  const int ch = tid & 7;
  const T* ga[4];
  const T* gb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = (tid >> 3) + 32 * i;
    ga[i] = A + (int64_t)min(m0 + r, p.M - 1) * p.lda + ch * KPF;
    int brw;
    if (PAIR != PAIR_NONE) {
      const int c = n0 + (r & 63);
      brw = r >= 64 ? c + pair_off : c;
    } else {
      brw = min(n0 + r, p.N - 1);
    }
    gb[i] = B + (int64_t)brw * p.ldb + ch * KPF;
  }
  uint4 ra[4], rb[4];
  bool gok = false;
  auto gload = [&](int st) {
    const int k0 = kbeg + st * KSTAGE;
    gok = k0 + ch * KPF < kend;
    const int kc = gok ? k0 : kbeg - ch * KPF;  // clamped: a valid address
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = ld16(ga[i] + kc);
      rb[i] = ld16(gb[i] + kc);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (tid >> 3) + 32 * i;
      st16(&As[buf][r * LROW + ch * 16], gok ? ra[i] : zero16());
      st16(&Bs[buf][r * LROW + ch * 16], gok ? rb[i] : zero16());
    }
  };

  f32x4_v acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  int brow_l[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    if (PAIR != PAIR_NONE)
      brow_l[nb] = (nb < 2 ? 0 : 64) + wn * 32 + (nb & 1) * 16 + r16;
    else
      brow_l[nb] = wn * 64 + nb * 16 + r16;
  }

  if (nstage > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int st = 0; st < nstage; ++st) {
    const int buf = st & 1;
    if (st + 1 < nstage) gload(st + 1);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint4 af[4], bf[4];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        af[mb] = *reinterpret_cast<const uint4*>(&As[buf][(wm * 64 + mb * 16 + r16) * LROW + ks * 64 + g * 16]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        bf[nb] = *reinterpret_cast<const uint4*>(&Bs[buf][brow_l[nb] * LROW + ks * 64 + g * 16]);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) mfma_step(acc[mb][nb], af[mb], bf[nb], T());
    }
    if (st + 1 < nstage) lstore(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int grow = m0 + wm * 64 + mb * 16 + 4 * g + i;
      if (grow >= p.M) continue;
      if (PAIR != PAIR_NONE) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int gcol = n0 + wn * 32 + nb * 16 + r16;
          epilogue_store<EPI, T>(p, z, split, grow, gcol, acc[mb][nb][i], acc[mb][nb + 2][i]);
        }
      } else {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          const int gcol = n0 + wn * 64 + nb * 16 + r16;
          if (gcol < p.N) epilogue_store<EPI, T>(p, z, split, grow, gcol, acc[mb][nb][i], 0.f);
        }
      }
    }
  }
}

// --------------------------------------------------------------------------
// tiled, bf16, direct global->LDS pipeline.  Same 128x128 workgroup tile and
// 2x2 waves of 64x64 as gemm_tiled, but each 64-element K stage (128 bytes of
// every A and B row) is copied by global_load_lds_dwordx4 (1 KB of whole rows
// per instruction) instead of through registers.  NS = 2: double-buffered,
// 64 KB of LDS, two workgroups per CU (the other workgroup's MFMAs cover a
// stage's copy latency); NS = 4: a ring of four stages, three in flight, one
// workgroup per CU.  Two stages measured faster at the batch-32 shapes.
// 16-byte chunks are XOR-swizzled (RFX_GSWZ).  K and the split length must be
// multiples of 64 (no partial stage to zero-fill).  M32: each wave's 64x64
// block as 2x2 32x32x16 MFMAs (four accumulators) instead of 4x4 16x16x32
// ones (sixteen): the same LDS fragment bytes and matrix-core cycles in half
// the instructions, which one wave per SIMD issues closer to the unit's rate
// (gate|up on the long context 12.9 -> 12.3 us; the 32-stage down projection
// at 32 envs measured slower, 22.4 -> 22.8 us, and keeps 16x16x32).
// --------------------------------------------------------------------------
constexpr int DST = 64;                  // K elements per stage
constexpr int DROWB = DST * 2;           // bytes per stage row (128)
constexpr int DSTAGE = (TBM + TBN) * DROWB;  // bytes per stage (32 KB)

// chunk swizzle of stage row r: 16 distinct bank positions over 16
// consecutive 128-byte rows (the row parity picks the half of the 256-byte
// bank window, the XOR the 16-byte slot)
#define RFX_GSWZ(r) (((r) & 7) ^ (((r) >> 3) & 1))

// Workgroup -> tile.  Workgroups are dispatched round-robin over the 8 XCDs,
// each with its own L2.  With a 1-D grid, XCD x receives the tiles
// [x*per, (x+1)*per) of the tile sequence in which the M tile varies fastest,
// so the workgroups sharing an L2 also share B (weight) tiles and a band of
// A tiles instead of touching every tile of both operands.
template <int PAIR, int BM>
RFX_DEV bool dma_tile(const GemmArgs& p, int& bx, int& by, int& bz) {
  const int nx = PAIR == PAIR_NONE ? (p.N + TBN - 1) / TBN : p.N / (PAIR == PAIR_N ? 64 : 128);
  const int ny = (p.M + BM - 1) / BM;
  const int total = nx * ny * p.batch * p.splits;
  const int per = (total + 7) / 8;
  const int t = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (t >= total) return false;
  by = t % ny;
  const int rest = t / ny;
  bx = rest % nx;
  bz = rest / nx;
  return true;
}

// s_waitcnt operand: wait until at most n vector-memory operations are
// outstanding (vmcnt bits [3:0] and [15:14]); expcnt and lgkmcnt left at their
// maxima (no wait)
constexpr int vmcnt_enc(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// BM (160, 128, 96 or 64) rows per tile: two waves along M hold BM/2 rows
// each (MB = BM/32 blocks of 16).  160- and 96-row tiles serve grids whose
// 128-row count just exceeds one wave of workgroups (two tiles on a few CUs
// would set the kernel time): 160-row tiles one per CU where they fit one
// wave, else 96-row tiles two per CU (340 of them cost 3/4 of that).
//
// KW = 2 (160-row tiles; 64-row tiles with a paired epilogue): eight waves,
// two per output block, each taking one of the two 32-wide k-steps of every
// stage, so that each SIMD holds two waves and one's MFMAs run while the
// other waits on LDS; each wave then finalizes half of the block's columns,
// so the epilogue work is shared too.  QKV at 32 envs: 21.8 -> 18.3 us; QKV
// of the long context (64-row tiles): 11.7 -> 11.1 us.  With the fp32
// epilogue on 128-row (16x16 or 32x32 blocks) and 64-row tiles it was not
// faster (32 envs: output projection 15.1 -> 15.5, down 23.1 -> 23.1 us; long
// context: output projection 7.5 -> 8.2, down 10.3 -> 10.7 us).
template <int EPI, int NS, int NSTC, int BM = TBM, bool M32 = false, int KW = 1>
__global__ __launch_bounds__(256 * KW) void gemm_dma(GemmArgs p) {
  using T = bf16_t;
  constexpr int PAIR = EpiPair<EPI>::value;
  // BM / 32: 16-row blocks per wave, and A copies (8 rows each) per wave per
  // stage
  static_assert(NS == 2 || NS == 4, "two or four stages");
  static_assert(BM == 160 || BM == 128 || BM == 96 || BM == 64, "160-, 128-, 96- or 64-row tiles");
  static_assert(KW == 1 || (KW == 2 && NS == 4 && NSTC > 0 && !M32), "K-split waves: unrolled pipeline, 16x16 blocks");
  constexpr int CPS = BM / 32 + 4;          // copy instructions per output block per stage
  constexpr int CPW = (CPS + KW - 1) / KW;  // copy instructions per wave per stage
  // stages sized for at least 128 rows (a 96-row tile uses 28 of the 32 KB)
  constexpr int STB = ((BM > TBM ? BM : TBM) + TBN) * DROWB;
  __shared__ __attribute__((aligned(16))) unsigned char st0[STB];
  __shared__ __attribute__((aligned(16))) unsigned char st1[STB];
  __shared__ __attribute__((aligned(16))) unsigned char st2[NS == 4 ? STB : 16];
  __shared__ __attribute__((aligned(16))) unsigned char st3[NS == 4 ? STB : 16];

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  // output block wq (2 x 2 over the tile); with KW = 2 two waves share it,
  // wave wk taking k-step wk (elements 32wk .. 32wk + 31) of every stage
  const int wq = wave & 3, wk = wave >> 2;
  const int wm = wq >> 1, wn = wq & 1;
  int bx, by, bz;
  if (!dma_tile<PAIR, BM>(p, bx, by, bz)) return;
  const int z = bz / p.splits, split = bz % p.splits;
  const int m0 = by * BM;
  int n0, pair_off;
  if constexpr (PAIR == PAIR_HEAD) {
    const int half = p.qkv.head_dim >> 1, per_head = half / 64;
    const int h = bx / per_head;
    n0 = h * p.qkv.head_dim + (bx - h * per_head) * 64;
    pair_off = half;
  } else if constexpr (PAIR == PAIR_N) {
    n0 = bx * 64;
    pair_off = p.N;
  } else {
    n0 = bx * TBN;
    pair_off = 0;
  }
  const int kbeg = split * p.k_per_split;
  const int kend = min(p.K, kbeg + p.k_per_split);
  // NSTC > 0: the stage count is a compile-time constant and the stage loop is
  // fully unrolled, so the compiler tracks which LDS buffer every copy in
  // flight targets (a loop would merge that knowledge at its header and make
  // it wait for all copies there)
  const int nst = NSTC > 0 ? NSTC : (kend - kbeg) / DST;

  const T* A = reinterpret_cast<const T*>(p.A) + (int64_t)z * p.a_bstride;
  const T* B = reinterpret_cast<const T*>(p.B) + (int64_t)z * p.b_bstride;

  // DMA, with NA = BM/32: wave w, instruction j covers stage rows
  // 8*(NA*w + j) + (lane >> 3) of A (j < NA) or 8*(4w + j - NA) + (lane >> 3)
  // of B (j >= NA); physical chunk lane & 7 holds logical chunk
  // (lane & 7) ^ swizzle(row)
  // The copies of output block wq are split over its KW waves: wave wk issues
  // instructions j = wk*CPW + i.  With KW = 2 and an odd count the second
  // wave's last instruction repeats its previous one (same bytes to the same
  // place), so every wave issues CPW copies per stage and waits on one count.
  const T* gsrc[9];  // the first CPW are used (a bound that depends on BM breaks the lambda capture)
  int lrow[9];       // LDS stage row of copy i (wave-uniform)
  {
    const int rr = lane >> 3, pc = lane & 7;
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int j = KW == 1 ? i : min(wk * CPW + i, CPS - 1);
      const bool isa = j < (BM / 32);
      const int row0 = isa ? 8 * ((BM / 32) * wq + j) : 8 * (4 * wq + j - (BM / 32));
      const int row = row0 + rr;
      lrow[i] = isa ? row0 : BM + row0;
      const int lc = pc ^ RFX_GSWZ(row);
      if (isa) {
        gsrc[i] = A + (int64_t)min(m0 + row, p.M - 1) * p.lda + kbeg + lc * 8;
      } else {
        int brw;
        if (PAIR != PAIR_NONE) {
          const int c = n0 + (row & 63);
          brw = row >= 64 ? c + pair_off : c;
        } else {
          brw = min(n0 + row, p.N - 1);
        }
        gsrc[i] = B + (int64_t)brw * p.ldb + kbeg + lc * 8;
      }
    }
  }
  // stage layout: A rows 0..BM-1 then B rows 0..127, 128 bytes each
  auto issue = [&](int st, unsigned char* buf) __attribute__((always_inline)) {
    const int k0 = st * DST;
#pragma unroll
    for (int i = 0; i < CPW; ++i) __builtin_amdgcn_global_load_lds(gsrc[i] + k0, buf + lrow[i] * DROWB, 16, 0, 0);
  };

  static_assert(!M32 || BM % 64 == 0, "32x32 blocks need 32-row wave halves");
  constexpr int MB2 = M32 ? BM / 64 : 1;  // 32-row blocks per wave
  f32x4_v acc[(BM / 32)][4];              // 16x16x32: C^T blocks [16-row block][16-column block]
  f32x16_v acc2[MB2][2];                  // 32x32x16: C^T blocks [32-row block][32-column block]
  if constexpr (M32) {
#pragma unroll
    for (int a = 0; a < MB2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) acc2[a][b] = f32x16_v{};
  } else {
#pragma unroll
    for (int a = 0; a < (BM / 32); ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = f32x4_v{0.f, 0.f, 0.f, 0.f};
  }
  // 32x32x16: lane l reads row l & 31 of a 32-row block (32-aligned, so the
  // swizzle is that of l & 31), chunk 2kk + (l >> 5) of k-step kk; column
  // block 1 of a pair holds the paired columns of block 0
  const int r32 = lane & 31, h32 = lane >> 5;
  int foff2[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) foff2[kk] = r32 * DROWB + ((2 * kk + h32) ^ RFX_GSWZ(r32)) * 16;
  int brow2[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) brow2[nb] = PAIR != PAIR_NONE ? nb * 64 + wn * 32 : wn * 64 + nb * 32;

  // fragment offsets: row r (r & 7 == r16 & 7), k-step kk of the stage,
  // chunk 4kk + g at (4kk + g) ^ (r16 & 7)
  int foff[2 / KW];  // k-step kk = kh + wk*2/KW
#pragma unroll
  for (int kh = 0; kh < 2 / KW; ++kh) {
    const int kk = kh + wk * (2 / KW);
    foff[kh] = r16 * DROWB + ((4 * kk + g) ^ RFX_GSWZ(r16)) * 16;
  }
  int brow_l[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    if (PAIR != PAIR_NONE)
      brow_l[nb] = (nb < 2 ? 0 : 64) + wn * 32 + (nb & 1) * 16;
    else
      brow_l[nb] = wn * 64 + nb * 16;
  }

  // four stages: st, st+1, st+2 in flight at the start of stage st (CPS
  // instructions each, completing in order); two stages: only st
  auto step = [&](int st, const unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt)
                  __attribute__((always_inline)) {
    if (NS == 4 && st + 2 < nst)
      __builtin_amdgcn_s_waitcnt(vmcnt_enc(2 * CPW));
    else if (NS == 4 && st + 1 < nst)
      __builtin_amdgcn_s_waitcnt(vmcnt_enc(CPW));
    else
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    // every wave's share of stage st is in LDS and every wave has finished
    // stage st-1, whose buffer the next copy overwrites
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (st + NS - 1 < nst) issue(st + NS - 1, nxt);
    if constexpr (M32) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        uint4 af[MB2], bf[2];
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          bf[nb] = *reinterpret_cast<const uint4*>(cur + (BM + brow2[nb]) * DROWB + foff2[kk]);
#pragma unroll
        for (int mb = 0; mb < MB2; ++mb)
          af[mb] = *reinterpret_cast<const uint4*>(cur + (wm * (BM / 2) + mb * 32) * DROWB + foff2[kk]);
#pragma unroll
        for (int mb = 0; mb < MB2; ++mb)
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) mfma32_step(acc2[mb][nb], bf[nb], af[mb]);  // C^T blocks
      }
      return;
    }
#pragma unroll
    for (int kh = 0; kh < 2 / KW; ++kh) {
      uint4 af[(BM / 32)], bf[4];
#pragma unroll
      for (int mb = 0; mb < (BM / 32); ++mb)
        af[mb] = *reinterpret_cast<const uint4*>(cur + (wm * (BM / 2) + mb * 16) * DROWB + foff[kh]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        bf[nb] = *reinterpret_cast<const uint4*>(cur + (BM + brow_l[nb]) * DROWB + foff[kh]);
#pragma unroll
      for (int mb = 0; mb < (BM / 32); ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) mfma_step(acc[mb][nb], bf[nb], af[mb], T());  // C^T blocks
    }
  };

  if constexpr (NSTC > 0) {
    static_assert(NS == 4, "unrolled pipeline uses four stages");
    unsigned char* const bufs[4] = {st0, st1, st2, st3};
    issue(0, bufs[0]);
    if (NSTC > 1) issue(1, bufs[1]);
    if (NSTC > 2) issue(2, bufs[2]);
#pragma unroll
    for (int st = 0; st < NSTC; ++st) step(st, bufs[st & 3], bufs[(st + 3) & 3]);
  } else if constexpr (NS == 4) {
    if (nst > 0) issue(0, st0);
    if (nst > 1) issue(1, st1);
    if (nst > 2) issue(2, st2);
    for (int st = 0; st < nst; st += 4) {
      step(st, st0, st3);
      if (st + 1 < nst) step(st + 1, st1, st0);
      if (st + 2 < nst) step(st + 2, st2, st1);
      if (st + 3 < nst) step(st + 3, st3, st2);
    }
  } else {
    if (nst > 0) issue(0, st0);
    for (int st = 0; st < nst; st += 2) {
      step(st, st0, st1);
      if (st + 1 < nst) step(st + 1, st1, st0);
    }
  }

  if constexpr (KW == 2) {
    // The two waves of an output block hold partial sums over their halves of
    // every stage.  Each finalizes half of the block's columns: it hands the
    // other half to its partner through LDS (the stage buffer numbered like
    // the block: after this barrier every copy has landed and every fragment
    // read is done) and adds what the partner hands over.  a + b = b + a, so
    // both orders give the same sum.
    constexpr int NX = (BM / 32) * 2;  // float4s handed over per lane
    static_assert(2 * NX * 64 * 16 <= STB, "hand-over fits one stage buffer");
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    unsigned char* const xb = wq == 0 ? st0 : (wq == 1 ? st1 : (wq == 2 ? st2 : st3));
    float4* const sendp = reinterpret_cast<float4*>(xb) + wk * (NX * 64) + lane;
    const float4* const recvp = reinterpret_cast<const float4*>(xb) + (1 - wk) * (NX * 64) + lane;
    // wave wk finalizes two of the four column blocks, slot s2 being block
    // nbA(s2) for wave 0 and nbB(s2) for wave 1 (with pairs: a first-half
    // block and the block of its paired columns)
#pragma unroll
    for (int mb = 0; mb < (BM / 32); ++mb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int nbA = PAIR != PAIR_NONE ? 2 * s2 : s2, nbB = PAIR != PAIR_NONE ? 1 + 2 * s2 : 2 + s2;
        const f32x4_v v = wk ? acc[mb][nbA] : acc[mb][nbB];
        sendp[(mb * 2 + s2) * 64] = make_float4(v[0], v[1], v[2], v[3]);
      }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    f32x4_v fin[(BM / 32)][2];
#pragma unroll
    for (int mb = 0; mb < (BM / 32); ++mb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int nbA = PAIR != PAIR_NONE ? 2 * s2 : s2, nbB = PAIR != PAIR_NONE ? 1 + 2 * s2 : 2 + s2;
        const float4 r = recvp[(mb * 2 + s2) * 64];
        fin[mb][s2] = (wk ? acc[mb][nbB] : acc[mb][nbA]) + f32x4_v{r.x, r.y, r.z, r.w};
      }
#pragma unroll
    for (int mb = 0; mb < (BM / 32); ++mb) {
      const int grow = m0 + wm * (BM / 2) + mb * 16 + r16;
      if (grow >= p.M) continue;
      if (PAIR != PAIR_NONE) {
        const int gcol = n0 + wn * 32 + wk * 16 + 4 * g;
        const float v[4] = {fin[mb][0][0], fin[mb][0][1], fin[mb][0][2], fin[mb][0][3]};
        const float u[4] = {fin[mb][1][0], fin[mb][1][1], fin[mb][1][2], fin[mb][1][3]};
        epilogue_store4<EPI>(p, z, split, grow, gcol, v, u);
      } else {
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const int gcol = n0 + wn * 64 + (2 * wk + s2) * 16 + 4 * g;
          const float v[4] = {fin[mb][s2][0], fin[mb][s2][1], fin[mb][s2][2], fin[mb][s2][3]};
          if (gcol + 3 < p.N) {
            epilogue_store4<EPI>(p, z, split, grow, gcol, v, v);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (gcol + e < p.N) epilogue_store<EPI, T>(p, z, split, grow, gcol + e, v[e], 0.f);
          }
        }
      }
    }
    return;
  }
  if constexpr (M32) {
    // acc2[mb][nb] holds the transposed 32x32 block: lane l has output row
    // m0 + wm*BM/2 + mb*32 + (l & 31) and, for q4 < 4, the four consecutive
    // columns 8*q4 + 4*(l >> 5) .. +3 of column block nb
#pragma unroll
    for (int mb = 0; mb < MB2; ++mb) {
      const int grow = m0 + wm * (BM / 2) + mb * 32 + r32;
      if (grow >= p.M) continue;
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        if (PAIR != PAIR_NONE) {
          const int gcol = n0 + wn * 32 + 8 * q4 + 4 * h32;
          const float v[4] = {acc2[mb][0][4 * q4], acc2[mb][0][4 * q4 + 1], acc2[mb][0][4 * q4 + 2],
                              acc2[mb][0][4 * q4 + 3]};
          const float u[4] = {acc2[mb][1][4 * q4], acc2[mb][1][4 * q4 + 1], acc2[mb][1][4 * q4 + 2],
                              acc2[mb][1][4 * q4 + 3]};
          epilogue_store4<EPI>(p, z, split, grow, gcol, v, u);
        } else {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
            const int gcol = n0 + wn * 64 + nb * 32 + 8 * q4 + 4 * h32;
            const float v[4] = {acc2[mb][nb][4 * q4], acc2[mb][nb][4 * q4 + 1], acc2[mb][nb][4 * q4 + 2],
                                acc2[mb][nb][4 * q4 + 3]};
            if (gcol + 3 < p.N) {
              epilogue_store4<EPI>(p, z, split, grow, gcol, v, v);
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (gcol + e < p.N) epilogue_store<EPI, T>(p, z, split, grow, gcol + e, v[e], 0.f);
            }
          }
        }
      }
    }
    return;
  }
  // acc[mb][nb] holds the transposed 16x16 block: lane (r16, g) has output
  // row m0 + wm*64 + mb*16 + r16, columns 4g .. 4g+3 of column block nb
#pragma unroll
  for (int mb = 0; mb < (BM / 32); ++mb) {
    const int grow = m0 + wm * (BM / 2) + mb * 16 + r16;
    if (grow >= p.M) continue;
    if (PAIR != PAIR_NONE) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int gcol = n0 + wn * 32 + nb * 16 + 4 * g;
        const float v[4] = {acc[mb][nb][0], acc[mb][nb][1], acc[mb][nb][2], acc[mb][nb][3]};
        const float u[4] = {acc[mb][nb + 2][0], acc[mb][nb + 2][1], acc[mb][nb + 2][2], acc[mb][nb + 2][3]};
        epilogue_store4<EPI>(p, z, split, grow, gcol, v, u);
      }
    } else {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int gcol = n0 + wn * 64 + nb * 16 + 4 * g;
        const float v[4] = {acc[mb][nb][0], acc[mb][nb][1], acc[mb][nb][2], acc[mb][nb][3]};
        if (gcol + 3 < p.N) {
          epilogue_store4<EPI>(p, z, split, grow, gcol, v, v);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (gcol + e < p.N) epilogue_store<EPI, T>(p, z, split, grow, gcol + e, v[e], 0.f);
        }
      }
    }
  }
}

// --------------------------------------------------------------------------
// tiled, bf16, 256x256 workgroup tile for the large-M shapes (the batched
// projections, the frame projection, the conditioning MLPs).  Eight waves in
// 2 (M) x 4 (N), each a 128x64 block of 16x16x32 MFMAs (C^T blocks, 32
// accumulators of four floats per lane).  The copy into LDS per K stage is
// (256 + 256) rows x 128 bytes = 64 KB for 256x256x64x2 flops, half the bytes
// per flop of the 128x128 tile: with every CU copying from L2 at once, the
// copy rate and not the MFMA rate bounds the smaller tile.  Double-buffered
// (128 KB of LDS, one workgroup per CU).  Pairs (gated GELU, rotate-half
// RoPE) put 128 first-half and the matching 128 second-half columns in one
// tile; a wave holds 32 + 32 of them.
// --------------------------------------------------------------------------
constexpr int GBM = 256, GBN = 256;
constexpr int GSTAGE = (GBM + GBN) * DROWB;  // 64 KB

// Tiles of one XCD (a contiguous range of the tile sequence) in groups of up
// to 8 M tiles by every N tile, M fastest within a group: the 32 tiles an XCD
// runs at once then cover 8 M x 4 N tiles, whose A and B panels they read in
// step, instead of 32 M tiles of one N panel, which re-read A for every tile
// (the frame projection at 32 envs: 96 x 36 tiles with a 1 MB A panel each).
template <int PAIR>
RFX_DEV bool big_tile(const GemmArgs& p, int& bx, int& by, int& bz) {
  constexpr int GM = 8;
  const int nx = PAIR == PAIR_NONE ? (p.N + GBN - 1) / GBN : (PAIR == PAIR_N ? p.N / 128 : p.N / 256);
  const int ny = (p.M + GBM - 1) / GBM;
  const int total = nx * ny * p.batch * p.splits;
  const int per = (total + 7) / 8;
  const int t = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (t >= total) return false;
  const int tz = nx * ny;
  bz = t / tz;
  const int tt = t - bz * tz;
  const int grp = tt / (GM * nx);
  const int m0 = grp * GM;
  const int gm = min(GM, ny - m0);
  const int r = tt - grp * GM * nx;
  by = m0 + r % gm;
  bx = r / gm;
  return true;
}

template <int EPI>
__global__ __launch_bounds__(512) void gemm_big(GemmArgs p) {
  using T = bf16_t;
  constexpr int PAIR = EpiPair<EPI>::value;
  __shared__ __attribute__((aligned(16))) unsigned char st0[GSTAGE];
  __shared__ __attribute__((aligned(16))) unsigned char st1[GSTAGE];

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int wm = wave >> 2, wn = wave & 3;
  int bx, by, bz;
  if (!big_tile<PAIR>(p, bx, by, bz)) return;
  const int z = bz / p.splits, split = bz % p.splits;
  const int m0 = by * GBM;
  int n0, pair_off;
  if constexpr (PAIR == PAIR_HEAD) {
    const int half = p.qkv.head_dim >> 1, per_head = half / 128;
    const int h = bx / per_head;
    n0 = h * p.qkv.head_dim + (bx - h * per_head) * 128;
    pair_off = half;
  } else if constexpr (PAIR == PAIR_N) {
    n0 = bx * 128;
    pair_off = p.N;
  } else {
    n0 = bx * GBN;
    pair_off = 0;
  }
  const int kbeg = split * p.k_per_split;
  const int kend = min(p.K, kbeg + p.k_per_split);
  const int nst = (kend - kbeg) / DST;

  const T* A = reinterpret_cast<const T*>(p.A) + (int64_t)z * p.a_bstride;
  const T* B = reinterpret_cast<const T*>(p.B) + (int64_t)z * p.b_bstride;

  // DMA: wave w, instruction j covers stage rows 8*(4w + (j & 3)) + (lane >> 3)
  // of A (j < 4) or B (j >= 4): 8 waves x 4 x 8 = 256 rows of each; physical
  // chunk lane & 7 holds logical chunk (lane & 7) ^ swizzle(row)
  const T* gsrc[8];
  {
    const int rr = lane >> 3, pc = lane & 7;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = 8 * (4 * wave + (j & 3)) + rr;
      const int lc = pc ^ RFX_GSWZ(row);
      if (j < 4) {
        gsrc[j] = A + (int64_t)min(m0 + row, p.M - 1) * p.lda + kbeg + lc * 8;
      } else {
        int brw;
        if (PAIR != PAIR_NONE) {
          const int c = n0 + (row & 127);
          brw = row >= 128 ? c + pair_off : c;
        } else {
          brw = min(n0 + row, p.N - 1);
        }
        gsrc[j] = B + (int64_t)brw * p.ldb + kbeg + lc * 8;
      }
    }
  }
  auto issue = [&](int st, unsigned char* buf) __attribute__((always_inline)) {
    const int k0 = st * DST;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = 8 * (4 * wave + (j & 3));
      __builtin_amdgcn_global_load_lds(gsrc[j] + k0, buf + ((j >= 4 ? GBM : 0) + row) * DROWB, 16, 0, 0);
    }
  };

  f32x4_v acc[8][4];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  int foff[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) foff[kk] = r16 * DROWB + ((4 * kk + g) ^ RFX_GSWZ(r16)) * 16;
  int brow_l[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    if (PAIR != PAIR_NONE)
      brow_l[nb] = (nb < 2 ? 0 : 128) + wn * 32 + (nb & 1) * 16;
    else
      brow_l[nb] = wn * 64 + nb * 16;
  }

  auto step = [&](int st, const unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt)
                  __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0): this wave's share of stage st
    // every wave's share is in LDS, and every wave is done with stage st-1,
    // whose buffer the next copy overwrites
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (st + 1 < nst) issue(st + 1, nxt);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      uint4 bf[4];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        bf[nb] = *reinterpret_cast<const uint4*>(cur + (GBM + brow_l[nb]) * DROWB + foff[kk]);
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        const uint4 af = *reinterpret_cast<const uint4*>(cur + (wm * 128 + mb * 16) * DROWB + foff[kk]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) mfma_step(acc[mb][nb], bf[nb], af, T());  // C^T blocks
      }
    }
  };

  if (nst > 0) issue(0, st0);
  for (int st = 0; st < nst; st += 2) {
    step(st, st0, st1);
    if (st + 1 < nst) step(st + 1, st1, st0);
  }

  // acc[mb][nb]: lane (r16, g) holds output row m0 + wm*128 + mb*16 + r16,
  // columns 4g .. 4g+3 of column block nb
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) {
    const int grow = m0 + wm * 128 + mb * 16 + r16;
    if (grow >= p.M) continue;
    if (PAIR != PAIR_NONE) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int gcol = n0 + wn * 32 + nb * 16 + 4 * g;
        const float v[4] = {acc[mb][nb][0], acc[mb][nb][1], acc[mb][nb][2], acc[mb][nb][3]};
        const float u[4] = {acc[mb][nb + 2][0], acc[mb][nb + 2][1], acc[mb][nb + 2][2], acc[mb][nb + 2][3]};
        epilogue_store4<EPI>(p, z, split, grow, gcol, v, u);
      }
    } else {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int gcol = n0 + wn * 64 + nb * 16 + 4 * g;
        const float v[4] = {acc[mb][nb][0], acc[mb][nb][1], acc[mb][nb][2], acc[mb][nb][3]};
        if (gcol + 3 < p.N) {
          epilogue_store4<EPI>(p, z, split, grow, gcol, v, v);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (gcol + e < p.N) epilogue_store<EPI, T>(p, z, split, grow, gcol + e, v[e], 0.f);
        }
      }
    }
  }
}

// --------------------------------------------------------------------------
// 256x256 tile with 32-element K stages: 32 KB per stage, five stages (the
// whole 160 KB of LDS) and four copies in flight.  With 64-element stages
// only one 64 KB copy is in flight per CU while a stage is computed, and the
// copy latency, not the bandwidth, sets the pace.  A 64-byte stage row holds
// four 16-byte chunks; chunk c of row r sits at c ^ ((r >> 2) & 3), so the 16
// rows a fragment read touches with one chunk each fall on distinct banks.
// NST (stages per workgroup) is a compile-time constant and the stage loop
// fully unrolled, so the compiler knows which buffer every copy in flight
// targets and does not wait for all copies before reading LDS.
// --------------------------------------------------------------------------
constexpr int HROWB = 64;                       // bytes per stage row
constexpr int HSTAGE = (GBM + GBN) * HROWB;     // 32 KB
#define RFX_HSWZ(r) (((r) >> 2) & 3)

template <int EPI, int NST>
__global__ __launch_bounds__(512) void gemm_big5(GemmArgs p) {
  using T = bf16_t;
  constexpr int PAIR = EpiPair<EPI>::value;
  constexpr int NS = 5;
  __shared__ __attribute__((aligned(16))) unsigned char st0[HSTAGE];
  __shared__ __attribute__((aligned(16))) unsigned char st1[HSTAGE];
  __shared__ __attribute__((aligned(16))) unsigned char st2[HSTAGE];
  __shared__ __attribute__((aligned(16))) unsigned char st3[HSTAGE];
  __shared__ __attribute__((aligned(16))) unsigned char st4[HSTAGE];

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int wm = wave >> 2, wn = wave & 3;
  int bx, by, bz;
  if (!big_tile<PAIR>(p, bx, by, bz)) return;
  const int z = bz / p.splits, split = bz % p.splits;
  const int m0 = by * GBM;
  int n0, pair_off;
  if constexpr (PAIR == PAIR_HEAD) {
    const int half = p.qkv.head_dim >> 1, per_head = half / 128;
    const int h = bx / per_head;
    n0 = h * p.qkv.head_dim + (bx - h * per_head) * 128;
    pair_off = half;
  } else if constexpr (PAIR == PAIR_N) {
    n0 = bx * 128;
    pair_off = p.N;
  } else {
    n0 = bx * GBN;
    pair_off = 0;
  }
  const int kbeg = split * p.k_per_split;

  const T* A = reinterpret_cast<const T*>(p.A) + (int64_t)z * p.a_bstride;
  const T* B = reinterpret_cast<const T*>(p.B) + (int64_t)z * p.b_bstride;

  // DMA: wave w, instruction j covers stage rows 16*(2w + (j & 1)) + (lane >> 2)
  // of A (j < 2) or B (j >= 2): 8 waves x 2 x 16 = 256 rows of each; physical
  // chunk lane & 3 holds logical chunk (lane & 3) ^ swizzle(row)
  const T* gsrc[4];
  {
    const int rr = lane >> 2, pc = lane & 3;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = 16 * (2 * wave + (j & 1)) + rr;
      const int lc = pc ^ RFX_HSWZ(row);
      if (j < 2) {
        gsrc[j] = A + (int64_t)min(m0 + row, p.M - 1) * p.lda + kbeg + lc * 8;
      } else {
        int brw;
        if (PAIR != PAIR_NONE) {
          const int c = n0 + (row & 127);
          brw = row >= 128 ? c + pair_off : c;
        } else {
          brw = min(n0 + row, p.N - 1);
        }
        gsrc[j] = B + (int64_t)brw * p.ldb + kbeg + lc * 8;
      }
    }
  }
  auto issue = [&](int st, unsigned char* buf) __attribute__((always_inline)) {
    const int k0 = st * 32;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = 16 * (2 * wave + (j & 1));
      __builtin_amdgcn_global_load_lds(gsrc[j] + k0, buf + ((j >= 2 ? GBM : 0) + row) * HROWB, 16, 0, 0);
    }
  };

  f32x4_v acc[8][4];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  // fragment rows are 16-aligned, so the swizzle of row r16 + 16i is that of r16
  const int foff = r16 * HROWB + (g ^ RFX_HSWZ(r16)) * 16;
  int brow_l[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    if (PAIR != PAIR_NONE)
      brow_l[nb] = (nb < 2 ? 0 : 128) + wn * 32 + (nb & 1) * 16;
    else
      brow_l[nb] = wn * 64 + nb * 16;
  }

  auto step = [&](int st, const unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt)
                  __attribute__((always_inline)) {
    // stage st is complete once at most (stages issued after it) x 4 of this
    // wave's copies are outstanding
    const int after = (st + NS - 2 < NST ? st + NS - 2 : NST - 1) - st;
    if (after >= 3)
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8) | 12);
    else if (after == 2)
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8) | 8);
    else if (after == 1)
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8) | 4);
    else
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
    // every wave's share of stage st is in LDS, and every wave is done with
    // stage st-1, whose buffer the next copy overwrites
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (st + NS - 1 < NST) issue(st + NS - 1, nxt);
    uint4 bf[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      bf[nb] = *reinterpret_cast<const uint4*>(cur + (GBM + brow_l[nb]) * HROWB + foff);
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const uint4 af = *reinterpret_cast<const uint4*>(cur + (wm * 128 + mb * 16) * HROWB + foff);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) mfma_step(acc[mb][nb], bf[nb], af, T());  // C^T blocks
    }
  };

  unsigned char* const bufs[NS] = {st0, st1, st2, st3, st4};
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < NST) issue(st, bufs[st]);
#pragma unroll
  for (int st = 0; st < NST; ++st) step(st, bufs[st % NS], bufs[(st + NS - 1) % NS]);

#pragma unroll
  for (int mb = 0; mb < 8; ++mb) {
    const int grow = m0 + wm * 128 + mb * 16 + r16;
    if (grow >= p.M) continue;
    if (PAIR != PAIR_NONE) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int gcol = n0 + wn * 32 + nb * 16 + 4 * g;
        const float v[4] = {acc[mb][nb][0], acc[mb][nb][1], acc[mb][nb][2], acc[mb][nb][3]};
        const float u[4] = {acc[mb][nb + 2][0], acc[mb][nb + 2][1], acc[mb][nb + 2][2], acc[mb][nb + 2][3]};
        epilogue_store4<EPI>(p, z, split, grow, gcol, v, u);
      }
    } else {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int gcol = n0 + wn * 64 + nb * 16 + 4 * g;
        const float v[4] = {acc[mb][nb][0], acc[mb][nb][1], acc[mb][nb][2], acc[mb][nb][3]};
        epilogue_store4<EPI>(p, z, split, grow, gcol, v, v);
      }
    }
  }
}

// --------------------------------------------------------------------------
// host side
// --------------------------------------------------------------------------
static int skinny_mb(int M) { return M <= 16 ? 1 : (M <= 32 ? 2 : 4); }

int gemm_pick_splits(int M, int N, int K, int elem_bytes) {
  const int ks = 64 / elem_bytes;
  if (M <= 64) {
    const int cols = 32;
    const int base = (N + cols - 1) / cols;
    int maxs = K / (ks * 4 * 2);  // at least two k-steps per wave
    if (maxs < 1) maxs = 1;
    int s = (256 + base - 1) / base;
    if (s > 8) s = 8;
    return s < 1 ? 1 : (s > maxs ? maxs : s);
  }
  const int base = ((N + TBN - 1) / TBN) * ((M + TBM - 1) / TBM);
  if (elem_bytes == 2) {
    // bf16 tiled path: the largest power-of-two split that keeps one wave of
    // workgroups (<= 256, one per CU for the four-stage pipeline) and at
    // least 8 stages of 64 per split
    int s = 1;
    while (base * s * 2 <= 256 && K % (64 * s * 2) == 0 && K / (s * 2) >= 512) s *= 2;
    // the same with 64-row tiles (which the launcher takes when they fit one
    // wave): fewer splits, so fewer fp32 partials for the residual to read,
    // if every split's K range is still a four-stage count of at most 16
    // stages (a 32-stage loop on 64-row tiles, 8 accumulators per wave, was
    // slower than two splits on 128-row tiles).  Down projection at 8 envs:
    // 4 splits instead of 8.
    const int base64 = ((N + TBN - 1) / TBN) * ((M + 63) / 64);
    int s64 = 1;
    while (base64 * s64 * 2 <= 256 && K % (64 * s64 * 2) == 0 && K / (s64 * 2) >= 512) s64 *= 2;
    const int nst64 = K % (64 * s64) == 0 ? K / (64 * s64) : 0;
    if (s64 < s && (nst64 == 8 || nst64 == 16)) s = s64;
    return s;
  }
  if (base >= 256 || K < 1024) return 1;
  int s = (256 + base - 1) / base;
  const int maxs = K / 512;
  return s > maxs ? maxs : s;
}

template <typename T, int MB, int EPI>
static void launch_skinny_cfg(const GemmArgs& a, hipStream_t s) {
  constexpr int PAIR = EpiPair<EPI>::value;
  constexpr int NB = PAIR ? 1 : 2;
  int nx;
  if (PAIR == PAIR_HEAD)
    nx = a.N / 32;  // (N / head_dim) heads x (head_dim/2 / 16) strips
  else if (PAIR == PAIR_N)
    nx = a.N / 16;
  else
    nx = (a.N + 16 * NB - 1) / (16 * NB);
  const int mch = (a.M + 16 * MB - 1) / (16 * MB);
  dim3 grid(nx, mch * a.splits, a.batch);
  // eight waves when a workgroup's K range has at least 32 k-steps: every
  // wave then issues all its loads in one round trip
  const int ks = 64 / (int)sizeof(T);
  if (a.k_per_split >= 32 * ks && a.K >= 32 * ks)
    RFX_LAUNCH((gemm_skinny<T, MB, NB, EPI, 8>), grid, dim3(512), 0, s, a);
  else
    RFX_LAUNCH((gemm_skinny<T, MB, NB, EPI, 4>), grid, dim3(256), 0, s, a);
}

// dynamic LDS above the default 64 KB limit must be allowed per kernel, once
template <typename K>
static void allow_large_lds(K kernel) {
  static const hipError_t once =
      hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  (void)once;
}

template <int MB, int EPI>
static void launch_skinny_lds_pick(const GemmArgs& a, hipStream_t s) {
  constexpr int PAIR = EpiPair<EPI>::value;
  constexpr int NB = PAIR ? 1 : 2;
  // eight waves when every wave gets at least two k-steps
  const int nw = a.k_per_split >= 16 * 32 ? 8 : 4;
  if (nw == 8)
    allow_large_lds(gemm_skinny_lds<MB, NB, EPI, 8>);
  else
    allow_large_lds(gemm_skinny_lds<MB, NB, EPI, 4>);
  launch_skinny_lds_cfg<MB, EPI>(a, s, nw);
}

template <typename T, int EPI>
static void launch_skinny(const GemmArgs& a, hipStream_t s) {
  // bf16 with the activation K range fitting in LDS: stage it there
  const int klen = a.k_per_split < a.K ? a.k_per_split : a.K;  // LDS holds one split's K range
  if (sizeof(T) == 2 && (size_t)16 * skinny_mb(a.M) * ((klen * 2 + 127) & ~127) <= 160 * 1024 &&
      a.k_per_split % 32 == 0 &&
      a.K % 32 == 0) {
    // an unsplit GEMM with few column strips (QKV at one env: 80) takes its
    // rows in two 32-row halves: twice the workgroups, each copying half the
    // activation rows; both halves of a strip land on the same XCD (nx is a
    // multiple of 8), so its weights come from HBM once
    constexpr int PAIR = EpiPair<EPI>::value;
    const int nx = PAIR == PAIR_HEAD ? a.N / 32 : (PAIR == PAIR_N ? a.N / 16 : (a.N + 31) / 32);
    if (skinny_mb(a.M) == 4 && a.splits == 1 && nx < 128 && nx % 8 == 0) {
      launch_skinny_lds_pick<2, EPI>(a, s);
      return;
    }
    switch (skinny_mb(a.M)) {
      case 1: launch_skinny_lds_pick<1, EPI>(a, s); return;
      case 2: launch_skinny_lds_pick<2, EPI>(a, s); return;
      default: launch_skinny_lds_pick<4, EPI>(a, s); return;
    }
  }
  switch (skinny_mb(a.M)) {
    case 1: launch_skinny_cfg<T, 1, EPI>(a, s); break;
    case 2: launch_skinny_cfg<T, 2, EPI>(a, s); break;
    default: launch_skinny_cfg<T, 4, EPI>(a, s); break;
  }
}

template <typename T, int EPI>
static void launch_tiled(const GemmArgs& a, hipStream_t s) {
  constexpr int PAIR = EpiPair<EPI>::value;
  const int nx = PAIR == PAIR_NONE ? (a.N + TBN - 1) / TBN : a.N / (PAIR == PAIR_N ? 64 : 128);
  dim3 grid(nx, (a.M + TBM - 1) / TBM, a.batch * a.splits);
  // (vector epilogue stores: output rows start 16-byte aligned)
  if (sizeof(T) == 2 && a.K % DST == 0 && a.k_per_split % DST == 0 && a.N % 4 == 0 && a.ldo % 4 == 0) {
    const int total = grid.x * grid.y * grid.z;
    // 256x256 tiles when there are at least 512 rows and the large tiles
    // alone give at least half a wave of workgroups
    const bool pair_ok = (PAIR == PAIR_NONE && a.N % GBN == 0) || (PAIR == PAIR_N && a.N % 128 == 0) ||
                         (PAIR == PAIR_HEAD && (a.qkv.head_dim / 2) % 128 == 0);
    const int bx = PAIR == PAIR_NONE ? (a.N + GBN - 1) / GBN : (PAIR == PAIR_N ? a.N / 128 : a.N / 256);
    const int btotal = bx * ((a.M + GBM - 1) / GBM) * a.batch * a.splits;
    if (pair_ok && a.M >= 512 && btotal >= 128 && a.k_per_split / DST >= 8) {
      const dim3 g((btotal + 7) / 8 * 8);
      // K range of every split (one split may be given a range past K)
      const int kr = a.splits == 1 ? a.K : (a.K == a.k_per_split * a.splits ? a.k_per_split : 0);
      if (kr == 1024)
        RFX_LAUNCH((gemm_big5<EPI, 32>), g, dim3(512), 0, s, a);
      else if (kr == 2048)
        RFX_LAUNCH((gemm_big5<EPI, 64>), g, dim3(512), 0, s, a);
      else
        RFX_LAUNCH((gemm_big<EPI>), g, dim3(512), 0, s, a);
      return;
    }
    // four-stage unrolled pipeline (one workgroup per CU) when one wave of
    // workgroups covers the grid; else the two-stage one (two per CU).  The
    // stage count is that of every split's K range (a single split may be
    // given a range past K: its range is then K).
    const int kr1 = a.splits == 1 ? a.K : (a.K == a.k_per_split * a.splits ? a.k_per_split : 0);
    const int nst = kr1 % DST == 0 ? kr1 / DST : 0;
    // just over one wave of 128-row tiles with a 16-stage K range: 160-row
    // tiles on the four-stage pipeline when they fit one wave, one per CU
    // (QKV at 32 envs: 220 workgroups instead of 340 96-row ones two per CU,
    // 23.5 -> 21.2 us; the two-stage 160-row kernel took 26.6 us), with two
    // waves per output block (21.8 -> 18.3 us)
    const int total160 = nx * ((a.M + 159) / 160) * a.batch * a.splits;
    if (total > 256 && total160 <= 256 && nst == 16) {
      RFX_LAUNCH((gemm_dma<EPI, 4, 16, 160, false, 2>), dim3((total160 + 7) / 8 * 8), dim3(512), 0, s, a);
      return;
    }
    if (total > 256) {
      // just over one wave of 128-row tiles: 96-row tiles, two per CU, when
      // they fit in two waves' worth (the busiest CU then holds 2 x 96 rows
      // instead of 2 x 128)
      const int total96 = nx * ((a.M + 95) / 96) * a.batch * a.splits;
      if (total <= 512 && total96 <= 512)
        RFX_LAUNCH((gemm_dma<EPI, 2, 0, 96>), dim3((total96 + 7) / 8 * 8), dim3(256), 0, s, a);
      else
        RFX_LAUNCH((gemm_dma<EPI, 2, 0>), dim3((total + 7) / 8 * 8), dim3(256), 0, s, a);
    } else if (nst == 8 || nst == 16 || nst == 32) {
      // 64-row tiles when even those stay within one wave of workgroups:
      // more CUs, each with half the K loop's work (QKV at 8 envs: 140
      // workgroups instead of 80)
      const int total64 = nx * ((a.M + 63) / 64) * a.batch * a.splits;
      const dim3 g64((total64 + 7) / 8 * 8), g128((total + 7) / 8 * 8);
      const bool t64 = total64 <= 256;
      // 64-row tiles with a paired epilogue (RoPE, gated GELU, K/V scatter)
      // run two waves per output block, as the 160-row tiles do: the QKV of
      // the long context 11.7 -> 11.1 us; with the fp32 epilogue it was not
      // faster
      constexpr int KE = (EPI == EPI_ROPE || EPI == EPI_GELU || EPI == EPI_KV) ? 2 : 1;
      if (nst == 8) {
        if (t64) RFX_LAUNCH((gemm_dma<EPI, 4, 8, 64, false, KE>), g64, dim3(256 * KE), 0, s, a);
        else RFX_LAUNCH((gemm_dma<EPI, 4, 8, 128, true>), g128, dim3(256), 0, s, a);
      } else if (nst == 16) {
        if (t64) RFX_LAUNCH((gemm_dma<EPI, 4, 16, 64, false, KE>), g64, dim3(256 * KE), 0, s, a);
        else RFX_LAUNCH((gemm_dma<EPI, 4, 16, 128, true>), g128, dim3(256), 0, s, a);
      } else {
        if (t64) RFX_LAUNCH((gemm_dma<EPI, 4, 32, 64, false, KE>), g64, dim3(256 * KE), 0, s, a);
        else RFX_LAUNCH((gemm_dma<EPI, 4, 32>), g128, dim3(256), 0, s, a);
      }
    } else {
      RFX_LAUNCH((gemm_dma<EPI, 2, 0>), dim3((total + 7) / 8 * 8), dim3(256), 0, s, a);
    }
  }
  else
    RFX_LAUNCH((gemm_tiled<T, EPI>), grid, dim3(256), 0, s, a);
}

template <typename T, int EPI>
static void launch_pick(const GemmArgs& a, hipStream_t s) {
  bool skinny = a.M <= 64;
  // paired tiles of the tiled kernel hold 64 first-half columns of one head
  if ((EPI == EPI_ROPE || EPI == EPI_KV) && a.qkv.head_dim < 128) skinny = true;
  if (skinny)
    launch_skinny<T, EPI>(a, s);
  else
    launch_tiled<T, EPI>(a, s);
}

template <typename T>
hipError_t launch_gemm(const GemmArgs& a, int epi, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return hipErrorInvalidValue;
  if (epi == EPI_GELU && a.N % 64) return hipErrorInvalidValue;
  if ((epi == EPI_ROPE || epi == EPI_KV) && (a.qkv.head_dim % 64 || a.N % a.qkv.head_dim))
    return hipErrorInvalidValue;
  if (epi == EPI_KV && (a.N % (2 * a.qkv.head_dim) || a.M % a.kv.F)) return hipErrorInvalidValue;
  if (epi != EPI_F32 && a.splits != 1) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_F32: launch_pick<T, EPI_F32>(a, s); break;
    case EPI_MOD: launch_pick<T, EPI_MOD>(a, s); break;
    case EPI_SILU: launch_pick<T, EPI_SILU>(a, s); break;
    case EPI_GELU: launch_pick<T, EPI_GELU>(a, s); break;
    case EPI_ROPE: launch_pick<T, EPI_ROPE>(a, s); break;
    case EPI_KV: launch_pick<T, EPI_KV>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_gemm<float>(const GemmArgs&, int, hipStream_t);
template hipError_t launch_gemm<bf16_t>(const GemmArgs&, int, hipStream_t);

}  // namespace reflex
