// MFMA GEMMs for the dense projections of the action expert: packed QKV,
// output projection, packed gate|up with the gated-GELU epilogue, down
// projection, the conditioning MLPs and the frame K/V projection
// (Section 3.4 "Operator Fusion": packed W_QKV and packed gate/up).
//
// C[M][N] = A[M][K] * B[N][K]^T, both operands K-contiguous, fp32 accumulate.
//
// Two regimes:
//  * gemm_skinny (M <= 64): weight streaming.  At one environment the
//    activations are 51 rows while every weight byte is read once per Euler
//    step, so the kernel is bound by HBM bandwidth on the weights.  A workgroup
//    owns a 16- or 32-column strip and a K range; its four waves interleave
//    k-steps so that, per weight row, the wave group reads 256 contiguous
//    bytes per round; fragments go straight from global memory into MFMA
//    operands (no LDS staging: every weight byte is used by all rows in the
//    same instruction).  The four waves' partial tiles are summed through LDS.
//    K may be split across workgroups; the split partials are summed by the
//    consumer kernel (attention for QKV, the residual/norm kernel for the
//    output and down projections), so no atomics and no extra launch.
//  * gemm_tiled (M > 64): 128x128 workgroup tiles, 2x2 waves of 64x64, two
//    k-steps (128 bytes of K per row) per LDS stage, double-buffered LDS with
//    the next stage's global loads in flight during the MFMAs.
#include "common.h"
#include "kernels.h"

namespace reflex {

template <int EPI, typename T>
RFX_DEV void epilogue_store(const GemmArgs& p, int z, int split, int row, int col, float v, float u) {
  if (EPI == EPI_F32 || EPI == EPI_MOD) {
    if (EPI == EPI_MOD && p.mod_width > 0 && col >= p.mod_width) v = (col < 2 * p.mod_width) ? 0.f : 1.f;
    float* o = reinterpret_cast<float*>(p.out) + (int64_t)z * p.o_bstride +
               (int64_t)split * p.o_split_stride + (int64_t)row * p.ldo + col;
    *o = v;
  } else {
    T* o = reinterpret_cast<T*>(p.out) + (int64_t)z * p.o_bstride + (int64_t)row * p.ldo + col;
    if (EPI == EPI_SILU)
      *o = from_f<T>(silu(v));
    else
      *o = from_f<T>(gelu_tanh(v) * u);
  }
}

// --------------------------------------------------------------------------
// skinny: M <= 16*MB rows per workgroup chunk, NB 16-col blocks per strip
// --------------------------------------------------------------------------
template <typename T, int MB, int NB, bool DUAL, int EPI>
__global__ __launch_bounds__(256) void gemm_skinny(GemmArgs p) {
  constexpr int KPF = ElemT<T>::kPerFrag;
  constexpr int KS = 4 * KPF;             // elements per k-step
  constexpr int NBT = DUAL ? 2 * NB : NB; // B fragments per k-step
  constexpr int COLS = 16 * NB;           // output columns per workgroup
  constexpr int RCOLS = 16 * NBT + 1;     // LDS reduction row (padded)
  __shared__ float red[4][MB * 16][RCOLS];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int z = blockIdx.z;
  const int mchunk = blockIdx.y / p.splits, split = blockIdx.y % p.splits;
  const int m0 = mchunk * (16 * MB), n0 = blockIdx.x * COLS;
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
    const int c = min(n0 + (nb % NB) * 16 + r16, p.N - 1);
    const int brw = (DUAL && nb >= NB) ? p.N + c : c;
    brow[nb] = B + (int64_t)brw * p.ldb + g * KPF;
  }

  f32x4_v acc[MB][NBT];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb) acc[mb][nb] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  const int nsteps = (kend - kbeg + KS - 1) / KS;
  constexpr int U = 2;
  for (int s0 = wave; s0 < nsteps; s0 += 4 * U) {
    uint4 bf[U][NBT], af[U][MB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kbeg + (s0 + 4 * u) * KS;
      const bool ok = (s0 + 4 * u < nsteps) && (k + g * KPF < kend);
#pragma unroll
      for (int nb = 0; nb < NBT; ++nb) bf[u][nb] = ok ? ld16(brow[nb] + k) : zero16();
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) af[u][mb] = ok ? ld16(arow[mb] + k) : zero16();
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBT; ++nb) mfma_step(acc[mb][nb], af[u][mb], bf[u][nb], T());
  }

#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBT; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][mb * 16 + 4 * g + i][nb * 16 + r16] = acc[mb][nb][i];
  __syncthreads();

  for (int e = threadIdx.x; e < MB * 16 * COLS; e += 256) {
    const int row = e / COLS, col = e % COLS;
    const int grow = m0 + row, gcol = n0 + col;
    if (grow >= p.M || gcol >= p.N) continue;
    float v = red[0][row][col] + red[1][row][col] + red[2][row][col] + red[3][row][col];
    float u = 0.f;
    if (DUAL) u = red[0][row][col + COLS] + red[1][row][col + COLS] + red[2][row][col + COLS] +
                  red[3][row][col + COLS];
    epilogue_store<EPI, T>(p, z, split, grow, gcol, v, u);
  }
}

// --------------------------------------------------------------------------
// tiled: 128 x 128 workgroup tile (DUAL: 128 rows x 64 gate + 64 up columns)
// --------------------------------------------------------------------------
constexpr int TBM = 128, TBN = 128, TROWB = 128, TPAD = 16;  // bytes of K per stage row

template <typename T, bool DUAL, int EPI>
__global__ __launch_bounds__(256) void gemm_tiled(GemmArgs p) {
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
  const int ncols = DUAL ? TBN / 2 : TBN;  // output columns per tile
  const int n0 = blockIdx.x * ncols;
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
    if (DUAL) {
      const int c = min(n0 + (r & 63), p.N - 1);
      brw = (r >= 64) ? p.N + c : c;
    } else {
      brw = min(n0 + r, p.N - 1);
    }
    gb[i] = B + (int64_t)brw * p.ldb + ch * KPF;
  }
  uint4 ra[4], rb[4];
  auto gload = [&](int st) {
    const int k = kbeg + st * KSTAGE + ch * KPF;
    const bool ok = k < kend;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = ok ? ld16(ga[i] + (k - ch * KPF)) : zero16();
      rb[i] = ok ? ld16(gb[i] + (k - ch * KPF)) : zero16();
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (tid >> 3) + 32 * i;
      st16(&As[buf][r * LROW + ch * 16], ra[i]);
      st16(&Bs[buf][r * LROW + ch * 16], rb[i]);
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
    if (DUAL)
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
      if (DUAL) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int gcol = n0 + wn * 32 + nb * 16 + r16;
          if (gcol < p.N) epilogue_store<EPI, T>(p, z, split, grow, gcol, acc[mb][nb][i], acc[mb][nb + 2][i]);
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
// host side
// --------------------------------------------------------------------------
static int skinny_mb(int M) { return M <= 16 ? 1 : (M <= 32 ? 2 : 4); }

int gemm_pick_splits(int M, int N, int K, int elem_bytes) {
  const int ks = 64 / elem_bytes;
  if (M <= 64) {
    const int cols = 32;  // two 16-column blocks per strip
    const int base = (N + cols - 1) / cols;
    int maxs = K / (ks * 4);
    if (maxs < 1) maxs = 1;
    int s = (512 + base - 1) / base;
    return s < 1 ? 1 : (s > maxs ? maxs : s);
  }
  const int base = ((N + TBN - 1) / TBN) * ((M + TBM - 1) / TBM);
  if (base >= 256 || K < 1024) return 1;
  int s = (256 + base - 1) / base;
  const int maxs = K / 512;
  return s > maxs ? maxs : s;
}

template <typename T, int MB, bool DUAL, int EPI>
static void launch_skinny_cfg(const GemmArgs& a, hipStream_t s) {
  constexpr int NB = DUAL ? 1 : 2;
  const int cols = 16 * NB;
  const int mch = (a.M + 16 * MB - 1) / (16 * MB);
  dim3 grid((a.N + cols - 1) / cols, mch * a.splits, a.batch);
  RFX_LAUNCH((gemm_skinny<T, MB, NB, DUAL, EPI>), grid, dim3(256), 0, s, a);
}

template <typename T, bool DUAL, int EPI>
static void launch_skinny(const GemmArgs& a, hipStream_t s) {
  switch (skinny_mb(a.M)) {
    case 1: launch_skinny_cfg<T, 1, DUAL, EPI>(a, s); break;
    case 2: launch_skinny_cfg<T, 2, DUAL, EPI>(a, s); break;
    default: launch_skinny_cfg<T, 4, DUAL, EPI>(a, s); break;
  }
}

template <typename T, bool DUAL, int EPI>
static void launch_tiled(const GemmArgs& a, hipStream_t s) {
  const int ncols = DUAL ? TBN / 2 : TBN;
  dim3 grid((a.N + ncols - 1) / ncols, (a.M + TBM - 1) / TBM, a.batch * a.splits);
  RFX_LAUNCH((gemm_tiled<T, DUAL, EPI>), grid, dim3(256), 0, s, a);
}

template <typename T>
hipError_t launch_gemm(const GemmArgs& a, int epi, hipStream_t s) {
  const bool skinny = a.M <= 64;
  switch (epi) {
    case EPI_F32:
      skinny ? launch_skinny<T, false, EPI_F32>(a, s) : launch_tiled<T, false, EPI_F32>(a, s);
      break;
    case EPI_MOD:
      skinny ? launch_skinny<T, false, EPI_MOD>(a, s) : launch_tiled<T, false, EPI_MOD>(a, s);
      break;
    case EPI_SILU:
      skinny ? launch_skinny<T, false, EPI_SILU>(a, s) : launch_tiled<T, false, EPI_SILU>(a, s);
      break;
    case EPI_GELU:
      skinny ? launch_skinny<T, true, EPI_GELU>(a, s) : launch_tiled<T, true, EPI_GELU>(a, s);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_gemm<float>(const GemmArgs&, int, hipStream_t);
template hipError_t launch_gemm<bf16_t>(const GemmArgs&, int, hipStream_t);

}  // namespace reflex
