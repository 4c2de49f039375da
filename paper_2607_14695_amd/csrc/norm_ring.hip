// Row kernels of the denoise step and the cache writers:
//  * token embedding fused with the first AdaRMSNorm,
//  * residual update fused with the next AdaRMSNorm (it also sums the split-K
//    partials of the producing projection, so those GEMMs need no reduction),
//  * the last residual + final AdaRMSNorm + action head + Euler update,
//  * RoPE (cos, sin) tables with angles formed in double,
//  * conditioning rows [sinusoidal(tau_k); state] for the modulation MLPs,
//  * the ring / static-prefix writer (RoPE on K, V stored transposed).
//
// AdaRMSNorm (Eq. 2, Section 3.2): y = x * rsqrt(mean(x^2) + eps) * (1 + scale)
// + shift with the mean of squares accumulated in fp32 (the paper's mixed-
// precision guardrail); h stays fp32, y is rounded once to the GEMM operand
// type.  One workgroup per row: one read of h, one write of h and y.
#include "common.h"
#include "kernels.h"

namespace reflex {

// 4 consecutive elements as fp32 (8-byte bf16 or 16-byte fp32 load)
RFX_DEV float4 ld4f(const float* p) { return *reinterpret_cast<const float4*>(p); }
RFX_DEV float4 ld4f(const bf16_t* p) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                     __uint_as_float(v.y & 0xffff0000u));
}
RFX_DEV void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
RFX_DEV void st4(bf16_t* p, float4 v) {
  uint2 w;
  w.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
  w.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
  *reinterpret_cast<uint2*>(p) = w;
}
RFX_DEV float4 f4add(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }

// sum of nparts split-K partial rows in index order.  The loads of a group
// of G partials are all issued before any is added, so up to G partials cost
// one memory round trip (a loop with a dynamic trip count would wait for each
// group's loads before issuing the next).
template <int G>
RFX_DEV float4 sum_parts_g(const float* pp, int64_t stride, int nparts) {
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < nparts; s0 += G) {
    float4 a[G];
#pragma unroll
    for (int i = 0; i < G; ++i) a[i] = ld4f(pp + (int64_t)min(s0 + i, nparts - 1) * stride);  // clamped: valid, unused
#pragma unroll
    for (int i = 0; i < G; ++i)
      if (s0 + i < nparts) acc = f4add(acc, a[i]);
  }
  return acc;
}
RFX_DEV float4 sum_parts(const float* pp, int64_t stride, int nparts) {
  if (nparts <= 2) return sum_parts_g<2>(pp, stride, nparts);
  if (nparts <= 4) return sum_parts_g<4>(pp, stride, nparts);
  return sum_parts_g<8>(pp, stride, nparts);
}

// bf16 rounding of an fp32 value (round to nearest even), kept in fp32
RFX_DEV float rbf(float x) { return bf2f(f2bf(x)); }
RFX_DEV float4 rbf4(float4 v) { return make_float4(rbf(v.x), rbf(v.y), rbf(v.z), rbf(v.w)); }

// sum of squares of 4 values added to ss: fp32, or bf16 arithmetic with every
// product and every partial sum rounded
RFX_DEV float add_ssq(float ss, float4 v, bool bf) {
  if (!bf) return ss + v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  ss = rbf(ss + rbf(v.x * v.x));
  ss = rbf(ss + rbf(v.y * v.y));
  ss = rbf(ss + rbf(v.z * v.z));
  return rbf(ss + rbf(v.w * v.w));
}

// Block sum of the 256 per-thread partials and the inverse RMS 1/sqrt(ss/D +
// eps).  In bf16 arithmetic every partial sum, the mean and the result are
// rounded.
RFX_DEV float inv_rms(float ss, int D, float eps, bool bf, float* red) {
  if (!bf) return rsqrtf(block_sum_256(ss, red) / (float)D + eps);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss = rbf(ss + __shfl_xor(ss, off, 64));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  const float tot = rbf(rbf(red[0] + red[1]) + rbf(red[2] + red[3]));
  return rbf(rsqrtf(rbf(rbf(tot / (float)D) + eps)));
}

// y = v * r * (1 + scale) + shift for 4 columns
RFX_DEV float4 ada4(float4 v, float r, float4 sc, float4 sh) {
  return make_float4(v.x * r * (1.f + sc.x) + sh.x, v.y * r * (1.f + sc.y) + sh.y, v.z * r * (1.f + sc.z) + sh.z,
                     v.w * r * (1.f + sc.w) + sh.w);
}

// ---------------------------------------------------------------------------
// embedding + first norm: row m = b*T + t; t = 0 is the state token
// ---------------------------------------------------------------------------
// h = embed_scale * W in and y = ada(h) for token row m = b*T + t (t = 0:
// the state through W_s, else an action through W_ain), its n_in inputs
// already in LDS (`in`, visible to every thread).  hs: D floats of LDS; red:
// 4 floats of LDS for the norm's block reduction.  Shared by the embedding
// kernel and the final kernel's next-step epilogue.
// GROUPED: a thread issues the weight loads of up to 32 inputs (16 in fp32)
// of its four columns before it uses any (one L2 round trip per round, not
// per column and group of inputs).  Taken for a few rows; with many rows the
// per-column form keeps more rows resident (batch 32: 13.6 against 17.8 us
// for an earlier grouped form).  Each column sums its inputs in order, one
// group of four at a time (for a multiple of 8 inputs, the same arithmetic
// either way).
template <typename T, bool GROUPED>
RFX_DEV void embed_row(const EmbedArgs& p, int64_t m, int b, int t, const float* in, float* hs, float* red) {
  const int n_in = (t == 0) ? p.ds : p.da;
  const T* W = reinterpret_cast<const T*>(t == 0 ? p.w_state : p.w_ain);
  float ss = 0.f;
  if constexpr (GROUPED) {
    constexpr int CH = 64 / (int)sizeof(T);  // inputs per round of loads: 32 bf16 / 16 fp32
    for (int cb = 0; cb < p.D; cb += 1024) {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      const T* w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)  // clamped column: a valid address, result unused
        w[u] = W + (int64_t)min(cb + (int)threadIdx.x + 256 * u, p.D - 1) * n_in;
      if ((n_in & 3) == 0) {
        // every load of a round is issued before any is used; the sum adds
        // one group of four inputs at a time, in input order
        for (int e0 = 0; e0 < n_in; e0 += CH) {
          float4 wv[4][CH / 4];
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < CH / 4; ++j) wv[u][j] = ld4f(w[u] + min(e0 + 4 * j, n_in - 4));  // clamped: unused
#pragma unroll
          for (int j = 0; j < CH / 4; ++j) {
            const int e = e0 + 4 * j;
            if (e < n_in) {
#pragma unroll
              for (int u = 0; u < 4; ++u)
                acc[u] += wv[u][j].x * in[e] + wv[u][j].y * in[e + 1] + wv[u][j].z * in[e + 2] + wv[u][j].w * in[e + 3];
            }
          }
        }
      } else {
        for (int e = 0; e < n_in; ++e)
#pragma unroll
          for (int u = 0; u < 4; ++u) acc[u] += to_f(w[u][e]) * in[e];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb + threadIdx.x + 256 * u;
        if (c < p.D) {
          float v = acc[u] * p.embed_scale;
          if (p.norm_mode != NORM_FP32) v = rbf(v);  // bf16 residual stream
          hs[c] = v;
          ss = add_ssq(ss, make_float4(v, 0.f, 0.f, 0.f), p.norm_mode == NORM_BF16);
        }
      }
    }
  } else {
    for (int c = threadIdx.x; c < p.D; c += 256) {
      const T* w = W + (int64_t)c * n_in;
      float acc = 0.f;
      int e = 0;
      if ((n_in & 3) == 0) {
        for (; e + 8 <= n_in; e += 8) {
          const float4 w0 = ld4f(w + e), w1 = ld4f(w + e + 4);
          acc += w0.x * in[e] + w0.y * in[e + 1] + w0.z * in[e + 2] + w0.w * in[e + 3];
          acc += w1.x * in[e + 4] + w1.y * in[e + 5] + w1.z * in[e + 6] + w1.w * in[e + 7];
        }
      }
      for (; e < n_in; ++e) acc += to_f(w[e]) * in[e];
      acc *= p.embed_scale;
      if (p.norm_mode != NORM_FP32) acc = rbf(acc);  // bf16 residual stream
      hs[c] = acc;
      ss = add_ssq(ss, make_float4(acc, 0.f, 0.f, 0.f), p.norm_mode == NORM_BF16);
    }
  }
  const float r = inv_rms(ss, p.D, p.eps, p.norm_mode == NORM_BF16, red);
  const float* mod = p.mod + (int64_t)b * 3 * p.D;
  for (int c = threadIdx.x; c < p.D; c += 256) {
    p.h[(int64_t)m * p.D + c] = hs[c];
    const float xr = p.norm_mode == NORM_BF16 ? rbf(hs[c] * r) : hs[c] * r;
    const float y = xr * (1.f + mod[c]) + mod[p.D + c];
    reinterpret_cast<T*>(p.y)[(int64_t)m * p.D + c] = from_f<T>(y);
  }
}

template <typename T, bool GROUPED>
__global__ __launch_bounds__(256) void embed_norm_kernel(EmbedArgs p) {
  __shared__ float red[4];
  __shared__ float in[64];
  __shared__ float hs[16 * 256];
  const int m = blockIdx.x, b = m / p.T, t = m % p.T;
  const int n_in = (t == 0) ? p.ds : p.da;
  const float* src = (t == 0) ? p.state + (int64_t)b * p.ds : p.x + ((int64_t)b * (p.T - 1) + (t - 1)) * p.da;
  if (threadIdx.x < n_in) in[threadIdx.x] = src[threadIdx.x];
  __syncthreads();
  embed_row<T, GROUPED>(p, m, b, t, in, hs, red);
}

template <typename T>
hipError_t launch_embed_norm(const EmbedArgs& a, hipStream_t s) {
  if (a.D > 16 * 256 || a.ds > 64 || a.da > 64) return hipErrorInvalidValue;
  if (a.B * a.T <= 256)
    RFX_LAUNCH((embed_norm_kernel<T, true>), dim3(a.B * a.T), dim3(256), 0, s, a);
  else
    RFX_LAUNCH((embed_norm_kernel<T, false>), dim3(a.B * a.T), dim3(256), 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// residual + norm: one block per row, 4 columns per thread
// ---------------------------------------------------------------------------
template <typename T, int MAXC>  // MAXC 4-column chunks per thread: D <= 1024 * MAXC
__global__ __launch_bounds__(256) void resid_norm_kernel(ResidArgs p) {
  __shared__ float red[4];
  const int m = blockIdx.x, b = m / p.T;
  const float* gmod = p.gate_mod + (int64_t)b * 3 * p.D + 2 * p.D;
  const float* nmod = p.norm_mod + (int64_t)b * 3 * p.D;
  const int D4 = p.D >> 2;
  // everything this thread needs, the next site's scale and shift included,
  // is loaded before the row reduction: one memory round trip per row
  float4 v[MAXC], sc[MAXC], sh[MAXC];
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < MAXC; ++u) {
    const int c4 = threadIdx.x + 256 * u;
    if (c4 < D4) {
      const int c = c4 * 4;
      sc[u] = ld4f(nmod + c);
      sh[u] = ld4f(nmod + p.D + c);
      const float4 h = ld4f(p.h + (int64_t)m * p.D + c);
      const float4 gt = ld4f(gmod + c);
      const float4 acc = sum_parts(p.parts + (int64_t)m * p.D + c, p.part_stride, p.nparts);
      v[u] = make_float4(h.x + gt.x * acc.x, h.y + gt.y * acc.y, h.z + gt.z * acc.z, h.w + gt.w * acc.w);
      if (p.norm_mode != NORM_FP32) v[u] = rbf4(v[u]);  // bf16 residual stream
      ss = add_ssq(ss, v[u], p.norm_mode == NORM_BF16);
      st4(p.h + (int64_t)m * p.D + c, v[u]);
    }
  }
  const float r = inv_rms(ss, p.D, p.eps, p.norm_mode == NORM_BF16, red);
#pragma unroll
  for (int u = 0; u < MAXC; ++u) {
    const int c4 = threadIdx.x + 256 * u;
    if (c4 < D4) {
      const float4 x = v[u];
      const float4 y = p.norm_mode == NORM_BF16
                           ? ada4(rbf4(make_float4(x.x * r, x.y * r, x.z * r, x.w * r)), 1.f, sc[u], sh[u])
                           : ada4(x, r, sc[u], sh[u]);
      st4(reinterpret_cast<T*>(p.y) + (int64_t)m * p.D + c4 * 4, y);
    }
  }
}

template <typename T>
hipError_t launch_resid_norm(const ResidArgs& a, hipStream_t s) {
  if (a.D > 16 * 256 || (a.D & 3)) return hipErrorInvalidValue;
  // registers for only as many column chunks as the row needs
  if (a.D <= 1024)
    RFX_LAUNCH((resid_norm_kernel<T, 1>), dim3(a.M), dim3(256), 0, s, a);
  else if (a.D <= 2048)
    RFX_LAUNCH((resid_norm_kernel<T, 2>), dim3(a.M), dim3(256), 0, s, a);
  else
    RFX_LAUNCH((resid_norm_kernel<T, 4>), dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// last residual + final norm + action head + Euler: one block per action row.
// With fuse_next the kernel also starts the next Euler step: each action
// row's block embeds its new x and applies the next step's first norm (the
// embedding kernel's work for that row, in its grouped form), and one more
// block per env, after the action rows, does the same for the state token.
// The action rows read only their own h row, so writing it afterwards races
// with no other block.  Taken for a few rows only (final_fuses_embed: the
// launch-bound regime); at 32 envs the separate embedding kernel measured
// faster, and the other variants stay without the embedding's registers.
// ---------------------------------------------------------------------------
// GU: action-head weight loads a thread issues before using any; FUSE: the
// variant with the next step's embedding (p.fuse_next decides per launch)
template <typename T, int MAXC, int GU, bool FUSE>  // MAXC 4-column chunks per thread: D <= 1024 * MAXC
__global__ __launch_bounds__(256) void final_euler_kernel(FinalArgs p) {
  __shared__ float red[4];
  __shared__ float red2[4];
  __shared__ float xin[64];
  __shared__ float4 ys[4 * 256];
  __shared__ float vpart[4][64];
  const int H = p.T - 1;
  if (FUSE && blockIdx.x >= p.B * H) {  // the next step's state row of env b
    const int b = blockIdx.x - p.B * H;
    if (threadIdx.x < p.next.ds) xin[threadIdx.x] = p.next.state[(int64_t)b * p.next.ds + threadIdx.x];
    __syncthreads();
    embed_row<T, true>(p.next, (int64_t)b * p.T, b, 0, xin, reinterpret_cast<float*>(ys), red2);
    return;
  }
  const int b = blockIdx.x / H, i = blockIdx.x % H;
  const int64_t m = (int64_t)b * p.T + 1 + i;
  const float* gmod = p.gate_mod + (int64_t)b * 3 * p.D + 2 * p.D;
  const float* fmod = p.final_mod + (int64_t)b * 3 * p.D;
  const int D4 = p.D >> 2;
  float4 sc[MAXC], sh[MAXC];
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < MAXC; ++u) {
    const int c4 = threadIdx.x + 256 * u;
    if (c4 < D4) {
      const int c = c4 * 4;
      sc[u] = ld4f(fmod + c);  // loaded with the residual inputs: one round trip
      sh[u] = ld4f(fmod + p.D + c);
      const float4 h = ld4f(p.h + m * p.D + c);
      const float4 gt = ld4f(gmod + c);
      const float4 acc = sum_parts(p.parts + m * p.D + c, p.part_stride, p.nparts);
      float4 v = make_float4(h.x + gt.x * acc.x, h.y + gt.y * acc.y, h.z + gt.z * acc.z, h.w + gt.w * acc.w);
      if (p.norm_mode != NORM_FP32) v = rbf4(v);  // bf16 residual stream
      ys[c4] = v;
      ss = add_ssq(ss, v, p.norm_mode == NORM_BF16);
    }
  }
  const float r = inv_rms(ss, p.D, p.eps, p.norm_mode == NORM_BF16, red);
#pragma unroll
  for (int u = 0; u < MAXC; ++u) {
    const int c4 = threadIdx.x + 256 * u;
    if (c4 < D4) {
      const float4 v = ys[c4];
      ys[c4] = p.norm_mode == NORM_BF16
                   ? ada4(rbf4(make_float4(v.x * r, v.y * r, v.z * r, v.w * r)), 1.f, sc[u], sh[u])
                   : ada4(v, r, sc[u], sh[u]);
    }
  }
  __syncthreads();
  // v[a] = sum_c y[c] W[a][c]: eight threads per output, each a strided
  // eighth of the columns; the partial sums meet in three xor shuffles.  A
  // thread issues GU weight loads before it uses any (one L2 round trip per
  // GU columns instead of per column); the sum runs in column order.
  const T* W = reinterpret_cast<const T*>(p.w_aout);
  const int part = threadIdx.x & 7;
  for (int a0 = 0; a0 < p.da; a0 += 32) {
    const int a = a0 + (threadIdx.x >> 3);
    const int ar = a < p.da ? a : p.da - 1;  // clamped row: a valid address, result unused
    float acc = 0.f;
    for (int c0 = part; c0 < D4; c0 += 8 * GU) {
      float4 w[GU];
#pragma unroll
      for (int u = 0; u < GU; ++u) {
        const int c4 = min(c0 + 8 * u, D4 - 1);  // clamped column: a valid address, result unused
        w[u] = ld4f(W + (int64_t)ar * p.D + c4 * 4);
      }
#pragma unroll
      for (int u = 0; u < GU; ++u) {
        const int c4 = c0 + 8 * u;
        if (c4 < D4) {
          const float4 y = ys[c4];
          acc += w[u].x * y.x + w[u].y * y.y + w[u].z * y.z + w[u].w * y.w;
        }
      }
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    acc += __shfl_xor(acc, 4, 64);
    if (part == 0 && a < p.da) vpart[0][a] = acc;
  }
  __syncthreads();
  const int64_t xo = ((int64_t)b * H + i) * p.da;
  for (int a = threadIdx.x; a < p.da; a += 256) {
    const float x = p.x_in[xo + a] + p.dt * vpart[0][a];
    p.x_out[xo + a] = x;
    xin[a] = x;
    if (!__builtin_isfinite(x)) atomicOr(p.status, 1);
  }
  if (!FUSE || !p.fuse_next) return;
  __syncthreads();  // xin complete; every read of ys is done
  embed_row<T, true>(p.next, m, b, 1 + i, xin, reinterpret_cast<float*>(ys), red2);
}

bool final_fuses_embed(int B, int T, int D) { return B * T <= 256 && D <= 1024; }

template <typename T>
hipError_t launch_final_euler(const FinalArgs& a, hipStream_t s) {
  if (a.D > 16 * 256 || (a.D & 3) || a.da > 64) return hipErrorInvalidValue;
  if (a.fuse_next && (!final_fuses_embed(a.B, a.T, a.D) || a.next.D != a.D || a.next.B != a.B ||
                      a.next.T != a.T || a.next.da != a.da || a.next.ds > 64 || a.next.h != a.h))
    return hipErrorInvalidValue;
  // a few rows: every weight load of a thread in flight at once (32 for
  // D = 1024); many rows: groups of 8, fewer registers, more rows resident
  const dim3 grid(a.B * (a.T - 1));
  if (a.fuse_next)
    RFX_LAUNCH((final_euler_kernel<T, 1, 32, true>), dim3(a.B * a.T), dim3(256), 0, s, a);
  else if (a.D <= 1024 && grid.x <= 256)
    RFX_LAUNCH((final_euler_kernel<T, 1, 32, false>), grid, dim3(256), 0, s, a);
  else if (a.D <= 1024)
    RFX_LAUNCH((final_euler_kernel<T, 1, 8, false>), grid, dim3(256), 0, s, a);
  else if (a.D <= 2048)
    RFX_LAUNCH((final_euler_kernel<T, 2, 8, false>), grid, dim3(256), 0, s, a);
  else
    RFX_LAUNCH((final_euler_kernel<T, 4, 8, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// RoPE table: out[i][f] = (cos, sin)((pos0 + i) * theta^(-2f/d)), double angles
// ---------------------------------------------------------------------------
__global__ void rope_table_kernel(float2* out, const int64_t* pos0_dev, int64_t pos0, int n, int half,
                                  double theta) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * half) return;
  const int i = idx / half, f = idx % half;
  const int64_t base = pos0_dev ? *pos0_dev : pos0;
  const double inv = pow(theta, -2.0 * (double)f / (double)(2 * half));
  const double ang = (double)(base + i) * inv;
  double sn, cs;
  sincos(ang, &sn, &cs);
  out[idx] = make_float2((float)cs, (float)sn);
}

hipError_t launch_rope_table(float2* out, const int64_t* pos0_dev, int64_t pos0, int n, int head_dim,
                             double theta, hipStream_t s) {
  const int half = head_dim / 2;
  const int tot = n * half;
  if (tot <= 0) return hipSuccess;
  RFX_LAUNCH(rope_table_kernel, dim3((tot + 255) / 256), dim3(256), 0, s, out, pos0_dev, pos0, n, half,
                     theta);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// conditioning rows
// ---------------------------------------------------------------------------
template <typename T>
__global__ void cond_kernel(T* cond, const float* state, TauTable taus, int B, int D, int ds, double min_p,
                            double max_p) {
  const int row = blockIdx.x;  // k*B + b
  const int k = row / B, b = row % B;
  const int half = D / 2;
  const int C = D + ds;
  const double tau = (double)taus.tau[k];
  for (int c = threadIdx.x; c < C; c += blockDim.x) {
    float v;
    if (c < D) {
      const int i = c < half ? c : c - half;
      const double frac = half > 1 ? (double)i / (double)(half - 1) : 0.0;
      const double period = min_p * pow(max_p / min_p, frac);
      const double ang = 6.283185307179586 * tau / period;
      v = (float)(c < half ? sin(ang) : cos(ang));
    } else {
      v = state[(int64_t)b * ds + (c - D)];
    }
    cond[(int64_t)row * C + c] = from_f<T>(v);
  }
}

template <typename T>
hipError_t launch_cond(void* cond, const float* state, const TauTable& taus, int K, int B, int D, int ds,
                       double min_p, double max_p, hipStream_t s) {
  RFX_LAUNCH((cond_kernel<T>), dim3(K * B), dim3(256), 0, s, reinterpret_cast<T*>(cond), state, taus,
                     B, D, ds, min_p, max_p);
  return hipGetLastError();
}

__global__ void zero_kernel(uint4* p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  if (((uintptr_t)p & 15) || (bytes & 15)) return hipErrorInvalidValue;
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  RFX_LAUNCH(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, reinterpret_cast<uint4*>(p), n16);
  return hipGetLastError();
}

__global__ void tick_set_kernel(int64_t* tick, int64_t frames, int64_t n_valid, int64_t dyn_pos0,
                                int64_t hole_row) {
  if (threadIdx.x == 0) {
    tick[0] = frames;
    tick[1] = n_valid;
    tick[2] = dyn_pos0;
    tick[3] = hole_row;
  }
}

hipError_t launch_tick_set(int64_t* tick, int64_t frames, int64_t n_valid, int64_t dyn_pos0, int64_t hole_row,
                           hipStream_t s) {
  RFX_LAUNCH(tick_set_kernel, dim3(1), dim3(64), 0, s, tick, frames, n_valid, dyn_pos0, hole_row);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// ring / static writer.  Block = (64-token tile, layer, env).
// K: cache_k[b][l][row0 + j][d] = rope(k_j)[d]
// V: cache_vt[b][l][d][row0 + j] = v_j[d]   (transposed through LDS)
// ---------------------------------------------------------------------------
template <typename T, typename S, int DH>
__global__ __launch_bounds__(256) void ring_write_kernel(RingWriteArgs p) {
  constexpr int TJ = 32;  // tokens per block
  __shared__ float vt[TJ][DH + 1];
  const int j0 = blockIdx.x * TJ, l = blockIdx.y, b = blockIdx.z;
  if (p.tick && blockIdx.x == 0 && l == 0 && b == 0 && threadIdx.x == 0) {
    p.tick[0] = p.frames_written;
    p.tick[1] = (int64_t)p.n_valid;
    p.tick[2] = p.dyn_pos0;
    p.tick[3] = p.hole_row;
  }
  const S* sk = reinterpret_cast<const S*>(p.src_k) + (int64_t)b * p.sb + (int64_t)l * p.sl;
  const S* sv = reinterpret_cast<const S*>(p.src_v) + (int64_t)b * p.sb + (int64_t)l * p.sl;
  T* ck = reinterpret_cast<T*>(p.cache_k) + ((int64_t)b * p.L + l) * (int64_t)p.R * DH;
  T* cv = reinterpret_cast<T*>(p.cache_vt) + ((int64_t)b * p.L + l) * (int64_t)p.R * DH;
  const int ntok = min(TJ, p.n_tok - j0);
  constexpr int H2 = DH / 2;
  // vector accesses (4 elements per load, 8 tokens per V^T store) when every
  // base and stride they touch is aligned for them; else element by element.
  // The arithmetic per element is the same either way.
  const uintptr_t amask = (uintptr_t)(4 * sizeof(S)) - 1;
  const bool vec = (((uintptr_t)sk | (uintptr_t)sv) & amask) == 0 && (p.sj & 3) == 0 &&
                   (((uintptr_t)p.rope) & 15) == 0 && (((uintptr_t)ck | (uintptr_t)cv) & (8 * sizeof(T) - 1)) == 0 &&
                   (p.row0 & 7) == 0 && (p.R & 7) == 0;
  // K with RoPE: pairs (f, f + DH/2)
  if (vec) {
    for (int e = threadIdx.x; e < ntok * (H2 / 4); e += 256) {
      const int jj = e / (H2 / 4), f = (e % (H2 / 4)) * 4;
      const int j = j0 + jj;
      const S* src = sk + (int64_t)j * p.sj;
      const float4 lo = ld4f(src + f), hi = ld4f(src + f + H2);
      const float4* csp = reinterpret_cast<const float4*>(p.rope + (int64_t)j * H2 + f);
      const float4 c01 = csp[0], c23 = csp[1];  // (cos, sin) of f, f+1 and of f+2, f+3
      T* dst = ck + (int64_t)(p.row0 + j) * DH;
      st4(dst + f, make_float4(lo.x * c01.x - hi.x * c01.y, lo.y * c01.z - hi.y * c01.w, lo.z * c23.x - hi.z * c23.y,
                               lo.w * c23.z - hi.w * c23.w));
      st4(dst + f + H2, make_float4(hi.x * c01.x + lo.x * c01.y, hi.y * c01.z + lo.y * c01.w,
                                    hi.z * c23.x + lo.z * c23.y, hi.w * c23.z + lo.w * c23.w));
    }
  } else {
    for (int e = threadIdx.x; e < ntok * H2; e += 256) {
      const int jj = e / H2, f = e % H2;
      const int j = j0 + jj;
      const S* src = sk + (int64_t)j * p.sj;
      const float lo = to_f(src[f]), hi = to_f(src[f + H2]);
      const float2 cs = p.rope[(int64_t)j * H2 + f];
      T* dst = ck + (int64_t)(p.row0 + j) * DH;
      dst[f] = from_f<T>(lo * cs.x - hi * cs.y);
      dst[f + H2] = from_f<T>(hi * cs.x + lo * cs.y);
    }
  }
  // V transposed through LDS
  if (vec) {
    for (int e = threadIdx.x; e < ntok * (DH / 4); e += 256) {
      const int jj = e / (DH / 4), d = (e % (DH / 4)) * 4;
      const float4 v = ld4f(sv + (int64_t)(j0 + jj) * p.sj + d);
      vt[jj][d] = v.x;
      vt[jj][d + 1] = v.y;
      vt[jj][d + 2] = v.z;
      vt[jj][d + 3] = v.w;
    }
  } else {
    for (int e = threadIdx.x; e < ntok * DH; e += 256) {
      const int jj = e / DH, d = e % DH;
      vt[jj][d] = to_f(sv[(int64_t)(j0 + jj) * p.sj + d]);
    }
  }
  __syncthreads();
  if (vec && ntok == TJ) {
    // eight consecutive tokens of one d per thread
    for (int e = threadIdx.x; e < DH * (TJ / 8); e += 256) {
      const int d = e / (TJ / 8), j8 = (e % (TJ / 8)) * 8;
      T* dst = cv + (int64_t)d * p.R + p.row0 + j0 + j8;
      st4(dst, make_float4(vt[j8][d], vt[j8 + 1][d], vt[j8 + 2][d], vt[j8 + 3][d]));
      st4(dst + 4, make_float4(vt[j8 + 4][d], vt[j8 + 5][d], vt[j8 + 6][d], vt[j8 + 7][d]));
    }
  } else {
    for (int e = threadIdx.x; e < ntok * DH; e += 256) {
      const int d = e / ntok, jj = e % ntok;
      cv[(int64_t)d * p.R + p.row0 + j0 + jj] = from_f<T>(vt[jj][d]);
    }
  }
}

template <typename T, typename S>
hipError_t launch_ring_write(const RingWriteArgs& a, int head_dim, hipStream_t s) {
  dim3 grid((a.n_tok + 31) / 32, a.L, a.B);
  switch (head_dim) {
    case 64: RFX_LAUNCH((ring_write_kernel<T, S, 64>), grid, dim3(256), 0, s, a); break;
    case 128: RFX_LAUNCH((ring_write_kernel<T, S, 128>), grid, dim3(256), 0, s, a); break;
    case 256: RFX_LAUNCH((ring_write_kernel<T, S, 256>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_embed_norm<float>(const EmbedArgs&, hipStream_t);
template hipError_t launch_embed_norm<bf16_t>(const EmbedArgs&, hipStream_t);
template hipError_t launch_resid_norm<float>(const ResidArgs&, hipStream_t);
template hipError_t launch_resid_norm<bf16_t>(const ResidArgs&, hipStream_t);
template hipError_t launch_final_euler<float>(const FinalArgs&, hipStream_t);
template hipError_t launch_final_euler<bf16_t>(const FinalArgs&, hipStream_t);
template hipError_t launch_cond<float>(void*, const float*, const TauTable&, int, int, int, int, double, double,
                                       hipStream_t);
template hipError_t launch_cond<bf16_t>(void*, const float*, const TauTable&, int, int, int, int, double, double,
                                        hipStream_t);
template hipError_t launch_ring_write<float, float>(const RingWriteArgs&, int, hipStream_t);
template hipError_t launch_ring_write<bf16_t, bf16_t>(const RingWriteArgs&, int, hipStream_t);
template hipError_t launch_ring_write<bf16_t, float>(const RingWriteArgs&, int, hipStream_t);

}  // namespace reflex
