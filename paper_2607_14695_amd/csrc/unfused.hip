// Unfused passes for the operator-fusion ablation (Section 4.6, "Operator
// Fusion Impact").  The fused schedule applies RoPE and the gated GELU in the
// projection epilogues, adds the residual inside the norm kernel and the Euler
// update inside the action head; here each of those runs as its own kernel
// that reads its input from and writes its result to HBM.  The arithmetic is
// the same as in the fused kernels.
#include "common.h"
#include "kernels.h"

namespace reflex {

namespace {
RFX_DEV float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
}  // namespace

__global__ __launch_bounds__(256) void resid_add_kernel(ResidAddArgs p) {
  const int m = blockIdx.x, b = m / p.T;
  const float* gmod = p.gate_mod + (int64_t)b * 3 * p.D + 2 * p.D;
  for (int c = threadIdx.x * 4; c < p.D; c += 1024) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < p.nparts; ++s) {
      const float4 v = ld4(p.parts + s * p.part_stride + (int64_t)m * p.D + c);
      acc = make_float4(acc.x + v.x, acc.y + v.y, acc.z + v.z, acc.w + v.w);
    }
    float* h = p.h + (int64_t)m * p.D + c;
    const float4 hv = ld4(h), g = ld4(gmod + c);
    *reinterpret_cast<float4*>(h) =
        make_float4(hv.x + g.x * acc.x, hv.y + g.y * acc.y, hv.z + g.z * acc.z, hv.w + g.w * acc.w);
  }
}

hipError_t launch_resid_add(const ResidAddArgs& a, hipStream_t s) {
  if (a.D & 3) return hipErrorInvalidValue;
  RFX_LAUNCH(resid_add_kernel, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void norm_kernel(NormArgs p) {
  __shared__ float red[4];
  const int m = blockIdx.x, b = m / p.T;
  const float* h = p.h + (int64_t)m * p.D;
  float ss = 0.f;
  for (int c = threadIdx.x; c < p.D; c += 256) ss += h[c] * h[c];
  const float r = rsqrtf(block_sum_256(ss, red) / (float)p.D + p.eps);
  const float* mod = p.norm_mod + (int64_t)b * 3 * p.D;
  for (int c = threadIdx.x; c < p.D; c += 256)
    reinterpret_cast<T*>(p.y)[(int64_t)m * p.D + c] = from_f<T>(h[c] * r * (1.f + mod[c]) + mod[p.D + c]);
}

template <typename T>
hipError_t launch_norm(const NormArgs& a, hipStream_t s) {
  RFX_LAUNCH((norm_kernel<T>), dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void rope_scatter_kernel(RopeScatterArgs p) {
  const QkvOut& q = p.out;
  const int m = blockIdx.x, b = m / q.T, i = m - b * q.T;
  const int dh = q.head_dim, half = dh / 2, ncols = (q.Hq + 2) * dh;
  const float* row = p.qkv + (int64_t)m * ncols;
  // q heads and the k head: rotate-half pairs (f, f + half)
  for (int e = threadIdx.x; e < (q.Hq + 1) * half; e += 256) {
    const int head = e / half, f = e - head * half;
    const float lo = row[head * dh + f], hi = row[head * dh + f + half];
    const float2 cs = q.rope[i * half + f];
    T* dst = head < q.Hq ? reinterpret_cast<T*>(q.q) + ((int64_t)b * q.rows_pad + i * q.Hq + head) * dh
                         : reinterpret_cast<T*>(q.k) + ((int64_t)b * q.T + i) * dh;
    dst[f] = from_f<T>(lo * cs.x - hi * cs.y);
    dst[f + half] = from_f<T>(hi * cs.x + lo * cs.y);
  }
  // the v head, stored transposed (column i of [dh][tpad])
  T* vt = reinterpret_cast<T*>(q.vt) + (int64_t)b * dh * q.tpad;
  for (int d = threadIdx.x; d < dh; d += 256) vt[(int64_t)d * q.tpad + i] = from_f<T>(row[(q.Hq + 1) * dh + d]);
}

template <typename T>
hipError_t launch_rope_scatter(const RopeScatterArgs& a, hipStream_t s) {
  RFX_LAUNCH((rope_scatter_kernel<T>), dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void gelu_mul_kernel(GeluMulArgs p) {
  const int m = blockIdx.x;
  const float* u = p.u + (int64_t)m * 2 * p.F;
  for (int c = threadIdx.x; c < p.F; c += 256)
    reinterpret_cast<T*>(p.z)[(int64_t)m * p.F + c] = from_f<T>(gelu_tanh(u[c]) * u[p.F + c]);
}

template <typename T>
hipError_t launch_gelu_mul(const GeluMulArgs& a, hipStream_t s) {
  RFX_LAUNCH((gelu_mul_kernel<T>), dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

__global__ void euler_kernel(EulerArgs p) {
  const int H = p.T - 1;
  const int row = blockIdx.x, b = row / H, i = row - b * H;  // action row i of env b
  for (int a = threadIdx.x; a < p.da; a += blockDim.x) {
    const int64_t xo = ((int64_t)b * H + i) * p.da + a;
    p.x_out[xo] = p.x_in[xo] + p.dt * p.v[((int64_t)b * p.T + 1 + i) * p.da + a];
  }
}

hipError_t launch_euler(const EulerArgs& a, hipStream_t s) {
  RFX_LAUNCH(euler_kernel, dim3(a.B * (a.T - 1)), dim3(64), 0, s, a);
  return hipGetLastError();
}

template hipError_t launch_norm<float>(const NormArgs&, hipStream_t);
template hipError_t launch_norm<bf16_t>(const NormArgs&, hipStream_t);
template hipError_t launch_rope_scatter<float>(const RopeScatterArgs&, hipStream_t);
template hipError_t launch_rope_scatter<bf16_t>(const RopeScatterArgs&, hipStream_t);
template hipError_t launch_gelu_mul<float>(const GeluMulArgs&, hipStream_t);
template hipError_t launch_gelu_mul<bf16_t>(const GeluMulArgs&, hipStream_t);

}  // namespace reflex
