// Device-side helpers shared by the gfx950 kernels: storage types, bf16
// rounding, 16-byte fragments and the MFMA steps built on them.
//
// Fragment convention (CDNA3/CDNA4 16x16 MFMA): a wave multiplies a 16-row
// A block by a 16-column B block.  Lane l supplies row (l & 15) of A and
// column (l & 15) of B, each as one 16-byte "fragment" of consecutive
// contraction elements starting at element 4*(l >> 4) (fp32) or 8*(l >> 4)
// (bf16) of the current k-step.  A k-step therefore covers 64 bytes of every
// row: 32 bf16 (one v_mfma_f32_16x16x32_bf16) or 16 fp32 (four
// v_mfma_f32_16x16x4_f32, element t of every lane in the t-th instruction).
// The 16x16 fp32 result sits in lane l as rows 4*(l >> 4) + i, column (l & 15).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace reflex {

typedef uint16_t bf16_t;  // bfloat16 bit pattern
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;
typedef __attribute__((ext_vector_type(4))) float f32x4_v;
typedef __attribute__((ext_vector_type(16))) float f32x16_v;

#define RFX_DEV __device__ __forceinline__

RFX_DEV float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float -> bf16, round to nearest even (inputs are finite or inf; NaN kept NaN)
RFX_DEV bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> struct ElemT;
template <> struct ElemT<float> {
  static constexpr int kPerFrag = 4;  // elements per 16-byte fragment
  static RFX_DEV float to_f(float v) { return v; }
  static RFX_DEV float from_f(float v) { return v; }
};
template <> struct ElemT<bf16_t> {
  static constexpr int kPerFrag = 8;
  static RFX_DEV float to_f(bf16_t v) { return bf2f(v); }
  static RFX_DEV bf16_t from_f(float v) { return f2bf(v); }
};

template <typename T> RFX_DEV float to_f(T v) { return ElemT<T>::to_f(v); }
template <typename T> RFX_DEV T from_f(float v) { return ElemT<T>::from_f(v); }

// One k-step of a 16x16 MFMA tile from two 16-byte fragments.
RFX_DEV void mfma_step(f32x4_v& acc, const uint4& a, const uint4& b, bf16_t) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_v, a),
                                                __builtin_bit_cast(bf16x8_v, b), acc, 0, 0, 0);
}
RFX_DEV void mfma_step(f32x4_v& acc, const uint4& a, const uint4& b, float) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// One 32x32x16 bf16 MFMA: lane l supplies row / column (l & 31) and the 8
// contraction elements 8*(l >> 5) + [0, 8); the 32x32 fp32 result sits in lane
// l as rows 8*(q >> 2) + 4*(l >> 5) + (q & 3), q < 16, column (l & 31).
RFX_DEV void mfma32_step(f32x16_v& acc, const uint4& a, const uint4& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_v, a), __builtin_bit_cast(bf16x8_v, b), acc,
                                                0, 0, 0);
}

RFX_DEV uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
RFX_DEV void st16(void* p, const uint4& v) { *reinterpret_cast<uint4*>(p) = v; }
RFX_DEV uint4 zero16() { return make_uint4(0u, 0u, 0u, 0u); }

// Pack/unpack 16-byte fragments to/from fp32 values.
RFX_DEV void frag_to_f(const uint4& v, float* out, float) {
  out[0] = __uint_as_float(v.x); out[1] = __uint_as_float(v.y);
  out[2] = __uint_as_float(v.z); out[3] = __uint_as_float(v.w);
}
RFX_DEV void frag_to_f(const uint4& v, float* out, bf16_t) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(w[i] << 16);
    out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
RFX_DEV uint4 f_to_frag(const float* in, float) {
  return make_uint4(__float_as_uint(in[0]), __float_as_uint(in[1]), __float_as_uint(in[2]),
                    __float_as_uint(in[3]));
}
RFX_DEV uint4 f_to_frag(const float* in, bf16_t) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = (uint32_t)f2bf(in[2 * i]) | ((uint32_t)f2bf(in[2 * i + 1]) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

RFX_DEV float warp_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum over the 256 threads of a block; `red` needs 4 floats of shared memory.
RFX_DEV float block_sum_256(float v, float* red) {
  v = warp_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// GELU, tanh approximation: 0.5 u (1 + tanh(y)), y = sqrt(2/pi) (u + 0.044715 u^3).
// Evaluated in the equivalent logistic form u / (1 + exp(-2y)) (tanh(y) =
// 2 sigma(2y) - 1) with the hardware exp2 and reciprocal: relative error a few
// ulp; large |y| gives u or -0 without overflow trouble (1 + inf -> rcp 0).
RFX_DEV float gelu_tanh(float u) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float y = k0 * (u + 0.044715f * u * u * u);
  const float e = __builtin_amdgcn_exp2f(-2.0f * 1.4426950408889634f * y);  // exp(-2y)
  return u * __builtin_amdgcn_rcpf(1.0f + e);
}
RFX_DEV float silu(float u) { return u / (1.0f + __expf(-u)); }

}  // namespace reflex
