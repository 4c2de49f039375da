// Partitioned-region attention (Eq. 1, Section 3.1) for the dynamic rows.
//
// For every env, the T dynamic tokens x Hq query heads form T*Hq query rows
// that all read the single shared K/V head (multi-query).  The key sequence is
// [cached rows 0..Lc) ++ [dynamic rows 0..T), Lc = static_len +
// n_valid*frame_tokens read from device memory, so the same launch serves
// every tick.  Softmax is permutation-invariant over keys, so ring slots are
// read in physical order; the result equals one softmax over the concatenated
// context (Appendix A, Proposition A.1).
//
// Decomposition: blockIdx = (key split, 64-row query block, env).  A split
// owns a contiguous range of 64-key tiles; the dynamic tile comes last.  Each
// tile's K rows and V^T columns are staged in LDS once and reused by all 64
// query rows of the block (4 waves x 16 rows).
//
// Per wave the scores are computed transposed, S^T = K Q^T, with MFMA (A = K
// rows, B = the wave's 16 query rows held in registers).  In that layout each
// lane holds, for its query row, 4 consecutive keys of every 16-key block, so
// exp(S^T - m) is already the B operand of O^T = V^T P^T: the probabilities
// never leave registers.  V is stored transposed (d-major) in the cache so the
// A operand V^T[d][keys] is a contiguous LDS read.  Online softmax in base 2;
// row max / sum cross the 4 lane groups with two xor shuffles.
//
// With more than one split each block writes (O unnormalised, m, l) and a
// merge kernel combines the splits with log-sum-exp weights.
#include "common.h"
#include "kernels.h"

namespace reflex {

constexpr int AKT = 64;  // keys per tile

template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs p) {
  constexpr int ES = (int)sizeof(T);
  constexpr int KPF = ElemT<T>::kPerFrag;
  constexpr int KSD = 4 * KPF;       // head-dim elements per k-step
  constexpr int NKS = DH / KSD;      // k-steps over the head dim
  constexpr int NKB = AKT / 16;      // 16-key blocks per tile
  constexpr int NDB = DH / 16;       // 16-wide d blocks of the output
  constexpr int KROW = DH * ES + 16; // LDS bytes per K row
  constexpr int VROW = AKT * ES + 16;// LDS bytes per V^T row
  __shared__ __attribute__((aligned(16))) unsigned char Ks[AKT * KROW];
  __shared__ __attribute__((aligned(16))) unsigned char Vts[DH * VROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int split = blockIdx.x, rb = blockIdx.y, b = blockIdx.z;
  const int T_ = p.T, Hq = p.Hq;
  const int nrows = T_ * Hq;
  const int rq = rb * 64 + wave * 16 + r16;
  const bool qvalid = rq < nrows;
  const int iq = qvalid ? rq / Hq : 0;
  const int jq = qvalid ? rq % Hq : 0;
  const int64_t ldq = (int64_t)(Hq + 2) * DH;
  const int64_t mrow0 = (int64_t)b * T_;

  // ---- query fragments with RoPE at the dynamic position --------------------
  uint4 qf[NKS];
  {
    float q[NKS][KPF];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int e = 0; e < KPF; ++e) q[ks][e] = 0.f;
    if (qvalid) {
      for (int sp = 0; sp < p.qkv_splits; ++sp) {
        const float* src = p.qkv + sp * p.qkv_split_stride + (mrow0 + iq) * ldq + jq * DH + g * KPF;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
          for (int e = 0; e < KPF; e += 4) {
            const float4 v = *reinterpret_cast<const float4*>(src + ks * KSD + e);
            q[ks][e] += v.x; q[ks][e + 1] += v.y; q[ks][e + 2] += v.z; q[ks][e + 3] += v.w;
          }
      }
      const float2* rope = p.rope + (int64_t)iq * (DH / 2);
#pragma unroll
      for (int ks = 0; ks < NKS / 2; ++ks)
#pragma unroll
        for (int e = 0; e < KPF; ++e) {
          const float2 cs = rope[ks * KSD + g * KPF + e];
          const float lo = q[ks][e], hi = q[ks + NKS / 2][e];
          q[ks][e] = lo * cs.x - hi * cs.y;
          q[ks + NKS / 2][e] = hi * cs.x + lo * cs.y;
        }
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = f_to_frag(q[ks], T());
  }

  // ---- key range of this split ---------------------------------------------
  const int Lc = p.static_len + (*p.n_valid) * p.frame_tokens;
  const int n_ct = (Lc + AKT - 1) / AKT;
  const int n_dt = (T_ + AKT - 1) / AKT;
  const int total = n_ct + n_dt;
  const int per = (total + p.nsplit - 1) / p.nsplit;
  const int t_beg = split * per;
  const int t_end = min(total, t_beg + per);

  const T* ck = reinterpret_cast<const T*>(p.cache_k) + (int64_t)b * p.ck_bstride;
  const T* cvt = reinterpret_cast<const T*>(p.cache_vt) + (int64_t)b * p.ck_bstride;
  const float scale = rsqrtf((float)DH) * 1.4426950408889634f;  // 1/sqrt(d) * log2(e)

  f32x4_v o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4_v{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  for (int t = t_beg; t < t_end; ++t) {
    const bool dyn = t >= n_ct;
    __syncthreads();  // previous tile fully consumed
    if (!dyn) {
      const int r0 = t * AKT;
      constexpr int KCH = DH * ES / 16;  // 16-byte chunks per K row
      for (int c = tid; c < AKT * KCH; c += 256) {
        const int kr = c / KCH, cc = c % KCH;
        const int r = r0 + kr;
        uint4 v = zero16();
        if (r < Lc) v = ld16(reinterpret_cast<const unsigned char*>(ck + (int64_t)r * DH) + cc * 16);
        st16(&Ks[kr * KROW + cc * 16], v);
      }
      constexpr int VCH = AKT * ES / 16;  // 16-byte chunks per V^T row
      for (int c = tid; c < DH * VCH; c += 256) {
        const int d = c / VCH, cc = c % VCH;
        const int key = r0 + cc * (16 / ES);
        uint4 v = zero16();
        if (key < Lc) v = ld16(reinterpret_cast<const unsigned char*>(cvt + (int64_t)d * p.R + key));
        st16(&Vts[d * VROW + cc * 16], v);
      }
    } else {
      const int kd0 = (t - n_ct) * AKT;
      for (int c = tid; c < AKT * (DH / 2); c += 256) {
        const int kr = c / (DH / 2), f = c % (DH / 2);
        const int kd = kd0 + kr;
        float klo = 0.f, khi = 0.f, vlo = 0.f, vhi = 0.f;
        if (kd < T_) {
          for (int sp = 0; sp < p.qkv_splits; ++sp) {
            const float* src = p.qkv + sp * p.qkv_split_stride + (mrow0 + kd) * ldq + (int64_t)Hq * DH;
            klo += src[f];
            khi += src[f + DH / 2];
            vlo += src[DH + f];
            vhi += src[DH + f + DH / 2];
          }
          const float2 cs = p.rope[(int64_t)kd * (DH / 2) + f];
          const float a = klo * cs.x - khi * cs.y;
          khi = khi * cs.x + klo * cs.y;
          klo = a;
        }
        T* krow = reinterpret_cast<T*>(&Ks[kr * KROW]);
        krow[f] = from_f<T>(klo);
        krow[f + DH / 2] = from_f<T>(khi);
        reinterpret_cast<T*>(&Vts[f * VROW])[kr] = from_f<T>(vlo);
        reinterpret_cast<T*>(&Vts[(f + DH / 2) * VROW])[kr] = from_f<T>(vhi);
      }
    }
    __syncthreads();

    // S^T = K Q^T for this tile: s[kb][i] = score(key kb*16 + 4g + i, query r16)
    f32x4_v s[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      s[kb] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const uint4 a = *reinterpret_cast<const uint4*>(&Ks[(kb * 16 + r16) * KROW + ks * 64 + g * 16]);
        mfma_step(s[kb], a, qf[ks], T());
      }
    }
    // scale + mask, tile max
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kidx = kb * 16 + 4 * g + i;
        bool ok;
        if (!dyn) {
          ok = t * AKT + kidx < Lc;
        } else {
          const int kd = (t - n_ct) * AKT + kidx;
          ok = kd < T_ && (iq > 0 || kd == 0);
        }
        const float v = ok ? s[kb][i] * scale : -INFINITY;
        s[kb][i] = v;
        mt = fmaxf(mt, v);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = exp2f(s[kb][i] - m_use);
        s[kb][i] = e;
        psum += e;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * corr + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] *= corr;

    // O^T += V^T P^T
    if constexpr (ES == 2) {
#pragma unroll
      for (int c = 0; c < NKB / 2; ++c) {
        float pv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) { pv[i] = s[2 * c][i]; pv[4 + i] = s[2 * c + 1][i]; }
        const uint4 pf = f_to_frag(pv, T());
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const unsigned char* vr = &Vts[(db * 16 + r16) * VROW];
          const uint2 lo = *reinterpret_cast<const uint2*>(vr + ((2 * c) * 16 + 4 * g) * ES);
          const uint2 hi = *reinterpret_cast<const uint2*>(vr + ((2 * c + 1) * 16 + 4 * g) * ES);
          mfma_step(o[db], make_uint4(lo.x, lo.y, hi.x, hi.y), pf, T());
        }
      }
    } else {
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        float pv[4] = {s[kb][0], s[kb][1], s[kb][2], s[kb][3]};
        const uint4 pf = f_to_frag(pv, T());
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const uint4 a =
              *reinterpret_cast<const uint4*>(&Vts[(db * 16 + r16) * VROW + (kb * 16 + 4 * g) * ES]);
          mfma_step(o[db], a, pf, T());
        }
      }
    }
  }

  if (!qvalid) return;
  if (p.nsplit == 1) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    T* dst = reinterpret_cast<T*>(p.out) + (mrow0 + iq) * (int64_t)(Hq * DH) + jq * DH;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[db * 16 + 4 * g + i] = from_f<T>(o[db][i] * inv);
  } else {
    const int64_t prow = ((int64_t)b * p.nsplit + split) * p.rows_pad + rq;
    float* dst = p.part_o + prow * DH;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      *reinterpret_cast<float4*>(dst + db * 16 + 4 * g) = make_float4(o[db][0], o[db][1], o[db][2], o[db][3]);
    if (g == 0) {
      p.part_ml[prow * 2] = m_run;
      p.part_ml[prow * 2 + 1] = l_run;
    }
  }
}

// Merge the key splits: o = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs p) {
  constexpr int RPB = 256 / DH;  // rows per block
  const int b = blockIdx.y;
  const int rq = blockIdx.x * RPB + threadIdx.x / DH;
  const int d = threadIdx.x % DH;
  const int nrows = p.T * p.Hq;
  if (rq >= nrows) return;
  float M = -INFINITY;
  for (int s = 0; s < p.nsplit; ++s)
    M = fmaxf(M, p.part_ml[(((int64_t)b * p.nsplit + s) * p.rows_pad + rq) * 2]);
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float L = 0.f, acc = 0.f;
  for (int s = 0; s < p.nsplit; ++s) {
    const int64_t prow = ((int64_t)b * p.nsplit + s) * p.rows_pad + rq;
    const float w = exp2f(p.part_ml[prow * 2] - Mu);
    L += w * p.part_ml[prow * 2 + 1];
    acc += w * p.part_o[prow * DH + d];
  }
  const int i = rq / p.Hq, j = rq % p.Hq;
  T* dst = reinterpret_cast<T*>(p.out) + ((int64_t)b * p.T + i) * (int64_t)(p.Hq * DH) + j * DH + d;
  *dst = from_f<T>(L > 0.f ? acc / L : 0.f);
}

int attention_pick_splits(int B, int rows, int max_keys, int head_dim) {
  (void)head_dim;
  const int rbs = (rows + 63) / 64;
  const int base = B * rbs;
  const int tiles = (max_keys + AKT - 1) / AKT + 1;
  int s = (256 + base - 1) / base;
  const int cap = (tiles + 1) / 2;
  if (s > cap) s = cap;
  return s < 1 ? 1 : s;
}

template <typename T, int DH>
static void launch_attn_dh(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.nsplit, (a.T * a.Hq + 63) / 64, a.B);
  RFX_LAUNCH((attn_kernel<T, DH>), grid, dim3(256), 0, s, a);
}

template <typename T>
hipError_t launch_attention(const AttnArgs& a, int head_dim, hipStream_t s) {
  switch (head_dim) {
    case 64: launch_attn_dh<T, 64>(a, s); break;
    case 128: launch_attn_dh<T, 128>(a, s); break;
    case 256: launch_attn_dh<T, 256>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int DH>
static void launch_merge_dh(const AttnArgs& a, hipStream_t s) {
  constexpr int RPB = 256 / DH;
  dim3 grid((a.T * a.Hq + RPB - 1) / RPB, a.B);
  RFX_LAUNCH((attn_merge_kernel<T, DH>), grid, dim3(256), 0, s, a);
}

template <typename T>
hipError_t launch_attn_merge(const AttnArgs& a, int head_dim, hipStream_t s) {
  switch (head_dim) {
    case 64: launch_merge_dh<T, 64>(a, s); break;
    case 128: launch_merge_dh<T, 128>(a, s); break;
    case 256: launch_merge_dh<T, 256>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_attention<float>(const AttnArgs&, int, hipStream_t);
template hipError_t launch_attention<bf16_t>(const AttnArgs&, int, hipStream_t);
template hipError_t launch_attn_merge<float>(const AttnArgs&, int, hipStream_t);
template hipError_t launch_attn_merge<bf16_t>(const AttnArgs&, int, hipStream_t);

}  // namespace reflex
