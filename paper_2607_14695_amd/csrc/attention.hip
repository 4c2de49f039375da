// Partitioned-region attention (Eq. 1, Section 3.1) for the dynamic rows.
//
// For every env, the T dynamic tokens x Hq query heads form T*Hq query rows
// that all read the single shared K/V head (multi-query).  The key sequence is
// [cached rows 0..Lc) ++ [dynamic rows 0..T), Lc = static_len +
// n_valid*frame_tokens read from device memory, so the same launch serves
// every tick.  Softmax is permutation-invariant over keys, so ring slots are
// read in physical order; the result equals one softmax over the concatenated
// context (Appendix A, Proposition A.1).  A pipelined ring holds one spare
// slot, the one the next frame is being written into while this launch runs;
// the cached rows are then read around it (logical row j at physical row
// j + frame_tokens from *hole_row on), again from device memory.
//
// Inputs come ready from the QKV projection's epilogue: RoPE-rotated q rows
// and dynamic keys, and transposed dynamic values zero-padded to 64 columns,
// so the dynamic tile is staged exactly like a cached tile.
//
// Decomposition and placement.  A workgroup owns one query block of one env
// (64 rows on the fp32 path; up to 128 rows as eight 16-row waves, the env's
// row waves spread evenly over its blocks, or 32 rows as one wave pair, on
// the bf16 path) and a contiguous range of 64-key tiles (a key split); the
// dynamic tile comes last.  All query blocks of one (env,
// split) group share the same K/V tiles, so the 1-D grid is laid out such
// that a group's blocks are dispatched to the same XCD (workgroups go
// round-robin over the 8 XCDs): the tiles then come from HBM once and from
// that XCD's L2 for the other blocks.  Each tile's K rows and V^T columns are
// staged in LDS and reused by every row of the block.  The fp32 kernel loads
// the next tile into registers during the current one's MFMAs; the bf16
// kernels copy it into a second LDS stage with global_load_lds, and the
// software-pipelined one also computes the next tile's scores and softmax
// under the current tile's P.V.
//
// Per wave the scores are computed transposed, S^T = K Q^T (A = K rows from
// LDS, B = the wave's 16 query rows held in registers).  In that layout each
// lane holds, for its query row, 4 consecutive keys of every 16-key block, so
// exp(S^T - m) is already the B operand of O^T = V^T P^T: the probabilities
// never leave registers.  V is stored transposed (d-major) so V^T[d][keys] is
// a contiguous LDS read.  Online softmax in base 2; the row max / sum cross
// the 4 lane groups with two xor shuffles (lane swaps on the pipelined
// kernel).
//
// With more than one key split each block writes (O unnormalised, m, l) and a
// merge kernel combines the splits with log-sum-exp weights in a fixed order.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace reflex {

constexpr int AKT = 64;  // keys per tile

// (group, query block) of a workgroup in the XCD-aware 1-D grid; false if
// the workgroup is padding.
RFX_DEV bool attn_decode(int bid, int groups, int nrb, int& group, int& rb) {
  const int xcd = bid & 7, slot = bid >> 3;
  const int gx = slot / nrb;
  rb = slot - gx * nrb;
  group = gx * 8 + xcd;
  return group < groups;
}

template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs p) {
  constexpr int ES = (int)sizeof(T);
  constexpr int KPF = ElemT<T>::kPerFrag;
  constexpr int KSD = 4 * KPF;        // head-dim elements per k-step
  constexpr int NKS = DH / KSD;       // k-steps over the head dim
  constexpr int NKB = AKT / 16;       // 16-key blocks per tile
  constexpr int NDB = DH / 16;        // 16-wide d blocks of the output
  constexpr int KROW = DH * ES + 16;  // LDS bytes per K row
  constexpr int VROW = AKT * ES + 8;  // LDS bytes per V^T row (8-byte pad: the 16 rows a
                                      // lane group reads start on distinct banks)
  constexpr int KCH = DH * ES / 16;   // 16-byte chunks per K row
  constexpr int VCH = AKT * ES / 16;  // 16-byte chunks per V^T row (one tile)
  constexpr int NKL = AKT * KCH / 256;  // K chunks per thread
  constexpr int NVL = DH * VCH / 256;   // V^T chunks per thread
  __shared__ __attribute__((aligned(16))) unsigned char Ks[AKT * KROW];
  __shared__ __attribute__((aligned(16))) unsigned char Vts[DH * VROW];

  int group, rb;
  if (!attn_decode(blockIdx.x, p.B * p.nsplit, p.rows_pad / 64, group, rb)) return;
  const int b = group / p.nsplit, split = group - b * p.nsplit;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int T_ = p.T, Hq = p.Hq;
  const int nrows = T_ * Hq;
  const int rq = rb * 64 + wave * 16 + r16;
  const bool qvalid = rq < nrows;
  const int iq = qvalid ? rq / Hq : 0;
  const int jq = qvalid ? rq % Hq : 0;
  const int64_t mrow0 = (int64_t)b * T_;

  // ---- query fragments (RoPE applied by the projection epilogue) -----------
  uint4 qf[NKS];
  {
    const T* qrow =
        reinterpret_cast<const T*>(p.q) + ((int64_t)b * p.rows_pad + (qvalid ? rq : 0)) * DH + g * KPF;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = ld16(qrow + ks * KSD);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = qvalid ? qf[ks] : zero16();
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
  const T* kdb = reinterpret_cast<const T*>(p.kd) + (int64_t)b * T_ * DH;
  const T* vdb = reinterpret_cast<const T*>(p.vdt) + (int64_t)b * DH * p.tpad;
  const float scale = rsqrtf((float)DH) * 1.4426950408889634f;  // 1/sqrt(d) * log2(e)
  const int hole = *p.hole_row, skip = p.frame_tokens;

  // global -> register staging of one tile.  Loads are unconditional from
  // clamped (in-range) addresses and the out-of-range chunks are zeroed when
  // they are written to LDS: a conditional load would make the compiler wait
  // for every outstanding load at the branch join and serialise the prefetch.
  uint4 rk[NKL], rv[NVL];
  uint32_t kmask = 0, vmask = 0;
  auto gload = [&](int t) {
    const bool dyn = t >= n_ct;
    const int base = dyn ? (t - n_ct) * AKT : t * AKT;
    const int lim = dyn ? T_ : Lc;
    const T* ksrc = dyn ? kdb : ck;
    kmask = 0;
    vmask = 0;
#pragma unroll
    for (int i = 0; i < NKL; ++i) {
      const int c = tid + 256 * i;
      const int kr = c / KCH, cc = c % KCH;
      const int r = base + kr;
      const bool ok = r < lim;
      kmask |= ok ? (1u << i) : 0u;
      int rr = ok ? r : 0;
      rr += (!dyn && rr >= hole) ? skip : 0;
      rk[i] = ld16(reinterpret_cast<const unsigned char*>(ksrc + (int64_t)rr * DH) + cc * 16);
    }
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int c = tid + 256 * i;
      const int d = c / VCH, cc = c % VCH;
      const int key = base + cc * (16 / ES);
      // dynamic values are padded to tpad columns and zero beyond T
      const bool ok = dyn || key < lim;
      vmask |= ok ? (1u << i) : 0u;
      const T* vsrc = dyn ? vdb + (int64_t)d * p.tpad : cvt + (int64_t)d * p.R;
      int kk = ok ? key : 0;
      kk += (!dyn && kk >= hole) ? skip : 0;
      rv[i] = ld16(reinterpret_cast<const unsigned char*>(vsrc + kk));
    }
  };

  f32x4_v o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4_v{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  if (t_beg < t_end) gload(t_beg);
  for (int t = t_beg; t < t_end; ++t) {
    const bool dyn = t >= n_ct;
    __syncthreads();  // previous tile fully consumed
#pragma unroll
    for (int i = 0; i < NKL; ++i) {
      const int c = tid + 256 * i;
      st16(&Ks[(c / KCH) * KROW + (c % KCH) * 16], (kmask >> i) & 1u ? rk[i] : zero16());
    }
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int c = tid + 256 * i;
      const uint4 v = (vmask >> i) & 1u ? rv[i] : zero16();
      unsigned char* dst = &Vts[(c / VCH) * VROW + (c % VCH) * 16];  // 8-byte aligned rows
      *reinterpret_cast<uint2*>(dst) = make_uint2(v.x, v.y);
      *reinterpret_cast<uint2*>(dst + 8) = make_uint2(v.z, v.w);
    }
    __syncthreads();
    if (t + 1 < t_end) gload(t + 1);  // in flight during this tile's math

    // S^T = K Q^T for this tile: s[kb][i] = score(key kb*16 + 4g + i, query r16)
    f32x4_v s[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) s[kb] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const uint4 a = *reinterpret_cast<const uint4*>(&Ks[(kb * 16 + r16) * KROW + ks * 64 + g * 16]);
        mfma_step(s[kb], a, qf[ks], T());
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
          const unsigned char* vr = &Vts[(db * 16 + r16) * VROW + (kb * 16 + 4 * g) * ES];
          const uint2 lo = *reinterpret_cast<const uint2*>(vr);
          const uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
          mfma_step(o[db], make_uint4(lo.x, lo.y, hi.x, hi.y), pf, T());
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
    return;
  }
  const int64_t prow = ((int64_t)b * p.nsplit + split) * p.rows_pad + rq;
  float* dst = p.part_o + prow * DH;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
    *reinterpret_cast<float4*>(dst + db * 16 + 4 * g) = make_float4(o[db][0], o[db][1], o[db][2], o[db][3]);
  if (g == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(m_run, l_run);
}


// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// releases global memory, which makes the compiler wait for every outstanding
// vector-memory operation, including the LDS DMA of the next tile that is
// meant to stay in flight; DMA completion is awaited explicitly instead.
RFX_DEV void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// ---------------------------------------------------------------------------
// bf16 variant: eight waves of 16 query rows (16x16x32 MFMAs), two waves per
// SIMD.  With 16 rows a wave holds its Q fragments (32 registers), its O^T
// accumulator (64) and the scores (16) with room to keep eight LDS fragment
// reads in flight, and the second wave on the SIMD covers the latency the
// first one waits on.  A workgroup covers 128 query rows, like the launch
// geometry of the other variants, and stages each 64-key tile once in LDS for
// all eight waves.
//
// Tiles reach LDS by global_load_lds_dwordx4 into two stages (tile t+1 in
// flight during tile t).  16-byte chunks are XOR-swizzled on the global side
// of the DMA: K chunk c of row r sits at c ^ RFX_KSWZ(r), V^T chunk c of row d at
// c ^ (d mod 8).  Every per-lane LDS offset takes at most eight values, the
// rest being instruction immediates.
//
// Key order.  S^T block kb = 2j + e (16 keys x 16 queries) takes as its A
// operand row r the key 32j + 8*(r >> 2) + 4e + (r & 3).  Its result then
// leaves lane l (g = l >> 4) holding keys 32j + 8g + 4e + i, i < 4: over the
// two blocks of chunk j the lane owns the 8 consecutive keys 32j + 8g + [0, 8),
// which is exactly the contraction slice a B operand lane supplies to the
// 16x16x32 MFMA of O^T = V^T P^T.  The probabilities are used where they were
// computed, and each V^T fragment is one 16-byte chunk of one V^T row.
// ---------------------------------------------------------------------------
// K swizzle: 16 distinct values over the 16 rows a block's lanes read
// (8 for 64-wide heads, whose rows have 8 chunks)
#define RFX_KSWZ(r, kch) ((kch) >= 16 ? (((r) & 3) | (((r) >> 1) & 12)) : (((r) & 3) | (((r) >> 1) & 4)))

RFX_DEV uint32_t pack_bf16x2(float a, float b) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_v;
  const bf16x2_v v = {(__bf16)a, (__bf16)b};  // v_cvt_pk_bf16_f32, round to nearest even
  return __builtin_bit_cast(uint32_t, v);
}

template <int DH>
__global__ __launch_bounds__(512) void attn16_kernel(AttnArgs p) {
  using T = bf16_t;
  constexpr int NW = 8;
  constexpr int NKS = DH / 32;            // 32-wide d steps of S^T
  constexpr int NDB = DH / 16;            // 16-wide d blocks of O^T
  constexpr int KRB = DH * 2;             // bytes per K row in LDS
  constexpr int KCH = DH / 8;             // 16-byte chunks per K row
  constexpr int NKO = KCH >= 16 ? 4 : 2;  // distinct per-lane K chunk offsets per parity
  constexpr int VRB = AKT * 2;            // bytes per V^T row (128)
  constexpr int KBYTES = AKT * KRB;
  constexpr int VBYTES = DH * VRB;
  constexpr int STAGE = KBYTES + VBYTES;
  constexpr int NIK = KBYTES / 1024 / NW;  // 1-KB DMA instructions per wave, K
  constexpr int NIV = VBYTES / 1024 / NW;  // same for V^T
  static_assert(NIK >= 1 && NIV >= 1, "tile smaller than one DMA round");
  __shared__ __attribute__((aligned(16))) unsigned char stage0[STAGE];
  __shared__ __attribute__((aligned(16))) unsigned char stage1[STAGE];

  int group, rb;
  if (!attn_decode(blockIdx.x, p.B * p.nsplit, p.rows_pad / 128, group, rb)) return;
  const int b = group / p.nsplit, split = group - b * p.nsplit;

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int T_ = p.T, Hq = p.Hq;
  const int nrows = T_ * Hq;
  // rows of the block as in attn16p_kernel (the row waves of an env spread
  // evenly over its blocks), so both kernels group the same rows into a wave
  // and take the same lazy-rescale decisions; waves past the block's count
  // compute on row 0's data and store nothing
  const int nrb = p.rows_pad / 128, nw16 = (nrows + 15) / 16;
  const int wbase = nw16 / nrb, wextra = nw16 - wbase * nrb;
  const int nwb = wbase + (rb < wextra ? 1 : 0);
  const int rq = 16 * (rb * wbase + min(rb, wextra)) + wave * 16 + r16;
  const bool qvalid = wave < nwb && rq < nrows;
  const int iq = qvalid ? rq / Hq : 0;
  const int jq = qvalid ? rq % Hq : 0;

  uint4 qf[NKS];
  {
    // rows past the valid range compute on row 0's data and are never stored
    const T* qrow = reinterpret_cast<const T*>(p.q) + ((int64_t)b * p.rows_pad + (qvalid ? rq : 0)) * DH + g * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = ld16(qrow + ks * 32);
  }

  const int Lc = p.static_len + (*p.n_valid) * p.frame_tokens;
  const int n_ct = (Lc + AKT - 1) / AKT;
  const int n_dt = (T_ + AKT - 1) / AKT;
  const int total = n_ct + n_dt;
  const int per = (total + p.nsplit - 1) / p.nsplit;
  const int t_beg = split * per;
  const int t_end = min(total, t_beg + per);

  const T* ck = reinterpret_cast<const T*>(p.cache_k) + (int64_t)b * p.ck_bstride;
  const T* cvt = reinterpret_cast<const T*>(p.cache_vt) + (int64_t)b * p.ck_bstride;
  const T* kdb = reinterpret_cast<const T*>(p.kd) + (int64_t)b * T_ * DH;
  const T* vdb = reinterpret_cast<const T*>(p.vdt) + (int64_t)b * DH * p.tpad;
  const float scale = rsqrtf((float)DH) * 1.4426950408889634f;
  const int tpad = p.tpad, Rrow = p.R;  // copied: a lambda must not capture the kernel argument
  const int hole = __builtin_amdgcn_readfirstlane(*p.hole_row), skip = p.frame_tokens;
  constexpr int RPI = 64 / KCH;         // K rows per DMA instruction

  // DMA of tile t into stage sk.  Per-lane offsets are rebuilt from an opaque
  // copy of the lane id on every call so they are not hoisted into registers.
  auto issue = [&](int t, unsigned char* sk) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const bool dyn = t >= n_ct;
    const int base = dyn ? (t - n_ct) * AKT : t * AKT;
    const int last = (dyn ? T_ : Lc) - 1;
    unsigned char* sv = sk + KBYTES;
    const int kl = ln % KCH, kr = ln / KCH;
    const int vd = ln >> 3, vc = ln & 7;
    if (dyn) {
#pragma unroll
      for (int j = 0; j < NIK; ++j) {
        const int row = RPI * (wave * NIK + j) + kr;
        const int r = min(base + row, last);
        __builtin_amdgcn_global_load_lds(kdb + r * DH + (kl ^ RFX_KSWZ(row, KCH)) * 8, sk + (wave * NIK + j) * 1024, 16,
                                         0, 0);
      }
#pragma unroll
      for (int j = 0; j < NIV; ++j) {
        const int d = (wave * NIV + j) * 8 + vd;
        __builtin_amdgcn_global_load_lds(vdb + d * tpad + base + (vc ^ (d & 7)) * 8, sv + (wave * NIV + j) * 1024, 16,
                                         0, 0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NIK; ++j) {
        const int row = RPI * (wave * NIK + j) + kr;
        int r = min(base + row, last);
        r += r >= hole ? skip : 0;
        __builtin_amdgcn_global_load_lds(ck + (int64_t)r * DH + (kl ^ RFX_KSWZ(row, KCH)) * 8,
                                         sk + (wave * NIK + j) * 1024, 16, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < NIV; ++j) {
        const int d = (wave * NIV + j) * 8 + vd;
        int key = base + (vc ^ (d & 7)) * 8;
        key = key <= last ? key : 0;
        key += key >= hole ? skip : 0;
        __builtin_amdgcn_global_load_lds(cvt + (int64_t)d * Rrow + key,
                                         sv + (wave * NIV + j) * 1024, 16, 0, 0);
      }
    }
  };

  f32x4_v o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4_v{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // per-lane LDS read offsets (bytes).  K: row rho = 8*(r16 >> 2) + 4e +
  // (r16 & 3) of a 32-key chunk, d-chunk 4*ks + g, the low bits of ks in x.
  // V^T: row db*16 + r16, key chunk 4j + g.
  int koff[2][NKO], voff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int rho = 8 * (r16 >> 2) + 4 * e + (r16 & 3);
#pragma unroll
    for (int x = 0; x < NKO; ++x) koff[e][x] = rho * KRB + ((4 * x + g) ^ RFX_KSWZ(rho, KCH)) * 16;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) voff[j] = r16 * VRB + ((4 * j + g) ^ (r16 & 7)) * 16;

  auto step = [&](int t, const unsigned char* cur, unsigned char* nxt) __attribute__((always_inline)) {
    const bool dyn = t >= n_ct;
    // tile t's DMA (the only one outstanding) completes; after the barrier
    // every wave's part of it is visible and every wave has finished reading
    // the other stage, which tile t+1 then overwrites during the math
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    lds_barrier();
    if (t + 1 < t_end) issue(t + 1, nxt);
    const unsigned char* sk = cur;
    const unsigned char* sv = cur + KBYTES;

    // S^T = K Q^T: four 16-key blocks, their accumulation chains interleaved
    f32x4_v s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) s[kb] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k0 = 0; k0 < NKS; k0 += 2) {
      uint4 a[2][4];
#pragma unroll
      for (int u = 0; u < 2 && k0 + u < NKS; ++u)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          const int ks = k0 + u;
          a[u][kb] = *reinterpret_cast<const uint4*>(sk + (kb >> 1) * 32 * KRB + (ks / NKO) * NKO * 64 +
                                                     koff[kb & 1][ks % NKO]);
        }
#pragma unroll
      for (int u = 0; u < 2 && k0 + u < NKS; ++u)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) mfma_step(s[kb], a[u][kb], qf[k0 + u], T());
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }

    // block kb = 2j + e holds keys 32j + 8g + 4e + i; visible iff below lim:
    // the cached rows below Lc; among the dynamic rows the state row (iq == 0)
    // sees only key 0
    const int lim = (dyn ? (iq > 0 ? T_ : 1) - (t - n_ct) * AKT : Lc - t * AKT) - 8 * g;
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = (kb >> 1) * 32 + 4 * (kb & 1) + i < lim ? s[kb][i] * scale : -INFINITY;
        s[kb][i] = v;
        mt = fmaxf(mt, v);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    // lazy rescaling: the running max only moves when some row's tile max
    // exceeds it by more than 8 (log2 units), so the probabilities stay below
    // 2^8 and the O rescale is rare
    if (__any(mt > m_run + 8.f)) {
      const float m_new = fmaxf(m_run, mt);
      const float corr = m_new == -INFINITY ? 1.f : exp2f(m_run - m_new);
      l_run *= corr;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= corr;
    }
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    // scores are at most m_run + 8: the plain hardware exp2 (no denormal
    // range handling) is exact enough; masked keys give exp2(-inf) = 0
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = __builtin_amdgcn_exp2f(s[kb][i] - m_use);
        s[kb][i] = e;
        psum += e;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run += psum;

    // O^T += V^T P^T, two 32-key chunks; slot 8g + 4e + i <-> key 32j + 8g + 4e + i
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint4 pf = make_uint4(pack_bf16x2(s[2 * j][0], s[2 * j][1]), pack_bf16x2(s[2 * j][2], s[2 * j][3]),
                                  pack_bf16x2(s[2 * j + 1][0], s[2 * j + 1][1]),
                                  pack_bf16x2(s[2 * j + 1][2], s[2 * j + 1][3]));
#pragma unroll
      for (int d0 = 0; d0 < NDB; d0 += 8) {
        uint4 vf[8];
#pragma unroll
        for (int u = 0; u < 8 && d0 + u < NDB; ++u)
          vf[u] = *reinterpret_cast<const uint4*>(sv + (d0 + u) * 16 * VRB + voff[j]);
#pragma unroll
        for (int u = 0; u < 8 && d0 + u < NDB; ++u) mfma_step(o[d0 + u], vf[u], pf, T());
        __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      }
    }
  };

  if (t_beg < t_end) issue(t_beg, stage0);
  for (int t = t_beg; t < t_end; t += 2) {
    step(t, stage0, stage1);
    if (t + 1 < t_end) step(t + 1, stage1, stage0);
  }

  if (!qvalid) return;
  if (p.nsplit == 1) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    T* dst = reinterpret_cast<T*>(p.out) + ((int64_t)b * T_ + iq) * (int64_t)(Hq * DH) + jq * DH + 4 * g;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      *reinterpret_cast<uint2*>(dst + db * 16) =
          make_uint2(pack_bf16x2(o[db][0] * inv, o[db][1] * inv), pack_bf16x2(o[db][2] * inv, o[db][3] * inv));
    return;
  }
  // bf16 partials: half the bytes of this kernel's largest write and of the
  // merge's reads; the merged output is bf16 too
  const int64_t prow = ((int64_t)b * p.nsplit + split) * p.rows_pad + rq;
  T* dst = reinterpret_cast<T*>(p.part_o) + prow * DH + 4 * g;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
    *reinterpret_cast<uint2*>(dst + db * 16) =
        make_uint2(pack_bf16x2(o[db][0], o[db][1]), pack_bf16x2(o[db][2], o[db][3]));
  if (g == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(m_run, l_run);
}

// ---------------------------------------------------------------------------
// Software-pipelined 16-row variant: the decomposition, layouts, key order
// and arithmetic of attn16_kernel, with the per-tile work reordered so that a
// wave's softmax runs under its own MFMAs.  Iteration i computes S^T of tile
// i+1, then O^T += V^T P^T of tile i interleaved with the softmax of tile
// i+1.  That softmax takes the running max as it stands; when some row's tile
// max exceeds it by more than 8 (the lazy-rescale test), O is rescaled after
// the P.V step and the tile's exponentials are recomputed with the new max.
// The operations and their order per row are those of attn16_kernel, so the
// results are the same bit for bit.
//
// K and V^T have separate double buffers: at the start of iteration i the
// copies of K(i+2) and V^T(i+1) go into the buffers K(i) and V^T(i-1) left,
// and both land before iteration i+1 (one copy round in flight, 128 KB of
// LDS as before).  Row max and row sum cross the four lane groups with the
// gfx950 lane swaps (VALU), not LDS permutes, so they interleave with the
// V^T fragment reads.
// ---------------------------------------------------------------------------
RFX_DEV float xmax16_32(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
RFX_DEV float xsum16_32(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Copy of 16 bytes per lane from global memory into LDS (global_load_lds,
// LDS destination from M0), issued through inline assembly: the compiler
// then does not track these LDS writes and waits for its own LDS reads with
// partial counts instead of draining every outstanding read first.  Every
// kernel that uses it orders the copies itself: a vmcnt(0) wait and a
// barrier come before any read of a stage, and no stage is overwritten
// before a barrier that follows its last read.  Outstanding copies it does
// not know of only make the compiler's own vmcnt waits stricter (loads
// complete in order).  M0 is a reserved register the compiler sets right
// before each instruction of its own that reads it, so it is not declared
// clobbered (it cannot be); the kernels using this helper contain no other
// M0 reader.
RFX_DEV void lds_dma16(const void* g, void* lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"((unsigned)(size_t)lds) : "memory");
}

template <int DH>
__global__ __launch_bounds__(512) void attn16p_kernel(AttnArgs p) {
  using T = bf16_t;
  constexpr int NW = 8;
  constexpr int NKS = DH / 32;            // 32-wide d steps of S^T
  constexpr int NDB = DH / 16;            // 16-wide d blocks of O^T
  constexpr int KRB = DH * 2;             // bytes per K row in LDS
  constexpr int KCH = DH / 8;             // 16-byte chunks per K row
  constexpr int NKO = KCH >= 16 ? 4 : 2;  // distinct per-lane K chunk offsets per parity
  constexpr int VRB = AKT * 2;            // bytes per V^T row (128)
  constexpr int KBYTES = AKT * KRB;
  constexpr int VBYTES = DH * VRB;
  constexpr int NIK = KBYTES / 1024 / NW;  // 1-KB DMA instructions per wave, K
  constexpr int NIV = VBYTES / 1024 / NW;  // same for V^T
  static_assert(NIK >= 1 && NIV >= 1, "tile smaller than one DMA round");
  __shared__ __attribute__((aligned(16))) unsigned char kbuf0[KBYTES];
  __shared__ __attribute__((aligned(16))) unsigned char kbuf1[KBYTES];
  __shared__ __attribute__((aligned(16))) unsigned char vbuf0[VBYTES];
  __shared__ __attribute__((aligned(16))) unsigned char vbuf1[VBYTES];

  int group, rb;
  if (!attn_decode(blockIdx.x, p.B * p.nsplit, p.rows_pad / 128, group, rb)) return;
  const int b = group / p.nsplit, split = group - b * p.nsplit;

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int T_ = p.T, Hq = p.Hq;
  const int nrows = T_ * Hq;
  // The ceil(nrows/16) row waves of an env are spread evenly over its blocks
  // (408 rows: 7, 7, 6 and 6 waves instead of 8, 8, 8 and 2), so no block has
  // more computing waves than it must.  A wave past its block's count still
  // issues its share of the tile copies and joins every barrier, but does no
  // math: the per-tile LDS reads of the busiest block set the kernel's pace.
  const int nrb = p.rows_pad / 128, nw16 = (nrows + 15) / 16;
  const int wbase = nw16 / nrb, wextra = nw16 - wbase * nrb;
  const int nwb = wbase + (rb < wextra ? 1 : 0);  // computing waves of this block
  const bool active = wave < nwb;
  const int rq = 16 * (rb * wbase + min(rb, wextra)) + wave * 16 + r16;
  const bool qvalid = active && rq < nrows;
  const int iq = qvalid ? rq / Hq : 0;
  const int jq = qvalid ? rq % Hq : 0;

  uint4 qf[NKS];
  {
    // rows past the valid range compute on row 0's data and are never stored
    const T* qrow = reinterpret_cast<const T*>(p.q) + ((int64_t)b * p.rows_pad + (qvalid ? rq : 0)) * DH + g * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = ld16(qrow + ks * 32);
  }

  const int Lc = p.static_len + (*p.n_valid) * p.frame_tokens;
  const int n_ct = (Lc + AKT - 1) / AKT;
  const int n_dt = (T_ + AKT - 1) / AKT;
  const int total = n_ct + n_dt;
  const int per = (total + p.nsplit - 1) / p.nsplit;
  const int t_beg = split * per;
  const int t_end = min(total, t_beg + per);
  const int n = t_end - t_beg;

  const T* ck = reinterpret_cast<const T*>(p.cache_k) + (int64_t)b * p.ck_bstride;
  const T* cvt = reinterpret_cast<const T*>(p.cache_vt) + (int64_t)b * p.ck_bstride;
  const T* kdb = reinterpret_cast<const T*>(p.kd) + (int64_t)b * T_ * DH;
  const T* vdb = reinterpret_cast<const T*>(p.vdt) + (int64_t)b * DH * p.tpad;
  const float scale = rsqrtf((float)DH) * 1.4426950408889634f;
  const int tpad = p.tpad, Rrow = p.R;  // copied: a lambda must not capture the kernel argument
  const int hole = __builtin_amdgcn_readfirstlane(*p.hole_row), skip = p.frame_tokens;
  constexpr int RPI = 64 / KCH;         // K rows per DMA instruction

  // DMA of tile t's K rows / V^T columns.  Per-lane offsets are rebuilt from
  // an opaque copy of the lane id on every call so they are not hoisted into
  // registers.
  auto issue_k = [&](int t, unsigned char* sk) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const bool dyn = t >= n_ct;
    const int base = dyn ? (t - n_ct) * AKT : t * AKT;
    const int last = (dyn ? T_ : Lc) - 1;
    const int kl = ln % KCH, kr = ln / KCH;
    if (dyn) {
#pragma unroll
      for (int j = 0; j < NIK; ++j) {
        const int row = RPI * (wave * NIK + j) + kr;
        const int r = min(base + row, last);
        lds_dma16(kdb + r * DH + (kl ^ RFX_KSWZ(row, KCH)) * 8, sk + (wave * NIK + j) * 1024);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NIK; ++j) {
        const int row = RPI * (wave * NIK + j) + kr;
        int r = min(base + row, last);
        r += r >= hole ? skip : 0;
        lds_dma16(ck + (int64_t)r * DH + (kl ^ RFX_KSWZ(row, KCH)) * 8, sk + (wave * NIK + j) * 1024);
      }
    }
  };
  auto issue_v = [&](int t, unsigned char* sv) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const bool dyn = t >= n_ct;
    const int base = dyn ? (t - n_ct) * AKT : t * AKT;
    const int last = (dyn ? T_ : Lc) - 1;
    const int vd = ln >> 3, vc = ln & 7;
    if (dyn) {
#pragma unroll
      for (int j = 0; j < NIV; ++j) {
        const int d = (wave * NIV + j) * 8 + vd;
        lds_dma16(vdb + d * tpad + base + (vc ^ (d & 7)) * 8, sv + (wave * NIV + j) * 1024);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NIV; ++j) {
        const int d = (wave * NIV + j) * 8 + vd;
        int key = base + (vc ^ (d & 7)) * 8;
        key = key <= last ? key : 0;
        key += key >= hole ? skip : 0;
        lds_dma16(cvt + (int64_t)d * Rrow + key, sv + (wave * NIV + j) * 1024);
      }
    }
  };

  f32x4_v o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = f32x4_v{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // per-lane LDS read offsets (bytes), as in attn16_kernel
  int koff[2][NKO], voff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int rho = 8 * (r16 >> 2) + 4 * e + (r16 & 3);
#pragma unroll
    for (int x = 0; x < NKO; ++x) koff[e][x] = rho * KRB + ((4 * x + g) ^ RFX_KSWZ(rho, KCH)) * 16;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) voff[j] = r16 * VRB + ((4 * j + g) ^ (r16 & 7)) * 16;

  // S^T = K Q^T of the tile in sk: four 16-key blocks, chains interleaved
  auto scores = [&](const unsigned char* sk, f32x4_v* s) __attribute__((always_inline)) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) s[kb] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k0 = 0; k0 < NKS; k0 += 2) {
      uint4 a[2][4];
#pragma unroll
      for (int u = 0; u < 2 && k0 + u < NKS; ++u)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          const int ks = k0 + u;
          a[u][kb] = *reinterpret_cast<const uint4*>(sk + (kb >> 1) * 32 * KRB + (ks / NKO) * NKO * 64 +
                                                     koff[kb & 1][ks % NKO]);
        }
#pragma unroll
      for (int u = 0; u < 2 && k0 + u < NKS; ++u)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) mfma_step(s[kb], a[u][kb], qf[k0 + u], T());
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }
  };
  // mask and scale tile t's scores in place; returns the row max over the tile
  auto mask_max = [&](int t, f32x4_v* s) __attribute__((always_inline)) {
    const bool dyn = t >= n_ct;
    const int lim = (dyn ? (iq > 0 ? T_ : 1) - (t - n_ct) * AKT : Lc - t * AKT) - 8 * g;
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = (kb >> 1) * 32 + 4 * (kb & 1) + i < lim ? s[kb][i] * scale : -INFINITY;
        s[kb][i] = v;
        mt = fmaxf(mt, v);
      }
    return xmax16_32(mt);
  };
  // exponentials against m_use, packed as the two P^T operands; returns the
  // row sum
  auto expo = [&](const f32x4_v* s, float m_use, uint4* pf) __attribute__((always_inline)) {
    float e[4][4];
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        e[kb][i] = __builtin_amdgcn_exp2f(s[kb][i] - m_use);
        psum += e[kb][i];
      }
#pragma unroll
    for (int j = 0; j < 2; ++j)
      pf[j] = make_uint4(pack_bf16x2(e[2 * j][0], e[2 * j][1]), pack_bf16x2(e[2 * j][2], e[2 * j][3]),
                         pack_bf16x2(e[2 * j + 1][0], e[2 * j + 1][1]),
                         pack_bf16x2(e[2 * j + 1][2], e[2 * j + 1][3]));
    return xsum16_32(psum);
  };
  // lazy rescale test for a tile whose exponentials were taken against the
  // running max; on a rescale they are taken again against the new one
  auto commit = [&](float mt, const f32x4_v* s, uint4* pf, float psum) __attribute__((always_inline)) {
    if (__any(mt > m_run + 8.f)) {
      const float m_new = fmaxf(m_run, mt);
      const float corr = m_new == -INFINITY ? 1.f : exp2f(m_run - m_new);
      l_run *= corr;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= corr;
      psum = expo(s, m_run == -INFINITY ? 0.f : m_run, pf);
    }
    l_run += psum;
  };
  // O^T += V^T P^T of the tile in sv; slot 8g + 4e + i <-> key 32j + 8g + 4e + i
  auto pv = [&](const unsigned char* sv, const uint4* pf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int d0 = 0; d0 < NDB; d0 += 8) {
        uint4 vf[8];
#pragma unroll
        for (int u = 0; u < 8 && d0 + u < NDB; ++u)
          vf[u] = *reinterpret_cast<const uint4*>(sv + (d0 + u) * 16 * VRB + voff[j]);
#pragma unroll
        for (int u = 0; u < 8 && d0 + u < NDB; ++u) mfma_step(o[d0 + u], vf[u], pf[j], T());
      }
  };

  uint4 pcur[2], pnext[2];
  // iteration i: S^T of tile i+1 (K in kn), then P.V of tile i (V^T in vc)
  // under tile i+1's softmax; K(i+2) goes to kf, V^T(i+1) to vn
  auto iter = [&](int i, const unsigned char* kn, unsigned char* kf, const unsigned char* vc, unsigned char* vn)
                  __attribute__((always_inline)) {
    // K(i+1) and V^T(i) complete; every wave is done with K(i) and V^T(i-1)
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    lds_barrier();
    if (i + 2 < n) issue_k(t_beg + i + 2, kf);
    issue_v(t_beg + i + 1, vn);
    if (!active) return;
    f32x4_v s[4];
    scores(kn, s);
    const float m_use = m_run == -INFINITY ? 0.f : m_run;
    const float mt = mask_max(t_beg + i + 1, s);
    const float psum = expo(s, m_use, pnext);
    pv(vc, pcur);
    commit(mt, s, pnext, psum);
    pcur[0] = pnext[0];
    pcur[1] = pnext[1];
  };

  if (n > 0) {
    issue_k(t_beg, kbuf0);
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    lds_barrier();
    if (n > 1) issue_k(t_beg + 1, kbuf1);
    issue_v(t_beg, vbuf0);
    if (active) {
      f32x4_v s[4];
      scores(kbuf0, s);
      const float mt = mask_max(t_beg, s);
      const float psum = expo(s, 0.f, pcur);
      commit(mt, s, pcur, psum);
    }
    // tile i's K sits in kbuf[i & 1] and its V^T in vbuf[i & 1]
    int i = 0;
    for (; i + 2 < n; i += 2) {
      iter(i, kbuf1, kbuf0, vbuf0, vbuf1);
      iter(i + 1, kbuf0, kbuf1, vbuf1, vbuf0);
    }
    if (i + 1 < n) {
      iter(i, kbuf1, kbuf0, vbuf0, vbuf1);
      ++i;
    }
    // last tile: its P.V only
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    lds_barrier();
    if (active) pv((i & 1) ? vbuf1 : vbuf0, pcur);
  }

  if (!qvalid) return;
  if (p.nsplit == 1) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    T* dst = reinterpret_cast<T*>(p.out) + ((int64_t)b * T_ + iq) * (int64_t)(Hq * DH) + jq * DH + 4 * g;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      *reinterpret_cast<uint2*>(dst + db * 16) =
          make_uint2(pack_bf16x2(o[db][0] * inv, o[db][1] * inv), pack_bf16x2(o[db][2] * inv, o[db][3] * inv));
    return;
  }
  const int64_t prow = ((int64_t)b * p.nsplit + split) * p.rows_pad + rq;
  T* dst = reinterpret_cast<T*>(p.part_o) + prow * DH + 4 * g;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
    *reinterpret_cast<uint2*>(dst + db * 16) =
        make_uint2(pack_bf16x2(o[db][0], o[db][1]), pack_bf16x2(o[db][2], o[db][3]));
  if (g == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(m_run, l_run);
}

// ---------------------------------------------------------------------------
// bf16 variant with wave pairs.  Two waves share 32 query rows (two 16-row
// blocks): for S^T = K Q^T wave h takes keys [32h, 32h + 32) of the tile, for
// O^T = V^T P^T it takes head dims [h*DH/2, (h+1)*DH/2) over all 64 keys.
// Every K row and V^T row fragment a wave reads from LDS thus feeds two
// MFMAs (one per row block), half the LDS bytes per query row of a 16-row
// wave, while a wave still holds only its Q fragments (2 x DH/32 x 4 VGPRs),
// its half of O^T (DH/32 x 2 x 4) and 16 scores, so two waves fit per SIMD.
//
// Per tile the pair exchanges, through LDS, (1) its per-row score maxima, so
// both waves use the same running max and make the same lazy-rescale
// decision, and (2) its probabilities, already in the B-operand layout of the
// P.V MFMA (the key permutation of the 16-row variant: over its two score
// blocks a lane holds 8 consecutive keys of the wave's 32).  The running
// row sums cover each wave's own keys and are added once at the end; the
// running max is identical in both waves, so the two halves share one scale.
// A workgroup is one pair.  This variant serves the latency-bound regime (a
// few envs, down to one key tile per split): 32-row blocks waste fewer
// padded rows than 128-row ones (416 against 512 for 408 rows), so more
// workgroups each finish one tile sooner.  With four pairs sharing a tile at
// 32 envs the two extra barriers per tile made it slower than the 16-row
// variant, which therefore keeps the large batches.
// ---------------------------------------------------------------------------
template <int DH>
__global__ __launch_bounds__(128) void attn_pair_kernel(AttnArgs p) {
  using T = bf16_t;
  constexpr int NW = 2;
  constexpr int NKS = DH / 32;            // 32-wide d steps of S^T
  constexpr int NDH = DH / 32;            // 16-wide d blocks in half a head
  constexpr int KRB = DH * 2;             // bytes per K row in LDS
  constexpr int KCH = DH / 8;             // 16-byte chunks per K row
  constexpr int NKO = KCH >= 16 ? 4 : 2;  // distinct per-lane K chunk offsets per parity
  constexpr int VRB = AKT * 2;            // bytes per V^T row (128)
  constexpr int KBYTES = AKT * KRB;
  constexpr int VBYTES = DH * VRB;
  constexpr int STAGE = KBYTES + VBYTES;
  constexpr int NIK = KBYTES / 1024 / NW;  // 1-KB DMA instructions per wave, K
  constexpr int NIV = VBYTES / 1024 / NW;  // same for V^T
  static_assert(NIK >= 1 && NIV >= 1, "tile smaller than one DMA round");
  __shared__ __attribute__((aligned(16))) unsigned char stage0[STAGE];
  __shared__ __attribute__((aligned(16))) unsigned char stage1[STAGE];
  __shared__ __attribute__((aligned(16))) uint4 pbuf[2][2][64];  // [half][row block][lane]
  __shared__ float xbuf[2][2][16];                               // [half][row block][row]

  const int T_ = p.T, Hq = p.Hq;
  const int nrows = T_ * Hq;
  const int nrb = (nrows + 31) / 32;
  int group, rb;
  if (!attn_decode(blockIdx.x, p.B * p.nsplit, nrb, group, rb)) return;
  const int b = group / p.nsplit, split = group - b * p.nsplit;

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = wave;
  const int r16 = lane & 15, g = lane >> 4;
  int rq[2], iq[2], jq[2];
  bool qvalid[2];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) {
    rq[rr] = rb * 32 + rr * 16 + r16;
    qvalid[rr] = rq[rr] < nrows;
    iq[rr] = qvalid[rr] ? rq[rr] / Hq : 0;
    jq[rr] = qvalid[rr] ? rq[rr] % Hq : 0;
  }

  uint4 qf[2][NKS];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) {
    // rows past the valid range compute on row 0's data and are never stored
    const T* qrow =
        reinterpret_cast<const T*>(p.q) + ((int64_t)b * p.rows_pad + (qvalid[rr] ? rq[rr] : 0)) * DH + g * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[rr][ks] = ld16(qrow + ks * 32);
  }

  const int Lc = p.static_len + (*p.n_valid) * p.frame_tokens;
  const int n_ct = (Lc + AKT - 1) / AKT;
  const int n_dt = (T_ + AKT - 1) / AKT;
  const int total = n_ct + n_dt;
  const int per = (total + p.nsplit - 1) / p.nsplit;
  const int t_beg = split * per;
  const int t_end = min(total, t_beg + per);

  const T* ck = reinterpret_cast<const T*>(p.cache_k) + (int64_t)b * p.ck_bstride;
  const T* cvt = reinterpret_cast<const T*>(p.cache_vt) + (int64_t)b * p.ck_bstride;
  const T* kdb = reinterpret_cast<const T*>(p.kd) + (int64_t)b * T_ * DH;
  const T* vdb = reinterpret_cast<const T*>(p.vdt) + (int64_t)b * DH * p.tpad;
  const float scale = rsqrtf((float)DH) * 1.4426950408889634f;
  const int tpad = p.tpad, Rrow = p.R;
  const int hole = __builtin_amdgcn_readfirstlane(*p.hole_row), skip = p.frame_tokens;
  constexpr int RPI = 64 / KCH;  // K rows per DMA instruction

  // DMA of tile t into stage sk, shared by the two waves (same layout and
  // swizzles as the 16-row variant)
  auto issue = [&](int t, unsigned char* sk) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const bool dyn = t >= n_ct;
    const int base = dyn ? (t - n_ct) * AKT : t * AKT;
    const int last = (dyn ? T_ : Lc) - 1;
    unsigned char* sv = sk + KBYTES;
    const int kl = ln % KCH, kr = ln / KCH;
    const int vd = ln >> 3, vc = ln & 7;
    if (dyn) {
#pragma unroll
      for (int j = 0; j < NIK; ++j) {
        const int row = RPI * (wave * NIK + j) + kr;
        const int r = min(base + row, last);
        __builtin_amdgcn_global_load_lds(kdb + r * DH + (kl ^ RFX_KSWZ(row, KCH)) * 8, sk + (wave * NIK + j) * 1024, 16,
                                         0, 0);
      }
#pragma unroll
      for (int j = 0; j < NIV; ++j) {
        const int d = (wave * NIV + j) * 8 + vd;
        __builtin_amdgcn_global_load_lds(vdb + d * tpad + base + (vc ^ (d & 7)) * 8, sv + (wave * NIV + j) * 1024, 16,
                                         0, 0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NIK; ++j) {
        const int row = RPI * (wave * NIK + j) + kr;
        int r = min(base + row, last);
        r += r >= hole ? skip : 0;
        __builtin_amdgcn_global_load_lds(ck + (int64_t)r * DH + (kl ^ RFX_KSWZ(row, KCH)) * 8,
                                         sk + (wave * NIK + j) * 1024, 16, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < NIV; ++j) {
        const int d = (wave * NIV + j) * 8 + vd;
        int key = base + (vc ^ (d & 7)) * 8;
        key = key <= last ? key : 0;
        key += key >= hole ? skip : 0;
        __builtin_amdgcn_global_load_lds(cvt + (int64_t)d * Rrow + key, sv + (wave * NIV + j) * 1024, 16, 0, 0);
      }
    }
  };

  f32x4_v o[NDH][2];
#pragma unroll
  for (int db = 0; db < NDH; ++db)
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) o[db][rr] = f32x4_v{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};

  // per-lane LDS read offsets (bytes).  K: row rho = 32h + 8*(r16 >> 2) + 4e +
  // (r16 & 3), d-chunk 4*ks + g, the low bits of ks in x.  V^T: row r16 of a
  // d block, key chunk 4j + g of the wave's own (j = h) and the partner's
  // (j = 1 - h) 32 keys.
  int koff[2][NKO];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int rho = 32 * h + 8 * (r16 >> 2) + 4 * e + (r16 & 3);
#pragma unroll
    for (int x = 0; x < NKO; ++x) koff[e][x] = rho * KRB + ((4 * x + g) ^ RFX_KSWZ(rho, KCH)) * 16;
  }
  const int voff_own = h * NDH * 16 * VRB + r16 * VRB + ((4 * h + g) ^ (r16 & 7)) * 16;
  const int voff_oth = h * NDH * 16 * VRB + r16 * VRB + ((4 * (1 - h) + g) ^ (r16 & 7)) * 16;

  auto step = [&](int t, const unsigned char* cur, unsigned char* nxt) __attribute__((always_inline)) {
    const bool dyn = t >= n_ct;
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0): this wave's share of tile t
    lds_barrier();
    if (t + 1 < t_end) issue(t + 1, nxt);
    const unsigned char* sk = cur;
    const unsigned char* sv = cur + KBYTES;

    // S^T for the wave's 32 keys x 32 rows: s[e][rr]
    f32x4_v s[2][2];
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int rr = 0; rr < 2; ++rr) s[e][rr] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k0 = 0; k0 < NKS; k0 += 2) {
      uint4 a[2][2];
#pragma unroll
      for (int u = 0; u < 2 && k0 + u < NKS; ++u)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int ks = k0 + u;
          a[u][e] = *reinterpret_cast<const uint4*>(sk + (ks / NKO) * NKO * 64 + koff[e][ks % NKO]);
        }
#pragma unroll
      for (int u = 0; u < 2 && k0 + u < NKS; ++u)
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
          for (int rr = 0; rr < 2; ++rr) mfma_step(s[e][rr], a[u][e], qf[rr][k0 + u], T());
    }

    // lane (r16, g) holds keys 32h + 8g + 4e + i of row r16 in block rr;
    // visible iff below lim (cached rows below Lc; the state row sees only
    // dynamic key 0)
    float mt[2];
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      const int lim = (dyn ? (iq[rr] > 0 ? T_ : 1) - (t - n_ct) * AKT : Lc - t * AKT) - 32 * h - 8 * g;
      float m = -INFINITY;
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = 4 * e + i < lim ? s[e][rr][i] * scale : -INFINITY;
          s[e][rr][i] = v;
          m = fmaxf(m, v);
        }
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      mt[rr] = m;
    }
    // (1) row maxima of the two key halves
    if (g == 0) {
      xbuf[h][0][r16] = mt[0];
      xbuf[h][1][r16] = mt[1];
    }
    lds_barrier();
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) mt[rr] = fmaxf(mt[rr], xbuf[1 - h][rr][r16]);

    // lazy rescaling, identical in both waves of the pair (same maxima, same
    // running max): the running max moves only when a row's tile max exceeds
    // it by more than 8 (log2 units)
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      if (__any(mt[rr] > m_run[rr] + 8.f)) {
        const float m_new = fmaxf(m_run[rr], mt[rr]);
        const float corr = m_new == -INFINITY ? 1.f : exp2f(m_run[rr] - m_new);
        l_run[rr] *= corr;
        m_run[rr] = m_new;
#pragma unroll
        for (int db = 0; db < NDH; ++db) o[db][rr] *= corr;
      }
    }
    uint4 pf[2];
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      const float m_use = (m_run[rr] == -INFINITY) ? 0.f : m_run[rr];
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = __builtin_amdgcn_exp2f(s[e][rr][i] - m_use);
          s[e][rr][i] = x;
          psum += x;
        }
      psum += __shfl_xor(psum, 16, 64);
      psum += __shfl_xor(psum, 32, 64);
      l_run[rr] += psum;
      pf[rr] = make_uint4(pack_bf16x2(s[0][rr][0], s[0][rr][1]), pack_bf16x2(s[0][rr][2], s[0][rr][3]),
                          pack_bf16x2(s[1][rr][0], s[1][rr][1]), pack_bf16x2(s[1][rr][2], s[1][rr][3]));
    }
    // (2) probabilities of the two key halves, as P.V B operands
    pbuf[h][0][lane] = pf[0];
    pbuf[h][1][lane] = pf[1];
    lds_barrier();
    uint4 po[2];
    po[0] = pbuf[1 - h][0][lane];
    po[1] = pbuf[1 - h][1][lane];

    // O^T (the wave's half of the head) += V^T P^T over the own and the
    // partner's 32 keys
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int voff = c == 0 ? voff_own : voff_oth;
#pragma unroll
      for (int d0 = 0; d0 < NDH; d0 += 4) {
        uint4 vf[4];
#pragma unroll
        for (int u = 0; u < 4 && d0 + u < NDH; ++u)
          vf[u] = *reinterpret_cast<const uint4*>(sv + (d0 + u) * 16 * VRB + voff);
#pragma unroll
        for (int u = 0; u < 4 && d0 + u < NDH; ++u)
#pragma unroll
          for (int rr = 0; rr < 2; ++rr) mfma_step(o[d0 + u][rr], vf[u], c == 0 ? pf[rr] : po[rr], T());
      }
    }
  };

  if (t_beg < t_end) issue(t_beg, stage0);
  for (int t = t_beg; t < t_end; t += 2) {
    step(t, stage0, stage1);
    if (t + 1 < t_end) step(t + 1, stage1, stage0);
  }

  // row sums over all keys: own half + the partner's half
  if (g == 0) {
    xbuf[h][0][r16] = l_run[0];
    xbuf[h][1][r16] = l_run[1];
  }
  lds_barrier();
  float l_tot[2];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) l_tot[rr] = l_run[rr] + xbuf[1 - h][rr][r16];

  const int dbase = h * (DH / 2) + 4 * g;
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) {
    if (!qvalid[rr]) continue;
    if (p.nsplit == 1) {
      const float inv = l_tot[rr] > 0.f ? 1.f / l_tot[rr] : 0.f;
      T* dst = reinterpret_cast<T*>(p.out) + ((int64_t)b * T_ + iq[rr]) * (int64_t)(Hq * DH) + jq[rr] * DH + dbase;
#pragma unroll
      for (int db = 0; db < NDH; ++db)
        *reinterpret_cast<uint2*>(dst + db * 16) =
            make_uint2(pack_bf16x2(o[db][rr][0] * inv, o[db][rr][1] * inv),
                       pack_bf16x2(o[db][rr][2] * inv, o[db][rr][3] * inv));
    } else {
      const int64_t prow = ((int64_t)b * p.nsplit + split) * p.rows_pad + rq[rr];
      T* dst = reinterpret_cast<T*>(p.part_o) + prow * DH + dbase;
#pragma unroll
      for (int db = 0; db < NDH; ++db)
        *reinterpret_cast<uint2*>(dst + db * 16) =
            make_uint2(pack_bf16x2(o[db][rr][0], o[db][rr][1]), pack_bf16x2(o[db][rr][2], o[db][rr][3]));
      if (h == 0 && g == 0) *reinterpret_cast<float2*>(p.part_ml + prow * 2) = make_float2(m_run[rr], l_tot[rr]);
    }
  }
}

// Merge the key splits: o = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,
// splits combined in index order.  One thread per (query row, VEC
// consecutive d): 16-byte accesses (8 bf16 or 4 fp32 values) when the grid
// still holds a wave of blocks, else 4-byte ones (2 bf16) for four times the
// blocks at a few envs (one env: 3.45 -> 3.13 us against 8-byte ones).
// The partial O_s are fp32 on the fp32 path and bf16 on the bf16 path.
constexpr int kMaxSplits = 16;

// MAXS: the split count it is compiled for (at least p.nsplit): the partials
// of every split are held in registers at once, so a bound of 16 for two
// splits would cost the occupancy a memory-bound kernel needs.
template <typename T, int DH, int VEC, int MAXS>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs p) {
  static_assert(VEC * sizeof(T) == 16 || VEC * sizeof(T) == 8 || VEC * sizeof(T) == 4, "4-, 8- or 16-byte accesses");
  using Raw = typename std::conditional<VEC * sizeof(T) == 16, uint4,
                                        typename std::conditional<VEC * sizeof(T) == 8, uint2, uint32_t>::type>::type;
  constexpr int TPR = DH / VEC;             // threads per row
  constexpr int RPB = 256 / TPR;            // rows per block
  const int b = blockIdx.y;
  const int rsub = threadIdx.x / TPR, d = (threadIdx.x % TPR) * VEC;
  const int rq = blockIdx.x * RPB + rsub;
  const int nrows = p.T * p.Hq;
  if (rq >= nrows) return;
  const int64_t base = (int64_t)b * p.nsplit * p.rows_pad + rq;
  // all loads of this thread are independent: one memory round trip
  // (the raw partials are converted only after every load is issued)
  float2 ml[MAXS];
  Raw raw[MAXS];
#pragma unroll
  for (int s = 0; s < MAXS; ++s) {
    if (s < p.nsplit) {
      const int64_t prow = base + (int64_t)s * p.rows_pad;
      ml[s] = *reinterpret_cast<const float2*>(p.part_ml + prow * 2);
      raw[s] = *reinterpret_cast<const Raw*>(reinterpret_cast<const T*>(p.part_o) + prow * DH + d);
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < MAXS; ++s)
    if (s < p.nsplit) M = fmaxf(M, ml[s].x);
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float L = 0.f;
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
#pragma unroll
  for (int s = 0; s < MAXS; ++s)
    if (s < p.nsplit) {
      const float w = exp2f(ml[s].x - Mu);
      L += w * ml[s].y;
      const uint32_t* wd = reinterpret_cast<const uint32_t*>(&raw[s]);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        float v;
        if constexpr (sizeof(T) == 2)
          v = __uint_as_float((e & 1) ? (wd[e >> 1] & 0xffff0000u) : (wd[e >> 1] << 16));
        else
          v = __uint_as_float(wd[e]);
        acc[e] += w * v;
      }
    }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const int i = rq / p.Hq, j = rq % p.Hq;
  T* dst = reinterpret_cast<T*>(p.out) + ((int64_t)b * p.T + i) * (int64_t)(p.Hq * DH) + j * DH + d;
  Raw outw;
  uint32_t* w = reinterpret_cast<uint32_t*>(&outw);
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int e = 0; e < VEC / 2; ++e)
      w[e] = (uint32_t)f2bf(acc[2 * e] * inv) | ((uint32_t)f2bf(acc[2 * e + 1] * inv) << 16);
  } else {
#pragma unroll
    for (int e = 0; e < VEC; ++e) w[e] = __float_as_uint(acc[e] * inv);
  }
  *reinterpret_cast<Raw*>(dst) = outw;
}

// Query rows per attention workgroup: 128 on the bf16 path, 64 on fp32.
int attention_rows_per_block(int elem_bytes) { return elem_bytes == 2 ? 128 : 64; }

// Kernel and key-split count for (B envs, rows query rows, up to max_keys
// cached keys).  One workgroup per CU is resident (LDS bound), so both aim
// for about one wave of workgroups over the 256 CUs.  The 16-row variants
// cover 128 rows per workgroup; when that grid would reach one key tile per
// split (a few envs, short context) the launch is latency-bound and the
// wave-pair variant (32 rows per workgroup, one tile per split) is used,
// otherwise the software-pipelined 16-row kernel.  `force` (ATTN_AUTO,
// ATTN_ROWS16, ATTN_PAIR or ATTN_ROWS16_PIPE) overrides the choice.
AttnPlan attention_plan(int B, int rows, int max_keys, int elem_bytes, int force) {
  const int tiles = (max_keys + AKT - 1) / AKT + 1;
  AttnPlan pl;
  pl.kernel = ATTN_ROWS16;
  const int rpb = attention_rows_per_block(elem_bytes);
  int base = B * ((rows + rpb - 1) / rpb);
  if (elem_bytes == 2) {
    const bool latency = 256 / base >= tiles;
    if (force == ATTN_PAIR || (force == ATTN_AUTO && latency)) {
      pl.kernel = ATTN_PAIR;
      base = B * ((rows + 31) / 32);
    } else if (force != ATTN_ROWS16) {
      pl.kernel = ATTN_ROWS16_PIPE;
    }
  }
  int s = 256 / base;
  if (s > tiles) s = tiles;
  if (s > kMaxSplits) s = kMaxSplits;
  pl.splits = s < 1 ? 1 : s;
  return pl;
}

template <typename T, int DH>
static void launch_attn_dh(const AttnArgs& a, hipStream_t s) {
  const int groups = a.B * a.nsplit;
  if constexpr (sizeof(T) == 2) {
    const int rows = a.T * a.Hq;
    const int g8 = ((groups + 7) / 8) * 8;
    if (a.kernel == ATTN_PAIR)
      RFX_LAUNCH((attn_pair_kernel<DH>), dim3(g8 * ((rows + 31) / 32)), dim3(128), 0, s, a);
    else if (a.kernel == ATTN_ROWS16_PIPE)
      RFX_LAUNCH((attn16p_kernel<DH>), dim3(g8 * (a.rows_pad / 128)), dim3(512), 0, s, a);
    else
      RFX_LAUNCH((attn16_kernel<DH>), dim3(g8 * (a.rows_pad / 128)), dim3(512), 0, s, a);
  } else {
    const int nwg = ((groups + 7) / 8) * 8 * (a.rows_pad / 64);
    RFX_LAUNCH((attn_kernel<T, DH>), dim3(nwg), dim3(256), 0, s, a);
  }
}

template <typename T, int DH, int VEC>
static void launch_merge_vec(const AttnArgs& a, dim3 grid, hipStream_t s) {
  if (a.nsplit <= 2)
    RFX_LAUNCH((attn_merge_kernel<T, DH, VEC, 2>), grid, dim3(256), 0, s, a);
  else if (a.nsplit <= 4)
    RFX_LAUNCH((attn_merge_kernel<T, DH, VEC, 4>), grid, dim3(256), 0, s, a);
  else if (a.nsplit <= 8)
    RFX_LAUNCH((attn_merge_kernel<T, DH, VEC, 8>), grid, dim3(256), 0, s, a);
  else
    RFX_LAUNCH((attn_merge_kernel<T, DH, VEC, kMaxSplits>), grid, dim3(256), 0, s, a);
}

template <typename T, int DH>
static void launch_merge_dh(const AttnArgs& a, hipStream_t s) {
  constexpr int V16 = 16 / (int)sizeof(T);
  constexpr int RPB16 = 256 / (DH / V16);
  const int rows = a.T * a.Hq;
  const int blocks16 = (rows + RPB16 - 1) / RPB16 * a.B;
  if (sizeof(T) == 4 || blocks16 >= 256) {
    launch_merge_vec<T, DH, V16>(a, dim3((rows + RPB16 - 1) / RPB16, a.B), s);
  } else {
    constexpr int RPB4 = 256 / (DH / 2);
    launch_merge_vec<T, DH, 2>(a, dim3((rows + RPB4 - 1) / RPB4, a.B), s);
  }
}

template <typename T>
hipError_t launch_attention(const AttnArgs& a, int head_dim, hipStream_t s) {
  if (a.nsplit < 1 || a.nsplit > kMaxSplits || a.rows_pad % 128) return hipErrorInvalidValue;
  if (a.kernel != ATTN_ROWS16 && a.kernel != ATTN_PAIR && a.kernel != ATTN_ROWS16_PIPE) return hipErrorInvalidValue;
  switch (head_dim) {
    case 64: launch_attn_dh<T, 64>(a, s); break;
    case 128: launch_attn_dh<T, 128>(a, s); break;
    case 256: launch_attn_dh<T, 256>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
hipError_t launch_attn_merge(const AttnArgs& a, int head_dim, hipStream_t s) {
  if (a.nsplit <= 1) return hipSuccess;
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
