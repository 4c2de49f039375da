// Internal launch interface between the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace reflex {

// Start/stop events attached to the next launch (profiling only).  With both
// null the launch is a plain dispatch; otherwise the runtime stamps the
// events from the kernel's own dispatch packet, so the elapsed time is the
// kernel's execution time without host-side launch overhead.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
extern thread_local LaunchEvents g_launch_events;

#define RFX_LAUNCH(kernel, grid, block, shm, stream, ...)                                            \
  hipExtLaunchKernelGGL(kernel, grid, block, shm, stream, ::reflex::g_launch_events.start,          \
                        ::reflex::g_launch_events.stop, 0, __VA_ARGS__)

enum Epi : int {
  EPI_F32 = 0,   // out_f32[z][split][row][col] = acc (split-K partial sums)
  EPI_SILU = 1,  // out_t[z][row][col] = silu(acc)
  EPI_GELU = 2,  // paired B rows c and N + c: out_t[row][c] = gelu_tanh(gate) * up
  EPI_MOD = 3,   // like EPI_F32 (one split); with mod_width > 0 the shift/gate
                 // columns are replaced by 0/1 (scale-only modulation)
  EPI_ROPE = 4,  // packed QKV, paired columns d and d + head_dim/2 of a head:
                 // RoPE on q and k heads, scattered to the attention layouts
  EPI_KV = 5,    // frame K/V projection, paired columns d and d + head_dim/2 of
                 // each layer's K or V block: RoPE on K, written straight into
                 // the cache (K rows, V^T columns) of the frame's ring slot
};

// Destinations of the EPI_ROPE epilogue (row m = b*T + i of the GEMM).
struct QkvOut {
  const float2* rope;  // [T][head_dim/2] (cos, sin) at the dynamic positions
  void* q;             // [B][rows_pad][head_dim], row i*Hq + j  (RoPE applied)
  void* k;             // [B][T][head_dim]                       (RoPE applied)
  void* vt;            // [B][head_dim][tpad], column i          (V transposed)
  int T, Hq, head_dim, rows_pad, tpad;
};

// Destinations of the EPI_KV epilogue (row m = b*F + j of the GEMM, column
// n = (2l + kv)*head_dim + d): K rows and V^T columns of ring rows row0 + j.
struct KvOut {
  const float2* rope;  // [F][head_dim/2] (cos, sin) at the frame's positions
  void* cache_k;       // [B][L][R][head_dim]
  void* cache_vt;      // [B][L][head_dim][R]
  int R, row0, F, L;
};

// C[M][N] = A[M][K] * B[N][K]^T (+ epilogue).
struct GemmArgs {
  const void* A;
  const void* B;
  void* out;
  int64_t lda, ldb, ldo;              // row strides in elements
  int64_t a_bstride, b_bstride;       // per blockIdx.z strides (elements)
  int64_t o_bstride, o_split_stride;  // output strides (elements)
  int M, N, K;
  int splits;        // K split across workgroups (EPI_F32 only)
  int k_per_split;   // multiple of the k-step
  int mod_width;     // EPI_MOD: width D, 0 = full modulation
  int batch;         // blockIdx.z extent
  QkvOut qkv;        // EPI_ROPE; EPI_KV uses qkv.head_dim only
  KvOut kv;          // EPI_KV only
};

template <typename T> hipError_t launch_gemm(const GemmArgs& a, int epi, hipStream_t s);
// Heuristic: number of K splits for an EPI_F32 GEMM.
int gemm_pick_splits(int M, int N, int K, int elem_bytes);

// Partitioned-region attention (Eq. 1) for the dynamic rows of every env.
struct AttnArgs {
  const void* q;          // [B][rows_pad][dh]  RoPE applied
  const void* kd;         // [B][T][dh]         dynamic keys, RoPE applied
  const void* vdt;        // [B][dh][tpad]      dynamic values, transposed, zero beyond T
  int tpad;
  const void* cache_k;    // layer base: [B] stride ck_bstride, rows [R][dh]
  const void* cache_vt;   // layer base: [B] stride ck_bstride, [dh][R]
  int64_t ck_bstride;     // elements between envs (= L*R*dh)
  const int32_t* n_valid; // device: frames visible in the ring
  // device: cached rows are read in logical order; logical row j >= *hole_row
  // sits one frame further in memory (the spare slot of a pipelined ring is
  // skipped).  A value past the visible rows means no skip.  Both are
  // multiples of 8 rows, so no 16-byte load straddles the skip.
  const int32_t* hole_row;
  int static_len, frame_tokens, R;
  int B, T, Hq;
  int nsplit;             // key splits (blockIdx.x)
  float* part_o;          // [B][nsplit][rows_pad][dh], fp32 (fp32 path) or bf16 (bf16 path)
  float* part_ml;         // [B][nsplit][rows_pad][2]
  int rows_pad;
  void* out;              // [B*T][Hq*dh]
  int kernel;             // bf16 path: ATTN_ROWS16, ATTN_PAIR or ATTN_ROWS16_PIPE
};
template <typename T> hipError_t launch_attention(const AttnArgs& a, int head_dim, hipStream_t s);
template <typename T> hipError_t launch_attn_merge(const AttnArgs& a, int head_dim, hipStream_t s);
int attention_rows_per_block(int elem_bytes);
// bf16 attention kernels: 16-row waves (128 rows per workgroup; plain or
// software-pipelined, equal bit for bit) or one wave pair per workgroup (32
// rows); ATTN_AUTO picks by the launch geometry
enum AttnKernel : int { ATTN_AUTO = 0, ATTN_ROWS16 = 1, ATTN_PAIR = 2, ATTN_ROWS16_PIPE = 3 };
struct AttnPlan {
  int kernel;
  int splits;
};
AttnPlan attention_plan(int B, int rows, int max_keys, int elem_bytes, int force);

// Precision of the residual stream and of the RMS statistics.  NORM_FP32 is
// the method (fp32 statistics, Section 3.2); the other two reproduce the
// baselines of the stability ablation: a bf16 residual stream with the
// statistics accumulated in bf16 (every product and partial sum rounded), or
// with fp32 statistics ("fp32 norm-only").
enum NormMode : int { NORM_FP32 = 0, NORM_BF16 = 1, NORM_BF16_FP32_STATS = 2 };

// Token embedding + first AdaRMSNorm: h = embed_scale*[s W_s^T ; x W_ain^T], y = ada(h).
struct EmbedArgs {
  const float* x;        // [B][H][da]
  const float* state;    // [B][ds]
  const void* w_state;   // [D][ds]
  const void* w_ain;     // [D][da]
  const float* mod;      // site block for this step: [B][3D]
  float* h;              // [B*T][D]
  void* y;               // [B*T][D]
  int B, T, D, ds, da;
  float embed_scale, eps;
  int norm_mode;         // NormMode
};
template <typename T> hipError_t launch_embed_norm(const EmbedArgs& a, hipStream_t s);

// h += gate (.) sum_s parts[s]; y = ada(h) with the next site's scale/shift.
struct ResidArgs {
  float* h;               // [M][D]
  const float* parts;     // [nparts][M][D]
  int64_t part_stride;
  int nparts;
  const float* gate_mod;  // [B][3D] block of the residual's site (gate at +2D)
  const float* norm_mod;  // [B][3D] block of the next norm site
  void* y;                // [M][D]
  int M, T, D;
  float eps;
  int norm_mode;          // NormMode
};
template <typename T> hipError_t launch_resid_norm(const ResidArgs& a, hipStream_t s);

// Last residual + final AdaRMSNorm + action head + Euler update.
struct FinalArgs {
  const float* h;         // [B*T][D]
  const float* parts;
  int64_t part_stride;
  int nparts;
  const float* gate_mod;  // [B][3D]
  const float* final_mod; // [B][3D]
  const void* w_aout;     // [da][D]
  const float* x_in;      // [B][H][da]
  float* x_out;           // [B][H][da]
  int B, T, D, da;
  float dt, eps;
  int norm_mode;          // NormMode
  int32_t* status;        // bit 0 set when an action leaves the kernel non-finite
  // fuse_next: also the next Euler step's token embedding and first norm
  // (`next` as for launch_embed_norm; its x is this kernel's x_out, taken from
  // LDS), one extra block per env for the state row.  next.h must be h; only
  // where final_fuses_embed holds.
  int fuse_next;
  EmbedArgs next;
};
template <typename T> hipError_t launch_final_euler(const FinalArgs& a, hipStream_t s);
// whether launch_final_euler takes fuse_next for B envs of T tokens, width D
bool final_fuses_embed(int B, int T, int D);

// RoPE (cos, sin) table for positions pos0 + i, i < n; pos0 from *pos0_dev
// when non-null.  Angles formed in double.
hipError_t launch_rope_table(float2* out, const int64_t* pos0_dev, int64_t pos0, int n, int head_dim,
                             double theta, hipStream_t s);

// Conditioning rows c[k*B + b] = [sinusoidal(tau_k) ; state_b].
struct TauTable { float tau[65]; };
template <typename T> hipError_t launch_cond(void* cond, const float* state, const TauTable& taus, int K,
                                             int B, int D, int ds, double min_p, double max_p,
                                             hipStream_t s);

// Separate passes used by the unfused schedule of the fusion ablation: the
// work the fused kernels do in GEMM epilogues and in the residual/norm kernel.
struct ResidAddArgs {        // h += gate (.) sum_s parts[s]
  float* h;
  const float* parts;
  int64_t part_stride;
  int nparts;
  const float* gate_mod;     // [B][3D], gate at +2D
  int M, T, D;
};
hipError_t launch_resid_add(const ResidAddArgs& a, hipStream_t s);
struct NormArgs {            // y = h / rms(h) * (1 + scale) + shift
  const float* h;
  const float* norm_mod;     // [B][3D]
  void* y;
  int M, T, D;
  float eps;
};
template <typename T> hipError_t launch_norm(const NormArgs& a, hipStream_t s);
struct RopeScatterArgs {     // RoPE on the q and k heads of fp32 [M][(Hq+2)*dh] rows, scattered like EPI_ROPE
  const float* qkv;
  QkvOut out;
  int M;
};
template <typename T> hipError_t launch_rope_scatter(const RopeScatterArgs& a, hipStream_t s);
struct GeluMulArgs {         // z[m][c] = gelu_tanh(u[m][c]) * u[m][F + c]
  const float* u;
  void* z;
  int M, F;
};
template <typename T> hipError_t launch_gelu_mul(const GeluMulArgs& a, hipStream_t s);
struct EulerArgs {           // x_out = x_in + dt * v (action rows 1..T-1 of v [B*T][da])
  const float* v;
  const float* x_in;
  float* x_out;
  int B, T, da;
  float dt;
};
hipError_t launch_euler(const EulerArgs& a, hipStream_t s);

// Zero `bytes` (a multiple of 16) at a 16-byte aligned device address with a
// kernel (no memset node, so the launch is safe inside a captured graph).
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

// Sets the device tick state {frames, n_valid, dyn_pos0, hole_row} that the
// next chunk on this stream reads (one thread; the chunk's kernels follow in
// stream order).
hipError_t launch_tick_set(int64_t* tick, int64_t frames, int64_t n_valid, int64_t dyn_pos0, int64_t hole_row,
                           hipStream_t s);

// Ring/static write: K rows get RoPE from the table, V is stored transposed.
struct RingWriteArgs {
  const void* src_k;     // element (b, l, j, d) at b*sb + l*sl + j*sj + d
  const void* src_v;
  int64_t sb, sl, sj;
  const float2* rope;    // [n_tok][dh/2]
  void* cache_k;         // cache base, [B][L][R][dh]
  void* cache_vt;        // cache base, [B][L][dh][R]
  int row0;              // first cache row written
  int n_tok, L, B, R;
  // tick state update (written by block 0 when tick != nullptr)
  int64_t* tick;
  int64_t frames_written, dyn_pos0, hole_row;
  int32_t n_valid;
};
template <typename T, typename S> hipError_t launch_ring_write(const RingWriteArgs& a, int head_dim,
                                                               hipStream_t s);

}  // namespace reflex
