// C ABI of the Reflex denoise hot path (declared in include/reflex.h).
//
// The context holds only host integers and the caller's device pointers; the
// ring bookkeeping (frame index, slot, positions, eviction count) follows the
// FIFO window of Section 3.1 and the circular pointer arithmetic of Section 3.4
// / Appendix B.2, and is mirrored into a small device "tick state" so the
// captured denoise graph reads the current window length and dynamic positions
// from memory and never needs re-capture when a frame arrives.
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "../../include/reflex.h"
#include "common.h"
#include "kernels.h"

using namespace reflex;

namespace reflex {
thread_local LaunchEvents g_launch_events;
}

namespace {

thread_local char g_hip_err[256] = "";

enum ProfClass {
  PC_EMBED = 0, PC_QKV, PC_ATTN, PC_MERGE, PC_O, PC_RESID, PC_GU, PC_DOWN, PC_FINAL, PC_MOD, PC_ROPE, PC_FRAME_PROJ,
  PC_RING, PC_N
};
const char* const kProfNames[PC_N] = {"embed_norm", "gemm_qkv",     "attention", "attn_merge",
                                      "gemm_o",     "resid_norm",   "gemm_gate_up", "gemm_down",
                                      "final_euler", "modulation",  "rope_table",   "frame_proj",
                                      "ring_write"};

struct SplitK {
  int splits = 1;
  int kps = 0;
};

struct GraphEntry {
  const float* state;
  const float* noise;
  float* out;
  int steps;
  float taus[REFLEX_MAX_STEPS + 1];
  int mode;
  // Standard mode bakes the window's slots and positions into the graph
  int64_t frames_written;
  std::vector<const void*> srcs;
  hipGraphExec_t exec;
};

struct Workspace {
  int64_t* tick;
  int32_t* status;  // bytes 32..35 of the tick block: bit 0 = a non-finite action was produced
  float2* rope_dyn;
  float2* rope_frame;
  void* cond;
  void* hid;
  float* mod;
  float* h;
  void* y;
  void* q;
  void* kd;
  void* vdt;
  void* o;
  float* part_o;
  float* part_ml;
  void* z;
  float* rparts;
  void* naive_k;   // [L][B][T][dh] dynamic K of the first Euler step (Naive mode)
  void* naive_vt;  // [L][B][dh][tpad] dynamic V^T of the first Euler step (Naive mode)
  float* uf_wide;  // [M][max(Nqkv, 2*mlp)] fp32 projection outputs (unfused schedule)
  float* uf_v;     // [M][da] fp32 action-head output (unfused schedule)
};

constexpr int kWsParts = 22;

struct Plan {
  int T, M, S, Nqkv, C, R, slots, rows_pad, tpad, eb;
  SplitK o, down;
  int attn_splits, attn_kernel;
  int max_parts;
  size_t naive_k_stride, naive_vt_stride;  // per-layer bytes of the Naive-mode dynamic K/V
  size_t cache_bytes, ws_bytes;
  size_t off[kWsParts];
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

SplitK make_split(int M, int K, int splits, int eb) {
  // skinny kernels step K in 64-byte k-steps, tiled kernels in 128-byte stages
  const int gran = (M <= 64 ? 64 : 128) / eb;
  SplitK s;
  if (splits < 1) splits = 1;
  int kps = (K + splits - 1) / splits;
  kps = (kps + gran - 1) / gran * gran;
  s.kps = kps;
  s.splits = (K + kps - 1) / kps;
  return s;
}

int validate(const reflex_config* c) {
  if (!c) return REFLEX_EINVAL;
  if (c->dtype != REFLEX_DTYPE_F32 && c->dtype != REFLEX_DTYPE_BF16) return REFLEX_EINVAL;
  if (c->mod_mode != REFLEX_MOD_FULL && c->mod_mode != REFLEX_MOD_SCALE_ONLY) return REFLEX_EINVAL;
  if (c->n_layers < 1 || c->n_layers > 1024) return REFLEX_EINVAL;
  if (c->width < 64 || c->width > 4096 || c->width % 64) return REFLEX_EINVAL;
  if (c->mlp_dim < 64 || c->mlp_dim % 64) return REFLEX_EINVAL;
  if (c->cond_hidden < 64 || c->cond_hidden % 64) return REFLEX_EINVAL;
  if (c->n_q_heads < 1 || c->n_q_heads > 64) return REFLEX_EINVAL;
  if (c->n_kv_heads != 1) return REFLEX_EINVAL;
  if (c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256) return REFLEX_EINVAL;
  if (c->dtype == REFLEX_DTYPE_F32 && c->head_dim > 128) return REFLEX_EINVAL;
  if (c->state_dim < 8 || c->state_dim > 64 || c->state_dim % 8) return REFLEX_EINVAL;
  if (c->action_dim < 1 || c->action_dim > 64) return REFLEX_EINVAL;
  if (c->action_horizon < 1 || c->action_horizon + 1 > 128) return REFLEX_EINVAL;
  if (c->static_len < 0 || c->static_len % 8) return REFLEX_EINVAL;
  if (c->frame_tokens < 8 || c->frame_tokens % 8) return REFLEX_EINVAL;
  if (c->window_frames < 1) return REFLEX_EINVAL;
  if (c->spare_slot != 0 && c->spare_slot != 1) return REFLEX_EINVAL;
  if (c->norm_precision < REFLEX_NORM_FP32 || c->norm_precision > REFLEX_NORM_BF16_FP32_STATS) return REFLEX_EINVAL;
  if (c->attn_kernel < REFLEX_ATTN_AUTO || c->attn_kernel > REFLEX_ATTN_ROWS16_PIPE) return REFLEX_EINVAL;
  if (c->frame_dim < 0 || c->frame_dim % 8) return REFLEX_EINVAL;
  if (c->batch < 1 || c->batch > 4096) return REFLEX_EINVAL;
  if (c->max_steps < 1 || c->max_steps > REFLEX_MAX_STEPS) return REFLEX_EINVAL;
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.0) || !(c->temb_min_period > 0.0) ||
      !(c->temb_max_period > 0.0))
    return REFLEX_EINVAL;
  const int64_t R = (int64_t)c->static_len + ((int64_t)c->window_frames + c->spare_slot) * c->frame_tokens;
  if (R > (1 << 24)) return REFLEX_EINVAL;
  return REFLEX_OK;
}

Plan make_plan(const reflex_config* c) {
  Plan p;
  const int eb = c->dtype == REFLEX_DTYPE_BF16 ? 2 : 4;
  p.eb = eb;
  p.T = 1 + c->action_horizon;
  p.M = c->batch * p.T;
  p.S = 2 * c->n_layers + 1;
  p.Nqkv = (c->n_q_heads + 2) * c->head_dim;
  p.C = c->width + c->state_dim;
  p.slots = c->window_frames + c->spare_slot;
  p.R = c->static_len + p.slots * c->frame_tokens;
  const int rows = p.T * c->n_q_heads;
  p.rows_pad = (rows + 127) / 128 * 128;
  p.tpad = (p.T + 63) / 64 * 64;
  p.o = make_split(p.M, c->n_q_heads * c->head_dim,
                   gemm_pick_splits(p.M, c->width, c->n_q_heads * c->head_dim, eb), eb);
  p.down = make_split(p.M, c->mlp_dim, gemm_pick_splits(p.M, c->width, c->mlp_dim, eb), eb);
  const AttnPlan ap = attention_plan(c->batch, rows, p.R, eb, c->attn_kernel);
  p.attn_splits = ap.splits;
  p.attn_kernel = ap.kernel;
  p.max_parts = p.o.splits > p.down.splits ? p.o.splits : p.down.splits;

  const size_t B = c->batch, L = c->n_layers, dh = c->head_dim, D = c->width, K = c->max_steps;
  p.cache_bytes = align256(B * L * p.R * dh * eb) * 2;
  size_t sz[kWsParts];
  sz[0] = 64;                                                             // tick
  sz[1] = (size_t)p.T * (dh / 2) * sizeof(float2);                        // rope_dyn
  sz[2] = (size_t)(c->static_len > c->frame_tokens ? c->static_len : c->frame_tokens) * (dh / 2) *
          sizeof(float2);                                                 // rope_frame
  sz[3] = K * B * p.C * eb;                                               // cond
  sz[4] = K * B * (size_t)p.S * c->cond_hidden * eb;                      // hid
  sz[5] = (size_t)p.S * K * B * 3 * D * sizeof(float);                    // mod
  sz[6] = (size_t)p.M * D * sizeof(float);                                // h
  sz[7] = (size_t)p.M * D * eb;                                           // y
  sz[8] = B * (size_t)p.rows_pad * dh * eb;                               // q
  sz[9] = B * (size_t)p.T * dh * eb;                                      // kd
  sz[10] = B * dh * (size_t)p.tpad * eb;                                  // vdt
  sz[11] = 0;  // (unused)
  sz[12] = (size_t)p.M * c->n_q_heads * dh * eb;                          // o
  sz[13] = B * p.attn_splits * (size_t)p.rows_pad * dh * sizeof(float);   // part_o
  sz[14] = B * p.attn_splits * (size_t)p.rows_pad * 2 * sizeof(float);    // part_ml
  sz[15] = (size_t)p.M * c->mlp_dim * eb;                                 // z
  sz[16] = (size_t)p.max_parts * p.M * D * sizeof(float);                 // rparts
  sz[17] = 0;  // (unused: the frame projection writes the cache from its epilogue)
  p.naive_k_stride = align256(sz[9]);
  p.naive_vt_stride = align256(sz[10]);
  sz[18] = L * p.naive_k_stride;                                          // naive_k
  sz[19] = L * p.naive_vt_stride;                                         // naive_vt
  sz[20] = (size_t)p.M * (p.Nqkv > 2 * c->mlp_dim ? p.Nqkv : 2 * c->mlp_dim) * sizeof(float);  // uf_wide
  sz[21] = (size_t)p.M * c->action_dim * sizeof(float);                   // uf_v
  size_t off = 0;
  for (int i = 0; i < kWsParts; ++i) {
    p.off[i] = off;
    off += align256(sz[i]);
  }
  p.ws_bytes = off;
  return p;
}

}  // namespace

struct reflex_ctx {
  reflex_config cfg;
  reflex_weights w;
  Plan plan;
  Workspace ws;
  void* cache_k;
  void* cache_vt;
  hipStream_t stream;
  int64_t frames_written;
  int alive;
  std::vector<GraphEntry> graphs;
  // profiling
  int prof_enabled;
  double prof_ms[PC_N];
  int32_t prof_launches[PC_N];
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> ev_pending;
  // in-graph timing: launches of the classes in stamp_mask (bit i: class i)
  // are bracketed by wall-clock stamps written to stamps[3 j .. 3 j + 2]
  uint32_t stamp_mask = 0;
  unsigned long long* stamps = nullptr;
  int32_t stamp_next = 0, stamp_cap = 0;
  // pipelined streaming (spare slot): completion events of the last two frame
  // writes (n = frame index) and of recent chunks (n = frames they read, one
  // record per distinct n, increasing), with a pool of free events
  struct EvRec {
    int64_t n;
    hipEvent_t ev;
    hipStream_t stream;
  };
  std::vector<EvRec> write_recs, chunk_recs;
  std::vector<hipEvent_t> pipe_free;
};

namespace {

int hip_fail(hipError_t e) {
  snprintf(g_hip_err, sizeof(g_hip_err), "HIP error %d: %s", (int)e, hipGetErrorString(e));
  return REFLEX_EHIP;
}

// Ring bookkeeping of writing frame f (Section 3.1 FIFO; Appendix B.2).  A
// ring with a spare slot places frame f in slot f mod (W + 1).
int plan_frame(const reflex_ctx* ctx, int64_t f, reflex_ring_step* stp) {
  const reflex_config& c = ctx->cfg;
  const int rc = reflex_ring_plan(f, c.window_frames, c.frame_tokens, c.static_len, stp);
  if (rc != REFLEX_OK) return rc;
  stp->slot = (int32_t)(f % ctx->plan.slots);
  return REFLEX_OK;
}

// Logical cached row from which the physical rows skip the spare slot, once n
// frames are written: the spare slot is the one frame n will be written into.
// Without a spare slot the rows are read in place (the value is past them).
int64_t hole_row(const reflex_ctx* ctx, int64_t n) {
  const reflex_config& c = ctx->cfg;
  if (!c.spare_slot) return ctx->plan.R;
  return (int64_t)c.static_len + (n % ctx->plan.slots) * c.frame_tokens;
}

hipEvent_t pipe_event(reflex_ctx* ctx) {
  if (!ctx->pipe_free.empty()) {
    hipEvent_t e = ctx->pipe_free.back();
    ctx->pipe_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
  return e;
}

// One thread writes the GPU's constant-rate wall clock: in a graph it runs
// after the previous launch has completed and before the next one starts.
__global__ __launch_bounds__(64) void stamp_kernel(unsigned long long* slot) {
  if (threadIdx.x == 0) *slot = (unsigned long long)wall_clock64();
}

struct Launcher {
  reflex_ctx* ctx;
  bool prof;
  size_t ev_next = 0;
  hipEvent_t take() {
    if (ev_next == ctx->ev_pool.size()) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      ctx->ev_pool.push_back(e);
    }
    return ctx->ev_pool[ev_next++];
  }
  hipError_t stamp(int k) {
    hipLaunchKernelGGL(stamp_kernel, dim3(1), dim3(64), 0, ctx->stream, ctx->stamps + ctx->stamp_next + k);
    return hipGetLastError();
  }
  template <typename F>
  int run(int cls, F&& f) {
    // in-graph timing: two adjacent stamps (their difference is the cost of a
    // launch boundary at this point of the graph), the launch, a third stamp
    const bool stamped = (ctx->stamp_mask >> cls) & 1u;
    if (stamped) {
      if (ctx->stamp_next + 3 > ctx->stamp_cap) return REFLEX_EINVAL;
      hipError_t e = stamp(0);
      if (e == hipSuccess) e = stamp(1);
      if (e != hipSuccess) return hip_fail(e);
    }
    hipEvent_t a = nullptr, b = nullptr;
    if (prof) {
      a = take();
      b = take();
      if (!a || !b) return hip_fail(hipErrorOutOfMemory);
      g_launch_events.start = a;
      g_launch_events.stop = b;
    }
    hipError_t e = f();
    g_launch_events = LaunchEvents{};
    if (e != hipSuccess) return hip_fail(e);
    if (prof) ctx->ev_pending.push_back({cls, {a, b}});
    if (stamped) {
      e = stamp(2);
      if (e != hipSuccess) return hip_fail(e);
      ctx->stamp_next += 3;
    }
    return REFLEX_OK;
  }
};

#define RFX_TRY(expr)           \
  do {                          \
    const int _rc = (expr);     \
    if (_rc != REFLEX_OK) return _rc; \
  } while (0)

template <typename T>
int write_static(reflex_ctx* ctx, const void* sk, const void* sv, bool publish, Launcher& L);
template <typename T>
int write_frame(reflex_ctx* ctx, const void* frame, const reflex_ring_step& stp, bool publish, Launcher& L,
                hipStream_t st);

// Standard mode (full history recomputation): the static prefix and every
// window frame are encoded into their cache rows again, with the kernels and
// positions of their first write, so the rows receive identical bytes.
template <typename T>
int reencode_history(reflex_ctx* ctx, const reflex_sources* src, Launcher& L) {
  const reflex_config& c = ctx->cfg;
  if (c.static_len > 0) RFX_TRY(write_static<T>(ctx, src->static_k, src->static_v, false, L));
  for (int i = 0; i < src->n_frames; ++i) {
    reflex_ring_step stp;
    RFX_TRY(plan_frame(ctx, ctx->frames_written - src->n_frames + i, &stp));
    RFX_TRY(write_frame<T>(ctx, src->frames[i], stp, false, L, ctx->stream));
  }
  return REFLEX_OK;
}

template <typename T>
int enqueue_chunk(reflex_ctx* ctx, const Workspace& W, const float* state, const float* noise, int steps,
                  const float* taus, float* out, bool prof, int mode, const reflex_sources* src) {
  const reflex_config& c = ctx->cfg;
  const Plan& P = ctx->plan;
  hipStream_t st = ctx->stream;
  Launcher L{ctx, prof};
  const int B = c.batch, Tn = P.T, M = P.M, D = c.width, dh = c.head_dim, Hq = c.n_q_heads;
  const int Kmax = c.max_steps;
  const int64_t site_stride = (int64_t)Kmax * B * 3 * D;
  auto mod_at = [&](int site, int k) { return W.mod + site * site_stride + (int64_t)k * B * 3 * D; };

  RFX_TRY(L.run(PC_ROPE, [&] { return launch_rope_table(W.rope_dyn, W.tick + 2, 0, Tn, dh, c.rope_theta, st); }));

  // conditioning MLPs for every step and site (hoisted: c depends on tau_k and s only)
  TauTable tt;
  memset(&tt, 0, sizeof(tt));
  for (int k = 0; k <= steps; ++k) tt.tau[k] = taus[k];
  RFX_TRY(L.run(PC_MOD, [&] {
    return launch_cond<T>(W.cond, state, tt, steps, B, D, c.state_dim, c.temb_min_period, c.temb_max_period, st);
  }));
  {
    GemmArgs g{};
    g.A = W.cond; g.lda = P.C;
    g.B = ctx->w.w_mod1; g.ldb = P.C;
    g.out = W.hid; g.ldo = (int64_t)P.S * c.cond_hidden;
    g.M = steps * B; g.N = P.S * c.cond_hidden; g.K = P.C;
    g.splits = 1; g.k_per_split = P.C + 64; g.batch = 1;
    RFX_TRY(L.run(PC_MOD, [&] { return launch_gemm<T>(g, EPI_SILU, st); }));
    GemmArgs h{};
    h.A = W.hid; h.lda = (int64_t)P.S * c.cond_hidden; h.a_bstride = c.cond_hidden;
    h.B = ctx->w.w_mod2; h.ldb = c.cond_hidden; h.b_bstride = (int64_t)3 * D * c.cond_hidden;
    h.out = W.mod; h.ldo = 3 * D; h.o_bstride = site_stride;
    h.M = steps * B; h.N = 3 * D; h.K = c.cond_hidden;
    h.splits = 1; h.k_per_split = c.cond_hidden + 64; h.batch = P.S;
    h.mod_width = c.mod_mode == REFLEX_MOD_SCALE_ONLY ? D : 0;
    RFX_TRY(L.run(PC_MOD, [&] { return launch_gemm<T>(h, EPI_MOD, st); }));
  }

  const size_t eb = sizeof(T);
  const char* wqkv = (const char*)ctx->w.w_qkv;
  const char* wo = (const char*)ctx->w.w_o;
  const char* wgu = (const char*)ctx->w.w_gu;
  const char* wdown = (const char*)ctx->w.w_down;
  const int64_t rpart_stride = (int64_t)M * D;

  // token embedding + first norm of step k (x_k, site 0 of step k).  With a
  // few rows (launch-bound) the final kernel of step k - 1 does it for k > 0.
  auto embed_args = [&](int k, const float* x) {
    return EmbedArgs{x, state, ctx->w.w_state, ctx->w.w_ain, mod_at(0, k), W.h, W.y,
                     B, Tn, D, c.state_dim, c.action_dim, c.embed_scale, c.rms_eps, c.norm_precision};
  };
  const bool fuse_embed = final_fuses_embed(B, Tn, D);
  for (int k = 0; k < steps; ++k) {
    const float* x_in = (k == 0) ? noise : out;
    if (mode == REFLEX_MODE_STANDARD) RFX_TRY(reencode_history<T>(ctx, src, L));
    if (k == 0 || !fuse_embed) {
      const EmbedArgs ea = embed_args(k, x_in);
      RFX_TRY(L.run(PC_EMBED, [&] { return launch_embed_norm<T>(ea, st); }));
    }
    for (int l = 0; l < c.n_layers; ++l) {
      GemmArgs q{};
      q.A = W.y; q.lda = D;
      q.B = wqkv + (size_t)l * P.Nqkv * D * eb; q.ldb = D;
      q.M = M; q.N = P.Nqkv; q.K = D; q.splits = 1; q.k_per_split = D + 128; q.batch = 1;
      // dynamic K/V read by the attention: this step's, or in Naive mode the
      // first step's, kept per layer
      void* kd = W.kd;
      void* vdt = W.vdt;
      if (mode == REFLEX_MODE_NAIVE) {
        kd = (char*)W.naive_k + (size_t)l * P.naive_k_stride;
        vdt = (char*)W.naive_vt + (size_t)l * P.naive_vt_stride;
      }
      const bool stale = mode == REFLEX_MODE_NAIVE && k > 0;
      q.qkv = QkvOut{W.rope_dyn, W.q, stale ? W.kd : kd, stale ? W.vdt : vdt, Tn, Hq, dh, P.rows_pad, P.tpad};
      RFX_TRY(L.run(PC_QKV, [&] { return launch_gemm<T>(q, EPI_ROPE, st); }));

      AttnArgs aa{};
      aa.q = W.q; aa.kd = kd; aa.vdt = vdt; aa.tpad = P.tpad;
      aa.cache_k = (const char*)ctx->cache_k + (size_t)l * P.R * dh * eb;
      aa.cache_vt = (const char*)ctx->cache_vt + (size_t)l * P.R * dh * eb;
      aa.ck_bstride = (int64_t)c.n_layers * P.R * dh;
      aa.n_valid = reinterpret_cast<const int32_t*>(W.tick + 1);
      aa.hole_row = reinterpret_cast<const int32_t*>(W.tick + 3);
      aa.static_len = c.static_len; aa.frame_tokens = c.frame_tokens; aa.R = P.R;
      aa.B = B; aa.T = Tn; aa.Hq = Hq; aa.nsplit = P.attn_splits; aa.kernel = P.attn_kernel;
      aa.part_o = W.part_o; aa.part_ml = W.part_ml;
      aa.rows_pad = P.rows_pad; aa.out = W.o;
      RFX_TRY(L.run(PC_ATTN, [&] { return launch_attention<T>(aa, dh, st); }));
      if (P.attn_splits > 1) RFX_TRY(L.run(PC_MERGE, [&] { return launch_attn_merge<T>(aa, dh, st); }));

      GemmArgs og{};
      og.A = W.o; og.lda = (int64_t)Hq * dh;
      og.B = wo + (size_t)l * D * Hq * dh * eb; og.ldb = (int64_t)Hq * dh;
      og.out = W.rparts; og.ldo = D; og.o_split_stride = rpart_stride;
      og.M = M; og.N = D; og.K = Hq * dh; og.splits = P.o.splits; og.k_per_split = P.o.kps; og.batch = 1;
      RFX_TRY(L.run(PC_O, [&] { return launch_gemm<T>(og, EPI_F32, st); }));

      ResidArgs r1{W.h, W.rparts, rpart_stride, P.o.splits, mod_at(2 * l, k), mod_at(2 * l + 1, k), W.y,
                   M, Tn, D, c.rms_eps, c.norm_precision};
      RFX_TRY(L.run(PC_RESID, [&] { return launch_resid_norm<T>(r1, st); }));

      GemmArgs gu{};
      gu.A = W.y; gu.lda = D;
      gu.B = wgu + (size_t)l * 2 * c.mlp_dim * D * eb; gu.ldb = D;
      gu.out = W.z; gu.ldo = c.mlp_dim;
      gu.M = M; gu.N = c.mlp_dim; gu.K = D; gu.splits = 1; gu.k_per_split = D + 128; gu.batch = 1;
      RFX_TRY(L.run(PC_GU, [&] { return launch_gemm<T>(gu, EPI_GELU, st); }));

      GemmArgs dg{};
      dg.A = W.z; dg.lda = c.mlp_dim;
      dg.B = wdown + (size_t)l * D * c.mlp_dim * eb; dg.ldb = c.mlp_dim;
      dg.out = W.rparts; dg.ldo = D; dg.o_split_stride = rpart_stride;
      dg.M = M; dg.N = D; dg.K = c.mlp_dim; dg.splits = P.down.splits; dg.k_per_split = P.down.kps; dg.batch = 1;
      RFX_TRY(L.run(PC_DOWN, [&] { return launch_gemm<T>(dg, EPI_F32, st); }));

      if (l + 1 < c.n_layers) {
        ResidArgs r2{W.h, W.rparts, rpart_stride, P.down.splits, mod_at(2 * l + 1, k), mod_at(2 * l + 2, k),
                     W.y, M, Tn, D, c.rms_eps, c.norm_precision};
        RFX_TRY(L.run(PC_RESID, [&] { return launch_resid_norm<T>(r2, st); }));
      }
    }
    const float dt = (float)((double)taus[k + 1] - (double)taus[k]);
    FinalArgs fa{W.h, W.rparts, rpart_stride, P.down.splits, mod_at(2 * c.n_layers - 1, k),
                 mod_at(2 * c.n_layers, k), ctx->w.w_aout, x_in, out, B, Tn, D, c.action_dim, dt, c.rms_eps,
                 c.norm_precision, W.status, fuse_embed && k + 1 < steps ? 1 : 0,
                 embed_args(k + 1 < steps ? k + 1 : k, out)};
    RFX_TRY(L.run(PC_FINAL, [&] { return launch_final_euler<T>(fa, st); }));
  }
  return REFLEX_OK;
}

// The unfused schedule of the operator-fusion ablation (Section 4.6): the
// same chunk with the conditioning MLPs evaluated at every step instead of
// once per chunk, RoPE and the gated GELU applied by their own kernels to fp32
// projection outputs, the residual add, the norm, the action head and the
// Euler update as separate launches.  Attention and the token embedding are
// the fused path's.
template <typename T>
int enqueue_chunk_unfused(reflex_ctx* ctx, const float* state, const float* noise, int steps, const float* taus,
                          float* out, bool prof) {
  const reflex_config& c = ctx->cfg;
  const Plan& P = ctx->plan;
  const Workspace& W = ctx->ws;
  hipStream_t st = ctx->stream;
  Launcher L{ctx, prof};
  const int B = c.batch, Tn = P.T, M = P.M, D = c.width, dh = c.head_dim, Hq = c.n_q_heads, F = c.mlp_dim;
  const int64_t site_stride = (int64_t)c.max_steps * B * 3 * D;
  auto mod_at = [&](int site, int k) { return W.mod + site * site_stride + (int64_t)k * B * 3 * D; };
  const size_t eb = sizeof(T);
  const int64_t rpart_stride = (int64_t)M * D;

  RFX_TRY(L.run(PC_ROPE, [&] { return launch_rope_table(W.rope_dyn, W.tick + 2, 0, Tn, dh, c.rope_theta, st); }));
  for (int k = 0; k < steps; ++k) {
    // conditioning MLPs of this step only
    TauTable tt;
    memset(&tt, 0, sizeof(tt));
    tt.tau[0] = taus[k];
    RFX_TRY(L.run(PC_MOD, [&] {
      return launch_cond<T>(W.cond, state, tt, 1, B, D, c.state_dim, c.temb_min_period, c.temb_max_period, st);
    }));
    GemmArgs g1{};
    g1.A = W.cond; g1.lda = P.C;
    g1.B = ctx->w.w_mod1; g1.ldb = P.C;
    g1.out = W.hid; g1.ldo = (int64_t)P.S * c.cond_hidden;
    g1.M = B; g1.N = P.S * c.cond_hidden; g1.K = P.C;
    g1.splits = 1; g1.k_per_split = P.C + 64; g1.batch = 1;
    RFX_TRY(L.run(PC_MOD, [&] { return launch_gemm<T>(g1, EPI_SILU, st); }));
    GemmArgs g2{};
    g2.A = W.hid; g2.lda = (int64_t)P.S * c.cond_hidden; g2.a_bstride = c.cond_hidden;
    g2.B = ctx->w.w_mod2; g2.ldb = c.cond_hidden; g2.b_bstride = (int64_t)3 * D * c.cond_hidden;
    g2.out = mod_at(0, k); g2.ldo = 3 * D; g2.o_bstride = site_stride;
    g2.M = B; g2.N = 3 * D; g2.K = c.cond_hidden;
    g2.splits = 1; g2.k_per_split = c.cond_hidden + 64; g2.batch = P.S;
    g2.mod_width = c.mod_mode == REFLEX_MOD_SCALE_ONLY ? D : 0;
    RFX_TRY(L.run(PC_MOD, [&] { return launch_gemm<T>(g2, EPI_MOD, st); }));

    const float* x_in = (k == 0) ? noise : out;
    EmbedArgs ea{x_in, state, ctx->w.w_state, ctx->w.w_ain, mod_at(0, k), W.h, W.y,
                 B, Tn, D, c.state_dim, c.action_dim, c.embed_scale, c.rms_eps, c.norm_precision};
    RFX_TRY(L.run(PC_EMBED, [&] { return launch_embed_norm<T>(ea, st); }));
    for (int l = 0; l < c.n_layers; ++l) {
      GemmArgs q{};
      q.A = W.y; q.lda = D;
      q.B = (const char*)ctx->w.w_qkv + (size_t)l * P.Nqkv * D * eb; q.ldb = D;
      q.out = W.uf_wide; q.ldo = P.Nqkv;
      q.M = M; q.N = P.Nqkv; q.K = D; q.splits = 1; q.k_per_split = D + 128; q.batch = 1;
      RFX_TRY(L.run(PC_QKV, [&] { return launch_gemm<T>(q, EPI_F32, st); }));
      RopeScatterArgs rs{W.uf_wide, QkvOut{W.rope_dyn, W.q, W.kd, W.vdt, Tn, Hq, dh, P.rows_pad, P.tpad}, M};
      RFX_TRY(L.run(PC_ROPE, [&] { return launch_rope_scatter<T>(rs, st); }));

      AttnArgs aa{};
      aa.q = W.q; aa.kd = W.kd; aa.vdt = W.vdt; aa.tpad = P.tpad;
      aa.cache_k = (const char*)ctx->cache_k + (size_t)l * P.R * dh * eb;
      aa.cache_vt = (const char*)ctx->cache_vt + (size_t)l * P.R * dh * eb;
      aa.ck_bstride = (int64_t)c.n_layers * P.R * dh;
      aa.n_valid = reinterpret_cast<const int32_t*>(W.tick + 1);
      aa.hole_row = reinterpret_cast<const int32_t*>(W.tick + 3);
      aa.static_len = c.static_len; aa.frame_tokens = c.frame_tokens; aa.R = P.R;
      aa.B = B; aa.T = Tn; aa.Hq = Hq; aa.nsplit = P.attn_splits; aa.kernel = P.attn_kernel;
      aa.part_o = W.part_o; aa.part_ml = W.part_ml;
      aa.rows_pad = P.rows_pad; aa.out = W.o;
      RFX_TRY(L.run(PC_ATTN, [&] { return launch_attention<T>(aa, dh, st); }));
      if (P.attn_splits > 1) RFX_TRY(L.run(PC_MERGE, [&] { return launch_attn_merge<T>(aa, dh, st); }));

      GemmArgs og{};
      og.A = W.o; og.lda = (int64_t)Hq * dh;
      og.B = (const char*)ctx->w.w_o + (size_t)l * D * Hq * dh * eb; og.ldb = (int64_t)Hq * dh;
      og.out = W.rparts; og.ldo = D; og.o_split_stride = rpart_stride;
      og.M = M; og.N = D; og.K = Hq * dh; og.splits = P.o.splits; og.k_per_split = P.o.kps; og.batch = 1;
      RFX_TRY(L.run(PC_O, [&] { return launch_gemm<T>(og, EPI_F32, st); }));
      ResidAddArgs ra1{W.h, W.rparts, rpart_stride, P.o.splits, mod_at(2 * l, k), M, Tn, D};
      RFX_TRY(L.run(PC_RESID, [&] { return launch_resid_add(ra1, st); }));
      NormArgs n1{W.h, mod_at(2 * l + 1, k), W.y, M, Tn, D, c.rms_eps};
      RFX_TRY(L.run(PC_RESID, [&] { return launch_norm<T>(n1, st); }));

      GemmArgs gu{};
      gu.A = W.y; gu.lda = D;
      gu.B = (const char*)ctx->w.w_gu + (size_t)l * 2 * F * D * eb; gu.ldb = D;
      gu.out = W.uf_wide; gu.ldo = 2 * F;
      gu.M = M; gu.N = 2 * F; gu.K = D; gu.splits = 1; gu.k_per_split = D + 128; gu.batch = 1;
      RFX_TRY(L.run(PC_GU, [&] { return launch_gemm<T>(gu, EPI_F32, st); }));
      GeluMulArgs gm{W.uf_wide, W.z, M, F};
      RFX_TRY(L.run(PC_GU, [&] { return launch_gelu_mul<T>(gm, st); }));

      GemmArgs dg{};
      dg.A = W.z; dg.lda = F;
      dg.B = (const char*)ctx->w.w_down + (size_t)l * D * F * eb; dg.ldb = F;
      dg.out = W.rparts; dg.ldo = D; dg.o_split_stride = rpart_stride;
      dg.M = M; dg.N = D; dg.K = F; dg.splits = P.down.splits; dg.k_per_split = P.down.kps; dg.batch = 1;
      RFX_TRY(L.run(PC_DOWN, [&] { return launch_gemm<T>(dg, EPI_F32, st); }));
      ResidAddArgs ra2{W.h, W.rparts, rpart_stride, P.down.splits, mod_at(2 * l + 1, k), M, Tn, D};
      RFX_TRY(L.run(PC_RESID, [&] { return launch_resid_add(ra2, st); }));
      // the next site's norm: the next layer's attention norm, or the final one
      NormArgs n2{W.h, mod_at(2 * l + 2, k), W.y, M, Tn, D, c.rms_eps};
      RFX_TRY(L.run(PC_RESID, [&] { return launch_norm<T>(n2, st); }));
    }
    GemmArgs hg{};
    hg.A = W.y; hg.lda = D;
    hg.B = ctx->w.w_aout; hg.ldb = D;
    hg.out = W.uf_v; hg.ldo = c.action_dim;
    hg.M = M; hg.N = c.action_dim; hg.K = D; hg.splits = 1; hg.k_per_split = D + 128; hg.batch = 1;
    RFX_TRY(L.run(PC_FINAL, [&] { return launch_gemm<T>(hg, EPI_F32, st); }));
    EulerArgs eu{W.uf_v, x_in, out, B, Tn, c.action_dim, (float)((double)taus[k + 1] - (double)taus[k])};
    RFX_TRY(L.run(PC_FINAL, [&] { return launch_euler(eu, st); }));
  }
  return REFLEX_OK;
}

int enqueue_chunk_dispatch(reflex_ctx* ctx, const Workspace& W, const float* state, const float* noise, int steps,
                           const float* taus, float* out, bool prof, int mode, const reflex_sources* src) {
  if (mode == REFLEX_MODE_UNFUSED) {
    if (ctx->cfg.dtype == REFLEX_DTYPE_BF16)
      return enqueue_chunk_unfused<bf16_t>(ctx, state, noise, steps, taus, out, prof);
    return enqueue_chunk_unfused<float>(ctx, state, noise, steps, taus, out, prof);
  }
  if (ctx->cfg.dtype == REFLEX_DTYPE_BF16)
    return enqueue_chunk<bf16_t>(ctx, W, state, noise, steps, taus, out, prof, mode, src);
  return enqueue_chunk<float>(ctx, W, state, noise, steps, taus, out, prof, mode, src);
}

// publish: also set the device tick state to "no frame written" (the first
// write at init); a Standard-mode re-encode leaves the tick state alone.
template <typename T>
int write_static(reflex_ctx* ctx, const void* sk, const void* sv, bool publish, Launcher& L) {
  const reflex_config& c = ctx->cfg;
  const Plan& P = ctx->plan;
  hipError_t e;
  if (c.static_len > 0) {
    RFX_TRY(L.run(PC_ROPE, [&] {
      return launch_rope_table(ctx->ws.rope_frame, nullptr, 0, c.static_len, c.head_dim, c.rope_theta, ctx->stream);
    }));
  }
  RingWriteArgs a{};
  a.src_k = sk; a.src_v = sv;
  a.sb = (int64_t)c.n_layers * c.static_len * c.head_dim;
  a.sl = (int64_t)c.static_len * c.head_dim;
  a.sj = c.head_dim;
  a.rope = ctx->ws.rope_frame;
  a.cache_k = ctx->cache_k; a.cache_vt = ctx->cache_vt;
  a.row0 = 0; a.n_tok = c.static_len; a.L = c.n_layers; a.B = c.batch; a.R = P.R;
  a.tick = publish ? ctx->ws.tick : nullptr; a.frames_written = 0; a.n_valid = 0; a.dyn_pos0 = c.static_len;
  a.hole_row = hole_row(ctx, 0);
  if (c.static_len == 0) {
    if (!publish) return REFLEX_OK;
    // still publish the tick state; a one-token dummy write is not needed, so
    // set it with a tiny copy instead
    int64_t host_tick[4] = {0, 0, (int64_t)c.static_len, a.hole_row};
    e = hipMemcpyAsync(ctx->ws.tick, host_tick, sizeof(host_tick), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    return e == hipSuccess ? REFLEX_OK : hip_fail(e);
  }
  return L.run(PC_RING, [&] { return launch_ring_write<T, T>(a, c.head_dim, ctx->stream); });
}

// publish: advance the device tick state to this frame (a new frame); a
// Standard-mode re-encode of an older frame leaves the tick state alone.
template <typename T>
int write_frame(reflex_ctx* ctx, const void* frame, const reflex_ring_step& stp, bool publish, Launcher& L,
                hipStream_t st) {
  const reflex_config& c = ctx->cfg;
  const Plan& P = ctx->plan;
  RFX_TRY(L.run(PC_ROPE, [&] {
    return launch_rope_table(ctx->ws.rope_frame, nullptr, stp.pos0, c.frame_tokens, c.head_dim, c.rope_theta, st);
  }));
  RingWriteArgs a{};
  const int dh = c.head_dim;
  a.rope = ctx->ws.rope_frame;
  a.cache_k = ctx->cache_k; a.cache_vt = ctx->cache_vt;
  a.row0 = c.static_len + stp.slot * c.frame_tokens;
  a.n_tok = c.frame_tokens; a.L = c.n_layers; a.B = c.batch; a.R = P.R;
  a.tick = publish ? ctx->ws.tick : nullptr; a.frames_written = stp.frame_index + 1; a.n_valid = stp.n_valid;
  a.dyn_pos0 = stp.dyn_pos0;
  a.hole_row = hole_row(ctx, stp.frame_index + 1);
  if (c.frame_dim > 0) {
    // the frame K/V projection of every layer, RoPE on K and the transposed V
    // written by its epilogue straight into the slot's cache rows
    const int N = c.n_layers * 2 * dh;
    GemmArgs g{};
    g.A = frame; g.lda = c.frame_dim;
    g.B = ctx->w.w_kv; g.ldb = c.frame_dim;
    g.M = c.batch * c.frame_tokens; g.N = N; g.K = c.frame_dim;
    g.splits = 1; g.k_per_split = c.frame_dim + 128; g.batch = 1;
    g.qkv.head_dim = dh;
    g.kv = KvOut{ctx->ws.rope_frame, ctx->cache_k, ctx->cache_vt, P.R, a.row0, c.frame_tokens, c.n_layers};
    RFX_TRY(L.run(PC_FRAME_PROJ, [&] { return launch_gemm<T>(g, EPI_KV, st); }));
    if (publish)
      RFX_TRY(L.run(PC_RING, [&] {
        return launch_tick_set(ctx->ws.tick, a.frames_written, a.n_valid, a.dyn_pos0, a.hole_row, st);
      }));
  } else {
    a.src_k = frame;
    a.src_v = (const char*)frame + (size_t)c.frame_tokens * dh * sizeof(T);
    a.sb = (int64_t)c.n_layers * 2 * c.frame_tokens * dh;
    a.sl = (int64_t)2 * c.frame_tokens * dh;
    a.sj = dh;
    RFX_TRY(L.run(PC_RING, [&] { return launch_ring_write<T, T>(a, dh, st); }));
  }
  return REFLEX_OK;
}

// Sum the per-launch events of a profiled call into the per-class totals.
int collect_profile(reflex_ctx* ctx, hipStream_t st) {
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e);
  for (int i = 0; i < PC_N; ++i) {
    ctx->prof_ms[i] = 0.0;
    ctx->prof_launches[i] = 0;
  }
  int rc = REFLEX_OK;
  for (auto& pe : ctx->ev_pending) {
    float ms = 0.f;
    const hipError_t t = hipEventElapsedTime(&ms, pe.second.first, pe.second.second);
    if (t != hipSuccess) {
      // report the failure and leave no pending error behind for the caller's next HIP call
      rc = hip_fail(t);
      (void)hipGetLastError();
      break;
    }
    ctx->prof_ms[pe.first] += ms;
    ctx->prof_launches[pe.first] += 1;
  }
  ctx->ev_pending.clear();
  return rc;
}

// One frame write on stream st.  A write on the context's stream also
// publishes the device tick state for the next chunk there.  With a spare
// slot, chunks set their own tick state (a write on another stream must not
// touch the state a running chunk reads), and the write is ordered on the
// device after the previous write and after every chunk that still reads the
// frame in its target slot.
int write_entry(reflex_ctx* ctx, const void* frame, hipStream_t st, int64_t* frame_index_out,
                int32_t* evicted_tokens_out) {
  if (!frame) return REFLEX_EINVAL;
  const reflex_config& c = ctx->cfg;
  const int64_t f = ctx->frames_written;
  reflex_ring_step stp;
  int rc = plan_frame(ctx, f, &stp);
  if (rc != REFLEX_OK) return rc;
  const bool spare = c.spare_slot != 0;
  if (spare) {
    hipError_t e = hipSuccess;
    // the previous write shares the frame RoPE table and must finish first
    if (!ctx->write_recs.empty() && ctx->write_recs.back().stream != st)
      e = hipStreamWaitEvent(st, ctx->write_recs.back().ev, 0);
    // slot f mod (W+1) holds frame f-W-1, which the windows of chunks over
    // n in [f-W, f-1] frames contain; the latest chunk with n <= f-1 covers
    // all earlier ones (one stream)
    for (auto it = ctx->chunk_recs.rbegin(); e == hipSuccess && it != ctx->chunk_recs.rend(); ++it) {
      if (it->n <= f - 1) {
        if (it->stream != st) e = hipStreamWaitEvent(st, it->ev, 0);
        break;
      }
    }
    if (e != hipSuccess) return hip_fail(e);
  }
  const bool prof = ctx->prof_enabled != 0;
  if (prof) ctx->ev_pending.clear();
  {
    Launcher L{ctx, prof};
    const bool publish = st == ctx->stream;
    rc = c.dtype == REFLEX_DTYPE_BF16 ? write_frame<bf16_t>(ctx, frame, stp, publish, L, st)
                                      : write_frame<float>(ctx, frame, stp, publish, L, st);
  }
  if (rc == REFLEX_OK && prof) rc = collect_profile(ctx, st);
  if (rc != REFLEX_OK) return rc;
  if (spare) {
    hipEvent_t ev = pipe_event(ctx);
    if (!ev) return hip_fail(hipErrorOutOfMemory);
    const hipError_t e = hipEventRecord(ev, st);
    if (e != hipSuccess) {
      ctx->pipe_free.push_back(ev);
      return hip_fail(e);
    }
    ctx->write_recs.push_back({f, ev, st});
    if (ctx->write_recs.size() > 2) {
      ctx->pipe_free.push_back(ctx->write_recs.front().ev);
      ctx->write_recs.erase(ctx->write_recs.begin());
    }
    // every chunk so far read n <= f frames: for the next write only the
    // latest one matters
    while (ctx->chunk_recs.size() > 1) {
      ctx->pipe_free.push_back(ctx->chunk_recs.front().ev);
      ctx->chunk_recs.erase(ctx->chunk_recs.begin());
    }
  }
  ctx->frames_written += 1;
  if (frame_index_out) *frame_index_out = stp.frame_index;
  if (evicted_tokens_out) *evicted_tokens_out = stp.evicted;
  return REFLEX_OK;
}

}  // namespace

extern "C" {

int reflex_ring_plan(int64_t frames_written, int32_t window_frames, int32_t frame_tokens, int32_t static_len,
                     reflex_ring_step* out) {
  if (!out || frames_written < 0 || window_frames < 1 || frame_tokens < 1 || static_len < 0) return REFLEX_EINVAL;
  const int64_t f = frames_written;
  out->frame_index = f;
  out->slot = (int32_t)(f % window_frames);
  out->n_valid = (int32_t)(f + 1 < window_frames ? f + 1 : window_frames);
  out->pos0 = (int64_t)static_len + f * frame_tokens;
  out->dyn_pos0 = (int64_t)static_len + (f + 1) * frame_tokens;
  out->evicted = f >= window_frames ? frame_tokens : 0;
  out->reserved = 0;
  return REFLEX_OK;
}

int reflex_query_sizes(const reflex_config* cfg, size_t* cache_bytes, size_t* workspace_bytes) {
  const int rc = validate(cfg);
  if (rc != REFLEX_OK) return rc;
  if (!cache_bytes || !workspace_bytes) return REFLEX_EINVAL;
  const Plan p = make_plan(cfg);
  *cache_bytes = p.cache_bytes;
  *workspace_bytes = p.ws_bytes;
  return REFLEX_OK;
}

int reflex_cache_init(const reflex_config* cfg, const reflex_weights* w, void* cache_mem, void* workspace_mem,
                      const void* static_k, const void* static_v, void* stream, reflex_ctx** out) {
  int rc = validate(cfg);
  if (rc != REFLEX_OK) return rc;
  if (!w || !cache_mem || !workspace_mem || !out) return REFLEX_EINVAL;
  if (cfg->static_len > 0 && (!static_k || !static_v)) return REFLEX_EINVAL;
  if (!w->w_qkv || !w->w_o || !w->w_gu || !w->w_down || !w->w_state || !w->w_ain || !w->w_aout || !w->w_mod1 ||
      !w->w_mod2)
    return REFLEX_EINVAL;
  if (cfg->frame_dim > 0 && !w->w_kv) return REFLEX_EINVAL;
  if (((uintptr_t)cache_mem & 255) || ((uintptr_t)workspace_mem & 255)) return REFLEX_EINVAL;
  if (w->dtype != cfg->dtype) return REFLEX_EDTYPE;

  reflex_ctx* ctx = new (std::nothrow) reflex_ctx();
  if (!ctx) return REFLEX_EINVAL;
  ctx->cfg = *cfg;
  ctx->w = *w;
  ctx->plan = make_plan(cfg);
  ctx->stream = reinterpret_cast<hipStream_t>(stream);
  ctx->frames_written = 0;
  ctx->alive = 1;
  ctx->prof_enabled = 0;
  const Plan& P = ctx->plan;
  char* base = reinterpret_cast<char*>(workspace_mem);
  Workspace& W = ctx->ws;
  W.tick = reinterpret_cast<int64_t*>(base + P.off[0]);
  W.status = reinterpret_cast<int32_t*>(base + P.off[0] + 32);
  W.rope_dyn = reinterpret_cast<float2*>(base + P.off[1]);
  W.rope_frame = reinterpret_cast<float2*>(base + P.off[2]);
  W.cond = base + P.off[3];
  W.hid = base + P.off[4];
  W.mod = reinterpret_cast<float*>(base + P.off[5]);
  W.h = reinterpret_cast<float*>(base + P.off[6]);
  W.y = base + P.off[7];
  W.q = base + P.off[8];
  W.kd = base + P.off[9];
  W.vdt = base + P.off[10];
  W.o = base + P.off[12];
  W.part_o = reinterpret_cast<float*>(base + P.off[13]);
  W.part_ml = reinterpret_cast<float*>(base + P.off[14]);
  W.z = base + P.off[15];
  W.rparts = reinterpret_cast<float*>(base + P.off[16]);
  W.naive_k = base + P.off[18];
  W.naive_vt = base + P.off[19];
  W.uf_wide = reinterpret_cast<float*>(base + P.off[20]);
  W.uf_v = reinterpret_cast<float*>(base + P.off[21]);
  ctx->cache_k = cache_mem;
  ctx->cache_vt = reinterpret_cast<char*>(cache_mem) + P.cache_bytes / 2;

  // zeroed cache, as the paper's pre-allocated ring buffer (Appendix B.2)
  hipError_t e = hipMemsetAsync(cache_mem, 0, P.cache_bytes, ctx->stream);
  // the workspace starts zeroed: tick state and the zero padding of the
  // dynamic value columns beyond T
  if (e == hipSuccess) e = hipMemsetAsync(workspace_mem, 0, P.ws_bytes, ctx->stream);
  if (e != hipSuccess) {
    delete ctx;
    return hip_fail(e);
  }
  {
    Launcher L{ctx, false};
    rc = cfg->dtype == REFLEX_DTYPE_BF16 ? write_static<bf16_t>(ctx, static_k, static_v, true, L)
                                          : write_static<float>(ctx, static_k, static_v, true, L);
  }
  if (rc != REFLEX_OK) {
    delete ctx;
    return rc;
  }
  *out = ctx;
  return REFLEX_OK;
}

int reflex_cache_write_frame(reflex_ctx* ctx, const void* frame, int64_t* frame_index_out,
                             int32_t* evicted_tokens_out) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  return write_entry(ctx, frame, ctx->stream, frame_index_out, evicted_tokens_out);
}

int reflex_pipeline_write_frame(reflex_ctx* ctx, const void* frame, void* writer_stream, int64_t* frame_index_out,
                                int32_t* evicted_tokens_out) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  if (!ctx->cfg.spare_slot) return REFLEX_EINVAL;
  return write_entry(ctx, frame, reinterpret_cast<hipStream_t>(writer_stream), frame_index_out,
                     evicted_tokens_out);
}

}  // extern "C"

namespace {

constexpr int64_t kAllFrames = INT64_MIN;  // every frame written so far

int denoise_launch(reflex_ctx* ctx, int mode, const reflex_sources* src, std::vector<const void*> srcs,
                   const float* state, const float* noise, int32_t num_steps, const float* taus,
                   float* actions_out);
int denoise_launch_static(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                          const float* taus, float* actions_out);

// A caller's tau schedule in host memory, or copied from device memory (a
// stream-ordered copy on the context's stream, waited for).
int read_taus(reflex_ctx* ctx, const float* tau_schedule, int32_t num_steps, float* taus) {
  if (!tau_schedule) {
    for (int k = 0; k <= num_steps; ++k) taus[k] = (float)(1.0 - (double)k / (double)num_steps);
    return REFLEX_OK;
  }
  hipPointerAttribute_t attr;
  memset(&attr, 0, sizeof(attr));
  const hipError_t pe = hipPointerGetAttributes(&attr, tau_schedule);
  if (pe != hipSuccess) (void)hipGetLastError();  // an unregistered host pointer
  if (pe == hipSuccess && (attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged)) {
    hipError_t e = hipMemcpyAsync(taus, tau_schedule, sizeof(float) * (num_steps + 1), hipMemcpyDeviceToHost,
                                  ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(e);
  } else {
    for (int k = 0; k <= num_steps; ++k) taus[k] = tau_schedule[k];
  }
  return REFLEX_OK;
}

// n_req: the frames the chunk reads on a context with a spare slot (-1: the
// newest completed write, kAllFrames: all); ignored without a spare slot,
// where the tick state published by the last write is read.
int denoise_entry(reflex_ctx* ctx, int mode, const reflex_sources* src, const float* state, const float* noise,
                  int32_t num_steps, const float* tau_schedule, float* actions_out, int64_t n_req,
                  int64_t* n_out, bool use_static = false) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  if (!state || !noise || !actions_out) return REFLEX_EINVAL;
  if (num_steps < 1 || num_steps > ctx->cfg.max_steps) return REFLEX_EINVAL;
  if (mode != REFLEX_MODE_REFLEX && mode != REFLEX_MODE_STANDARD && mode != REFLEX_MODE_NAIVE &&
      mode != REFLEX_MODE_UNFUSED)
    return REFLEX_EINVAL;
  const bool spare = ctx->cfg.spare_slot != 0;
  if (spare && mode == REFLEX_MODE_STANDARD) return REFLEX_EINVAL;
  const int64_t F = ctx->frames_written;
  int64_t n = F;
  if (spare && n_req != kAllFrames) {
    if (n_req == -1) {
      // the newest frame whose write has completed (at most one is in flight
      // that a chunk may skip: the spare slot protects one)
      if (!ctx->write_recs.empty() && ctx->write_recs.back().n == F - 1) {
        const hipError_t q = hipEventQuery(ctx->write_recs.back().ev);
        if (q == hipErrorNotReady) n = F - 1;
        else if (q != hipSuccess) return hip_fail(q);
      }
    } else {
      n = n_req;
    }
    if (n < (F > 0 ? F - 1 : 0) || n > F) return REFLEX_EINVAL;
  }
  std::vector<const void*> srcs;
  if (mode == REFLEX_MODE_STANDARD) {
    const reflex_config& c = ctx->cfg;
    const int64_t n_valid = ctx->frames_written < c.window_frames ? ctx->frames_written : c.window_frames;
    if (!src || src->n_frames != n_valid || (n_valid > 0 && !src->frames)) return REFLEX_EINVAL;
    if (c.static_len > 0 && (!src->static_k || !src->static_v)) return REFLEX_EINVAL;
    srcs.push_back(src->static_k);
    srcs.push_back(src->static_v);
    for (int i = 0; i < src->n_frames; ++i) {
      if (!src->frames[i]) return REFLEX_EINVAL;
      srcs.push_back(src->frames[i]);
    }
  } else {
    src = nullptr;
  }
  float taus[REFLEX_MAX_STEPS + 1];
  RFX_TRY(read_taus(ctx, tau_schedule, num_steps, taus));

  if (spare) {
    // frame n-1 (and so every earlier frame) written, then this chunk's window
    hipError_t e = hipSuccess;
    for (const auto& w : ctx->write_recs)
      if (w.n == n - 1 && w.stream != ctx->stream) e = hipStreamWaitEvent(ctx->stream, w.ev, 0);
    if (e != hipSuccess) return hip_fail(e);
    const reflex_config& c = ctx->cfg;
    e = launch_tick_set(ctx->ws.tick, n, n < c.window_frames ? n : c.window_frames,
                        (int64_t)c.static_len + n * c.frame_tokens, hole_row(ctx, n), ctx->stream);
    if (e != hipSuccess) return hip_fail(e);
  }
  const int rc = use_static ? denoise_launch_static(ctx, state, noise, num_steps, taus, actions_out)
                            : denoise_launch(ctx, mode, src, std::move(srcs), state, noise, num_steps, taus, actions_out);
  if (rc != REFLEX_OK) return rc;
  if (spare) {
    hipError_t e;
    if (!ctx->chunk_recs.empty() && ctx->chunk_recs.back().n == n) {
      e = hipEventRecord(ctx->chunk_recs.back().ev, ctx->stream);
    } else {
      hipEvent_t ev = pipe_event(ctx);
      if (!ev) return hip_fail(hipErrorOutOfMemory);
      e = hipEventRecord(ev, ctx->stream);
      if (e == hipSuccess) ctx->chunk_recs.push_back({n, ev, ctx->stream});
      else ctx->pipe_free.push_back(ev);
    }
    if (e != hipSuccess) return hip_fail(e);
  }
  if (n_out) *n_out = n;
  return REFLEX_OK;
}

// The chunk's launches: eager with per-launch events when profiling, else
// one captured graph per distinct (pointers, steps, schedule, strategy).
int denoise_launch(reflex_ctx* ctx, int mode, const reflex_sources* src, std::vector<const void*> srcs,
                   const float* state, const float* noise, int32_t num_steps, const float* taus,
                   float* actions_out) {
  if (ctx->prof_enabled) {
    ctx->ev_pending.clear();
    int rc = enqueue_chunk_dispatch(ctx, ctx->ws, state, noise, num_steps, taus, actions_out, true, mode, src);
    if (rc != REFLEX_OK) return rc;
    return collect_profile(ctx, ctx->stream);
  }

  GraphEntry* hit = nullptr;
  for (auto& g : ctx->graphs) {
    if (g.state == state && g.noise == noise && g.out == actions_out && g.steps == num_steps &&
        g.mode == mode && memcmp(g.taus, taus, sizeof(float) * (num_steps + 1)) == 0 &&
        (mode != REFLEX_MODE_STANDARD || (g.frames_written == ctx->frames_written && g.srcs == srcs))) {
      hit = &g;
      break;
    }
  }
  if (!hit) {
    hipGraph_t graph;
    hipError_t e = hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) return hip_fail(e);
    int rc = enqueue_chunk_dispatch(ctx, ctx->ws, state, noise, num_steps, taus, actions_out, false, mode, src);
    e = hipStreamEndCapture(ctx->stream, &graph);
    if (rc != REFLEX_OK) {
      if (e == hipSuccess) (void)hipGraphDestroy(graph);
      return rc;
    }
    if (e != hipSuccess) return hip_fail(e);
    hipGraphExec_t exec;
    e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (e != hipSuccess) return hip_fail(e);
    if (ctx->graphs.size() >= 8) {
      (void)hipGraphExecDestroy(ctx->graphs.front().exec);
      ctx->graphs.erase(ctx->graphs.begin());
    }
    GraphEntry ge;
    ge.state = state; ge.noise = noise; ge.out = actions_out; ge.steps = num_steps;
    memset(ge.taus, 0, sizeof(ge.taus));
    memcpy(ge.taus, taus, sizeof(float) * (num_steps + 1));
    ge.mode = mode;
    ge.frames_written = ctx->frames_written;
    ge.srcs = std::move(srcs);
    ge.exec = exec;
    ctx->graphs.push_back(std::move(ge));
    hit = &ctx->graphs.back();
  }
  hipError_t e = hipGraphLaunch(hit->exec, ctx->stream);
  return e == hipSuccess ? REFLEX_OK : hip_fail(e);
}

// ---------------------------------------------------------------------------
// Allocation-free denoise: the chunk's transient buffers live in a static
// device array instead of the context's workspace, and the launches run
// eagerly (instantiating a graph allocates).  One array per device, shared by
// every such call on that device.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
void* g_scratch_dev[kMaxDevices];  // device address of `scratch` per device (null until set up)
std::mutex g_scratch_mu;

// Device address of this device's copy of the array, looked up once per
// device with that device current.
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  if (dev < 0 || dev >= kMaxDevices) return REFLEX_EINVAL;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e);
    if (!ptr) return hip_fail(hipErrorInvalidSymbol);
    g_scratch_dev[dev] = ptr;
  }
  *out = g_scratch_dev[dev];
  return REFLEX_OK;
}

// Bytes of static scratch a chunk of this context needs: workspace parts 1..16
// (the RoPE tables through the split-K partials), laid out as in the workspace.
size_t static_scratch_bytes(const Plan& P) { return P.off[17] - P.off[1]; }

int denoise_launch_static(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                          const float* taus, float* actions_out) {
  const Plan& P = ctx->plan;
  void* base = nullptr;
  RFX_TRY(scratch_address(&base));
  Workspace W = ctx->ws;  // tick state, status word and the frame path's tables stay in the workspace
  char* b = reinterpret_cast<char*>(base) - P.off[1];
  W.rope_dyn = reinterpret_cast<float2*>(b + P.off[1]);
  W.cond = b + P.off[3];
  W.hid = b + P.off[4];
  W.mod = reinterpret_cast<float*>(b + P.off[5]);
  W.h = reinterpret_cast<float*>(b + P.off[6]);
  W.y = b + P.off[7];
  W.q = b + P.off[8];
  W.kd = b + P.off[9];
  W.vdt = b + P.off[10];
  W.o = b + P.off[12];
  W.part_o = reinterpret_cast<float*>(b + P.off[13]);
  W.part_ml = reinterpret_cast<float*>(b + P.off[14]);
  W.z = b + P.off[15];
  W.rparts = reinterpret_cast<float*>(b + P.off[16]);
  // the array keeps the previous call's bytes: the dynamic value columns
  // beyond T must read as zero (the attention multiplies them by p = 0)
  const hipError_t e = launch_zero(W.vdt, P.off[11] - P.off[10], ctx->stream);
  if (e != hipSuccess) return hip_fail(e);
  return enqueue_chunk_dispatch(ctx, W, state, noise, num_steps, taus, actions_out, false, REFLEX_MODE_REFLEX,
                                nullptr);
}

}  // namespace

extern "C" {

int reflex_denoise_chunk(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                         const float* tau_schedule, float* actions_out) {
  return denoise_entry(ctx, REFLEX_MODE_REFLEX, nullptr, state, noise, num_steps, tau_schedule, actions_out,
                       kAllFrames, nullptr);
}

int reflex_denoise_chunk_baseline(reflex_ctx* ctx, int32_t mode, const reflex_sources* src, const float* state,
                                  const float* noise, int32_t num_steps, const float* tau_schedule,
                                  float* actions_out) {
  return denoise_entry(ctx, mode, src, state, noise, num_steps, tau_schedule, actions_out, kAllFrames, nullptr);
}

int reflex_pipeline_denoise_chunk(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                                  const float* tau_schedule, float* actions_out, int64_t n_frames,
                                  int64_t* n_frames_out) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  if (!ctx->cfg.spare_slot || n_frames < -1) return REFLEX_EINVAL;
  return denoise_entry(ctx, REFLEX_MODE_REFLEX, nullptr, state, noise, num_steps, tau_schedule, actions_out,
                       n_frames, n_frames_out);
}

int reflex_denoise_chunk_static(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                                const float* tau_schedule, float* actions_out) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  if (static_scratch_bytes(ctx->plan) > kScratchBytes) return REFLEX_ESCRATCH;
  return denoise_entry(ctx, REFLEX_MODE_REFLEX, nullptr, state, noise, num_steps, tau_schedule, actions_out,
                       kAllFrames, nullptr, true);
}

int reflex_check_status(reflex_ctx* ctx) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  int32_t st = 0;
  const int32_t zero = 0;
  hipError_t e = hipMemcpyAsync(&st, ctx->ws.status, sizeof(st), hipMemcpyDeviceToHost, ctx->stream);
  if (e == hipSuccess) e = hipMemcpyAsync(ctx->ws.status, &zero, sizeof(zero), hipMemcpyHostToDevice, ctx->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return hip_fail(e);
  return (st & 1) ? REFLEX_ENONFINITE : REFLEX_OK;
}

int reflex_destroy(reflex_ctx* ctx) {
  if (!ctx) return REFLEX_OK;
  ctx->alive = 0;
  for (auto& g : ctx->graphs) (void)hipGraphExecDestroy(g.exec);
  ctx->graphs.clear();
  for (auto e : ctx->ev_pool) (void)hipEventDestroy(e);
  ctx->ev_pool.clear();
  for (auto& r : ctx->write_recs) (void)hipEventDestroy(r.ev);
  for (auto& r : ctx->chunk_recs) (void)hipEventDestroy(r.ev);
  for (auto e : ctx->pipe_free) (void)hipEventDestroy(e);
  delete ctx;
  return REFLEX_OK;
}

const char* reflex_strerror(int status) {
  switch (status) {
    case REFLEX_OK: return "ok";
    case REFLEX_EINVAL: return "invalid argument or unsupported configuration";
    case REFLEX_EDTYPE: return "weight dtype does not match the configured compute dtype";
    case REFLEX_EHIP: return g_hip_err[0] ? g_hip_err : "HIP error";
    case REFLEX_ESTATE: return "context not initialised or destroyed";
    case REFLEX_ENONFINITE: return "a denoise produced a non-finite action since the last status check";
    case REFLEX_ESCRATCH: return "the call needs more scratch than the library's static device array holds";
    default: return "unknown status";
  }
}

int64_t reflex_frames_written(const reflex_ctx* ctx) {
  if (!ctx) return REFLEX_ESTATE;
  return ctx->frames_written;
}

int reflex_profile_enable(reflex_ctx* ctx, int enable) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  ctx->prof_enabled = enable ? 1 : 0;
  return REFLEX_OK;
}

int reflex_profile_read(reflex_ctx* ctx, const char** names, double* ms, int32_t* launches, int32_t* n_classes) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  if (!names || !ms || !launches || !n_classes) return REFLEX_EINVAL;
  const int n = *n_classes < PC_N ? *n_classes : PC_N;
  for (int i = 0; i < n; ++i) {
    names[i] = kProfNames[i];
    ms[i] = ctx->prof_ms[i];
    launches[i] = ctx->prof_launches[i];
  }
  *n_classes = n;
  return REFLEX_OK;
}

int reflex_profile_graph(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                         const float* tau_schedule, float* actions_out, uint32_t class_mask, int32_t reps,
                         double* ms_per_replay, int32_t* launches) {
  if (!ctx || !ctx->alive) return REFLEX_ESTATE;
  if (!state || !noise || !actions_out || !ms_per_replay || !launches) return REFLEX_EINVAL;
  if (num_steps < 1 || num_steps > ctx->cfg.max_steps || reps < 1 || (class_mask & ((1u << PC_N) - 1)) == 0)
    return REFLEX_EINVAL;
  float taus[REFLEX_MAX_STEPS + 1];
  RFX_TRY(read_taus(ctx, tau_schedule, num_steps, taus));
  int dev = 0, khz = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
  if (e != hipSuccess) return hip_fail(e);
  if (khz <= 0) return hip_fail(hipErrorInvalidValue);

  // room for three stamps per launch of the chunk (a bound on its launches:
  // at most 12 per layer and step plus the per-chunk ones), and one slot for
  // the two stamps that open the graph
  const reflex_config& c = ctx->cfg;
  const int cap = 3 * (num_steps * (12 * c.n_layers + 8) + 16);
  unsigned long long* stamps = nullptr;
  e = hipMalloc(&stamps, sizeof(unsigned long long) * (cap + 1));
  if (e != hipSuccess) return hip_fail(e);
  std::vector<unsigned long long> host(cap);

  // the whole chunk, the selected classes' launches stamped
  hipGraph_t graph;
  hipGraphExec_t exec = nullptr;
  int rc = REFLEX_OK;
  e = hipStreamBeginCapture(ctx->stream, hipStreamCaptureModeThreadLocal);
  if (e == hipSuccess) {
    // two uncounted stamps open the graph: a measured bracket never starts
    // at a replay's first node, whose boundary is not the chunk's
    hipError_t le = hipSuccess;
    for (int i = 0; le == hipSuccess && i < 2; ++i) {
      hipLaunchKernelGGL(stamp_kernel, dim3(1), dim3(64), 0, ctx->stream, stamps + cap);
      le = hipGetLastError();
    }
    if (le == hipSuccess) {
      ctx->stamp_mask = class_mask;
      ctx->stamps = stamps;
      ctx->stamp_next = 0;
      ctx->stamp_cap = cap;
      rc = enqueue_chunk_dispatch(ctx, ctx->ws, state, noise, num_steps, taus, actions_out, false,
                                  REFLEX_MODE_REFLEX, nullptr);
      ctx->stamp_mask = 0;
      ctx->stamps = nullptr;
    }
    // the capture is always ended, whatever failed inside it
    e = hipStreamEndCapture(ctx->stream, &graph);
    if (e == hipSuccess && (rc != REFLEX_OK || le != hipSuccess)) (void)hipGraphDestroy(graph);
    if (e == hipSuccess && rc == REFLEX_OK && le == hipSuccess) {
      e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
    }
    if (e == hipSuccess) e = le;
  }
  const int n = ctx->stamp_next / 3;
  double ticks = 0.0;
  // one untimed replay, then reps replays, the stamps read back after each
  if (rc == REFLEX_OK && e == hipSuccess) e = hipGraphLaunch(exec, ctx->stream);
  for (int r = 0; rc == REFLEX_OK && e == hipSuccess && r < reps; ++r) {
    e = hipGraphLaunch(exec, ctx->stream);
    if (e == hipSuccess)
      e = hipMemcpyAsync(host.data(), stamps, sizeof(unsigned long long) * 3 * n, hipMemcpyDeviceToHost,
                         ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    for (int j = 0; e == hipSuccess && j < n; ++j) {
      const double t0 = (double)host[3 * j], t1 = (double)host[3 * j + 1], t2 = (double)host[3 * j + 2];
      ticks += (t2 - t1) - (t1 - t0);
    }
  }
  if (exec) (void)hipGraphExecDestroy(exec);
  const hipError_t f = hipFree(stamps);
  if (rc != REFLEX_OK) return rc;
  if (e == hipSuccess) e = f;
  if (e != hipSuccess) {
    const int r = hip_fail(e);
    (void)hipGetLastError();  // leave no pending error for the caller's next call
    return r;
  }
  *ms_per_replay = ticks / reps / (double)khz;  // kHz: ticks per millisecond
  *launches = n;
  return REFLEX_OK;
}

}  // extern "C"
