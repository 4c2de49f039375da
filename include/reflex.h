/*
 * reflex.h -- C ABI of the MI355X (gfx950) Reflex denoise hot path.
 *
 * The library computes the per-denoising-step forward of a flow-matching
 * action expert over a three-region KV cache, following the paper "Reflex:
 * Real-Time Vision-Language-Action Control through Streaming Inference":
 *
 *   - a pinned static prefix (language tokens), written once (Section 3.1);
 *   - a sliding FIFO window of the last W observation frames, held in a
 *     pre-allocated ring and overwritten in O(1) per frame (Section 3.1,
 *     Section 3.4 "Ring Buffer Architecture", Appendix B.1-B.2);
 *   - a dynamic suffix (one state token + H action tokens) recomputed at every
 *     Euler step; attention over [static; window; dynamic] is Eq. 1 and equals
 *     full-batch attention (Appendix A, Proposition A.1).
 *
 * Every layer uses AdaRMSNorm with fp32 statistics (Eq. 2, Section 3.2),
 * packed QKV and gate|up projections (Section 3.4 "Operator Fusion"), and the
 * chunk is integrated with explicit Euler from noise at tau = 1 to actions at
 * tau = 0.
 *
 * Memory ownership: the caller allocates and owns every device buffer
 * (weights, cache, workspace, inputs, outputs).  The library never allocates
 * or frees device memory; it owns only the host-side context.  All device
 * work is enqueued on the stream given to reflex_cache_init and is
 * asynchronous unless stated otherwise.  A context is bound to one stream and
 * is not thread-safe.
 *
 * Status codes: 0 on success, a negative REFLEX_E* value on failure;
 * reflex_strerror() describes a code (and the last HIP error for
 * REFLEX_EHIP).  On failure no context state changes.
 */
#ifndef REFLEX_H
#define REFLEX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REFLEX_OK 0
#define REFLEX_EINVAL (-1)   /* null pointer, bad shape or unsupported size */
#define REFLEX_EDTYPE (-2)   /* weight dtype differs from the config's dtype */
#define REFLEX_EHIP (-3)     /* a HIP call or kernel launch failed */
#define REFLEX_ESTATE (-4)   /* context not initialised or already destroyed */
#define REFLEX_ENONFINITE (-5) /* reflex_check_status: a denoise produced a non-finite action */
#define REFLEX_ESCRATCH (-6) /* reflex_denoise_chunk_static: the chunk needs more scratch than
                                the library's static device array holds */

#define REFLEX_DTYPE_F32 0
#define REFLEX_DTYPE_BF16 1

#define REFLEX_MOD_FULL 0        /* y = n(x)(1+scale)+shift; h += gate * f(y) */
#define REFLEX_MOD_SCALE_ONLY 1  /* shift = 0, gate = 1: Eq. 2 exactly */

#define REFLEX_MAX_STEPS 64

/* Precision of the residual stream and of the RMS statistics of every
 * AdaRMSNorm.  REFLEX_NORM_FP32 is the method (fp32 statistics, Section 3.2).
 * The other two reproduce the baselines of the stability stress test
 * (Section 4.6): a bf16 residual stream with the statistics accumulated in
 * bf16 (every product and partial sum rounded to bf16), and a bf16 residual
 * stream with fp32 statistics ("FP32 norm-only"). */
#define REFLEX_NORM_FP32 0
#define REFLEX_NORM_BF16 1
#define REFLEX_NORM_BF16_FP32_STATS 2

/* Attention kernel of the bf16 path.  All compute the same masked softmax
 * over [static; ring window; dynamic] (Eq. 1) and agree to rounding.
 * REFLEX_ATTN_AUTO picks by the launch geometry: one wave pair per 32 query
 * rows when the launch would reach one key tile per split (a few envs and a
 * short context), otherwise 16-row waves sharing each key tile over 128
 * query rows, software-pipelined (a tile's scores and softmax run under the
 * previous tile's P.V MFMAs).  REFLEX_ATTN_ROWS16 forces the 16-row kernel
 * without that pipelining (the same results bit for bit); the other values
 * force one kernel (tests, tuning).  The fp32 path has one kernel and
 * ignores the field. */
#define REFLEX_ATTN_AUTO 0
#define REFLEX_ATTN_ROWS16 1
#define REFLEX_ATTN_PAIR 2
#define REFLEX_ATTN_ROWS16_PIPE 3

/*
 * Shape of the action expert and of the cache.
 *
 * Model: n_layers transformer layers of width `width`; a gated-GELU MLP of
 * width mlp_dim; n_q_heads query heads sharing n_kv_heads K/V heads of size
 * head_dim; one state token (state_dim) and action_horizon action tokens
 * (action_dim each) form the dynamic region (T = 1 + action_horizon rows).
 * The conditioning MLP of each AdaRMSNorm site maps c = [sinusoidal(tau) (width
 * values); state] through cond_hidden SiLU units to 3*width outputs
 * (scale, shift, gate).  Sites: 2*l (attention norm of layer l), 2*l+1 (MLP norm
 * of layer l), 2*n_layers (final norm before the action head).
 *
 * Cache: static_len prefix tokens; window_frames ring slots of frame_tokens
 * tokens, plus one spare slot when spare_slot = 1 (the pipelined ring of the
 * reflex_pipeline_* calls: frame f then goes to slot f mod (window_frames + 1),
 * and a chunk still sees exactly window_frames frames).
 * frame_dim > 0: frames arrive as [frame_tokens, frame_dim]
 * embeddings and K/V come from the per-layer frame projection w_kv;
 * frame_dim == 0: frames arrive as pre-RoPE per-layer K/V.  batch independent
 * environments advance in lockstep and share the weights.
 *
 * Numerics: dtype is the storage/compute type of weights, cache and GEMM
 * operands (accumulation, statistics, residual stream and actions are fp32).
 * RoPE: rotate-half, base rope_theta; positions are absolute: static
 * 0..static_len-1, frame f token j at static_len + f*frame_tokens + j, dynamic
 * token i at static_len + frames_written*frame_tokens + i.  The token embeddings
 * are multiplied by embed_scale.
 *
 * Supported by this build: n_kv_heads == 1; head_dim in {64, 128, 256};
 * width, mlp_dim, cond_hidden multiples of 64; state_dim, action_dim, frame_dim
 * multiples of 8; dynamic rows T <= 128 per env.
 */
typedef struct reflex_config {
  int32_t n_layers;
  int32_t width;
  int32_t mlp_dim;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t state_dim;
  int32_t action_dim;
  int32_t action_horizon;
  int32_t cond_hidden;
  int32_t static_len;
  int32_t frame_tokens;
  int32_t window_frames;
  int32_t frame_dim;
  int32_t batch;
  int32_t dtype;       /* REFLEX_DTYPE_* */
  int32_t mod_mode;    /* REFLEX_MOD_* */
  int32_t max_steps;   /* largest num_steps a denoise call may use (<= 64) */
  float rms_eps;
  float embed_scale;
  double rope_theta;
  double temb_min_period;
  double temb_max_period;
  int32_t spare_slot;      /* 0 or 1, see "Cache" above */
  int32_t norm_precision;  /* REFLEX_NORM_*: REFLEX_NORM_FP32 for the method */
  int32_t attn_kernel;     /* REFLEX_ATTN_*: REFLEX_ATTN_AUTO unless forcing one */
} reflex_config;

/*
 * Device pointers to the weights, row-major, rows are output features
 * (y = x W^T), element type `dtype`.  The library reads them in place; they
 * must stay valid and unchanged for the life of the context.
 *
 *   w_qkv  [n_layers][(Hq + 2) * head_dim][width]  rows: q heads, k, v
 *   w_o    [n_layers][width][Hq * head_dim]
 *   w_gu   [n_layers][2 * mlp_dim][width]           rows: gate, then up
 *   w_down [n_layers][width][mlp_dim]
 *   w_state[width][state_dim]
 *   w_ain  [width][action_dim]
 *   w_aout [action_dim][width]
 *   w_mod1 [2*n_layers+1][cond_hidden][width + state_dim]
 *   w_mod2 [2*n_layers+1][3 * width][cond_hidden]  rows: scale, shift, gate
 *   w_kv   [n_layers][2 * head_dim][frame_dim]     rows: k, then v; NULL when
 *                                                   frame_dim == 0
 *
 * dtype: the element type the caller's framework reports for the output
 * projection w_o (the dtype probe of Section 3.2 "Robust Dtype Inference").
 */
typedef struct reflex_weights {
  const void* w_qkv;
  const void* w_o;
  const void* w_gu;
  const void* w_down;
  const void* w_state;
  const void* w_ain;
  const void* w_aout;
  const void* w_mod1;
  const void* w_mod2;
  const void* w_kv;
  int32_t dtype;
} reflex_weights;

/* Host-side bookkeeping of one FIFO write (Section 3.1; Appendix B.1). */
typedef struct reflex_ring_step {
  int64_t frame_index; /* f: index of the frame being written (0-based)      */
  int32_t slot;        /* ring slot f mod W                                   */
  int32_t n_valid;     /* frames visible after the write: min(f + 1, W)       */
  int64_t pos0;        /* absolute position of the frame's first token        */
  int64_t dyn_pos0;    /* absolute position of dynamic token 0 afterwards     */
  int32_t evicted;     /* tokens evicted by the write: frame_tokens if f >= W */
  int32_t reserved;
} reflex_ring_step;

typedef struct reflex_ctx reflex_ctx;

/*
 * Bytes the caller must allocate for the cache and the workspace.  Pure host
 * function (no device calls).  Both buffers need 256-byte alignment.
 *
 * Cache layout (element type `dtype`), R = static_len + (window_frames + spare_slot)*frame_tokens:
 *   K at offset 0:           [batch][n_layers][R][head_dim]   RoPE applied
 *   V at offset K bytes:     [batch][n_layers][head_dim][R]   stored transposed
 * Rows [0, static_len) hold the static prefix; ring slot s holds rows
 * [static_len + s*frame_tokens, static_len + (s+1)*frame_tokens).
 * The first 32 bytes of the workspace hold the device tick state as four
 * int64 values {frames_written, n_valid, dyn_pos0, hole_row} (read-only for
 * callers): the frames, window length and dynamic position the next chunk
 * uses, and the logical cached row from which the physical rows skip the
 * spare slot (a value past the window means no skip).  Bytes 32..35 hold the
 * status word that reflex_check_status reads.  The rest of the workspace is
 * private scratch of the library.
 * The caller allocates both buffers once, before the control loop: no
 * allocation happens per frame or per chunk (the pre-allocated ring and
 * buffers of Section 3.4 and Appendix B.2).
 * Returns REFLEX_EINVAL for an unsupported config.
 */
int reflex_query_sizes(const reflex_config* cfg, size_t* cache_bytes, size_t* workspace_bytes);

/*
 * Validate the config, check the weights' dtype against cfg->dtype (dtype
 * probe, Section 3.2), bind the caller's buffers and write the pinned static
 * prefix: K rows get RoPE at positions 0..static_len-1, V rows are copied.
 *
 * static_k, static_v: device, [batch][n_layers][static_len][head_dim], pre-RoPE,
 * element type dtype; read during this call's stream work only.
 * cache_mem / workspace_mem: device buffers of the sizes reflex_query_sizes
 * returned.  stream: a hipStream_t (NULL = the null stream).
 * On success *out receives a new context with frames_written = 0.
 * Errors: REFLEX_EINVAL, REFLEX_EDTYPE, REFLEX_EHIP; *out untouched on error.
 */
int reflex_cache_init(const reflex_config* cfg, const reflex_weights* w, void* cache_mem,
                      void* workspace_mem, const void* static_k, const void* static_v,
                      void* stream, reflex_ctx** out);

/*
 * Write one new frame for all envs (FIFO, incremental prefill of the newest
 * frame only, Section 3.1): slot f mod W is overwritten; K gets RoPE at
 * positions static_len + f*frame_tokens + j.
 *
 * frame: device, element type dtype;
 *   frame_dim > 0:  [batch][frame_tokens][frame_dim] embeddings;
 *   frame_dim == 0: [batch][n_layers][2][frame_tokens][head_dim] pre-RoPE K, V.
 * frame_index_out / evicted_tokens_out (nullable host pointers) receive f and
 * the evicted token count (the eviction count of add_new_prefix, Appendix B.1).
 * The host metadata is returned synchronously; the device work is async.
 * Errors: REFLEX_EINVAL, REFLEX_ESTATE, REFLEX_EHIP; on error f is not advanced.
 */
int reflex_cache_write_frame(reflex_ctx* ctx, const void* frame, int64_t* frame_index_out,
                             int32_t* evicted_tokens_out);

/*
 * Denoise one action chunk per env over the current cache (static prefix +
 * the n_valid written frames + the dynamic region), num_steps Euler steps.
 *
 * state:  device fp32 [batch][state_dim]
 * noise:  device fp32 [batch][action_horizon][action_dim], x at tau_0
 * actions_out: device fp32 [batch][action_horizon][action_dim], x at tau_K;
 *         may alias noise.
 * tau_schedule: fp32 array of num_steps + 1 values, tau_0 = 1 > ... >
 *         tau_K = 0, or NULL for tau_k = 1 - k/num_steps (the uniform Euler
 *         grid from noise at tau = 1, Section 3.2).  Host memory, or device
 *         memory: a device array is copied to the host on the context's
 *         stream and that copy is waited for, so the call then blocks until
 *         the stream's earlier work is done.
 * The cache is only read (timestep invariance, Section 3.1).  An empty ring
 * is allowed.  Launches are captured once into a HIP graph per distinct
 * (pointers, num_steps, schedule) and replayed.
 * Timing: a wait for this chunk queued on another stream while the chunk
 * runs (an event wait in another hardware queue) lengthens the gaps between
 * its kernels: a batch-1 pi0 chunk took 9.78 ms against 8.73 ms without one.
 * Queue work that depends on the result on this context's stream, or order
 * other streams after it once it has completed.
 * Errors: REFLEX_EINVAL (null pointer, num_steps outside [1, max_steps]),
 * REFLEX_ESTATE, REFLEX_EHIP.
 */
int reflex_denoise_chunk(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                         const float* tau_schedule, float* actions_out);

/* Cache strategies of the comparison in Section 4 (Baselines) and the
 * partitioned-attention ablation table of Section 4.6. */
#define REFLEX_MODE_REFLEX 0   /* the method: cached regions read, dynamic K/V fresh at every step */
#define REFLEX_MODE_STANDARD 1 /* full history recomputation: before every Euler step the static
                                  prefix and every window frame are encoded into the cache again */
#define REFLEX_MODE_NAIVE 2    /* a K/V cache that ignores the timestep: the dynamic K/V computed at
                                  the first Euler step are reused at every later step */
#define REFLEX_MODE_UNFUSED 3  /* the method without operator fusion (the fusion ablation of Section
                                  4.6): conditioning MLPs at every step, RoPE, gated GELU, residual add,
                                  norm, action head and Euler update as separate launches */

/* Sources the Standard strategy re-encodes at every step. */
typedef struct reflex_sources {
  const void* static_k;       /* device, as given to reflex_cache_init (may be NULL if static_len == 0) */
  const void* static_v;
  const void* const* frames;  /* host array of n_frames device pointers, each laid out as the frame
                                 argument of reflex_cache_write_frame, oldest first: frames[i] is frame
                                 number frames_written - n_frames + i */
  int32_t n_frames;           /* must equal n_valid = min(frames_written, window_frames) */
  int32_t reserved;
} reflex_sources;

/*
 * reflex_denoise_chunk under a chosen cache strategy, for the comparisons of
 * Section 4: the full-recomputation "Standard" baseline and the "Naive Cache"
 * negative control.  Arguments as reflex_denoise_chunk, plus:
 *   mode: REFLEX_MODE_REFLEX (identical to reflex_denoise_chunk),
 *         REFLEX_MODE_STANDARD, REFLEX_MODE_NAIVE or REFLEX_MODE_UNFUSED;
 *   src:  required for REFLEX_MODE_STANDARD, ignored otherwise (may be NULL).
 *         The frame and static buffers are read by the device work of this
 *         call and must stay unchanged until it completes.
 * Standard re-writes every window frame into its own slot at its own absolute
 * positions and the static prefix at positions 0..static_len-1 before each
 * step, with the same kernels as reflex_cache_write_frame; the cache bytes
 * therefore end up unchanged and the actions equal those of the method.  The
 * graph of a Standard call is also keyed by frames_written and the source
 * pointers.  Naive keeps one set of dynamic K/V per layer in the workspace.
 * Errors: REFLEX_EINVAL (unknown mode, missing or inconsistent sources, and as
 * reflex_denoise_chunk), REFLEX_ESTATE, REFLEX_EHIP.
 */
int reflex_denoise_chunk_baseline(reflex_ctx* ctx, int32_t mode, const reflex_sources* src,
                                  const float* state, const float* noise, int32_t num_steps,
                                  const float* tau_schedule, float* actions_out);

/*
 * Asynchronous pipeline (Section 3.3): a producer writes frames on a stream of
 * its own while the context's stream denoises chunks over frames whose write
 * has completed, so the two overlap on the GPU.  Both calls need a context
 * created with cfg.spare_slot = 1: the ring then has window_frames + 1 slots
 * and the frame being written never lands in a slot that an in-flight chunk
 * reads.  Ordering between the two streams is done on the device with events;
 * neither call blocks the host.
 *
 * reflex_pipeline_write_frame: reflex_cache_write_frame with the device work
 * enqueued on writer_stream (a hipStream_t; may be the context's stream).  On
 * the device it first waits for the previous frame write and for every chunk,
 * enqueued earlier, whose window contains the frame in the target slot.  It
 * does not change the frames a chunk sees: each chunk picks its window.
 * The frame buffer must stay unchanged until the write has completed.
 *
 * reflex_pipeline_denoise_chunk: reflex_denoise_chunk on the context's stream
 * over the window of the first n_frames frames (frames max(0, n_frames - W) ..
 * n_frames - 1, dynamic tokens at positions static_len + n_frames*frame_tokens
 * + i).  With F frames written so far, n_frames must lie in [max(0, F - 1), F];
 * the context's stream waits on the device for the write of frame
 * n_frames - 1.  n_frames = -1 takes F if the newest write has completed when
 * the call is made, else F - 1 (the consumer querying the latest cache state;
 * the host never waits).  *n_frames_out (nullable) receives the value used.
 * reflex_denoise_chunk on such a context is this call with n_frames = F.
 *
 * Errors: REFLEX_EINVAL (cfg.spare_slot == 0, n_frames outside the range, and
 * as the calls they extend), REFLEX_ESTATE, REFLEX_EHIP.  The Standard
 * strategy of reflex_denoise_chunk_baseline is not available on a context
 * with a spare slot (it would re-encode frames on the context's stream while
 * the writer stream uses the same scratch); the Naive strategy is.
 */
int reflex_pipeline_write_frame(reflex_ctx* ctx, const void* frame, void* writer_stream,
                                int64_t* frame_index_out, int32_t* evicted_tokens_out);
int reflex_pipeline_denoise_chunk(reflex_ctx* ctx, const float* state, const float* noise,
                                  int32_t num_steps, const float* tau_schedule, float* actions_out,
                                  int64_t n_frames, int64_t* n_frames_out);

/*
 * reflex_denoise_chunk for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * chunk, with the same kernels and the same results, but the chunk's
 * transient buffers (modulation, residual stream, activations, attention and
 * split-K partials) live in one static device array of the library
 * (64 MiB, allocated with the library's code on each device it runs on and
 * held until the process ends) instead of the context's workspace, and the
 * launches are enqueued directly on the context's stream (no graph is
 * instantiated).  No hipMalloc, hipFree or allocating library routine is
 * called.  Arguments, the tau schedule and the window as for
 * reflex_denoise_chunk; only the method's strategy is offered.
 * Every call on a device shares that device's array: calls that overlap on
 * one device (two contexts on two streams, or a call while another's work is
 * still in flight on another stream) race and give wrong results; calls in
 * stream order, on any contexts, are safe.  The array keeps the last call's
 * contents; the call clears what its kernels need zeroed.
 * Errors: REFLEX_ESCRATCH when the chunk needs more than 64 MiB (16 MiB at
 * batch 1 at the pi0 shapes with max_steps 10, so up to batch 4 fits; the
 * transient bytes grow with batch and max_steps), and as reflex_denoise_chunk.
 */
int reflex_denoise_chunk_static(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                                const float* tau_schedule, float* actions_out);

/*
 * Status of the chunks denoised on this context since the last check: waits
 * for the context's stream, reads and clears the device status word, and
 * returns REFLEX_ENONFINITE when any action written by the method's final
 * kernel was NaN or infinite (the NaN/Inf events that the BF16 stability
 * comparison of Section 4.6 counts), else 0.  Denoise calls stay
 * asynchronous; the check is the one synchronizing call.
 * Errors: REFLEX_ESTATE, REFLEX_EHIP.
 */
int reflex_check_status(reflex_ctx* ctx);

/* Release the host context and its captured graphs; never frees caller
 * memory (the caller-owned cache and workspace of Section 3.4's
 * pre-allocated buffers outlive it).  NULL is a no-op.  Returns 0. */
int reflex_destroy(reflex_ctx* ctx);

/* Text for a status code (for REFLEX_EHIP, the last HIP error string). */
const char* reflex_strerror(int status);

/*
 * Bookkeeping of writing frame number frames_written into a ring of
 * window_frames slots (pure host function, Section 3.1 FIFO; Appendix B.2).
 * Errors: REFLEX_EINVAL for a null out, a negative frames_written or
 * non-positive sizes.
 */
int reflex_ring_plan(int64_t frames_written, int32_t window_frames, int32_t frame_tokens,
                     int32_t static_len, reflex_ring_step* out);

/* Frames written so far into the context (host mirror).  Returns a negative
 * status for a NULL context. */
int64_t reflex_frames_written(const reflex_ctx* ctx);

/*
 * Per-kernel-class device timing (diagnostics).  While enabled, every
 * reflex_denoise_chunk and reflex_cache_write_frame runs its launches eagerly
 * (no graph) with hipEvents around each launch and synchronizes the context's
 * stream before returning; reflex_profile_read then returns the summed
 * milliseconds and launch counts per class of the last such call (the class
 * names are "embed_norm", "gemm_qkv", "attention", "attn_merge", "gemm_o",
 * "resid_norm", "gemm_gate_up", "gemm_down", "final_euler", "modulation",
 * "rope_table", "frame_proj", "ring_write").
 * n_classes in/out: capacity of the arrays in, number written out.
 */
int reflex_profile_enable(reflex_ctx* ctx, int enable);
int reflex_profile_read(reflex_ctx* ctx, const char** names, double* ms, int32_t* launches,
                        int32_t* n_classes);

/*
 * Device time of some kernel classes inside the chunk's graph (diagnostics;
 * the launch-level timing of Appendix D's measurement).  One
 * reflex_denoise_chunk call (same arguments and rules; it computes and writes
 * actions_out) is captured into a HIP graph in which every launch of a class
 * whose bit is set in class_mask (bit i: class i in reflex_profile_read's
 * order) is bracketed by one-thread kernels that write the GPU's wall clock:
 * two back to back before it, one after.  Per launch the time is (t2 - t1) -
 * (t1 - t0), the bracket minus the cost of a launch boundary measured at the
 * same point of the graph, so every kernel runs in the chunk's own order and
 * cache state.  The graph is replayed once untimed and then reps times, the
 * stamps read back after each.  Out: the summed milliseconds of the selected
 * classes per chunk (mean over the replays) and their launches per chunk (0
 * and 0 when they launch nothing).  Allocates and frees a stamp buffer;
 * synchronizes the stream.  Errors: REFLEX_ESTATE, REFLEX_EINVAL (null
 * pointers, num_steps out of range, reps < 1, no known class selected),
 * REFLEX_EHIP.
 */
int reflex_profile_graph(reflex_ctx* ctx, const float* state, const float* noise, int32_t num_steps,
                         const float* tau_schedule, float* actions_out, uint32_t class_mask, int32_t reps,
                         double* ms_per_replay, int32_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* REFLEX_H */
