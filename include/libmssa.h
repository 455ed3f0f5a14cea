/*
 * libmssa -- Multi-Scale Self-Attention (MSSA) over a Multi-Scale
 * Patchification (MSP) rolling window, for AMD Instinct MI355X (gfx950).
 *
 * Method: Ms. Forcing, Sec. 4.1.  A rolling window (Sec. 3.1, Eq. 2) holds
 * T states; state l carries F latent frames tokenized at patch scale p_l
 * (a power-of-two multiple of the native patch, nondecreasing in l), so a
 * frame of H x W native tokens becomes a ceil(H/p_l) x ceil(W/p_l) grid
 * (Eq. 3).  Queries at scale s attend to (Eq. 4)
 *     [ sink frames at native density
 *     | history frames average-pooled to scale s
 *     | every window frame b at scale max(s, p_b), pooled from p_b ]
 * with softmax(scale * q k^T) v per head.  Frames coarser than the query keep
 * their own scale; the sink is never resampled.  A pooled cell averages the
 * cells of its f x f block that exist (ragged edges average fewer cells).
 *
 * Conventions shared by every entry point
 *   - Tensors are token-major, contiguous [tokens, num_heads, head_dim], in
 *     the plan's dtype (bf16 or fp32), 16-byte aligned device pointers.
 *     Window tokens are ordered (state 1..T, frame, row, col) at the state's
 *     scale; sink and history tokens are (frame, row, col) at native scale,
 *     history oldest first.
 *   - The caller owns all device memory (inputs, output, workspace).  The
 *     library never allocates or frees device memory; a plan owns only host
 *     memory.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Device entry points only enqueue work on it and never synchronise; a
 *     fault inside a kernel surfaces at the caller's next synchronisation.
 *   - Every entry point validates its arguments before enqueuing anything
 *     and returns a status; no C++ exception crosses this boundary.
 *     mssa_last_error() returns a thread-local message for the last failure.
 *   - A plan is immutable after creation and may be shared between threads
 *     and streams; concurrent calls need one workspace each.
 *   - Kernels use fixed reduction orders and no atomics: results are
 *     bitwise reproducible run to run.
 */
#ifndef LIBMSSA_H
#define LIBMSSA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MSSA_MAX_STATES 8

typedef struct mssa_plan_s* mssa_plan;

typedef enum {
  MSSA_OK = 0,
  MSSA_ERR_INVALID_ARG = 1, /* null pointer, bad size, inconsistent argument */
  MSSA_ERR_UNSUPPORTED = 2, /* valid descriptor this build does not run */
  MSSA_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
  MSSA_ERR_DEVICE = 4,      /* HIP launch or runtime error */
  MSSA_ERR_NO_MEMORY = 5    /* host allocation failed */
} mssa_status;

typedef enum { MSSA_BF16 = 0, MSSA_F32 = 1 } mssa_dtype;

/* Static problem description (Sec. 4.1 problem statement; Sec. 5.1 sizes). */
typedef struct {
  int32_t num_states;               /* T, 1..MSSA_MAX_STATES */
  int32_t scales[MSSA_MAX_STATES];  /* p_l / p for l = 1..T: powers of two in
                                       [1, 64], nondecreasing (Sec. 4.1) */
  int32_t grid_h, grid_w;           /* native token grid of a latent frame */
  int32_t frames_per_state;         /* F latent frames per window state */
  int32_t sink_frames;              /* S native sink frames (>= 0) */
  int32_t hist_frames;              /* Hh native history frames (>= 0) */
  int32_t num_heads;                /* >= 1 */
  int32_t head_dim;                 /* 64 or 128 */
  int32_t dtype;                    /* mssa_dtype of every tensor */
  float softmax_scale;              /* <= 0 selects 1/sqrt(head_dim) */
  int32_t flags;                    /* MSSA_PLAN_* bits, 0 for the plain path */
} mssa_plan_desc;

/* Plan flag: the history pooled to every query scale s > 1 lives in
 * caller-owned pooled-history rings (one K and one V ring per such scale)
 * that the cache roll keeps up to date, instead of being pooled from native
 * history by every mssa_pool_kv.  Such a plan pools only window frames in
 * mssa_pool_kv and is run with mssa_forward_ring / mssa_hist_append_ring. */
#define MSSA_PLAN_POOLED_HIST_RING 1

/* Plan flag: resample by stride instead of by block mean (the literal reading
 * of Eq. 4's Subsample and of the stride-2 probe of Sec. 3.2).  Every pooled
 * token is the first cell (row f*Y, column f*X) of its f x f block on the
 * source frame's grid, copied bit for bit.  Grids, context tables and
 * attention are unchanged; only what mssa_pool_kv / mssa_pool_hist_ring write
 * differs.  Combines with MSSA_PLAN_POOLED_HIST_RING. */
#define MSSA_PLAN_STRIDED_SUBSAMPLE 2

/* Plan flag (with MSSA_PLAN_POOLED_HIST_RING, bf16, scales[0] == 1): the
 * cache roll moves no data.  Window state 1's K/V are written by their
 * producer straight into spare slots of the native history ring, and
 * mssa_pool_kv_head_ring pools them into the same slots of every pooled
 * ring; the attention reads state 1 from there, and mssa_head_ring_roll only
 * advances the ring state.  See "Cache roll without copies" below. */
#define MSSA_PLAN_HEAD_IN_RING 4

/* Plan flag: every q_win passed with this plan holds the queries already
 * multiplied by softmax_scale * log2(e), i.e. Eq. 4's scaled scores
 * scale q k^T taken into the base-2 exponent domain, so that
 * softmax(scale q k^T) = 2^(q' k^T) / sum 2^(q' k^T) for q' = scale log2(e) q.
 * A producer can fold the factor into its own epilogue before its single
 * rounding to the plan dtype (the query projection's weights, or the query
 * norm's gain), and the bf16 attention then spends no instruction per score
 * on the scale.  Outputs and lse are those of the unscaled queries q; the
 * backward's dq_win is the gradient with respect to q' (dL/dq' = dL/dq /
 * (softmax_scale log2(e))).  softmax_scale still names the factor. */
#define MSSA_PLAN_Q_PRESCALED 8

/* Sizes derived by the plan.  Group g is the g-th distinct query scale in
 * window token order; its queries are the contiguous range
 * [q_begin[g], q_end[g]) and its context has n_kv[g] tokens per head.
 * The pooled K/V that group g reads (history pooled to its scale, then the
 * window frames finer than its scale pooled to it, in context order) live in
 * the workspace at byte offsets pooled_k_offset[g] / pooled_v_offset[g],
 * pooled_tokens[g] tokens each, laid out [tokens, num_heads, head_dim]. */
typedef struct {
  int64_t n_q;              /* window (query) tokens */
  int64_t n_sink_tok;       /* sink_frames * grid_h * grid_w */
  int64_t n_hist_tok;       /* hist_frames * grid_h * grid_w */
  int64_t workspace_bytes;  /* minimum workspace for pool_kv / forward */
  int64_t pairs_per_head;   /* sum over groups of queries * n_kv */
  int64_t flops_alg;        /* 4 * head_dim * num_heads * pairs_per_head */
  int64_t pool_bytes_alg;   /* bytes pool_kv must read once and write once */
  int32_t n_groups;
  int32_t group_scale[MSSA_MAX_STATES];
  int32_t q_begin[MSSA_MAX_STATES];
  int32_t q_end[MSSA_MAX_STATES];
  int64_t n_kv[MSSA_MAX_STATES];
  int64_t pooled_k_offset[MSSA_MAX_STATES];
  int64_t pooled_v_offset[MSSA_MAX_STATES];
  int64_t pooled_tokens[MSSA_MAX_STATES];
} mssa_plan_info;

/* Build the static plan: MSP grids (Eq. 3), query groups, the per-scale
 * context segment tables (Eq. 4), pool jobs and the kernel work list.
 * Host only.  Returns MSSA_ERR_INVALID_ARG for a malformed descriptor or
 * null pointer, MSSA_ERR_UNSUPPORTED for a schedule that is not made of
 * nondecreasing powers of two, head_dim not in {64, 128}, or sizes beyond
 * the 32-bit token indexing of the kernels.  *out is set only on success;
 * release it with mssa_plan_destroy. */
mssa_status mssa_plan_create(const mssa_plan_desc* desc, mssa_plan* out);

/* mssa_plan_create with the number of persistent attention blocks of the
 * bf16 forward chosen by the caller.  The forward's work (every query scale,
 * head and 256-query tile, each a sequence of 64-key tiles) is cut into
 * attention_blocks equal shares, one per block; a share may end inside an
 * item, whose pieces are then merged in a fixed order.  attention_blocks ==
 * 0 takes one block per resident slot of the current device (512 without a
 * device), as mssa_plan_create does; fewer leaves compute units to other
 * streams, more runs in several waves.  The plan's workspace size depends on
 * it.  MSSA_ERR_INVALID_ARG for attention_blocks < 0; otherwise as
 * mssa_plan_create. */
mssa_status mssa_plan_create_ex(const mssa_plan_desc* desc, int32_t attention_blocks, mssa_plan* out);

/* Release a plan (NULL is ignored).  The caller must not use it afterwards
 * and must have no work using it still pending on any stream. */
void mssa_plan_destroy(mssa_plan plan);

/* Copy the derived sizes into *info (host). */
mssa_status mssa_plan_query(mssa_plan plan, mssa_plan_info* info);

/* Export the plan tables as int64 values (host):
 *   [n_grid, n_qgrp, n_seg,
 *    GRID rows  {scale, gh, gw, tokens}                        x n_grid,
 *    QGRP rows  {q_scale, q_begin, q_end, n_kv}                x n_qgrp,
 *    SEG rows   {q_scale, kind, frame, src_scale, eff_scale,
 *                factor, n_tok, kv_begin}                      x n_seg,
 *    TOTAL      {n_q, pairs_per_head}]
 * kind: 0 sink, 1 history, 2 window; frame: index within its kind (window
 * frames counted across states).  SEG rows are in context order: sink,
 * history oldest first, window state 1..T (Eq. 4).  *needed receives the
 * number of int64 values; if cap < *needed nothing is written and
 * MSSA_ERR_INVALID_ARG is returned (dst may be NULL to query the size). */
mssa_status mssa_plan_tables(mssa_plan plan, int64_t* dst, int64_t cap, int64_t* needed);

/* K/V resampling (Eq. 4 "Subsample", read as an average pool): for every
 * query scale s > 1, average-pool each history frame from native and each
 * window frame with p_b < s from p_b to scale s, over the cells that exist
 * in each block, for K and V alike, every head and channel.  fp32
 * accumulation; results rounded to the plan dtype (round-to-nearest-even)
 * into the workspace at the offsets mssa_plan_query reports.
 *   k_hist, v_hist  [n_hist_tok, H, D] device (NULL iff hist_frames == 0)
 *   k_win, v_win    [n_q, H, D] device
 *   workspace       device, >= workspace_bytes, 256-byte aligned
 * Enqueues on `stream`; a plan with a single query scale 1 enqueues
 * nothing. */
mssa_status mssa_pool_kv(mssa_plan plan, const void* k_hist, const void* v_hist,
                         const void* k_win, const void* v_win, void* workspace,
                         int64_t workspace_bytes, void* stream);

/* Multi-scale self-attention forward (Eq. 4): for every head and query
 * scale s, out = softmax(softmax_scale * q k^T) v over the context of s,
 * reading sink/history/window K/V directly and the pooled K/V that
 * mssa_pool_kv wrote to `workspace` earlier on the same stream.  bf16 plans
 * use bf16 matrix cores with fp32 accumulation and an fp32 online softmax;
 * fp32 plans compute in fp32 throughout.
 *   q_win            [n_q, H, D] device
 *   k_sink, v_sink   [n_sink_tok, H, D] device (NULL iff sink_frames == 0)
 *   k_hist, v_hist   [n_hist_tok, H, D] device (NULL iff hist_frames == 0)
 *   k_win, v_win     [n_q, H, D] device
 *   workspace        as passed to mssa_pool_kv
 *   out              [n_q, H, D] device, same dtype, must not alias inputs */
mssa_status mssa_forward(mssa_plan plan, const void* q_win, const void* k_sink,
                         const void* v_sink, const void* k_hist, const void* v_hist,
                         const void* k_win, const void* v_win, const void* workspace,
                         int64_t workspace_bytes, void* out, void* stream);

/* ------------------------------------------------------ no allocation
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): pool +
 * forward of one pass with the library's own scratch as the workspace.
 *
 * mssa_attention_noalloc(plan, ...) enqueues exactly what mssa_pool_kv
 * followed by mssa_forward enqueue (the same kernels, bitwise the same
 * output), with the workspace in a device array of
 * MSSA_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends.  It calls no device allocation routine.  The
 * scratch of the current device is found on the first call on that device;
 * `stream` must belong to the current device.  Every call on a GPU shares
 * that GPU's scratch, which keeps the last call's contents (nothing in it
 * needs to start at zero): calls that overlap on one GPU (two streams, or
 * host threads) race and must be ordered by the caller.
 *   arguments  as for mssa_forward, without the workspace
 * MSSA_ERR_WORKSPACE if the plan's workspace_bytes exceed
 * MSSA_NOALLOC_SCRATCH_BYTES (e.g. the 40-head 720p layer);
 * MSSA_ERR_UNSUPPORTED for plans with MSSA_PLAN_POOLED_HIST_RING; otherwise
 * the errors of mssa_pool_kv and mssa_forward, all checked before anything
 * is enqueued. */
#define MSSA_NOALLOC_SCRATCH_BYTES (256ll << 20)

mssa_status mssa_attention_noalloc(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                                   const void* k_hist, const void* v_hist, const void* k_win, const void* v_win,
                                   void* out, void* stream);

/* ----------------------------------------------------------------- training
 * The window is trained through its attention (Sec. 3.1; Alg. 1 updates the
 * model by gradient steps on the rolling window), so the backward of Eq. 4:
 * per head and query scale s, with P = softmax(softmax_scale q k_s^T) and dO
 * the gradient of the output,
 *   dV_s = P^T dO,  dS = P * (dO V_s^T - rowsum(dO * out)),
 *   dQ = softmax_scale dS K_s,  dK_s = softmax_scale dS^T Q,
 * and each context row's gradient goes back to the sink, history or window
 * token(s) it was made from (block mean: g / c to each of the block's c
 * cells; strided plans: g to the block's first cell), summed over the query
 * scales whose contexts hold it.  Plans with MSSA_PLAN_POOLED_HIST_RING are
 * not supported (MSSA_ERR_UNSUPPORTED). */

/* mssa_forward that also writes lse [H, n_q] (fp32, device, head-major):
 * lse[h * n_q + i] = log sum_j exp(softmax_scale q_i . k_j) over query i's
 * context, natural log (q the unscaled queries also for
 * MSSA_PLAN_Q_PRESCALED plans).  Same arguments and errors as mssa_forward; lse must
 * be non-null and 16-byte aligned. */
mssa_status mssa_forward_lse(mssa_plan plan, const void* q_win, const void* k_sink,
                             const void* v_sink, const void* k_hist, const void* v_hist,
                             const void* k_win, const void* v_win, const void* workspace,
                             int64_t workspace_bytes, void* out, float* lse, void* stream);

/* Bytes of device workspace mssa_backward needs (>= workspace_bytes: the
 * pooled K/V sit at the same offsets as for mssa_forward, followed by the
 * backward's own buffers: fp32 row statistics and context gradients, and for
 * bf16 plans the bf16 dS = P * (dP - rowsum) of as many whole heads as fit
 * in 8 GiB (at least one; the backward runs the heads in such chunks), i.e.
 * about 2 bytes per (query, context token) pair of each head of a chunk). */
mssa_status mssa_backward_workspace_size(mssa_plan plan, int64_t* bytes);

/* Gradients of MSSA with respect to all seven inputs.
 *   q_win .. v_win   the forward's inputs (as for mssa_forward)
 *   out, lse         the forward's output and mssa_forward_lse's lse
 *   d_out            [n_q, H, D] device, gradient of the output
 *   workspace        device, >= mssa_backward_workspace_size bytes,
 *                    256-byte aligned, whose pooled K/V are what
 *                    mssa_pool_kv wrote for these inputs (the forward's
 *                    workspace can be reused as is)
 *   dq_win .. dv_win device outputs shaped like the inputs, plan dtype,
 *                    written (not accumulated; dq_win is the gradient with
 *                    respect to q_win as passed, i.e. the scaled queries of
 *                    a MSSA_PLAN_Q_PRESCALED plan); dk_sink / dv_sink may be
 *                    NULL iff sink_frames == 0, dk_hist / dv_hist iff
 *                    hist_frames == 0; no gradient may alias an input.
 * bf16 plans use bf16 matrix cores with fp32 accumulation (probabilities
 * and dS rounded to bf16 as matrix operands); fp32 plans compute in fp32.
 * Enqueues on `stream`; deterministic (fixed summation orders, no atomics).
 * MSSA_ERR_WORKSPACE for a small workspace. */
mssa_status mssa_backward(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                          const void* k_hist, const void* v_hist, const void* k_win, const void* v_win,
                          const void* out, const float* lse, const void* d_out, void* workspace,
                          int64_t workspace_bytes, void* dq_win, void* dk_sink, void* dv_sink, void* dk_hist,
                          void* dv_hist, void* dk_win, void* dv_win, void* stream);

/* --------------------------------------------------------------- MSP tiers
 * The steps on either side of the attention (Sec. 4.1, Multi-Scale
 * Patchification): window state l is tokenized with patch p * p_l by its
 * tier's own patch embedding (each (p p_l) x (p p_l) patch of all latent
 * channels, flattened in (channel, row, column) order, times the tier's
 * weights, plus bias: a 2-D convolution with kernel = stride = p p_l); the
 * de-embedding maps tokens back to pixels; the attention's q, k, v are one
 * linear projection of the tokens.  Patches past a ragged frame edge see
 * zeros; de-embedded pixels past it are dropped.  bf16 plans only (fp32
 * accumulation); MSSA_ERR_UNSUPPORTED for fp32 plans or when
 * C * (p * scale)^2 is not a multiple of 8. */
typedef struct {
  int32_t latent_channels;  /* C */
  int32_t patch;            /* p: native patch size in latent pixels (the plan's grid is in patches) */
  int32_t hidden;           /* model width (heads x head_dim for the attention), multiple of 8 */
} mssa_tier_desc;

/* Device workspace bytes of mssa_patch_embed / mssa_patch_unembed. */
mssa_status mssa_tier_workspace_size(mssa_plan plan, const mssa_tier_desc* tier, int64_t* bytes);

/* latent [T*F, C, grid_h * p, grid_w * p] bf16 (window frames in window
 * order) -> tokens [n_q, hidden] bf16 in the attention's window token order.
 * w_embed[g] / b_embed[g]: query group g's tier (mssa_plan_info order, scale
 * s = group_scale[g]), [hidden, C * (p s)^2] and [hidden] bf16, device. */
mssa_status mssa_patch_embed(mssa_plan plan, const mssa_tier_desc* tier, const void* latent,
                             const void* const* w_embed, const void* const* b_embed, void* workspace,
                             int64_t workspace_bytes, void* tokens, void* stream);

/* tokens [n_q, hidden] -> latent [T*F, C, grid_h * p, grid_w * p] (bf16):
 * w_out[g] [C * (p s)^2, hidden], b_out[g] [C * (p s)^2]. */
mssa_status mssa_patch_unembed(mssa_plan plan, const mssa_tier_desc* tier, const void* tokens,
                               const void* const* w_out, const void* const* b_out, void* workspace,
                               int64_t workspace_bytes, void* latent, void* stream);

/* q, k, v = x W_qkv^T + b_qkv split in three blocks of `hidden` features:
 * x [n_tokens, hidden], w_qkv [3 * hidden, hidden], b_qkv [3 * hidden],
 * q, k, v [n_tokens, hidden] (= [n_tokens, heads, head_dim]), all bf16,
 * device; outputs must not alias x. */
mssa_status mssa_qkv_project(int64_t n_tokens, int32_t hidden, const void* x, const void* w_qkv,
                             const void* b_qkv, void* q, void* k, void* v, void* stream);

/* mssa_qkv_project with the queries multiplied by q_scale: q = (x W_q^T +
 * b_q) * q_scale, taken on the fp32 sum and rounded to bf16 once; k and v
 * as mssa_qkv_project writes them.  With q_scale = softmax_scale * log2(e)
 * it hands over the queries of a MSSA_PLAN_Q_PRESCALED plan (Eq. 4's score
 * scale folded into the query projection's epilogue) with no second
 * rounding.  MSSA_ERR_INVALID_ARG also for a non-finite q_scale. */
mssa_status mssa_qkv_project_scaled(int64_t n_tokens, int32_t hidden, const void* x, const void* w_qkv,
                                    const void* b_qkv, float q_scale, void* q, void* k, void* v, void* stream);

/* Streaming cache roll (Sec. 3.1, Eq. 2; Alg. 1 KV-cache update): after a
 * rolling pass the head state (window state 1, which must be at native
 * scale: scales[0] == 1) is emitted, and its F native frames of K and V
 * become the newest history frames.  They are copied from the first
 * F * grid_h * grid_w tokens of k_win / v_win into a caller-owned ring of
 * ring_cap_frames native frames ([ring_cap_frames * grid_h * grid_w, H, D],
 * plan dtype).  The ring holds *ring_count valid frames: while it is not
 * full they are slots [0, count) and the frames are appended at slot count;
 * once full, the oldest frames (starting at slot *ring_head) are overwritten
 * and *ring_head advances.  The valid frames are therefore always slots
 * [0, count), which a plan with hist_frames == count reads as its history
 * (attention is invariant to the order of its context frames).
 *   k_win, v_win     [n_q, H, D] device, this pass's window K/V
 *   k_ring, v_ring   device ring buffers (must not overlap k_win / v_win)
 *   ring_head, ring_count  host in/out; 0 <= count <= cap, 0 <= head < cap,
 *                    head == 0 unless count == cap
 * Enqueues device-to-device copies on `stream`; MSSA_ERR_UNSUPPORTED if
 * scales[0] != 1 or ring_cap_frames < frames_per_state. */
mssa_status mssa_hist_append(mssa_plan plan, const void* k_win, const void* v_win, void* k_ring,
                             void* v_ring, int32_t ring_cap_frames, int32_t* ring_head,
                             int32_t* ring_count, void* stream);

/* Streaming with incrementally pooled history (Sec. 3.1, Eq. 2 cache roll;
 * Eq. 4 history at the query scale), for plans created with
 * MSSA_PLAN_POOLED_HIST_RING.  For query group g (mssa_plan_info order) with
 * scale s = group_scale[g] > 1, the pooled-history ring of K (V) is a
 * caller-owned device buffer of ring_cap_frames slots of tok_s tokens
 * ([ring_cap_frames * tok_s, H, D], plan dtype, tok_s the tokens of a frame
 * at scale s); slot f holds the native ring's slot f pooled to s.  Arrays
 * k_*_pooled / v_*_pooled have one entry per query group; entries of groups
 * with scale 1 are ignored and may be NULL.  The history the plan reads is
 * slots [0, hist_frames), as for the native ring.  Pooled frames equal, bit
 * for bit, what mssa_pool_kv computes from the native frames; the attention
 * outputs agree with the plain path up to the kernel's rounding (the
 * pooled history is a key run of its own, so key tiles fall differently). */

/* Pool native ring slots [0, hist_frames) to every query scale s > 1 into
 * the pooled rings (once, to start from an existing native history).
 * MSSA_ERR_UNSUPPORTED for a plan without the flag. */
mssa_status mssa_pool_hist_ring(mssa_plan plan, const void* k_ring, const void* v_ring, void* const* k_ring_pooled,
                                void* const* v_ring_pooled, void* stream);

/* mssa_forward for a MSSA_PLAN_POOLED_HIST_RING plan: group g with scale > 1
 * reads its history from k_hist_pooled[g] / v_hist_pooled[g]; everything else
 * (and workspace, which holds this pass's pooled window frames) as in
 * mssa_forward.  MSSA_ERR_UNSUPPORTED for a plan without the flag. */
mssa_status mssa_forward_ring(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                              const void* k_hist, const void* v_hist, const void* const* k_hist_pooled,
                              const void* const* v_hist_pooled, const void* k_win, const void* v_win,
                              const void* workspace, int64_t workspace_bytes, void* out, void* stream);

/* mssa_hist_append for a MSSA_PLAN_POOLED_HIST_RING plan: the head state's F
 * native frames go to the native ring as there, and the same frames pooled
 * to each scale s > 1, which this pass's mssa_pool_kv left in `workspace`,
 * go to the same slots of the pooled rings.  Enqueues device-to-device
 * copies on `stream` (after this pass's mssa_forward, which reads the
 * rings).  MSSA_ERR_UNSUPPORTED for a plan without the flag. */
mssa_status mssa_hist_append_ring(mssa_plan plan, const void* k_win, const void* v_win, const void* workspace,
                                  int64_t workspace_bytes, void* k_ring, void* v_ring, void* const* k_ring_pooled,
                                  void* const* v_ring_pooled, int32_t ring_cap_frames, int32_t* ring_head,
                                  int32_t* ring_count, void* stream);

/* ------------------------------------------------ cache roll without copies
 * For plans created with MSSA_PLAN_HEAD_IN_RING (Sec. 3.1, Eq. 2: the head
 * state emitted by a pass becomes the newest history; Alg. 1's KV-cache
 * update).  The native ring and every pooled ring (one per query group with
 * scale s > 1, as for MSSA_PLAN_POOLED_HIST_RING) have ring_frames slots of
 * one frame each; ring_frames - F is the FIFO cap of the history (F =
 * frames_per_state), and both ring_frames and the cap are multiples of F.
 * The ring state is (ring_count, ring_spare):
 *   - the history is ring_count frames (the plan's hist_frames), oldest
 *     first, in slots ring_spare - ring_count .. ring_spare - 1 (mod
 *     ring_frames);
 *   - slots ring_spare .. ring_spare + F - 1 hold window state 1 of the
 *     current pass: its producer writes the native K/V there (frame f of the
 *     state in slot ring_spare + f), in place of the first F frames of the
 *     window K/V;
 *   - ring_spare is a multiple of F in [0, ring_frames).
 * A fresh ring starts with its history in slots [0, count) and ring_spare =
 * count (mssa_pool_hist_ring fills the pooled rings from it).  A pass is
 * mssa_pool_kv_head_ring, mssa_forward_head_ring, mssa_head_ring_roll; the
 * roll copies nothing.
 *   k_win, v_win   window K/V of states 2..T only: [n_q - F * grid_h *
 *                  grid_w, H, D] device (the window tokens after state 1)
 *   k_ring, v_ring the native ring, [ring_frames * grid_h * grid_w, H, D]
 *   k_ring_pooled, v_ring_pooled  per query group (mssa_plan_info order):
 *                  [ring_frames * tok_s, H, D] for scale s > 1, else ignored
 * MSSA_ERR_UNSUPPORTED for a plan without the flag; MSSA_ERR_INVALID_ARG
 * for a ring state that breaks the rules above or ring_count !=
 * hist_frames. */

/* Pool window state 1 (read from the native ring's spare slots) into the
 * spare slots of every pooled ring, and the window frames of states 2..T
 * that are finer than a query scale into the workspace (Eq. 4). */
mssa_status mssa_pool_kv_head_ring(mssa_plan plan, const void* k_ring, const void* v_ring, const void* k_win,
                                   const void* v_win, void* const* k_ring_pooled, void* const* v_ring_pooled,
                                   void* workspace, int64_t workspace_bytes, int32_t ring_frames,
                                   int32_t ring_count, int32_t ring_spare, void* stream);

/* Attention of the pass (Eq. 4): as mssa_forward, with the history and
 * window state 1 read from the rings. */
mssa_status mssa_forward_head_ring(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                                   const void* k_ring, const void* v_ring, const void* const* k_ring_pooled,
                                   const void* const* v_ring_pooled, const void* k_win, const void* v_win,
                                   const void* workspace, int64_t workspace_bytes, void* out, int32_t ring_frames,
                                   int32_t ring_count, int32_t ring_spare, void* stream);

/* The cache roll after a pass (host only, nothing enqueued): state 1 joins
 * the history, whose oldest frames leave once it exceeds the cap.
 * *ring_count becomes min(count + F, ring_frames - F) and *ring_spare
 * (spare + F) mod ring_frames. */
mssa_status mssa_head_ring_roll(mssa_plan plan, int32_t ring_frames, int32_t* ring_count, int32_t* ring_spare);

/* Name of a status code (static string). */
const char* mssa_status_string(mssa_status s);

/* Detail of the last non-OK status returned on this thread ("" if none). */
const char* mssa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBMSSA_H */
