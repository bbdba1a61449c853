/*
 * statekv.h — C ABI of the StateKV per-frame streaming video-prefill step on
 * AMD Instinct MI355X (gfx950).
 *
 * Method: "Linear Scaling Video VLMs for Long Video Understanding" (StateKV).
 * For every layer, the T query tokens of frame n attend over the layer's
 * compressed state C_{n-1} (capacity B, the only cross-frame context, Eq. 4)
 * followed by the frame's own keys, causal inside the frame (Eq. 5, mask M_n).
 * The same pass sums, for every candidate key, the attention mass it receives
 * from the frame's queries of all query heads sharing its KV head, divided by
 * T (the score instantiation of the "attention-driven selection" paragraph).
 * The B best candidates (ties: lowest position) become C_n (Eq. 6); the frame's
 * K/V rows are appended to the per-layer decode cache D (Eq. 4, the detailed
 * state), which prefill never reads.  Token positions derive from the virtual
 * length L_n (virtual sequence length paragraph).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers named q, k, v, out are DEVICE pointers owned by the caller, 16-byte
 *   aligned (the kernels move 16-byte chunks); a misaligned one is
 *   SKV_ERR_INVALID_ARG.
 * - Every device operation is enqueued on the HIP stream given to skv_init and
 *   is stream-ordered; no call blocks the host except skv_timing_stop.
 * - Errors are returned as skv_status.  Argument, order and capacity errors are
 *   found before anything is enqueued and leave the context unchanged.  A launch
 *   failure (SKV_ERR_DEVICE from skv_frame_step, skv_decode_step or skv_state_view) can come
 *   after earlier kernels of the same call were enqueued: the context is then
 *   marked, and every later frame or decode step returns SKV_ERR_DEVICE until
 *   skv_reset or skv_seek restarts the stream.  Asynchronous device faults
 *   surface at the caller's next synchronisation.
 * - All device memory of a context is allocated once in skv_init and released
 *   in skv_destroy; skv_frame_step allocates nothing.
 * - A context is not thread-safe: calls on one context must be serialised.
 */
#ifndef STATEKV_H
#define STATEKV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SKV_OK = 0,
  SKV_ERR_INVALID_ARG = -1,   /* null pointer, bad size, unsupported combination */
  SKV_ERR_OUT_OF_MEMORY = -2, /* device allocation failed in skv_init */
  SKV_ERR_CAPACITY = -3,      /* decode cache full: frame >= max_frames */
  SKV_ERR_ORDER = -4,         /* layer_begin is not the next layer of the current frame */
  SKV_ERR_DEVICE = -5,        /* HIP runtime or launch error */
  SKV_ERR_UNSUPPORTED = -6    /* valid request the library does not implement */
} skv_status;

typedef enum { SKV_BF16 = 0, SKV_F32 = 1 } skv_dtype;

/* What the cross-frame context of a layer is (selection paragraph of the
 * method, and the two baselines of the evaluation):
 *   SKV_POLICY_STATEKV  the compressed state C_n: the B candidates of state and
 *                       frame with the highest importance score (Eq. 6), ties
 *                       to the lowest position;
 *   SKV_POLICY_RECENT   the B most recent tokens (the recency-window baseline,
 *                       ReKV-style: a window of the last B / T frames when T
 *                       divides B); importance scores are still computed and
 *                       reported, but do not decide;
 *   SKV_POLICY_FULL     no compression: frame n attends to every earlier token,
 *                       read from the decode cache D (streaming full
 *                       self-attention, the Full SA baseline); capacity is
 *                       ignored, no scores are computed and the state stays
 *                       empty. */
typedef enum { SKV_POLICY_STATEKV = 0, SKV_POLICY_RECENT = 1, SKV_POLICY_FULL = 2 } skv_policy;

/* Rotary position embedding applied inside the step (virtual sequence length
 * paragraph: positions come from L_n, not from the cache size; RoPE scaling
 * paragraph: one scaling for cache building and decoding).  With SKV_ROPE_NONE
 * the inputs are used as given.  Otherwise the library rotates Q and K of every
 * frame (and of every decoded token) at their virtual positions
 * p = pos_offset + n*T + t (decoded tokens continue after the frames done),
 * and the compressed state and the decode cache hold the rotated keys.
 * Pairing is half-split: dimension j < d/2 rotates with j + d/2 by the angle
 * p * f_j, f_j = rope_theta^(-2j/d):
 *   x'_j = x_j cos - x_{j+d/2} sin,   x'_{j+d/2} = x_{j+d/2} cos + x_j sin.
 * SKV_ROPE_YARN uses YaRN's frequencies and temperature with scale s =
 * rope_factor and original context rope_orig_max: per dimension, r_j =
 * rope_orig_max * f_j / (2 pi), g_j = clamp((r_j - 1) / (32 - 1), 0, 1),
 * f'_j = (1 - g_j) f_j / s + g_j f_j, and cos and sin are multiplied by
 * 0.1 ln(s) + 1.  Angles are reduced in double precision on the host (a
 * table of cos/sin per position); rotated values are rounded to the config
 * dtype. */
typedef enum { SKV_ROPE_NONE = 0, SKV_ROPE_PLAIN = 1, SKV_ROPE_YARN = 2 } skv_rope;

/* Problem statement of the method: head counts and head dimension d_h (Eq. 5),
 * T tokens per frame, capacity B of the compressed state (Eq. 4), layer count,
 * and the decode-cache length, which grows by T per frame. */
typedef struct {
  int32_t n_layers;         /* L >= 1 */
  int32_t n_q_heads;        /* H_q, a multiple of n_kv_heads (grouped-query attention) */
  int32_t n_kv_heads;       /* H_kv >= 1; query head h reads KV head h / (H_q / H_kv) */
  int32_t head_dim;         /* d_h: 64 or 128 */
  int32_t tokens_per_frame; /* T >= 1 */
  int32_t capacity;         /* B >= 0 */
  int32_t max_frames;       /* frames the decode cache holds, >= 1 */
  int32_t dtype;            /* skv_dtype of Q, K, V, the output and both caches */
  float softmax_scale;      /* logit scale; 0 selects 1/sqrt(head_dim) */
  int64_t pos_offset;       /* virtual position of the first video token (room for a text prefix) */
  int32_t policy;           /* skv_policy; 0 (a zeroed config) is StateKV */
  int32_t max_decode_tokens; /* rows of D kept for tokens decoded after the video (>= 0) */
  int32_t rope;             /* skv_rope; 0 (a zeroed config): no rotation */
  float rope_theta;         /* RoPE base (> 0 when rope != 0), e.g. 10000 or 1e6 */
  float rope_factor;        /* YaRN scale s >= 1 (SKV_ROPE_YARN only) */
  int32_t rope_orig_max;    /* YaRN original context length (> 0, SKV_ROPE_YARN only) */
  int32_t split_refresh;    /* 0 (a zeroed config): the refresh of a frame step is one launch (selection
                               and state update in one set of workgroups, the decode-cache append in
                               another); 1: three launches, selection, state update, append, so that each
                               stage can be timed (skv_timing_*) and profiled on its own.  The results
                               are the same bit for bit. */
  int32_t key_split_mode;   /* calls too small to fill the device split the attention's keys into ranges
                               whose row statistics are merged before the output: 0 (a zeroed config):
                               one launch, in which the workgroups of a row range exchange their ranges'
                               statistics (each waits a bounded time for the others and computes any
                               that has not arrived); 1: two launches, statistics then output; 2: one
                               launch in which every workgroup computes every range's statistics itself.
                               The results are the same bit for bit. */
} skv_config;

typedef struct skv_ctx skv_ctx;

/* Validates cfg, allocates and zeroes every device buffer of one video stream
 * (compressed state and decode cache of all layers, scratch), and binds the
 * context to hip_stream (a hipStream_t; NULL means the default stream).
 * Limits: pos_offset + max_frames * T + max_decode_tokens < 2^31; B + T <= 16384
 * (STATEKV and RECENT); policy one of skv_policy, split_refresh 0 or 1 and
 * key_split_mode 0, 1 or 2, else SKV_ERR_INVALID_ARG.
 * Returns SKV_OK and *out, or an error and *out = NULL. */
skv_status skv_init(const skv_config* cfg, void* hip_stream, skv_ctx** out);

/* Runs layers [layer_begin, layer_begin + layer_count) of the current frame n:
 * attention with fused importance scoring (Eq. 5 and the score), Top-B refresh
 * of each layer's compressed state (Eq. 6), and append of the frame's K/V to
 * each layer's decode cache.  Under SKV_POLICY_RECENT the refresh keeps the B
 * most recent candidates; under SKV_POLICY_FULL the frame attends to all
 * n * T cached tokens plus itself (causal), and only the append follows.  Layers of one frame must be stepped in order;
 * the frame counter advances after the last layer.  layer_count = n_layers
 * runs the whole stack in one launch per stage.
 * Calls too small to fill the device (e.g. one layer of the 7B shape) split the
 * keys of the attention over more workgroups.  When such a call covers only part
 * of the stack, its selection and state update are not enqueued by the call
 * itself: they run beside the attention of the next such call on other layers
 * (the next layer of the real-model calling pattern), or are enqueued on their
 * own by the next call that needs the state, by skv_state_view or by a context
 * whose split_refresh is 1.  The frame's rows are read back from the decode
 * cache for them, so k and v may be reused once the call's work is done.  The
 * attention output, the decode-cache append and every result are the same as
 * without the deferral.
 * Device layouts (row-major, dtype of the config):
 *   q   [layer_count][H_q ][T][d]
 *   k,v [layer_count][H_kv][T][d]
 *   out [layer_count][H_q ][T][d]   attention output, written
 * Errors: SKV_ERR_INVALID_ARG (null pointer, count out of range),
 * SKV_ERR_ORDER, SKV_ERR_CAPACITY (n >= max_frames), SKV_ERR_DEVICE. */
skv_status skv_frame_step(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count,
                          const void* q, const void* k, const void* v, void* out);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): skv_frame_step with the
 * same arguments, layouts, results (bit for bit) and errors, except that the
 * per-call scratch of the step (column-sum partials, key-split row statistics and
 * output shares, admit lists) lives in one static device array of the library,
 * 64 MiB per device, instead of the context's buffers.  The call allocates and
 * frees nothing and calls no allocating routine.  A call needing more than 64 MiB
 * of scratch returns SKV_ERR_UNSUPPORTED with nothing enqueued (e.g. all 80 layers
 * of the 72B-shaped stack in one call; one layer per call fits).  Every call on a
 * device shares that device's array and leaves it holding its own partial
 * results; nothing in it has to start at zero.  Calls that overlap on one device
 * (contexts on different streams) race on the array: serialise them.  Since the
 * array is reused by the next call, this entry point never defers a selection
 * (see skv_frame_step); it enqueues one that an earlier skv_frame_step deferred.
 * A captured call is one frame of one stream: its launches carry the frame's
 * sizes and positions (and a key-split launch its exchange epoch), so a graph
 * holding it must not be replayed as a later frame. */
skv_status skv_frame_step_noalloc(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count,
                                  const void* q, const void* k, const void* v, void* out);

/* Decoding after (or between) frames reads the detailed state D, not C (the
 * decoding paragraph of the method).  Runs layers [layer_begin, layer_begin +
 * layer_count) for n_tokens new tokens: each attends to every video token of
 * D (T * frames done), every token decoded before, and the new tokens up to
 * itself (causal), with the grouped-query mapping of skv_frame_step; then the
 * new tokens' K/V are appended to D's decode rows.  Split-key ("flash
 * decoding") kernel plus a combine kernel; the whole read of D is the cost.
 * Layers must be stepped in order, and not while a frame is half done; the
 * decode counter advances after the last layer.
 * Device layouts (row-major, dtype of the config):
 *   q   [layer_count][H_q ][n_tokens][d]
 *   k,v [layer_count][H_kv][n_tokens][d]
 *   out [layer_count][H_q ][n_tokens][d]
 * Errors: SKV_ERR_INVALID_ARG, SKV_ERR_ORDER, SKV_ERR_CAPACITY (more than
 * max_decode_tokens decoded tokens), SKV_ERR_UNSUPPORTED (fp32 contexts),
 * SKV_ERR_DEVICE. */
skv_status skv_decode_step(skv_ctx* ctx, int32_t layer_begin, int32_t layer_count, int32_t n_tokens,
                           const void* q, const void* k, const void* v, void* out);

/* Borrowed view of one layer's compressed state C (Eq. 4) and of the last
 * step's candidate pool.  Slots are unordered; pos gives each slot's virtual
 * position.  Pointers stay valid until skv_destroy; contents change with the
 * next skv_frame_step.  The caller may write k, v, pos and score between steps
 * (used to force a given state); the first `size` slots of every KV head are
 * the state.  A selection deferred by a one-layer call (see skv_frame_step) is
 * enqueued on the context's stream first: synchronise that stream before
 * reading or writing through the view.  Errors: SKV_ERR_INVALID_ARG,
 * SKV_ERR_DEVICE (that launch failed). */
typedef struct {
  void* k;                 /* [H_kv][capacity][d] */
  void* v;                 /* [H_kv][capacity][d] */
  int32_t* pos;            /* [H_kv][capacity] virtual positions */
  float* score;            /* [H_kv][capacity] score at the frame that last selected the slot */
  int32_t size;            /* valid slots per KV head = min(B, T * frames done by this layer) */
  int32_t capacity;        /* B */
  int64_t frame;           /* frames this layer has completed */
  const float* pool_score; /* [H_kv][pool_stride] scores of the last step's candidates:
                              state slots 0..size_before-1 first, then frame tokens 0..T-1 */
  const int32_t* pool_pos; /* [H_kv][pool_stride] their virtual positions */
  int32_t pool_size;       /* candidates in the last step (0 before the first) */
  int32_t pool_stride;
} skv_state_view_t;

skv_status skv_state_view(skv_ctx* ctx, int32_t layer, skv_state_view_t* out);

/* Borrowed view of one layer's decode cache D (Eq. 4): video token rows in
 * stream order, then the rows of tokens decoded after the video; row r of KV
 * head g at k + (g * max_tokens + r) * d.  Valid until skv_destroy. */
typedef struct {
  void* k;               /* [H_kv][max_tokens][d] */
  void* v;               /* [H_kv][max_tokens][d] */
  int64_t n_tokens;      /* video rows written = T * frames done by this layer */
  int64_t max_tokens;    /* row stride: T * max_frames + max_decode_tokens */
  int32_t n_kv_heads;
  int32_t head_dim;
  int64_t decode_row0;   /* first decode row = T * max_frames */
  int64_t decode_tokens; /* decode rows written by this layer */
} skv_cache_view_t;

skv_status skv_decode_cache_view(skv_ctx* ctx, int32_t layer, skv_cache_view_t* out);

/* Starts a new video on the same context: frame counter, decoded-token count
 * and L_n return to 0, every state becomes empty, and a context marked by a
 * failed launch is usable again.  Device contents are left as they are
 * (nothing is enqueued; a deferred selection is dropped). */
skv_status skv_reset(skv_ctx* ctx);

/* Sets the frame counter to `frame` (0 <= frame < max_frames) at layer 0, so
 * that a caller can force a state through skv_state_view and run one step
 * from it.  The state size becomes min(B, T * frame); the decoded-token count
 * becomes 0; a context marked by a failed launch is usable again; a deferred
 * selection is dropped. */
skv_status skv_seek(skv_ctx* ctx, int64_t frame);

/* Kernel timing with HIP events on the context's stream.  skv_timing_start
 * creates events for up to max_steps subsequent skv_frame_step or
 * skv_decode_step calls (created here, never in the step).  skv_timing_stop
 * synchronises the stream and writes ms[i * SKV_N_STAGES + s] for step i and
 * stage s, *n_steps the number of steps recorded, then releases the events.
 * Stages of skv_frame_step:
 *   SKV_STAGE_ATTENTION     the attention launch(es): attention and column sums of P
 *                           (with RoPE, the key rotation before them);
 *   SKV_STAGE_REFRESH       the refresh launch: score finalisation, Top-B selection
 *                           and state update, with the decode-cache append running
 *                           in the same launch; with split_refresh, the selection
 *                           launch only (score finalisation, Top-B, admit lists);
 *   SKV_STAGE_STATE_UPDATE  split_refresh only: the admitted rows into their slots;
 *   SKV_STAGE_APPEND        split_refresh only: the frame's K/V into the decode cache.
 * Stages that a step does not run read 0.  Stages of
 * skv_decode_step: SKV_STAGE_ATTENTION (the split-key kernel and its combine) and
 * SKV_STAGE_APPEND (the new tokens' K/V into the decode cache). */
enum {
  SKV_STAGE_ATTENTION = 0,
  SKV_STAGE_REFRESH = 1,
  SKV_STAGE_STATE_UPDATE = 2,
  SKV_STAGE_APPEND = 3,
  SKV_N_STAGES = 4
};
skv_status skv_timing_start(skv_ctx* ctx, int32_t max_steps);
/* After skv_timing_start: record events on every stride-th step only (steps 0,
 * stride, 2 stride, ... of those that follow); the others run without events and
 * do not count towards max_steps.  Each skv_timing_start resets the stride to 1.
 * Event records between launches cost the device time (about 3.5% of a
 * whole-stack 7B frame with three per step), so sampling perturbs less.
 * Errors: SKV_ERR_INVALID_ARG (NULL ctx, stride < 1). */
skv_status skv_timing_stride(skv_ctx* ctx, int32_t stride);
skv_status skv_timing_stop(skv_ctx* ctx, int32_t* n_steps, float* ms, int32_t ms_capacity);

/* Frees every device buffer of the context; NULL is a no-op.  The caller must
 * make sure no enqueued work of the context is still running. */
void skv_destroy(skv_ctx* ctx);

/* Static, NUL-terminated name of a status. */
const char* skv_status_string(skv_status s);

/* Last error detail recorded on the calling thread (static storage). */
const char* skv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* STATEKV_H */
