/*
 * vla_prefix.h -- C ABI of the MI355X (gfx950) GPU-resident prefix of
 * block-layer partitioned vision-language-action inference.
 *
 * What it computes (the paper's Sec. IV-B, Eq. (5)): for a partition point k
 * (a count of whole transformer blocks), the boundary hidden state
 *     h^(k) = B_k( ... B_1( E(x) ) )
 * of one frame, together with the KV cache those k decoder blocks wrote, and
 * hands both to pinned host memory: the cross-device transfer T(.) of Eq. (6),
 * whose size for the hidden state is S_hid = B * L * D * b bytes (Eq. (11)).
 * The visual encoder's transformer blocks (the ViT on the GPU, Sec. IV-A) are
 * a second stack run by vla_run_encoder.  Frame identities survive the handoff
 * (Sec. IV-C, producer-consumer pipeline), so a consumer can pair every
 * boundary with its input frame while the GPU already works on the next one.
 *
 * Conventions for every call:
 *  - Every function returns vla_status; nothing throws or aborts across the
 *    ABI.  On failure the context keeps a message (vla_last_error) until the
 *    next call on it succeeds.
 *  - Validation happens before any launch: a rejected call enqueues nothing.
 *  - Tensors are row-major, innermost index last.  bf16 means IEEE bfloat16
 *    bit patterns (uint16_t); f32 means IEEE binary32.
 *  - "host or device" pointers are classified with hipPointerGetAttributes.
 *  - A context belongs to one device and is not thread-safe: serialise calls
 *    on one context externally.
 *  - Streams are hipStream_t values passed as void*.  NULL asks the library
 *    to create its own non-blocking streams (default priority).
 */
#ifndef VLA_PREFIX_H
#define VLA_PREFIX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct vla_ctx vla_ctx;

typedef enum {
  VLA_OK = 0,
  VLA_ERR_INVALID_ARG = -1, /* NULL pointer, bad enum, k_begin > k_end, ... */
  VLA_ERR_SHAPE = -2,       /* sizes exceed the context's limits or a buffer is too small */
  VLA_ERR_NOT_LOADED = -3,  /* a block in the requested range has no weights */
  VLA_ERR_NOT_PINNED = -4,  /* an output host buffer is not page-locked (hipHostMalloc) */
  VLA_ERR_OOM = -5,         /* the caller's device arena is smaller than vla_query_sizes asked */
  VLA_ERR_TIMEOUT = -6,     /* vla_wait_boundary gave up; the work is still in flight */
  VLA_ERR_HIP = -7,         /* a HIP runtime call failed; vla_last_error has its text */
  VLA_ERR_UNSUPPORTED = -8, /* a shape the kernels do not implement (see vla_stack_cfg) */
  VLA_ERR_UNKNOWN_FRAME = -9 /* no in-flight or finished frame has this id */
} vla_status;

typedef enum { VLA_BF16 = 0, VLA_F32 = 1 } vla_dtype;
typedef enum { VLA_STACK_LLM = 0, VLA_STACK_ENC = 1 } vla_stack;

/*
 * Shape of one stack of transformer blocks held on the GPU.
 *  n_blocks   blocks resident on the GPU (the largest partition point the
 *             context can run; GPU memory grows with it, Table V's trade-off).
 *  max_tokens largest tokens per sequence L; max_batch largest batch B
 *             (images for the encoder).  Workspace is sized for B*L rows.
 *  LLM stacks: RMSNorm, RoPE (rotate-half, angles from rope_base), causal
 *             attention with grouped KV heads, SwiGLU MLP, no biases.
 *  Encoder stacks: LayerNorm (with shift), bidirectional attention, GELU
 *             (erf) MLP, biases on every projection.
 *  dtype      VLA_BF16: bf16 weights and activations, fp32 accumulation,
 *             fp32 residual stream and reductions.  VLA_F32: the fp32 debug
 *             path, no reduced precision anywhere.
 * bf16 stacks need head_dim in {64, 128} and d_model, n_heads*head_dim,
 * d_ff multiples of 64; fp32 stacks need head_dim <= 128 and even.
 */
typedef struct {
  int n_blocks, d_model, n_heads, n_kv_heads, head_dim, d_ff;
  int max_tokens, max_batch;
  int norm_is_layernorm, mlp_is_gelu, causal, use_rope, has_bias;
  float norm_eps, rope_base;
  vla_dtype dtype;
} vla_stack_cfg;

/*
 * Host weights of one block, nn.Linear convention W[out][in], element type
 * = the stack's dtype (norm gains/shifts and biases too).  Shapes, with
 * d = d_model, hd = n_heads*head_dim, kvd = n_kv_heads*head_dim, F = d_ff:
 *   w_q[hd][d] w_k[kvd][d] w_v[kvd][d] w_o[d][hd]   norm1_g[d] norm2_g[d]
 *   LLM:     w_gate[F][d] w_up[F][d] w_down[d][F]
 *   encoder: w_fc1[F][d] b_fc1[F] w_fc2[d][F] b_fc2[d] b_qkv[hd+2kvd] b_o[d]
 *            norm1_b[d] norm2_b[d]
 * Fields a stack does not use must be NULL.  The library copies (and
 * re-lays-out) everything into its arena; the caller may free them on return.
 */
typedef struct {
  const void *w_q, *w_k, *w_v, *w_o, *b_qkv, *b_o;
  const void *w_gate, *w_up, *w_down;
  const void *w_fc1, *b_fc1, *w_fc2, *b_fc2;
  const void *norm1_g, *norm1_b, *norm2_g, *norm2_b;
} vla_block_weights;

/*
 * Caller-owned, caller-allocated PINNED host memory receiving one frame's
 * handoff.  hidden: [B][L][d] in out_dtype (either dtype for either stack;
 * f32 from a bf16 stack is the un-rounded fp32 residual).
 * kv: [k_end-k_begin][2][B][n_kv_heads][L][head_dim] in the stack's dtype,
 * K after RoPE, V as projected; may be NULL (kv_bytes 0) to skip the KV copy.
 * frame_id is written by the library.  The buffers must stay untouched until
 * vla_wait_boundary(frame_id) returns VLA_OK.
 */
typedef struct {
  void *hidden;
  size_t hidden_bytes;
  void *kv;
  size_t kv_bytes;
  vla_dtype out_dtype;
  uint64_t frame_id;
} vla_boundary;

/* Device arena bytes a context needs for these stacks (enc may be NULL), and
 * the hidden / KV handoff sizes of a run of k blocks at batch B, length L:
 * hidden_bytes = S_hid = B * L * D * b of Eq. (11) (b the stack dtype's
 * element bytes), kv_bytes = k * 2 * B * n_kv_heads * L * head_dim * b.
 * Negative B, L or k: VLA_ERR_INVALID_ARG; nothing is allocated. */
vla_status vla_query_sizes(const vla_stack_cfg *llm, const vla_stack_cfg *enc, int B, int L, int k,
                           size_t *arena_bytes, size_t *hidden_bytes, size_t *kv_bytes);

/* Create a context on `device` over a caller-owned device arena of
 * arena_bytes (>= vla_query_sizes' answer; the library never calls hipMalloc
 * after this point).  llm may be NULL for an encoder-only context and vice
 * versa.  compute_stream runs the decoder blocks, copy_stream the handoff.
 * encoder_stream runs the encoder blocks; NULL puts them on compute_stream,
 * one frame after the other.  Each stack has its own workspace in the arena,
 * so with a stream of its own the encoder of frame f+1 runs concurrently with
 * the prefix of frame f (the pipelining of Sec. IV-C on one GPU); the
 * library orders the two stacks as vla_run_encoder states. */
vla_status vla_create(const vla_stack_cfg *llm, const vla_stack_cfg *enc, int device, void *dev_arena,
                      size_t arena_bytes, void *compute_stream, void *encoder_stream, void *copy_stream,
                      vla_ctx **out);

/* Copy block `block` (0-based, < n_blocks) of stack `which` from host memory
 * into the arena.  Synchronous.  Re-loading a block replaces it. */
vla_status vla_load_block_weights(vla_ctx *ctx, vla_stack which, int block, const vla_block_weights *w);

/* Encoder: all n_blocks encoder blocks over patches[n_img][L_img][d_enc]
 * (host or device, stack dtype), each image attended independently; result
 * to out_dev[n_img][L_img][d_enc] (device, stack dtype).  Enqueued on the
 * encoder stream; returns after launch.  Ordering with the decoder, also
 * with an encoder stream of its own: a later vla_run_prefix / vla_run_blocks
 * on this context starts only after this run's output is written (so out_dev
 * may be its tokens), and this run writes out_dev only after the latest
 * earlier prefix has read its input (so one buffer may carry every frame).
 * Other readers of out_dev order themselves after the encoder stream. */
vla_status vla_run_encoder(vla_ctx *ctx, uint64_t frame_id, const void *patches, int n_img, int L_img,
                           void *out_dev);

/*
 * Front and back of the visual encoder: E(x_t) of Eq. (5) from the frame's
 * camera images (Eq. (1)), the part of the GPU stage that Sec. IV-A puts
 * before the backbone.  The paper does not describe either end; this library
 * computes the common ViT patch embedding and a LLaVA-style projector:
 *   images [n_img][channels][img_h][img_w] (stack dtype; normalised pixels)
 *   -> per image, patch x patch squares in row-major grid order (gh x gw,
 *      gh = img_h / patch, gw = img_w / patch), each flattened channel first,
 *      then pixel row, then pixel column, times w_patch^T, + b_patch
 *      + pos[grid index]                  (a stride-patch convolution)
 *   -> every block of the encoder stack (each image attended on its own)
 *   -> LayerNorm(post_g, post_b)
 *   -> merge of merge x merge neighbouring patches into one token: token
 *      (ty, tx) of an image, row-major over (gh/merge) x (gw/merge), holds the
 *      features of patches (ty*merge + dy, tx*merge + dx), dy outer, dx
 *      inner, side by side (merge*merge*d_enc wide)
 *   -> GELU(m w_c1^T + b_c1) w_c2^T + b_c2  = the visual tokens, d_out wide.
 * Needs: img_h, img_w multiples of patch; gh, gw multiples of merge;
 * gh * gw <= the encoder's max_tokens; bf16: d_hidden, d_out multiples of 64;
 * fp32: d_out a multiple of 4.
 */
typedef struct {
  int channels, img_h, img_w, patch, merge;
  int d_hidden; /* connector MLP width */
  int d_out;    /* token width (the decoder's d_model) */
  float norm_eps;
} vla_vision_cfg;

/* Host weights of the vision front, the encoder stack's dtype, all required:
 * w_patch[d_enc][channels*patch*patch] b_patch[d_enc] pos[gh*gw][d_enc]
 * post_g[d_enc] post_b[d_enc] w_c1[d_hidden][merge*merge*d_enc] b_c1[d_hidden]
 * w_c2[d_out][d_hidden] b_c2[d_out].  Copied (and re-laid-out) on load. */
typedef struct {
  const void *w_patch, *b_patch, *pos, *post_g, *post_b, *w_c1, *b_c1, *w_c2, *b_c2;
} vla_vision_weights;

/* Device bytes vla_attach_vision needs for this encoder stack and vision
 * front: weights plus scratch for max_batch images. */
vla_status vla_query_vision_sizes(const vla_stack_cfg *enc, const vla_vision_cfg *vis, size_t *bytes);

/* Give a context with an encoder stack a vision front, in caller-owned device
 * memory dev_mem of `bytes` (>= vla_query_vision_sizes, 256-byte aligned;
 * the library allocates nothing).  Waits for the context's work in flight;
 * attaching again replaces the previous front (its weights must be loaded
 * again).  The memory must outlive the context or the next attach. */
vla_status vla_attach_vision(vla_ctx *ctx, const vla_vision_cfg *vis, void *dev_mem, size_t bytes);

/* Copy the vision front's weights from host memory.  Synchronous. */
vla_status vla_load_vision_weights(vla_ctx *ctx, const vla_vision_weights *w);

/* One frame's backbone input, E(x_t): images[n_img][channels][img_h][img_w]
 * (host or device, n_img <= the encoder's max_batch) through the stem, the
 * encoder blocks and the connector into tokens_dev rows [0, V), V = n_img *
 * (gh/merge) * (gw/merge), camera by camera; then text[L_text][d_out] (host
 * or device, may be NULL when L_text = 0) into rows [V, V + L_text).
 * tokens_dev: device memory, 16-byte aligned, tokens_bytes >= (V + L_text) *
 * d_out * element size, in the encoder stack's dtype -- with a decoder stack
 * of the same dtype and d_model = d_out it is vla_run_prefix's input as it
 * is (B = 1, L = V + L_text).  Runs on the encoder stream and orders itself
 * with the decoder as vla_run_encoder does.  Enqueued; returns after launch. */
vla_status vla_run_vision(vla_ctx *ctx, uint64_t frame_id, const void *images, int n_img, const void *text,
                          int L_text, void *tokens_dev, size_t tokens_bytes);

/* Prefix: decoder blocks [0, k) over tokens[B][L][d] (host or device, stack
 * dtype) as one causal prefill; the boundary h^(k) and the KV cache of the k
 * blocks are copied to `out` on the copy stream, each layer's KV as soon as
 * that layer has written it.  k = 0 hands back the input (Eq. (5) with no
 * blocks).  Enqueued; returns after launch.  Equivalent to
 * vla_run_blocks(ctx, frame_id, tokens, <stack dtype>, B, L, 0, k, out). */
vla_status vla_run_prefix(vla_ctx *ctx, uint64_t frame_id, const void *tokens, int B, int L, int k,
                          vla_boundary *out);

/* Decoder blocks [k_begin, k_end) over an intermediate state h^(k_begin)
 * given as `tokens` in element type in_dtype (positions still start at 0):
 * one stage of the block pipeline of Eq. (6).  An f32 input continues the
 * fp32 residual stream exactly, so chaining f32 boundaries of adjacent
 * ranges reproduces one run over their union bit for bit.  KV in `out` covers
 * the blocks run. */
vla_status vla_run_blocks(vla_ctx *ctx, uint64_t frame_id, const void *tokens, vla_dtype in_dtype, int B, int L,
                          int k_begin, int k_end, vla_boundary *out);

/* One decode step across the boundary: decoder blocks [0, k) for one new
 * token of each of B <= 4 sequences (bf16 stacks).  x[B][d] (host or device,
 * bf16) are the tokens' inputs at position pos; each sequence attends over
 * its cached keys and values [0, pos) plus its own, and appends its key
 * (after RoPE) and value at pos.
 * kv_cache: caller-owned DEVICE memory [k][2][B][n_kv_heads][L_cap][head_dim]
 * bf16 (the layout of vla_boundary's kv with sequence stride L_cap instead of
 * L), rows [0, pos) filled (for instance with a prefix's KV handoff copied
 * in).  Needs pos < L_cap and, with RoPE, pos < max_tokens.
 * out->hidden receives h^(k) of the new tokens [B][d] in out_dtype; out->kv
 * must be NULL.  Frame ids, vla_wait_boundary and vla_frame_times work as for
 * vla_run_prefix.  Enqueued; returns after launch.  VLA_ERR_SHAPE when the
 * context's workspace (sized by max_tokens) cannot hold the step's scratch. */
vla_status vla_decode_step(vla_ctx *ctx, uint64_t frame_id, const void *x, int B, int pos, int k, void *kv_cache,
                           int L_cap, vla_boundary *out);

/* vla_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same arguments, result and errors, but every scratch buffer of the step
 * (residual, QKV rows, split-key attention partials, gate/up rows, attention
 * output, gated activation, input and boundary staging) lies in a fixed
 * device array of 4 MiB that the library holds on each GPU it runs on until
 * the process ends, instead of the context's workspace; the call allocates
 * nothing.  Larger steps fail with VLA_ERR_SHAPE before any launch (the
 * 7B-shaped stack fits up to position ~6400 at B = 4, ~30000 at B = 1;
 * ~6270 and ~30460 with split operands, whose gated activation carries its
 * remainder rows too).
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents (nothing in it needs to start at zero): calls from different
 * contexts or streams that overlap on one GPU race.  Within one context a
 * step waits for the context's earlier copies before it writes the array. */
vla_status vla_decode_step_static(vla_ctx *ctx, uint64_t frame_id, const void *x, int B, int pos, int k,
                                  void *kv_cache, int L_cap, vla_boundary *out);

/* The consumer side of the producer-consumer handoff (Sec. IV-C): block the
 * host until frame_id's handoff is complete (its host buffers are then
 * readable), or timeout_ms elapses (< 0: wait forever).  VLA_ERR_TIMEOUT
 * leaves the frame in flight, so a later wait can still collect it;
 * VLA_ERR_UNKNOWN_FRAME for an id neither in flight nor among the last 256
 * finished frames. */
vla_status vla_wait_boundary(vla_ctx *ctx, uint64_t frame_id, int timeout_ms);

/* Stage times of a completed frame (Eq. (8)-(9)): t_gpu_ms from the start of
 * the frame's prefix to its last block on the compute stream (T_G); t_xfer_ms
 * of the boundary hidden-state copy alone (T_X); t_total_ms from the prefix
 * start until every copy of the frame, KV included, finished.  Any output
 * pointer may be NULL. */
vla_status vla_frame_times(vla_ctx *ctx, uint64_t frame_id, float *t_gpu_ms, float *t_xfer_ms,
                           float *t_total_ms);

/* Kernel classes timed by the profiler, per stack. */
typedef enum {
  VLA_K_NORM = 0,     /* RMSNorm / LayerNorm (both per block) */
  VLA_K_QKV = 1,      /* QKV projection + RoPE + cache write */
  VLA_K_ATTN = 2,     /* attention */
  VLA_K_OPROJ = 3,    /* output projection + residual */
  VLA_K_MLP_UP = 4,   /* gate/up + SwiGLU, or fc1 + GELU */
  VLA_K_MLP_DOWN = 5, /* down / fc2 + residual */
  VLA_K_OTHER = 6,    /* intake, boundary cast (fp32 path: its extra kernels) */
  VLA_K_STEM = 7,     /* vision front: patch rows + patch embedding GEMM */
  VLA_K_CONNECTOR = 8, /* vision back: final norm + merge, connector MLP */
  VLA_K_COUNT = 9
} vla_kernel_class;

/* Start (enable != 0, clearing previous totals) or stop timing every kernel
 * launch with a pair of HIP events on the stream it runs on.  Launches of
 * the two stacks that overlap in time are each timed over the overlap. */
vla_status vla_profile(vla_ctx *ctx, int enable);
/* Totals since vla_profile(ctx, 1) for one stack and class: summed kernel
 * time in ms and launch count.  Synchronises the compute and encoder streams. */
vla_status vla_profile_read(vla_ctx *ctx, vla_stack which, vla_kernel_class cls, double *ms_total, int *launches);

/*
 * Precision of the activation operands of a bf16 decoder stack's QKV,
 * gate/up and down products.  Sec. IV-B rests the partitioned model's
 * fidelity on computing the same blocks (Eq. (5)-(6)); with bf16 operands
 * every product input is rounded to 8 significant bits, and with random-init
 * d=4096 blocks that rounding alone moves the boundary h^(k) away from an
 * fp32 computation by more than 1e-2 (relative L2) beyond about 8 blocks.
 *  VLA_PREC_BF16   (default) each operand is one bf16 value.
 *  VLA_PREC_SPLIT  the RMSNorm outputs and the gated activation are carried
 *                  as hi = bf16(v) and lo = bf16(v - hi), and each product
 *                  is hi W^T + lo W^T accumulated in fp32: a 16-bit
 *                  significand in place of 8, for twice the MFMA work of
 *                  those three products.  Weights, the attention path, the
 *                  KV cache and the boundary are unchanged.
 * Applies to prefix and block runs (vla_run_prefix, vla_run_blocks) and to
 * decode steps (vla_decode_step and its static variant) enqueued after the
 * call; a decode step stages each sequence's hi and lo rows side by side and
 * streams the weights once, so its cost stays that of the weight stream.
 * VLA_ERR_UNSUPPORTED for encoder stacks and fp32 stacks (the fp32 debug
 * path has no reduced precision).
 */
typedef enum { VLA_PREC_BF16 = 0, VLA_PREC_SPLIT = 1 } vla_precision;
vla_status vla_set_precision(vla_ctx *ctx, vla_stack which, vla_precision prec);

/* Fault injection for the error paths (tests and harnesses): after
 * `launches` further kernel launches have been enqueued, the next launch is
 * not made and its call fails with VLA_ERR_HIP as a failing launch would;
 * launches < 0 switches it off.  The failure takes the frame's work as far
 * as it was enqueued, waits for it, and forgets the frame id: every kernel
 * still runs to completion and later frames run normally. */
vla_status vla_inject_fault(vla_ctx *ctx, long launches);

/* Bytes of the arena in use after the loads so far (weights + workspace). */
vla_status vla_arena_used(const vla_ctx *ctx, size_t *bytes);

const char *vla_status_string(vla_status s);
/* Message of the last failure on ctx (ctx NULL: of the last failed
 * vla_create / vla_query_sizes on this thread). */
const char *vla_last_error(const vla_ctx *ctx);
/* Wait for all enqueued work, then release the context (not the arena or
 * caller streams). */
void vla_destroy(vla_ctx *ctx);

#ifdef __cplusplus
}
#endif
#endif /* VLA_PREFIX_H */
