/*
 * vla_suffix.h -- host (CPU) side of the block-layer partition and the
 * cross-frame asynchronous pipeline.
 *
 * The partitioned model of the paper's Eq. (6) applies the blocks after the
 * partition point on the CPU to the boundary state the GPU prefix handed over:
 *     F_p(x) = H( B_N( ... B_{p+1}( T(h^(p)) ) ) ).
 * vla_suffix runs B_{k_begin+1..k_end} (0-based blocks [k_begin, k_end)) on
 * the host.  vla_pipeline is the producer-consumer flow of Sec. IV-C: the
 * caller keeps enqueuing GPU prefixes of successive frames while a consumer
 * thread runs the suffix of earlier frames, in frame order and with frame
 * identities preserved, so the steady-state interval approaches
 * max(T_G, T_X + T_C) (Eq. (13)) instead of their sum (Eq. (12)).
 *
 * vla_sched is the boundary-adaptive controller Phi of Sec. IV-D: it picks
 * each frame's partition point inside a dynamic zone of blocks from the
 * runtime state z_t = [u_gpu, u_cpu, q_t] (Eq. (15)-(17)).
 *
 * The action head H is model-specific and not part of this library: the
 * suffix returns the hidden state after block k_end - 1.
 *
 * Same conventions as vla_prefix.h (status codes, row-major tensors, bf16 =
 * IEEE bfloat16 bit patterns).
 */
#ifndef VLA_SUFFIX_H
#define VLA_SUFFIX_H

#include "vla_prefix.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct vla_suffix vla_suffix;
typedef struct vla_pipeline vla_pipeline;

/* Host executor of decoder blocks [k_begin, k_end) of an LLM stack (the cfg's
 * n_blocks, max_tokens and max_batch are not used; dtype must be VLA_BF16 and
 * the stack an LLM stack: RMSNorm, RoPE, causal GQA attention, SwiGLU, no
 * biases).  Arithmetic as on the GPU: bf16 matrix-product operands with fp32
 * accumulation, fp32 residual stream, reductions and softmax.
 * n_threads worker threads (<= 0: one per hardware thread).
 * Needs a CPU with AVX-512 F/BW/VL and BF16 (VLA_ERR_UNSUPPORTED otherwise). */
vla_status vla_suffix_create(const vla_stack_cfg *llm, int k_begin, int k_end, int n_threads, vla_suffix **out);

/* Weights of block `block` in [k_begin, k_end), the same host layout as
 * vla_load_block_weights (bf16).  Copied and re-laid-out; the caller may free
 * them on return. */
vla_status vla_suffix_load_block_weights(vla_suffix *s, int block, const vla_block_weights *w);

/* Run the blocks over h^(k_begin) given in host memory as [B][L][d] bf16 or
 * f32 (in_dtype); positions start at 0.  Writes h^(k_end) as f32 [B][L][d]
 * to out (host).  Synchronous; uses the executor's threads.  Not thread-safe
 * per executor. */
vla_status vla_suffix_run(vla_suffix *s, const void *h, vla_dtype in_dtype, int B, int L, float *out);

/* As vla_suffix_run over blocks [k, k_end) only, k_begin <= k <= k_end, for
 * a frame whose GPU prefix ran blocks [0, k) (a partition point that moved
 * inside the dynamic zone).  k == k_end copies the boundary through. */
vla_status vla_suffix_run_from(vla_suffix *s, int k, const void *h, vla_dtype in_dtype, int B, int L, float *out);

/* Host KV caches for decode steps: capacity L_cap positions for B sequences
 * on each of the executor's blocks (B = 0 or L_cap = 0 frees them).  While
 * set, a vla_suffix_run / _run_from over B sequences of L <= L_cap tokens
 * records the keys (after RoPE) and values of the blocks it runs at
 * positions [0, L). */
vla_status vla_suffix_set_cache(vla_suffix *s, int B, int L_cap);

/* One decode step on the host: blocks [k, k_end) (k_begin <= k <= k_end) for
 * one new token of each of the cache's B sequences at position pos
 * (pos < L_cap), attending over cache rows [0, pos] and appending its own key
 * and value.  h[B][d] is the boundary state of the new tokens (bf16 or f32,
 * for instance the hidden output of vla_decode_step); out[B][d] f32 receives
 * the state after block k_end - 1.  VLA_ERR_SHAPE when B differs from the
 * cache's or pos is outside it. */
vla_status vla_suffix_decode_step(vla_suffix *s, int k, const void *h, vla_dtype in_dtype, int B, int pos,
                                  float *out);

/* Threads the executor uses. */
vla_status vla_suffix_threads(const vla_suffix *s, int *n);

void vla_suffix_destroy(vla_suffix *s);

/* Consumer of the boundaries of prefix context `ctx` (which stays the
 * caller's: the pipeline never calls into it from its thread).  Holds at most
 * `depth` frames between push and pop. */
vla_status vla_pipeline_create(vla_ctx *ctx, vla_suffix *s, int depth, vla_pipeline **out);

/* Hand frame `frame_id` to the consumer right after vla_run_prefix(ctx,
 * frame_id, ..., k, b) was enqueued on the same thread (the pipeline marks the
 * end of that frame's copies on ctx's copy stream).  The consumer waits for
 * the copy, runs suffix blocks [k, k_end) on b->hidden (its out_dtype, B, L as
 * given; k_begin <= k <= k_end) and writes h^(k_end) f32 [B][L][d] to `out`
 * (host).  b->hidden and out must stay valid and untouched until the frame is
 * popped.  Blocks while `depth` frames are pending. */
vla_status vla_pipeline_push(vla_pipeline *p, uint64_t frame_id, const vla_boundary *b, int B, int L, int k,
                             float *out);

/* Frames pushed and not yet popped (the backlog q_t of Eq. (15)). */
vla_status vla_pipeline_backlog(vla_pipeline *p, int *n);

/* Wait for the oldest pushed frame (frames complete in push order), up to
 * timeout_ms (< 0: forever).  Returns its id, the time the consumer waited
 * for its boundary after taking it up (t_wait_ms), and the suffix time T_C
 * (t_cpu_ms).  Any output pointer may be NULL. */
vla_status vla_pipeline_pop(vla_pipeline *p, uint64_t *frame_id, float *t_wait_ms, float *t_cpu_ms, int timeout_ms);

/* Stops the consumer after the frames already pushed; their results are
 * still written. */
void vla_pipeline_destroy(vla_pipeline *p);

typedef struct vla_sched vla_sched;

/* Controller over the dynamic zone [k_lo, k_hi] of an N-block backbone
 * (blocks below k_lo always on the GPU, from k_hi on always on the host),
 * starting at k_init.  Its stage model is linear in the blocks on each side
 * (Eq. (8)-(10)): T_G(k) = a + b k, T_X = x, T_C(k) = c (N - k), from the
 * priors a_ms, b_ms, c_ms, x_ms until frames are observed.  backlog_hi: a
 * consumer queue this long or longer stops moves towards the host. */
vla_status vla_sched_create(int n_blocks, int k_lo, int k_hi, int k_init, float a_ms, float b_ms, float c_ms,
                            float x_ms, int backlog_hi, vla_sched **out);

/* Fold in a finished frame that ran with partition point k: its GPU stage
 * T_G, transfer T_X and host stage T_C (ms; T_C is 0 when k = N).  a and b
 * are refitted by forgetting least squares once two distinct k were seen (a
 * single k only moves a), c is the mean host time per block, x the mean T_X. */
vla_status vla_sched_observe(vla_sched *s, int k, float t_g_ms, float t_x_ms, float t_c_ms);

/* Predicted stage times and stream interval (Eq. (13)) of partition point k
 * when other modules use fractions u_gpu, u_cpu in [0, 1) of the processors:
 * T_G / (1 - u_gpu), T_C / (1 - u_cpu), max(T_G', T_X + T_C').  Any output
 * pointer may be NULL. */
vla_status vla_sched_predict(const vla_sched *s, int k, float u_gpu, float u_cpu, float *t_g_ms, float *t_c_ms,
                             float *t_stream_ms);

/* pi_t = Phi(z_t) (Eq. (17)): the partition point of the next frame, at most
 * one block from the current one and inside the zone, with the shortest
 * predicted interval; ties keep fewer blocks on the GPU.  backlog is q_t (for
 * instance vla_pipeline_backlog).  gpu_budget_ms > 0 caps the predicted GPU
 * stage (reserving the rest of the GPU for other modules): a candidate within
 * the budget beats one outside it, and with none within, the one with the
 * shortest GPU stage is taken.  The decision becomes the current k. */
vla_status vla_sched_decide(vla_sched *s, float u_gpu, float u_cpu, int backlog, float gpu_budget_ms, int *k_out);

/* The current model (any output pointer may be NULL). */
vla_status vla_sched_model(const vla_sched *s, float *a_ms, float *b_ms, float *c_ms, float *x_ms);

void vla_sched_destroy(vla_sched *s);

#ifdef __cplusplus
}
#endif

#endif
