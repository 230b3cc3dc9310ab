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

/* Threads the executor uses. */
vla_status vla_suffix_threads(const vla_suffix *s, int *n);

void vla_suffix_destroy(vla_suffix *s);

/* Consumer of the boundaries of prefix context `ctx` (which stays the
 * caller's: the pipeline never calls into it from its thread).  Holds at most
 * `depth` frames between push and pop. */
vla_status vla_pipeline_create(vla_ctx *ctx, vla_suffix *s, int depth, vla_pipeline **out);

/* Hand frame `frame_id` to the consumer right after vla_run_prefix(ctx,
 * frame_id, ..., b) was enqueued on the same thread (the pipeline marks the
 * end of that frame's copies on ctx's copy stream).  The consumer waits for
 * the copy, runs the suffix on b->hidden (its out_dtype, B, L as given) and
 * writes h^(k_end) f32 [B][L][d] to `out` (host).  b->hidden and out must
 * stay valid and untouched until the frame is popped.  Blocks while `depth`
 * frames are pending. */
vla_status vla_pipeline_push(vla_pipeline *p, uint64_t frame_id, const vla_boundary *b, int B, int L, float *out);

/* Wait for the oldest pushed frame (frames complete in push order), up to
 * timeout_ms (< 0: forever).  Returns its id, the time the consumer waited
 * for its boundary after taking it up (t_wait_ms), and the suffix time T_C
 * (t_cpu_ms).  Any output pointer may be NULL. */
vla_status vla_pipeline_pop(vla_pipeline *p, uint64_t *frame_id, float *t_wait_ms, float *t_cpu_ms, int timeout_ms);

/* Stops the consumer after the frames already pushed; their results are
 * still written. */
void vla_pipeline_destroy(vla_pipeline *p);

#ifdef __cplusplus
}
#endif

#endif
