/*
 * vla_ops.h -- operator-level entry points of the VLA prefix library.
 *
 * The kernels that vla_prefix.h's block calls are built from, exposed one by
 * one on caller-owned DEVICE pointers so each can be checked and timed alone.
 * All are enqueued on `stream` (a hipStream_t as void*, NULL = the null
 * stream) and return after launch; shapes are validated first and a rejected
 * call launches nothing (VLA_ERR_INVALID_ARG / VLA_ERR_UNSUPPORTED).
 * bf16 = bfloat16 bit patterns.  Row-major, innermost index last.
 */
#ifndef VLA_OPS_H
#define VLA_OPS_H

#include "vla_prefix.h"

#ifdef __cplusplus
extern "C" {
#endif

/* C[M][N] (fp32) = A[M][K] (bf16) * W[N][K]^T (bf16): the projection of every
 * block's linear layers (bf16 MFMA, fp32 accumulation).  K % 64 == 0. */
vla_status vla_op_gemm_bf16(const void *A, const void *W, float *C, int M, int N, int K, void *stream);

/* Scaled dot-product attention of the blocks: o[B][L][H*dh] (bf16) =
 * softmax(q k^T / sqrt(dh), causal mask if `causal`) v per (b, head), query
 * head h reading KV head h / (H / Hkv).  q[B][H][L][dh], k[B][Hkv][L][dh],
 * vt[B][Hkv][dh][ldvt] = V transposed with the keys of every group of 16
 * stored in the order [0-3, 8-11, 4-7, 12-15] (column c holds key c with
 * bits 2 and 3 swapped), the order the MFMA consumes them; ldvt >= L rounded
 * up to 16, ldvt % 16 == 0; columns of keys >= L are never used.  All bf16.  dh in {64, 128}. */
vla_status vla_op_attention_bf16(const void *q, const void *k, const void *vt, int ldvt, void *o, int B, int H,
                                 int Hkv, int L, int dh, int causal, void *stream);

/* The fused-epilogue products below take their weights packed slab-major,
 * the layout the resident block weights use: W[N][K] (bf16 rows) cut into
 * slabs of 128 rows x 64 k, each one contiguous block,
 *   element (n, k) at ((k / 64 * nblk + n / 128) * 128 + n % 128) * 64 + k % 64,
 * nblk = N rounded up to a multiple of 256, divided by 128 (pad rows zero).
 * vla_op_packed_weight_elems gives the element count (0 for a shape the
 * products reject: N <= 0, K <= 0, K % 64 != 0);
 * vla_op_pack_weight_bf16 packs HOST row-major W into HOST memory Wp of
 * that many elements (no GPU work). */
size_t vla_op_packed_weight_elems(int N, int K);
vla_status vla_op_pack_weight_bf16(const void *W, void *Wp, int N, int K);

/* H[M][N] (fp32, in place) += A[M][K] (bf16) * W^T + bias[N] (fp32, NULL =
 * none), Wp packed as above: the residual products of the blocks (output
 * projection, down / fc2).  Each lane reads the residual of its accumulators
 * behind the last K slab; bias and residual are added in the accumulators
 * and the sums stored from them.  N % 4 == 0, K % 64 == 0. */
vla_status vla_op_gemm_residual_bf16(const void *A, const void *Wp, float *H, const float *bias, int M, int N, int K,
                                     void *stream);

/* out[M][N] (bf16) = f(A[M][K] * W^T + bias[N]), Wp packed as above, bias
 * fp32 or NULL, f = the exact GELU z * Phi(z) (erfc by Abramowitz & Stegun
 * 7.1.26, |error| <= 1.5e-7) when `gelu`, else the identity: the ViT fc1
 * product and the plain bias product.  N % 8 == 0, K % 64 == 0. */
vla_status vla_op_gemm_bias_bf16(const void *A, const void *Wp, void *out, const float *bias, int M, int N, int K,
                                 int gelu, void *stream);

/* y[M][d] (bf16) = RMSNorm(x[M][d] fp32; gain g[d] fp32, eps) -- or
 * LayerNorm with shift b[d] when b != NULL.  d % 4 == 0, d <= 8192. */
vla_status vla_op_norm_bf16(const float *x, const float *g, const float *b, float eps, void *y, int M, int d,
                            void *stream);

#ifdef __cplusplus
}
#endif
#endif /* VLA_OPS_H */
