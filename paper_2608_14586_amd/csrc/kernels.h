// Host-side launch wrappers of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace vla {

// ---------------------------------------------------------------- bf16 GEMMs
// Every GEMM computes acc[M][N] = A[M][K] * W[N][K]^T (bf16 in, fp32
// accumulate) and hands acc to an epilogue.  K % 64 == 0, lda % 8 == 0.
//
// Resident weights are packed slab-major: the GEMM moves W in slabs of
// SLAB_N rows x 64 k, and each slab is one contiguous 16 KB block, the blocks
// of one k range side by side:
//   element (n, k) at ((k / 64 * nblk + n / SLAB_N) * SLAB_N + n % SLAB_N) * 64 + k % 64
// nblk = slab_blocks(N) (N rounded up to whole pairs of blocks, pad rows
// zero).  At any moment the whole chip then streams one contiguous stretch of
// the weights, rather than 128-byte pieces of rows 2*K bytes apart.
constexpr int SLAB_N = 128;
inline int slab_blocks(int N) { return (N + 2 * SLAB_N - 1) / (2 * SLAB_N) * 2; }
// Host-side packing of row-major bf16 rows W[N][K] into that layout
// (dst: slab_blocks(N) * SLAB_N * K elements, pad rows zero).  K % 64 == 0.
inline void pack_slabs(const uint16_t* W, uint16_t* dst, int N, int K) {
  const int nblk = slab_blocks(N);
  for (size_t i = 0; i < (size_t)nblk * SLAB_N * K; ++i) dst[i] = 0;
  for (int kt = 0; kt < K / 64; ++kt)
    for (int n = 0; n < N; ++n)
      for (int j = 0; j < 64; ++j)
        dst[(((size_t)kt * nblk + n / SLAB_N) * SLAB_N + n % SLAB_N) * 64 + j] = W[(size_t)n * K + (size_t)kt * 64 + j];
}

// A weight operand: packed (nblk > 0, ld unused) or row-major with leading
// dimension ld (nblk == 0).
struct WOperand {
  const bf16_t* p;
  int ld;
  int nblk;
};

// C (fp32) = acc, W row-major [N][ldw] (ldw % 8 == 0)
hipError_t gemm_bf16_store_f32(const bf16_t* A, int lda, const bf16_t* W, int ldw, float* C, int ldc, int M,
                               int N, int K, hipStream_t s);
// The block GEMMs below take packed weights.  a_parts = 2 (split operand):
// A is [M][2K], a hi + lo pair of bf16 values per element side by side
// (columns [0, K) hi, [K, 2K) lo), and acc = hi * W^T + lo * W^T, twice the
// MFMA work of a plain bf16 operand and a 16-bit significand in its place.
// H (fp32 residual) += acc + bias (bias may be NULL)
hipError_t gemm_bf16_residual(const bf16_t* A, int lda, const WOperand& W, float* H, int ldh, const float* bias,
                              int M, int N, int K, hipStream_t s, int a_parts = 1);
// out (bf16) [M][N/2] = silu(gate) * up, W rows interleaved in groups of 32
// (32 gate rows, then the 32 up rows of the same features); N % 64 == 0.
// lo_col > 0: the remainder bf16(y - bf16(y)) of each output also goes to
// column lo_col + c of its row (lo_col >= N/2, ldo >= lo_col + N/2).
hipError_t gemm_bf16_swiglu(const bf16_t* A, int lda, const WOperand& W, bf16_t* out, int ldo, int M, int N, int K,
                            hipStream_t s, int a_parts = 1, int lo_col = 0);
// out (bf16) = gelu_erf(acc + bias)
hipError_t gemm_bf16_gelu(const bf16_t* A, int lda, const WOperand& W, bf16_t* out, int ldo, const float* bias,
                          int M, int N, int K, hipStream_t s);

// Fused QKV projection epilogue.  Packed weight rows: [q heads | k heads |
// v heads], each head's head_dim rows in 64-row groups that hold 32 rows of
// the first rotary half followed by their 32 partner rows of the second half
// (dims c*32..c*32+31 then dh/2+c*32..), so a wave owns every rotary pair.
struct QkvArgs {
  const float* bias;    // packed order, NULL if none
  const float* rope_cos;  // [max_tokens][dh/2], NULL: no rotary embedding
  const float* rope_sin;
  bf16_t* q;   // [B][H][L][dh]
  bf16_t* k;   // [B][Hkv][L][dh]
  bf16_t* v;   // [B][Hkv][L][dh], NULL: V rows not written (V^T still is)
  bf16_t* vt;  // [B][Hkv][dh][ldvt] (V transposed, keys of each 16-group in the order
               // [0-3, 8-11, 4-7, 12-15], for the attention's PV product)
  int ldvt;
  int L, H, Hkv, dh;
};
hipError_t gemm_bf16_qkv(const bf16_t* A, int lda, const WOperand& W, const QkvArgs& qa, int M, int N, int K,
                         hipStream_t s, int a_parts = 1);

// out (bf16) = acc + bias (bias may be NULL); N % 8 == 0, ldo % 8 == 0
hipError_t gemm_bf16_bias(const bf16_t* A, int lda, const WOperand& W, bf16_t* out, int ldo, const float* bias,
                          int M, int N, int K, hipStream_t s);

// ---------------------------------------------------------- vision stem
// Patch rows of n_img images [C][H][W] cut into p x p patches (row-major
// grid, gw = W / p across): A[i * L + l][k] for k < C*p*p is pixel
// (c, y, x) = (k / (p*p), k / p % p, k % p) of patch l, zero up to Kp;
// h[i * L + l][:] = pos[l][:] (fp32), the residual the stem GEMM adds to.
hipError_t patchify_bf16(const bf16_t* img, int n_img, int C, int H, int W, int p, bf16_t* A, int Kp,
                         const float* pos, float* h, int d, hipStream_t s);
hipError_t patchify_f32(const float* img, int n_img, int C, int H, int W, int p, float* A, int Kp, const float* pos,
                        float* h, int d, hipStream_t s);

// ---------------------------------------------------------- bf16 attention
// o[B][L][H*dh] = softmax(q k^T / sqrt(dh) [+ causal mask]) v per (b, head);
// query head h reads KV head h / (H / Hkv).  q [B][H][L][dh], k [B][Hkv][L][dh],
// vt [B][Hkv][dh][ldvt] in the key order of QkvArgs::vt, ldvt % 16 == 0.
// dh in {64, 128}.
hipError_t attention_bf16(const bf16_t* q, const bf16_t* k, const bf16_t* vt, int ldvt, bf16_t* o, int B, int H,
                          int Hkv, int L, int dh, bool causal, hipStream_t s);

// ------------------------------------------------------------ bf16 decode step
// One new token for each of B <= 4 sequences (decode_bf16.hip).  W operands
// are the packed resident weights; fp32 rows [B][...] throughout.  parts = 2
// carries the normalised rows (QKV, gate/up) and the gated activation (down)
// as split operands, hi = bf16(v) and lo = bf16(v - hi), whose products sum
// in fp32, as the prefill does under VLA_PREC_SPLIT.
// QKV (and gate/up): raw[b][n] = (RMSNorm(h[b]) g) . W[n], packed row order.
hipError_t decode_qkv(const float* h, const float* g, float eps, const WOperand& W, float* raw, int B, int N, int K,
                      hipStream_t s, int parts = 1);
// Attention of the token at position pos over cache rows [0, pos] of
// kc/vc [B][Hkv][L_cap][dh]: RoPE on q and the new key, the new key and value
// appended at pos, o[B][H*dh] (bf16).  Scratch: split-key partials, fp32,
// decode_attention_scratch(B, H, dh, pos) bytes.
size_t decode_attention_scratch(int B, int H, int dh, int pos);
hipError_t decode_attention(const float* qkv, int qkv_n, const float* rope_cos, const float* rope_sin, bf16_t* kc,
                            bf16_t* vc, int L_cap, int pos, int B, int H, int Hkv, int dh, float* part, bf16_t* o,
                            hipStream_t s);
// h[b] += o[b] . W^T (the O projection, o [B][K] bf16)
hipError_t decode_oproj(const bf16_t* o, int K, const WOperand& W, float* h, int B, int N, hipStream_t s);
// a[b] = bf16(swiglu(RMSNorm(h[b]) g . W^T)) over the interleaved gate/up
// rows (N = 2 fpad), the gated activation [B][parts * fpad] (parts = 2: its
// remainder in columns [fpad, 2 fpad)); gu [B][2 fpad] fp32 is scratch for
// inputs too wide to stage whole.
hipError_t decode_up(const float* h, const float* g, float eps, const WOperand& W, int fpad, float* gu, bf16_t* a,
                     int B, int K, hipStream_t s, int parts = 1);
// h[b] += a[b] . W^T (the down projection over the padded width fpad; a as
// decode_up writes it)
hipError_t decode_down(const bf16_t* a, int fpad, const WOperand& W, float* h, int B, int N, hipStream_t s,
                       int parts = 1);

// Fixed device scratch of the decode step that allocates nothing
// (static_scratch.hip): its size, and its address on `device` (resolved once
// per device; `device` must be the current device the first time).
size_t static_scratch_bytes();
hipError_t static_scratch_resolve(int device, void** out);

// ----------------------------------------------------- norms and elementwise
// y[M][d] = norm(x[M][d]) (fp32 in); RMSNorm when beta == NULL and !layernorm.
hipError_t rmsnorm_bf16(const float* x, const float* g, float eps, bf16_t* y, int M, int d, hipStream_t s);
// RMSNorm as a split operand: y[M][2d], columns [0, d) bf16(v), [d, 2d) the
// remainder bf16(v - bf16(v)) of the fp32 result v.
hipError_t rmsnorm_bf16_split(const float* x, const float* g, float eps, bf16_t* y, int M, int d, hipStream_t s);
hipError_t layernorm_bf16(const float* x, const float* g, const float* b, float eps, bf16_t* y, int M, int d,
                          hipStream_t s);
hipError_t rmsnorm_f32(const float* x, const float* g, float eps, float* y, int M, int d, hipStream_t s);
hipError_t layernorm_f32(const float* x, const float* g, const float* b, float eps, float* y, int M, int d,
                         hipStream_t s);
// LayerNorm of encoder rows, n_img images x gh*gw patches in row-major grid
// order, each written into the connector's merged layout: patch (gy, gx) of
// image i becomes feature block (gy % m) * m + gx % m (d wide) of token
// i * (gh/m) * (gw/m) + (gy/m) * (gw/m) + gx/m (m*m*d wide).
hipError_t layernorm_merge_bf16(const float* x, const float* g, const float* b, float eps, bf16_t* y, int n_img,
                                int gh, int gw, int m, int d, hipStream_t s);
hipError_t layernorm_merge_f32(const float* x, const float* g, const float* b, float eps, float* y, int n_img,
                               int gh, int gw, int m, int d, hipStream_t s);
hipError_t bf16_to_f32(const bf16_t* x, float* y, size_t n, hipStream_t s);
hipError_t f32_to_bf16(const float* x, bf16_t* y, size_t n, hipStream_t s);

// ------------------------------------------------------------- fp32 debug path
// C[M][N] (op) A[M][K] * W[N][K]^T in fp32 FMA; mode 0: C = acc + bias,
// mode 1: C += acc + bias.
hipError_t gemm_f32(const float* A, int lda, const float* W, int ldw, float* C, int ldc, const float* bias,
                    int mode, int M, int N, int K, hipStream_t s);
// qkv[M][(H+2Hkv)*dh] natural order -> q/k/v/vt (fp32) with rotary on q, k.
hipError_t qkv_split_f32(const float* qkv, const float* rope_cos, const float* rope_sin, float* q, float* k,
                         float* v, float* vt, int ldvt, int B, int L, int H, int Hkv, int dh, hipStream_t s);
hipError_t attention_f32(const float* q, const float* k, const float* v, float* o, int B, int H, int Hkv, int L,
                         int dh, bool causal, hipStream_t s);
// gu[M][2F] (gate | up) -> a[M][F] = silu(gate) * up
hipError_t swiglu_f32(const float* gu, float* a, int M, int F, hipStream_t s);
// x[M][F] = gelu(x)
hipError_t gelu_f32(float* x, size_t n, hipStream_t s);

}  // namespace vla
