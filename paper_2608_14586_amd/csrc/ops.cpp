// Operator-level entry points (include/vla_ops.h).
#include <hip/hip_runtime.h>

#include "../../include/vla_ops.h"
#include "kernels.h"

namespace {
vla_status status_of(hipError_t e) {
  if (e == hipSuccess) return VLA_OK;
  return e == hipErrorInvalidValue ? VLA_ERR_UNSUPPORTED : VLA_ERR_HIP;
}
}  // namespace

extern "C" {

vla_status vla_op_gemm_bf16(const void* A, const void* W, float* C, int M, int N, int K, void* stream) {
  if (!A || !W || !C || M < 0 || N < 0 || K <= 0) return VLA_ERR_INVALID_ARG;
  if (K % 64) return VLA_ERR_UNSUPPORTED;
  return status_of(vla::gemm_bf16_store_f32((const bf16_t*)A, K, (const bf16_t*)W, K, C, N, M, N, K,
                                            (hipStream_t)stream));
}

size_t vla_op_packed_weight_elems(int N, int K) {
  if (N <= 0 || K <= 0 || K % 64) return 0;
  return (size_t)vla::slab_blocks(N) * vla::SLAB_N * K;
}

vla_status vla_op_pack_weight_bf16(const void* W, void* Wp, int N, int K) {
  if (!W || !Wp || N <= 0 || K <= 0) return VLA_ERR_INVALID_ARG;
  if (K % 64) return VLA_ERR_UNSUPPORTED;
  vla::pack_slabs((const uint16_t*)W, (uint16_t*)Wp, N, K);
  return VLA_OK;
}

vla_status vla_op_gemm_residual_bf16(const void* A, const void* Wp, float* H, const float* bias, int M, int N, int K,
                                     void* stream) {
  if (!A || !Wp || !H || M < 0 || N <= 0 || K <= 0) return VLA_ERR_INVALID_ARG;
  if (K % 64 || N % 4) return VLA_ERR_UNSUPPORTED;
  const vla::WOperand w{(const bf16_t*)Wp, 0, vla::slab_blocks(N)};
  return status_of(vla::gemm_bf16_residual((const bf16_t*)A, K, w, H, N, bias, M, N, K, (hipStream_t)stream));
}

vla_status vla_op_gemm_bias_bf16(const void* A, const void* Wp, void* out, const float* bias, int M, int N, int K,
                                 int gelu, void* stream) {
  if (!A || !Wp || !out || M < 0 || N <= 0 || K <= 0) return VLA_ERR_INVALID_ARG;
  if (K % 64 || N % 8) return VLA_ERR_UNSUPPORTED;
  const vla::WOperand w{(const bf16_t*)Wp, 0, vla::slab_blocks(N)};
  hipError_t e = gelu ? vla::gemm_bf16_gelu((const bf16_t*)A, K, w, (bf16_t*)out, N, bias, M, N, K, (hipStream_t)stream)
                      : vla::gemm_bf16_bias((const bf16_t*)A, K, w, (bf16_t*)out, N, bias, M, N, K, (hipStream_t)stream);
  return status_of(e);
}

vla_status vla_op_attention_bf16(const void* q, const void* k, const void* vt, int ldvt, void* o, int B, int H,
                                 int Hkv, int L, int dh, int causal, void* stream) {
  if (!q || !k || !vt || !o || B < 0 || H <= 0 || Hkv <= 0 || L < 0) return VLA_ERR_INVALID_ARG;
  if (H % Hkv || (dh != 64 && dh != 128) || ldvt < (L + 15) / 16 * 16 || ldvt % 16) return VLA_ERR_UNSUPPORTED;
  return status_of(vla::attention_bf16((const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)vt, ldvt, (bf16_t*)o, B, H,
                                       Hkv, L, dh, causal != 0, (hipStream_t)stream));
}

vla_status vla_op_norm_bf16(const float* x, const float* g, const float* b, float eps, void* y, int M, int d,
                            void* stream) {
  if (!x || !g || !y || M < 0 || d <= 0) return VLA_ERR_INVALID_ARG;
  if (d % 4 || d > 8192) return VLA_ERR_UNSUPPORTED;
  hipError_t e = b ? vla::layernorm_bf16(x, g, b, eps, (bf16_t*)y, M, d, (hipStream_t)stream)
                   : vla::rmsnorm_bf16(x, g, eps, (bf16_t*)y, M, d, (hipStream_t)stream);
  return status_of(e);
}

}  // extern "C"
