// fp32 debug path: the same blocks with no reduced precision anywhere.  Plain
// VALU kernels; they exist to check the composition (rotary layout, cache
// layout, grouped heads, residual order) at a 1e-4 bar, not for speed.

#include <math.h>

#include "kernels.h"

namespace vla {
namespace {

// C = A * W^T (+ bias), or C += ..., 64x64 tile, 16-deep k slabs, 4x4 per thread.
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int lda,
                                                       const float* __restrict__ W, int ldw, float* __restrict__ C,
                                                       int ldc, const float* __restrict__ bias, int mode, int M,
                                                       int N, int K) {
  __shared__ float sA[16][64 + 4];
  __shared__ float sB[16][64 + 4];
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int e = tid; e < 64 * 16; e += 256) {
      int r = e / 16, kk = e % 16;
      int gm = m0 + r, gn = n0 + r, gk = k0 + kk;
      sA[kk][r] = (gm < M && gk < K) ? A[(size_t)gm * lda + gk] : 0.f;
      sB[kk][r] = (gn < N && gk < K) ? W[(size_t)gn * ldw + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int row = m0 + ty * 4 + i;
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int col = n0 + tx * 4 + j;
      if (col >= N) continue;
      float v = acc[i][j] + (bias ? bias[col] : 0.f);
      float* p = C + (size_t)row * ldc + col;
      *p = mode == 1 ? *p + v : v;
    }
  }
}

// one thread per (row, head-column pair) of the natural-order qkv matrix
__global__ void qkv_split_f32_kernel(const float* __restrict__ qkv, const float* __restrict__ rc,
                                     const float* __restrict__ rs, float* q, float* k, float* v, float* vt, int ldvt,
                                     int B, int L, int H, int Hkv, int dh) {
  const int half = dh / 2;
  const int npairs = (H + 2 * Hkv) * half;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)B * L * npairs) return;
  const int pr = (int)(idx % npairs);
  const int row = (int)(idx / npairs);
  const int b = row / L, pos = row % L;
  const int head_all = pr / half, i = pr % half;
  const int ncol = (H + 2 * Hkv) * dh;
  const float* src = qkv + (size_t)row * ncol + head_all * dh;
  float x1 = src[i], x2 = src[i + half];
  if (head_all < H + Hkv && rc != nullptr) {
    float c = rc[(size_t)pos * half + i], s = rs[(size_t)pos * half + i];
    float y1 = x1 * c - x2 * s, y2 = x2 * c + x1 * s;
    x1 = y1;
    x2 = y2;
  }
  if (head_all < H) {
    float* d = q + (((size_t)b * H + head_all) * L + pos) * dh;
    d[i] = x1;
    d[i + half] = x2;
  } else if (head_all < H + Hkv) {
    int hh = head_all - H;
    float* d = k + (((size_t)b * Hkv + hh) * L + pos) * dh;
    d[i] = x1;
    d[i + half] = x2;
  } else {
    int hh = head_all - H - Hkv;
    float* d = v + (((size_t)b * Hkv + hh) * L + pos) * dh;
    d[i] = x1;
    d[i + half] = x2;
    if (vt) {
      vt[(((size_t)b * Hkv + hh) * dh + i) * ldvt + pos] = x1;
      vt[(((size_t)b * Hkv + hh) * dh + i + half) * ldvt + pos] = x2;
    }
  }
}

// one thread per query; keys streamed through the cache, online softmax
template <int DHMAX>
__global__ __launch_bounds__(64) void attention_f32_kernel(const float* __restrict__ q, const float* __restrict__ k,
                                                           const float* __restrict__ v, float* __restrict__ o,
                                                           int B, int H, int Hkv, int L, int dh, int causal,
                                                           float scale) {
  const int qi = blockIdx.x * 64 + threadIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  if (qi >= L) return;
  const int hk = h / (H / Hkv);
  const float* qr = q + (((size_t)b * H + h) * L + qi) * dh;
  const float* kh = k + ((size_t)b * Hkv + hk) * (size_t)L * dh;
  const float* vh = v + ((size_t)b * Hkv + hk) * (size_t)L * dh;
  float qv[DHMAX], acc[DHMAX];
#pragma unroll
  for (int d = 0; d < DHMAX; ++d) {
    qv[d] = d < dh ? qr[d] : 0.f;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int kend = causal ? qi + 1 : L;
  for (int j = 0; j < kend; ++j) {
    const float* kr = kh + (size_t)j * dh;
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < DHMAX; ++d)
      if (d < dh) s = fmaf(qv[d], kr[d], s);
    s *= scale;
    float mn = fmaxf(m, s);
    float alpha = expf(m - mn);
    float p = expf(s - mn);
    l = l * alpha + p;
    const float* vr = vh + (size_t)j * dh;
#pragma unroll
    for (int d = 0; d < DHMAX; ++d)
      if (d < dh) acc[d] = fmaf(p, vr[d], acc[d] * alpha);
    m = mn;
  }
  float* orow = o + ((size_t)b * L + qi) * (size_t)(H * dh) + h * dh;
#pragma unroll
  for (int d = 0; d < DHMAX; ++d)
    if (d < dh) orow[d] = acc[d] / l;
}

__global__ void swiglu_f32_kernel(const float* __restrict__ gu, float* __restrict__ a, int M, int F) {
  size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)M * F) return;
  size_t row = idx / F, f = idx % F;
  float g = gu[row * 2 * F + f], u = gu[row * 2 * F + F + f];
  a[idx] = g / (1.f + expf(-g)) * u;
}

__global__ void gelu_f32_kernel(float* x, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float z = x[i];
  x[i] = z * 0.5f * erfcf(-z * 0.70710678118654752f);
}

}  // namespace

hipError_t gemm_f32(const float* A, int lda, const float* W, int ldw, float* C, int ldc, const float* bias, int mode,
                    int M, int N, int K, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, A, lda, W, ldw, C, ldc, bias, mode, M, N, K);
  return hipGetLastError();
}

hipError_t qkv_split_f32(const float* qkv, const float* rope_cos, const float* rope_sin, float* q, float* k,
                         float* v, float* vt, int ldvt, int B, int L, int H, int Hkv, int dh, hipStream_t s) {
  size_t n = (size_t)B * L * (H + 2 * Hkv) * (dh / 2);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(qkv_split_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, qkv, rope_cos,
                     rope_sin, q, k, v, vt, ldvt, B, L, H, Hkv, dh);
  return hipGetLastError();
}

hipError_t attention_f32(const float* q, const float* k, const float* v, float* o, int B, int H, int Hkv, int L,
                         int dh, bool causal, hipStream_t s) {
  if (B <= 0 || L <= 0) return hipSuccess;
  if (Hkv <= 0 || H % Hkv != 0 || dh > 128) return hipErrorInvalidValue;
  dim3 grid((L + 63) / 64, H, B);
  float scale = 1.f / sqrtf((float)dh);
  if (dh <= 64)
    hipLaunchKernelGGL((attention_f32_kernel<64>), grid, dim3(64), 0, s, q, k, v, o, B, H, Hkv, L, dh, causal ? 1 : 0,
                       scale);
  else
    hipLaunchKernelGGL((attention_f32_kernel<128>), grid, dim3(64), 0, s, q, k, v, o, B, H, Hkv, L, dh,
                       causal ? 1 : 0, scale);
  return hipGetLastError();
}

hipError_t swiglu_f32(const float* gu, float* a, int M, int F, hipStream_t s) {
  size_t n = (size_t)M * F;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, gu, a, M, F);
  return hipGetLastError();
}

hipError_t gelu_f32(float* x, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(gelu_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x, n);
  return hipGetLastError();
}

}  // namespace vla
