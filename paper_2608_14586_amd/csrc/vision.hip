// Front of the visual encoder: camera images -> patch rows for the stem GEMM.
//
// The stem is the ViT patch embedding, a stride-p convolution: patch l of an
// image is projected by the stem weights and the learned position embedding
// of its grid index is added.  This kernel lays each patch out as one GEMM
// row (channel, then pixel row, then pixel column: the element order of the
// convolution kernel) and writes the position embedding into the fp32
// residual; the stem is then the encoder's bias-and-residual GEMM, and the
// residual is the encoder's input as it is.  HBM-bound and small (an image is
// read once, its patch rows written once).

#include "kernels.h"

namespace vla {
namespace {

// one workgroup per patch row
template <class T>
__global__ __launch_bounds__(256) void patchify_kernel(const T* __restrict__ img, int C, int H, int W, int p, int gw,
                                                       int L, T* __restrict__ A, int Kp, const float* __restrict__ pos,
                                                       float* __restrict__ h, int d) {
  const int row = blockIdx.x;
  const int i = row / L, l = row % L, gy = l / gw, gx = l % gw;
  const int pp = p * p, K = C * pp;
  const T* base = img + (size_t)i * C * H * W + (size_t)gy * p * W + (size_t)gx * p;
  T* a = A + (size_t)row * Kp;
  for (int k = threadIdx.x; k < Kp; k += 256) {
    T v = T(0);
    if (k < K) {
      const int c = k / pp, y = (k / p) % p, x = k % p;
      v = base[((size_t)c * H + y) * W + x];
    }
    a[k] = v;
  }
  const float* ps = pos + (size_t)l * d;
  float* hr = h + (size_t)row * d;
  for (int j = threadIdx.x; j < d; j += 256) hr[j] = ps[j];
}

template <class T>
hipError_t launch_patchify(const T* img, int n_img, int C, int H, int W, int p, T* A, int Kp, const float* pos,
                           float* h, int d, hipStream_t s) {
  if (n_img <= 0) return hipSuccess;
  if (C <= 0 || p <= 0 || H <= 0 || W <= 0 || H % p || W % p || Kp < C * p * p || d <= 0) return hipErrorInvalidValue;
  const int gw = W / p, L = (H / p) * gw;
  hipLaunchKernelGGL((patchify_kernel<T>), dim3((unsigned)(n_img * L)), dim3(256), 0, s, img, C, H, W, p, gw, L, A,
                     Kp, pos, h, d);
  return hipGetLastError();
}

}  // namespace

hipError_t patchify_bf16(const bf16_t* img, int n_img, int C, int H, int W, int p, bf16_t* A, int Kp,
                         const float* pos, float* h, int d, hipStream_t s) {
  return launch_patchify(img, n_img, C, H, W, p, A, Kp, pos, h, d, s);
}

hipError_t patchify_f32(const float* img, int n_img, int C, int H, int W, int p, float* A, int Kp, const float* pos,
                        float* h, int d, hipStream_t s) {
  return launch_patchify(img, n_img, C, H, W, p, A, Kp, pos, h, d, s);
}

}  // namespace vla
