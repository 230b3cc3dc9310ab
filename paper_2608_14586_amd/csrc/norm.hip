// Row normalisations and casts (HBM-bound): one wave per row, float4 loads,
// the row kept in registers between the reduction and the scaled store.

#include "kernels.h"

namespace vla {
namespace {

// Where row r of the output starts: y + rows(r).
struct RowsPlain {
  int d;
  __device__ __forceinline__ size_t operator()(int r) const { return (size_t)r * d; }
};

// Encoder rows (images x gh*gw patches, row-major grid) placed in the
// connector's merged layout: patch (gy, gx) of image i is feature block
// (gy % m) * m + gx % m of token i * (gh/m) * (gw/m) + (gy/m) * (gw/m) + gx/m,
// a token being m*m*d wide.
struct RowsMerged {
  int d, gh, gw, m;
  __device__ __forceinline__ size_t operator()(int r) const {
    const int L = gh * gw, i = r / L, l = r % L, gy = l / gw, gx = l % gw, tw = gw / m;
    const size_t tok = (size_t)i * (gh / m) * tw + (size_t)(gy / m) * tw + gx / m;
    return tok * m * m * d + (size_t)((gy % m) * m + gx % m) * d;
  }
};

// lo > 0 (bf16 output only): the remainder bf16(v - bf16(v)) of each output
// v also goes to y + rows(row) + lo + column.
template <int NCH, bool LAYERNORM, class OutT, class Rows>
__global__ __launch_bounds__(256) void norm_kernel(const float* __restrict__ x, const float* __restrict__ g,
                                                   const float* __restrict__ bta, float eps, OutT* __restrict__ y,
                                                   int M, int d, Rows rows, int lo) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int n4 = d >> 2;
  const f32x4* xr = (const f32x4*)(x + (size_t)row * d);
  const f32x4* g4 = (const f32x4*)g;
  const f32x4* b4 = (const f32x4*)bta;
  f32x4 v[NCH], gv[NCH], bv[LAYERNORM ? NCH : 1];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    int i = lane + c * 64;
    v[c] = i < n4 ? xr[i] : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // the gains (and biases) load beside the row, not after its reduction
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    int i = lane + c * 64;
    gv[c] = i < n4 ? g4[i] : f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (LAYERNORM) bv[c] = i < n4 ? b4[i] : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int c = 0; c < NCH; ++c) s += (v[c][0] + v[c][1]) + (v[c][2] + v[c][3]);
  float mean = 0.f, rstd;
  if (LAYERNORM) {
    mean = warp_sum(s) / (float)d;
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      int i = lane + c * 64;
      if (i < n4)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float t = v[c][e] - mean;
          q += t * t;
        }
    }
    rstd = rsqrtf(warp_sum(q) / (float)d + eps);
  } else {
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) q += v[c][e] * v[c][e];
    rstd = rsqrtf(warp_sum(q) / (float)d + eps);
  }
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    int i = lane + c * 64;
    if (i >= n4) continue;
    const f32x4 gg = gv[c];
    f32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = (v[c][e] - mean) * rstd * gg[e];
    if constexpr (LAYERNORM) {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] += bv[c][e];
    }
    const size_t at = rows(row) + (size_t)i * 4;
    if constexpr (sizeof(OutT) == 2) {
      u32x2 w = {pack_bf2(o[0], o[1]), pack_bf2(o[2], o[3])};
      *(u32x2*)((bf16_t*)y + at) = w;
      if (lo) {
        const u32x2 r = {pack_bf2(o[0] - __uint_as_float(w[0] << 16), o[1] - __uint_as_float(w[0] & 0xFFFF0000u)),
                         pack_bf2(o[2] - __uint_as_float(w[1] << 16), o[3] - __uint_as_float(w[1] & 0xFFFF0000u))};
        *(u32x2*)((bf16_t*)y + at + lo) = r;
      }
    } else {
      *(f32x4*)((float*)y + at) = o;
    }
  }
}

template <bool LN, class OutT, class Rows>
hipError_t launch_norm(const float* x, const float* g, const float* b, float eps, OutT* y, int M, int d,
                       Rows rows, hipStream_t s, int lo = 0) {
  if (M <= 0) return hipSuccess;
  if (d % 4 != 0) return hipErrorInvalidValue;
  const int n4 = d / 4;
  dim3 grid((M + 3) / 4), block(256);
#define VLA_NORM(NCH) \
  hipLaunchKernelGGL((norm_kernel<NCH, LN, OutT, Rows>), grid, block, 0, s, x, g, b, eps, y, M, d, rows, lo)
  if (n4 <= 64) VLA_NORM(1);
  else if (n4 <= 128) VLA_NORM(2);
  else if (n4 <= 256) VLA_NORM(4);
  else if (n4 <= 512) VLA_NORM(8);
  else if (n4 <= 1024) VLA_NORM(16);
  else if (n4 <= 2048) VLA_NORM(32);
  else return hipErrorInvalidValue;
#undef VLA_NORM
  return hipGetLastError();
}

template <class OutT>
hipError_t launch_norm_merge(const float* x, const float* g, const float* b, float eps, OutT* y, int n_img, int gh,
                             int gw, int m, int d, hipStream_t s) {
  if (n_img <= 0 || gh <= 0 || gw <= 0 || m <= 0 || gh % m || gw % m) return hipErrorInvalidValue;
  return launch_norm<true>(x, g, b, eps, y, n_img * gh * gw, d, RowsMerged{d, gh, gw, m}, s);
}

__global__ void bf16_to_f32_kernel(const bf16_t* __restrict__ x, float* __restrict__ y, size_t n) {
  size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
  size_t stride = (size_t)gridDim.x * blockDim.x * 8;
  for (; i < n; i += stride) {
    if (i + 8 <= n) {
      u32x4 w = *(const u32x4*)(x + i);
      f32x4 a, b;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        a[2 * e] = __uint_as_float(w[e] << 16);
        a[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
        b[2 * e] = __uint_as_float(w[e + 2] << 16);
        b[2 * e + 1] = __uint_as_float(w[e + 2] & 0xFFFF0000u);
      }
      *(f32x4*)(y + i) = a;
      *(f32x4*)(y + i + 4) = b;
    } else {
      for (size_t j = i; j < n; ++j) y[j] = bf2f(x[j]);
    }
  }
}

__global__ void f32_to_bf16_kernel(const float* __restrict__ x, bf16_t* __restrict__ y, size_t n) {
  size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
  size_t stride = (size_t)gridDim.x * blockDim.x * 8;
  for (; i < n; i += stride) {
    if (i + 8 <= n) {
      f32x4 a = *(const f32x4*)(x + i), b = *(const f32x4*)(x + i + 4);
      u32x4 w = {pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]), pack_bf2(b[0], b[1]), pack_bf2(b[2], b[3])};
      *(u32x4*)(y + i) = w;
    } else {
      for (size_t j = i; j < n; ++j) y[j] = f2bf(x[j]);
    }
  }
}

inline unsigned ew_grid(size_t n) {
  size_t blocks = (n / 8 + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  return (unsigned)blocks;
}

}  // namespace

hipError_t rmsnorm_bf16(const float* x, const float* g, float eps, bf16_t* y, int M, int d, hipStream_t s) {
  return launch_norm<false>(x, g, (const float*)nullptr, eps, y, M, d, RowsPlain{d}, s);
}
hipError_t rmsnorm_bf16_split(const float* x, const float* g, float eps, bf16_t* y, int M, int d, hipStream_t s) {
  return launch_norm<false>(x, g, (const float*)nullptr, eps, y, M, d, RowsPlain{2 * d}, s, d);
}
hipError_t layernorm_bf16(const float* x, const float* g, const float* b, float eps, bf16_t* y, int M, int d,
                          hipStream_t s) {
  return launch_norm<true>(x, g, b, eps, y, M, d, RowsPlain{d}, s);
}
hipError_t rmsnorm_f32(const float* x, const float* g, float eps, float* y, int M, int d, hipStream_t s) {
  return launch_norm<false>(x, g, (const float*)nullptr, eps, y, M, d, RowsPlain{d}, s);
}
hipError_t layernorm_f32(const float* x, const float* g, const float* b, float eps, float* y, int M, int d,
                         hipStream_t s) {
  return launch_norm<true>(x, g, b, eps, y, M, d, RowsPlain{d}, s);
}

hipError_t layernorm_merge_bf16(const float* x, const float* g, const float* b, float eps, bf16_t* y, int n_img,
                                int gh, int gw, int m, int d, hipStream_t s) {
  return launch_norm_merge(x, g, b, eps, y, n_img, gh, gw, m, d, s);
}
hipError_t layernorm_merge_f32(const float* x, const float* g, const float* b, float eps, float* y, int n_img,
                               int gh, int gw, int m, int d, hipStream_t s) {
  return launch_norm_merge(x, g, b, eps, y, n_img, gh, gw, m, d, s);
}

hipError_t bf16_to_f32(const bf16_t* x, float* y, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(bf16_to_f32_kernel, dim3(ew_grid(n)), dim3(256), 0, s, x, y, n);
  return hipGetLastError();
}

hipError_t f32_to_bf16(const float* x, bf16_t* y, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(ew_grid(n)), dim3(256), 0, s, x, y, n);
  return hipGetLastError();
}

}  // namespace vla
