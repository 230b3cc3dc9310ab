// bf16 MFMA GEMM for gfx950 with fused epilogues.
//
// acc[M][N] = A[M][K] * W[N][K]^T.  Both operands are K-contiguous (the
// nn.Linear layout of the weights and the row-major activations), which is
// exactly the register layout v_mfma_f32_32x32x16_bf16 wants for both of its
// inputs: lane l holds 8 consecutive k of row (l % 32) in k-block (l / 32).
//
// Workgroup: NW waves over a BM x BN tile; each wave owns a WM x WN sub-tile
// of (WM/32) x (WN/32) MFMA 32x32 accumulators.  K advances in BK = 64 slabs
// moved global -> LDS by buffer_load ... lds (see the main loop below).
//
// Tile order: workgroup ids are first remapped so that each of the 8 XCDs
// (which take ids round-robin) receives a contiguous range of tiles, then
// walked M-fastest inside groups of GROUP_M tile rows, so the workgroups of
// one XCD share the same weight tiles in that XCD's L2.
//
// The MFMA 32x32 accumulator layout used by every epilogue: register r of
// lane l holds row (r/4)*8 + (l/32)*4 + (r%4), column l % 32.

#include "kernels.h"

namespace vla {
namespace {

constexpr int BK = 64;
constexpr int GROUP_M = 8;

template <int TM, int TN>
struct Acc {
  f32x16 v[TM][TN];
};

__device__ __forceinline__ int acc_row(int r, int lane) { return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3); }

// ------------------------------------------------------------------ epilogues

struct EpiStoreF32 {
  float* C;
  int ldc, M, N;
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>& a, int row0, int col0, int lane) const {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        int col = col0 + tn * 32 + (lane & 31);
        if (col >= N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int row = row0 + tm * 32 + acc_row(r, lane);
          if (row < M) C[(size_t)row * ldc + col] = a.v[tm][tn][r];
        }
      }
  }
};

struct EpiStoreBF16 {
  bf16_t* C;
  const float* bias;
  int ldc, M, N;
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>& a, int row0, int col0, int lane) const {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        int col = col0 + tn * 32 + (lane & 31);
        if (col >= N) continue;
        float b = bias ? bias[col] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int row = row0 + tm * 32 + acc_row(r, lane);
          if (row < M) C[(size_t)row * ldc + col] = f2bf(a.v[tm][tn][r] + b);
        }
      }
  }
};

struct EpiResidual {
  float* H;
  const float* bias;
  int ldh, M, N;
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>& a, int row0, int col0, int lane) const {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        int col = col0 + tn * 32 + (lane & 31);
        if (col >= N) continue;
        float b = bias ? bias[col] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int row = row0 + tm * 32 + acc_row(r, lane);
          if (row < M) {
            float* p = H + (size_t)row * ldh + col;
            *p = *p + (a.v[tm][tn][r] + b);
          }
        }
      }
  }
};

struct EpiGelu {
  bf16_t* out;
  const float* bias;
  int ldo, M, N;
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>& a, int row0, int col0, int lane) const {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        int col = col0 + tn * 32 + (lane & 31);
        if (col >= N) continue;
        float b = bias ? bias[col] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int row = row0 + tm * 32 + acc_row(r, lane);
          if (row < M) {
            float z = a.v[tm][tn][r] + b;
            // exact GELU: z * Phi(z), Phi(z) = 0.5 * erfc(-z / sqrt(2))
            float y = z * 0.5f * erfcf(-z * 0.70710678118654752f);
            out[(size_t)row * ldo + col] = f2bf(y);
          }
        }
      }
  }
};

// Pairs accumulator tiles (2p, 2p+1) = (gate, up) of the same 32 features.
struct EpiSwiGLU {
  bf16_t* out;
  int ldo, M, N;
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>& a, int row0, int col0, int lane) const {
    static_assert(TN % 2 == 0, "swiglu pairs tiles");
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tp = 0; tp < TN / 2; ++tp) {
        int pcol = col0 + tp * 64;
        if (pcol >= N) continue;
        int f = (pcol >> 1) + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int row = row0 + tm * 32 + acc_row(r, lane);
          if (row < M) {
            float g = a.v[tm][2 * tp][r], u = a.v[tm][2 * tp + 1][r];
            float s = g / (1.f + __expf(-g));
            out[(size_t)row * ldo + f] = f2bf(s * u);
          }
        }
      }
  }
};

struct EpiQKV {
  QkvArgs q;
  int M;
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>& a, int row0, int col0, int lane) const {
    static_assert(TN % 2 == 0, "qkv pairs tiles");
    const int dh = q.dh, L = q.L;
    const int i = lane & 31;
#pragma unroll
    for (int tp = 0; tp < TN / 2; ++tp) {
      const int p = col0 + tp * 64;  // packed column of this 64-wide group
      int kind, head, r;
      if (p < q.H * dh) {
        kind = 0; head = p / dh; r = p % dh;
      } else if (p < (q.H + q.Hkv) * dh) {
        kind = 1; head = (p - q.H * dh) / dh; r = (p - q.H * dh) % dh;
      } else if (p < (q.H + 2 * q.Hkv) * dh) {
        kind = 2; head = (p - (q.H + q.Hkv) * dh) / dh; r = (p - (q.H + q.Hkv) * dh) % dh;
      } else {
        continue;
      }
      const int c = r / 64;
      const int d1 = c * 32 + i, d2 = dh / 2 + c * 32 + i;
      const float b1 = q.bias ? q.bias[p + i] : 0.f;
      const float b2 = q.bias ? q.bias[p + 32 + i] : 0.f;
      const bool rot = (kind < 2) && q.rope_cos != nullptr;
      const int nh = kind == 0 ? q.H : q.Hkv;
      bf16_t* dst = kind == 0 ? q.q : (kind == 1 ? q.k : q.v);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float y1[4], y2[4];
          int rowb = row0 + tm * 32 + g * 8 + (lane >> 5) * 4;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            float x1 = a.v[tm][2 * tp][g * 4 + j] + b1;
            float x2 = a.v[tm][2 * tp + 1][g * 4 + j] + b2;
            int row = rowb + j;
            if (rot && row < M) {
              int pos = row % L;
              float cs = q.rope_cos[(size_t)pos * (dh / 2) + d1];
              float sn = q.rope_sin[(size_t)pos * (dh / 2) + d1];
              y1[j] = x1 * cs - x2 * sn;
              y2[j] = x2 * cs + x1 * sn;
            } else {
              y1[j] = x1;
              y2[j] = x2;
            }
            if (row < M) {
              int b = row / L, pos = row % L;
              size_t base = (((size_t)b * nh + head) * L + pos) * dh;
              dst[base + d1] = f2bf(y1[j]);
              dst[base + d2] = f2bf(y2[j]);
            }
          }
          if (kind == 2) {
            // V transposed: 4 consecutive positions of one dim per lane
            int b0 = rowb / L, pos0 = rowb % L;
            bool fast = (rowb + 3 < M) && (pos0 + 3 < L) && ((pos0 & 3) == 0) && ((q.ldvt & 3) == 0);
            if (fast) {
              size_t o1 = (((size_t)b0 * q.Hkv + head) * dh + d1) * q.ldvt + pos0;
              size_t o2 = (((size_t)b0 * q.Hkv + head) * dh + d2) * q.ldvt + pos0;
              u32x2 w1 = {pack_bf2(y1[0], y1[1]), pack_bf2(y1[2], y1[3])};
              u32x2 w2 = {pack_bf2(y2[0], y2[1]), pack_bf2(y2[2], y2[3])};
              *(u32x2*)(q.vt + o1) = w1;
              *(u32x2*)(q.vt + o2) = w2;
            } else {
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                int row = rowb + j;
                if (row >= M) continue;
                int b = row / L, pos = row % L;
                q.vt[(((size_t)b * q.Hkv + head) * dh + d1) * q.ldvt + pos] = f2bf(y1[j]);
                q.vt[(((size_t)b * q.Hkv + head) * dh + d2) * q.ldvt + pos] = f2bf(y2[j]);
              }
            }
          }
        }
      }
    }
  }
};

// ---------------------------------------------------------------- main loop
//
// The K slabs move global -> LDS with buffer_load ... lds (16 bytes per lane, written at M0 + 16 * lane), so no
// VGPRs or ds_write instructions are spent on staging and the next slab's
// loads run fully asynchronously behind the current slab's MFMAs.  LDS rows
// are 128 bytes (BK = 64 bf16) with the 16-byte chunks XOR-swizzled by
// ((row >> 1) & 7): each 16-lane phase of a fragment read covers all banks.
// Buffer resources clamp ragged M / N tiles: rows past the end read as zero.
// MFMA fragments are double buffered across the four k16 steps of a slab.

__device__ __forceinline__ void buffer_load_lds16(__amdgpu_buffer_rsrc_t r, void* lds, unsigned voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, 0, 0, 0);
}

template <int BM, int BN, int WM, int WN, int NW, class Epi>
__global__ __launch_bounds__(64 * NW) void gemm_bf16_dma_kernel(const bf16_t* __restrict__ A, int lda,
                                                                const bf16_t* __restrict__ W, int ldw, int M, int N,
                                                                int K, Epi epi) {
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int WAVES_N = BN / WN;
  static_assert((BM / WM) * (BN / WN) == NW, "wave grid must cover the tile");
  constexpr int ROWB = BK * 2;                             // bytes per LDS row (128)
  constexpr int A_INST = BM / (8 * NW), B_INST = BN / (8 * NW);  // 1 KB loads per wave per slab
  static_assert(A_INST >= 1 && B_INST >= 1, "tile too small for the wave count");
  __shared__ __attribute__((aligned(1024))) char smem[2 * (BM + BN) * ROWB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int nwg = gridDim.x;
  int id = blockIdx.x;
  if ((nwg & 7) == 0) id = (id & 7) * (nwg >> 3) + (id >> 3);
  const int group = GROUP_M * tiles_n;
  const int first_m = (id / group) * GROUP_M;
  const int gsz = min(tiles_m - first_m, GROUP_M);
  const int tile_m = first_m + (id % group) % gsz;
  const int tile_n = (id % group) / gsz;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  // buffer resources over the tile's rows; rows past M / N read as zero
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(A + (size_t)m0 * lda), (short)0, (int)((size_t)(M - m0) * lda * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(W + (size_t)n0 * ldw), (short)0, (int)((size_t)(N - n0) * ldw * 2), 0x00020000);

  // this lane's slot in each 1 KB load: row (lane / 8) of the 8-row group,
  // LDS chunk (lane % 8) holding global chunk (lane % 8) ^ key(tile row)
  const int lrow = lane >> 3, lslot = lane & 7;
  auto issue = [&](int k0, int buf) {
    char* base = smem + buf * (BM + BN) * ROWB;
#pragma unroll
    for (int j = 0; j < A_INST; ++j) {
      const int row = (wave * A_INST + j) * 8 + lrow;
      const int ch = lslot ^ ((row >> 1) & 7);
      buffer_load_lds16(ra, base + (wave * A_INST + j) * 1024, (unsigned)((row * lda + k0 + ch * 8) * 2));
    }
#pragma unroll
    for (int j = 0; j < B_INST; ++j) {
      const int row = (wave * B_INST + j) * 8 + lrow;
      const int ch = lslot ^ ((row >> 1) & 7);
      buffer_load_lds16(rb, base + BM * ROWB + (wave * B_INST + j) * 1024, (unsigned)((row * ldw + k0 + ch * 8) * 2));
    }
  };

  Acc<TM, TN> acc;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc.v[tm][tn][r] = 0.f;

  const int fi = lane & 31, fh = lane >> 5;
  const int a_row0 = (wm * WM + fi) * ROWB, b_row0 = BM * ROWB + (wn * WN + fi) * ROWB;
  const int key = (fi >> 1) & 7;
  bf16x8 fa[2][TM], fb[2][TN];
  auto frags = [&](int buf, int ks, int slot) {
    const char* base = smem + buf * (BM + BN) * ROWB;
    const int off = (((2 * ks + fh) ^ key) << 4);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) fa[slot][tm] = *(const bf16x8*)(base + a_row0 + tm * 32 * ROWB + off);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) fb[slot][tn] = *(const bf16x8*)(base + b_row0 + tn * 32 * ROWB + off);
  };

  const int nk = K / BK;
  issue(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  frags(0, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) issue((kt + 1) * BK, buf ^ 1);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < BK / 16) frags(buf, ks + 1, cur ^ 1);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          acc.v[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][tm], fb[cur][tn], acc.v[tm][tn], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kt + 1 < nk) frags(buf ^ 1, 0, 0);
  }

  epi(acc, m0 + wm * WM, n0 + wn * WN, lane);
}

template <class Epi>
hipError_t launch(const bf16_t* A, int lda, const bf16_t* W, int ldw, int M, int N, int K, const Epi& epi,
                  hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % BK != 0 || lda % 8 != 0 || ldw % 8 != 0) return hipErrorInvalidValue;
  // byte offsets inside a tile's buffer resource are 32-bit
  if ((size_t)256 * lda * 2 >= (1u << 31) || (size_t)256 * ldw * 2 >= (1u << 31)) return hipErrorInvalidValue;
  // 256x256 tiles (8 waves of 128x64) once they fill the chip at least twice;
  // otherwise 128x128 tiles (4 waves of 64x64, two workgroups per CU)
  const long tiles256 = (long)((M + 255) / 256) * ((N + 255) / 256);
  if (tiles256 >= 512) {
    int grid = ((M + 255) / 256) * ((N + 255) / 256);
    hipLaunchKernelGGL((gemm_bf16_dma_kernel<256, 256, 128, 64, 8, Epi>), dim3(grid), dim3(512), 0, s, A, lda, W,
                       ldw, M, N, K, epi);
  } else {
    int grid = ((M + 127) / 128) * ((N + 127) / 128);
    hipLaunchKernelGGL((gemm_bf16_dma_kernel<128, 128, 64, 64, 4, Epi>), dim3(grid), dim3(256), 0, s, A, lda, W, ldw,
                       M, N, K, epi);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_bf16_store_f32(const bf16_t* A, int lda, const bf16_t* W, int ldw, float* C, int ldc, int M, int N,
                               int K, hipStream_t s) {
  return launch(A, lda, W, ldw, M, N, K, EpiStoreF32{C, ldc, M, N}, s);
}

hipError_t gemm_bf16_store_bf16(const bf16_t* A, int lda, const bf16_t* W, int ldw, bf16_t* C, int ldc,
                                const float* bias, int M, int N, int K, hipStream_t s) {
  return launch(A, lda, W, ldw, M, N, K, EpiStoreBF16{C, bias, ldc, M, N}, s);
}

hipError_t gemm_bf16_residual(const bf16_t* A, int lda, const bf16_t* W, int ldw, float* H, int ldh,
                              const float* bias, int M, int N, int K, hipStream_t s) {
  return launch(A, lda, W, ldw, M, N, K, EpiResidual{H, bias, ldh, M, N}, s);
}

hipError_t gemm_bf16_swiglu(const bf16_t* A, int lda, const bf16_t* W, int ldw, bf16_t* out, int ldo, int M, int N,
                            int K, hipStream_t s) {
  if (N % 64 != 0) return hipErrorInvalidValue;
  return launch(A, lda, W, ldw, M, N, K, EpiSwiGLU{out, ldo, M, N}, s);
}

hipError_t gemm_bf16_gelu(const bf16_t* A, int lda, const bf16_t* W, int ldw, bf16_t* out, int ldo,
                          const float* bias, int M, int N, int K, hipStream_t s) {
  return launch(A, lda, W, ldw, M, N, K, EpiGelu{out, bias, ldo, M, N}, s);
}

hipError_t gemm_bf16_qkv(const bf16_t* A, int lda, const bf16_t* W, int ldw, const QkvArgs& qa, int M, int N, int K,
                         hipStream_t s) {
  if (qa.dh % 64 != 0 || N % 64 != 0) return hipErrorInvalidValue;
  return launch(A, lda, W, ldw, M, N, K, EpiQKV{qa, M}, s);
}

}  // namespace vla
