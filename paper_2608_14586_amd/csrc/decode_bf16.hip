// One decode step of the decoder blocks on the GPU: B <= 4 sequences, one
// new token each, attending over the KV cache the prefix handed over.
//
// With one token per sequence every projection is a skinny product whose
// cost is streaming the block's weights from HBM once, so the kernels are
// built around that stream:
//  * gemv_stream_kernel: each workgroup owns 16 output rows (8 when 16-row
//    tiles would leave fewer than two workgroups per CU) and streams their
//    weights over all of K from the packed slab-major layout (the rows' 128
//    bytes are contiguous per 64-k slab).  The input rows are staged into LDS
//    once, in bf16, before the main loop: RMSNorm is fused there (QKV,
//    gate/up; each workgroup recomputes the row's scale, d floats per row).
//    The gate/up product runs paired: a workgroup owns 16 features' gate
//    rows and their up rows and writes the gated bf16 activation, which the
//    down projection stages as it is, like the attention output for the O
//    projection.  (Gating inside the down projection's staging instead, from
//    the fp32 gate/up rows, reads four times the bytes per workgroup and
//    measured 14 us slower per launch.)
//    The main loop has no barrier, so two 1024-k chunks of weights
//    (up to 16 loads of 16 bytes per lane) stay in flight; slabs past K read
//    as zero through the buffer resource, so the loop has no branches.
//    Products and accumulation in fp32.  Epilogues: raw fp32 store or fp32
//    residual add.
//  * gemv_chunk_kernel: the same product staging the input chunk by chunk
//    (2048 k at a time, a barrier around each), for inputs too wide for the
//    streaming kernel's LDS (four rows of a d_ff-wide input) or too short to
//    fill its chunks.
//  * attn_decode_kernel: one workgroup per (sequence, head, 128-key split);
//    applies RoPE to q and to the new key at the token's position, appends the
//    new key and value to the cache, and writes (max, sum, unnormalised
//    output) partials that a small kernel combines into the bf16 attention
//    output.  (Combining in the last workgroup of each head, found with a
//    device-scope counter, needs an L2 write-back per workgroup on this
//    multi-XCD part and measured 3x slower than the extra launch.)
// Rounding points follow the prefill: normed activations, q and K/V after
// RoPE, the attention output and the gated activation are bf16.  With split
// operands each sequence's normed row and gated activation are staged twice,
// as bf16(v) and bf16(v - bf16(v)), and the two dot products of a weight row
// are added in fp32 (the weights still stream once).  The kernels take the
// number of staged rows per sequence, P, and the largest row count, MB, as
// template arguments.

#include "kernels.h"

namespace vla {
namespace {

constexpr int GV_KCH = 2048;       // K elements staged per chunk
constexpr int GV_MB = 4;           // largest batch
constexpr int ATT_KC = 128;        // keys per attention split

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
// the part of x that bf16(x) leaves out (rounded to bf16 by the caller)
__device__ __forceinline__ float lo_part(float x) { return x - bf2f(f2bf(x)); }

// acc + sum of the 8 products of bf16 pairs, two per v_dot2_f32_bf16: the
// bf16 operands go in as they are (no conversion to fp32) and every product
// is exact in fp32.  With several sequences each weight feeds several
// products, and converting both operands per product made the step VALU-bound.
// The pairs are taken by shuffling the 8-lane bf16 view of each operand:
// bit-casting the 32-bit words w[i] one by one instead compiled to a loop
// that read word 0 four times.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
__device__ __forceinline__ float dot8(const u32x4& w, const u32x4& x, float acc) {
  const bf16x8_t a = __builtin_bit_cast(bf16x8_t, w), b = __builtin_bit_cast(bf16x8_t, x);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 0, 1), __builtin_shufflevector(b, b, 0, 1), acc,
                                        false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 2, 3), __builtin_shufflevector(b, b, 2, 3), acc,
                                        false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 4, 5), __builtin_shufflevector(b, b, 4, 5), acc,
                                        false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 6, 7), __builtin_shufflevector(b, b, 6, 7), acc,
                                        false);
  return acc;
}

// ---------------------------------------------------------------- staging
// Each stage fills xs[b][0..n) (bf16) with columns [k0, k0 + n) of the
// product's input row b; prepare() runs once before the K loop.

// x = bf16(h * rsqrt(mean(h^2) + eps) * g), h fp32 [B][K]
struct StageNorm {
  const float* h;
  const float* g;
  float eps;
  // sc[b] = 1 / rms(h[b]) for the B rows at once: every row's 16-byte loads
  // are issued before any sum, and one pair of barriers serves all rows
  // (red: 4 x GV_MB floats)
  __device__ void prepare(float* sc, int B, int K, int tid, float* red) const {
    float s[GV_MB] = {0.f, 0.f, 0.f, 0.f};
    const int K4 = (K % 4 == 0) ? K : 0;  // rows 16-byte aligned
    for (int i = tid * 4; i < K4; i += 256 * 4) {
      f32x4 v[GV_MB];
#pragma unroll
      for (int b = 0; b < GV_MB; ++b)
        if (b < B) v[b] = *(const f32x4*)(h + (size_t)b * K + i);
#pragma unroll
      for (int b = 0; b < GV_MB; ++b)
        if (b < B) s[b] += v[b][0] * v[b][0] + v[b][1] * v[b][1] + v[b][2] * v[b][2] + v[b][3] * v[b][3];
    }
    for (int i = K4 + tid; i < K; i += 256)
#pragma unroll
      for (int b = 0; b < GV_MB; ++b)
        if (b < B) s[b] += h[(size_t)b * K + i] * h[(size_t)b * K + i];
#pragma unroll
    for (int b = 0; b < GV_MB; ++b) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) s[b] += __shfl_xor(s[b], o);
      if ((tid & 63) == 0) red[(tid >> 6) * GV_MB + b] = s[b];
    }
    __syncthreads();
    if (tid < B)
      sc[tid] = 1.f / sqrtf((red[tid] + red[GV_MB + tid] + red[2 * GV_MB + tid] + red[3 * GV_MB + tid]) / (float)K +
                            eps);
    __syncthreads();
  }
  // staged row bp = logical row bp / P; with P = 2 rows alternate between
  // the bf16 value (hi) and its remainder bf16(x - hi) (lo)
  __device__ void fill(bf16_t* xs, const float* sc, int Bp, int P, int K, int k0, int n, int tid) const {
    for (int bp = 0; bp < Bp; ++bp) {
      const int b = bp / P;
      const bool lo = bp % P;
      for (int i = tid; i < n; i += 256) {
        const float x = h[(size_t)b * K + k0 + i] * sc[b] * g[k0 + i];
        xs[bp * GV_KCH + i] = lo ? f2bf(lo_part(x)) : f2bf(x);
      }
    }
  }
  // dst[0, K) = row b normalised, or its remainder (part 1) (K % 4 == 0)
  __device__ void fill_row(bf16_t* dst, const float* sc, int b, int part, int K, int tid) const {
    const float s = sc[b];
    for (int i = tid * 4; i < K; i += 256 * 4) {
      const f32x4 x = *(const f32x4*)(h + (size_t)b * K + i), gg = *(const f32x4*)(g + i);
      f32x4 y = {x[0] * s * gg[0], x[1] * s * gg[1], x[2] * s * gg[2], x[3] * s * gg[3]};
      if (part)
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = lo_part(y[e]);
      *(u32x2*)(dst + i) = u32x2{pack_bf2(y[0], y[1]), pack_bf2(y[2], y[3])};
    }
  }
};

// x = a bf16 row already in global memory: row b at a + b * ld, its
// remainder row (split operands, part 1) lo elements further
struct StageCopy {
  const bf16_t* a;
  int ld, lo;
  __device__ void prepare(float*, int, int, int, float*) const {}
  __device__ void fill(bf16_t* xs, const float*, int Bp, int P, int K, int k0, int n, int tid) const {
    for (int bp = 0; bp < Bp; ++bp) {
      const bf16_t* src = a + (size_t)(bp / P) * ld + (bp % P) * lo + k0;
      for (int i = tid * 8; i < n; i += 256 * 8) *(u32x4*)(xs + bp * GV_KCH + i) = *(const u32x4*)(src + i);
    }
  }
  __device__ void fill_row(bf16_t* dst, const float*, int b, int part, int K, int tid) const {
    const bf16_t* src = a + (size_t)b * ld + part * lo;
    for (int i = tid * 8; i < K; i += 256 * 8) *(u32x4*)(dst + i) = *(const u32x4*)(src + i);
  }
};



// a[b][f] = bf16(silu(gate) * up) from the raw gate/up product gu[B][2*fpad]
// in the packed row order (each group of 64 rows: 32 gate rows, then their 32
// up rows).  Features past d_ff have zero weight rows, so they come out zero.
// Row b of a starts at a + b * ld; lo > 0 also writes bf16(y - bf16(y)) at
// column lo + f (split operands for the down projection).
__global__ __launch_bounds__(256) void swiglu_kernel(const float* __restrict__ gu, int fpad, int B,
                                                     bf16_t* __restrict__ a, int ld, int lo) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * fpad) return;
  const int b = i / fpad, f = i % fpad;
  const float* r = gu + (size_t)b * 2 * fpad + (f / 32) * 64 + f % 32;
  const float g = r[0];
  const float y = g / (1.f + __expf(-g)) * r[32];
  a[(size_t)b * ld + f] = f2bf(y);
  if (lo) a[(size_t)b * ld + lo + f] = f2bf(lo_part(y));
}

// ---------------------------------------------------------------- epilogues

struct EpiRaw {  // out[b][n] = acc
  float* out;
  int ld;
  __device__ void operator()(int b, int n, float v) const { out[(size_t)b * ld + n] = v; }
};

struct EpiAdd {  // h[b][n] += acc
  float* h;
  int ld;
  __device__ void operator()(int b, int n, float v) const { h[(size_t)b * ld + n] += v; }
};

// a[b][f] = bf16(silu(gate) * up), from the gate and up sums of feature f;
// lo > 0: also its remainder at a[b][lo + f]
struct EpiGated {
  bf16_t* a;
  int ld, lo;
  __device__ void operator()(int b, int f, float g, float u) const {
    const float y = g / (1.f + __expf(-g)) * u;
    a[(size_t)b * ld + f] = f2bf(y);
    if (lo) a[(size_t)b * ld + lo + f] = f2bf(lo_part(y));
  }
};

// out[b][n] for n in [blockIdx.x*ROWS, +ROWS), b < B: the dot of row n of
// the packed W [K/64][nblk][128][64] with the staged input row b.  Each
// logical row is staged as P rows (P = 2: hi and lo of split operands, whose
// products are summed), B * P <= MB.
template <int ROWS, int MB, int P, class Stage, class Epi>
__global__ __launch_bounds__(256) void gemv_chunk_kernel(Stage sg, const bf16_t* __restrict__ W, int nblk, int N, int K,
                                                   int B, Epi epi) {
  constexpr int GV_ROWS = ROWS, J = ROWS / 8;  // rows per workgroup, 8-row groups per lane
  __shared__ __attribute__((aligned(16))) bf16_t xs[MB * GV_KCH];
  __shared__ float red[4 * GV_ROWS * MB];
  __shared__ float sc[GV_MB];
  __shared__ float tmp[4 * GV_MB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * GV_ROWS;
  const int r8 = lane >> 3, c8 = lane & 7;
  // rows n0 + r8 + 8 j lie in the same 128-row block (ROWS | 128)
  const int blk = n0 / SLAB_N, ra = n0 % SLAB_N + r8;
  const int Bp = B * P;
  float acc[J][MB];
#pragma unroll
  for (int j = 0; j < J; ++j)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[j][b] = 0.f;
  // this wave's slabs of a chunk: wave, wave + 4, ...; a chunk's weight
  // loads (up to 16 per lane) are issued before the staging work they do not
  // depend on, so the HBM fetch overlaps it
  constexpr int U = GV_KCH / 64 / 4;
  u32x4 wv[U][J];
  auto load = [&](int k0) {
    const int s0 = k0 / 64, ns = min(GV_KCH, K - k0) / 64;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int sl = wave + 4 * u;
      if (sl < ns) {
        const bf16_t* base = W + (((size_t)(s0 + sl) * nblk + blk) * SLAB_N) * 64;
#pragma unroll
        for (int j = 0; j < J; ++j) wv[u][j] = *(const u32x4*)(base + (size_t)(ra + 8 * j) * 64 + c8 * 8);
      }
    }
  };
  load(0);
  sg.prepare(sc, B, K, tid, tmp);
  for (int k0 = 0; k0 < K; k0 += GV_KCH) {
    const int n = min(GV_KCH, K - k0), ns = n / 64;
    __syncthreads();  // the previous chunk's reads of xs are done
    sg.fill(xs, sc, Bp, P, K, k0, n, tid);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int sl = wave + 4 * u;
      if (sl < ns) {
#pragma unroll
        for (int b = 0; b < MB; ++b)
          if (b < Bp) {
            const u32x4 xv = *(const u32x4*)(xs + b * GV_KCH + sl * 64 + c8 * 8);
#pragma unroll
            for (int j = 0; j < J; ++j) acc[j][b] = dot8(wv[u][j], xv, acc[j][b]);
          }
      }
    }
    if (k0 + GV_KCH < K) load(k0 + GV_KCH);
  }
  // reduce over the 8 lanes of a row, then over the 4 waves
#pragma unroll
  for (int j = 0; j < J; ++j)
#pragma unroll
    for (int b = 0; b < MB; ++b) {
      float v = acc[j][b];
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 4);
      acc[j][b] = v;
    }
  if (c8 == 0)
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int b = 0; b < MB; ++b) red[(wave * GV_ROWS + r8 + 8 * j) * MB + b] = acc[j][b];
  __syncthreads();
  if (tid < GV_ROWS * GV_MB) {
    const int row = tid / GV_MB, b = tid % GV_MB;
    const int nn = n0 + row;
    if (b < B && nn < N) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w)
#pragma unroll
        for (int q = 0; q < P; ++q) v += red[(w * GV_ROWS + row) * MB + b * P + q];
      epi(b, nn, v);
    }
  }
}

constexpr int GS_KC = 1024;  // k per chunk of the streaming kernel: 16 slabs, 4 per wave
constexpr int GS_D = 2;      // chunks in flight per lane

__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// out[b][n] for n in [blockIdx.x*ROWS, +ROWS), b < B, over the input rows
// staged whole in LDS (xs[B][Kp], zero past K; Kp a multiple of KC*GS_D).
// PAIR: the gate/up product with SwiGLU in the epilogue.  Workgroup w owns
// features [16 w, 16 w + 16): their 16 gate rows and 16 up rows, 32 rows apart
// in the packed order (each 64-row group: 32 gate rows, then their 32 up
// rows), and epi(b, f, gate, up) writes the gated activation.
// Each logical row is staged as P rows (hi, lo with P = 2), B * P <= MB.
template <int ROWS, bool PAIR, int MB, int P, class Stage, class Epi>
__global__ __launch_bounds__(256) void gemv_stream_kernel(Stage sg, const bf16_t* __restrict__ W, int nblk, int N,
                                                          int K, int B, int Kp, Epi epi) {
  static_assert(!PAIR || ROWS == 32, "a paired workgroup owns 16 gate and 16 up rows");
  constexpr int J = ROWS / 8;
  constexpr int KC = PAIR ? GS_KC / 2 : GS_KC;  // the paired kernel keeps the same bytes in flight
  constexpr int U = KC / 64 / 4;
  constexpr int SPC = KC / 64;                 // slabs per chunk
  extern __shared__ __attribute__((aligned(16))) bf16_t xs[];
  __shared__ float red[4 * ROWS * MB];
  __shared__ float sc[GV_MB];
  __shared__ float tmp[4 * GV_MB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r8 = lane >> 3, c8 = lane & 7;
  // this lane's rows: block blk, rows rb + roff(j) inside it (all in one 128-row block)
  int blk, rb;
  if constexpr (PAIR) {
    const int w = blockIdx.x;
    blk = w / 4;
    rb = 64 * ((w / 2) % 2) + 16 * (w % 2) + r8;
  } else {
    const int n0 = blockIdx.x * ROWS;
    blk = n0 / SLAB_N;
    rb = n0 % SLAB_N + r8;
  }
  auto roff = [](int j) { return PAIR ? 8 * (j % 2) + 32 * (j / 2) : 8 * j; };
  // the whole packed matrix; slabs past K read as zero
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void*)W, (short)0, (int)((size_t)(K / 64) * nblk * SLAB_N * 64 * 2), 0x00020000);
  const unsigned slab_stride = (unsigned)nblk * SLAB_N * 64 * 2;
  const unsigned lane_off = (unsigned)(((size_t)blk * SLAB_N + rb) * 64 * 2 + c8 * 16);
  // chunk c, wave w: slabs c*SPC + w + 4u
  u32x4 wv[GS_D][U][J];
  auto issue = [&](int d, int c) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const unsigned sl = (unsigned)(c * SPC + wave + 4 * u);
#pragma unroll
      for (int j = 0; j < J; ++j) wv[d][u][j] = buffer_load16(rw, sl * slab_stride + lane_off + roff(j) * 64 * 2);
    }
  };
#pragma unroll
  for (int d = 0; d < GS_D; ++d) issue(d, d);
  // the input rows (these barriers also give the first chunks time to land)
  sg.prepare(sc, B, K, tid, tmp);
  const int Bp = B * P;
  for (int b = 0; b < Bp; ++b) {
    sg.fill_row(xs + (size_t)b * Kp, sc, b / P, b % P, K, tid);
    for (int i = K + tid; i < Kp; i += 256) xs[(size_t)b * Kp + i] = 0;
  }
  __syncthreads();
  float acc[J][MB];
#pragma unroll
  for (int j = 0; j < J; ++j)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[j][b] = 0.f;
  const int nch = Kp / KC;
  for (int c0 = 0; c0 < nch; c0 += GS_D) {
#pragma unroll
    for (int d = 0; d < GS_D; ++d) {
      const int c = c0 + d;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int sl = c * SPC + wave + 4 * u;
#pragma unroll
        for (int b = 0; b < MB; ++b)
          if (b < Bp) {
            const u32x4 xv = *(const u32x4*)(xs + (size_t)b * Kp + sl * 64 + c8 * 8);
#pragma unroll
            for (int j = 0; j < J; ++j) acc[j][b] = dot8(wv[d][u][j], xv, acc[j][b]);
          }
      }
      issue(d, c + GS_D);  // past the last chunk: reads past K, zero and unused
    }
  }
  // reduce over the 8 lanes of a row, then over the 4 waves; red row r8 + 8 j
  // is this lane's row j (paired: rows 0-15 gate, 16-31 their up partners)
#pragma unroll
  for (int j = 0; j < J; ++j)
#pragma unroll
    for (int b = 0; b < MB; ++b) {
      float v = acc[j][b];
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 4);
      acc[j][b] = v;
    }
  if (c8 == 0)
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int b = 0; b < MB; ++b) red[(wave * ROWS + r8 + 8 * j) * MB + b] = acc[j][b];
  __syncthreads();
  if constexpr (PAIR) {
    if (tid < 16 * GV_MB) {
      const int fl = tid / GV_MB, b = tid % GV_MB;
      if (b < B) {
        float g = 0.f, u = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
          for (int q = 0; q < P; ++q) {
            g += red[(w * ROWS + fl) * MB + b * P + q];
            u += red[(w * ROWS + 16 + fl) * MB + b * P + q];
          }
        epi(b, blockIdx.x * 16 + fl, g, u);
      }
    }
  } else {
    if (tid < ROWS * GV_MB) {
      const int row = tid / GV_MB, b = tid % GV_MB;
      const int nn = blockIdx.x * ROWS + row;
      if (b < B && nn < N) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
          for (int q = 0; q < P; ++q) v += red[(w * ROWS + row) * MB + b * P + q];
        epi(b, nn, v);
      }
    }
  }
}

// the streaming kernel's input rows: B * Kp bf16 in LDS
inline int stream_kp(int K) { return (K + GS_KC * GS_D - 1) / (GS_KC * GS_D) * (GS_KC * GS_D); }
// up to 48 KB the kernel runs several workgroups per CU; up to 96 KB (four
// d_ff-wide rows) one, and the grid then takes 16-row workgroups once 256 of
// them fill the CUs
constexpr size_t GS_LDS_SHARED = 48 * 1024, GS_LDS_MAX = 96 * 1024;
inline bool use_stream(int K, int B) { return K >= GS_KC && (size_t)B * stream_kp(K) * 2 <= GS_LDS_MAX; }
// dynamic LDS above the 64 KB default needs the kernel's attribute raised
template <class F>
hipError_t allow_lds(F* kernel, size_t bytes) {
  if (bytes <= 64 * 1024) return hipSuccess;
  return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}
// the buffer resource's size and the offsets (up to 16 slabs past Kp) fit in 31 bits
inline bool stream_offsets_ok(const WOperand& W, int Kp) {
  return (size_t)(Kp / 64 + 16) * W.nblk * SLAB_N * 64 * 2 < (1ull << 31);
}

// B logical rows, each staged as P rows (P = 2: split operands), B * P <= MB
template <int MB, int P, class Stage, class Epi>
hipError_t gemv_stream(const Stage& sg, const WOperand& W, int N, int K, int B, const Epi& epi, hipStream_t s) {
  const int Kp = stream_kp(K);
  const size_t lds = (size_t)B * P * Kp * 2;
  if (!stream_offsets_ok(W, Kp)) return hipErrorInvalidValue;
  if ((N + 15) / 16 >= (lds > GS_LDS_SHARED ? 256 : 512)) {
    hipError_t e = allow_lds(gemv_stream_kernel<16, false, MB, P, Stage, Epi>, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((gemv_stream_kernel<16, false, MB, P, Stage, Epi>), dim3((N + 15) / 16), dim3(256), lds, s, sg,
                       W.p, W.nblk, N, K, B, Kp, epi);
  } else {
    hipError_t e = allow_lds(gemv_stream_kernel<8, false, MB, P, Stage, Epi>, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((gemv_stream_kernel<8, false, MB, P, Stage, Epi>), dim3((N + 7) / 8), dim3(256), lds, s, sg,
                       W.p, W.nblk, N, K, B, Kp, epi);
  }
  return hipGetLastError();
}

template <int MB, int P, class Stage, class Epi>
hipError_t gemv_chunk(const Stage& sg, const WOperand& W, int N, int K, int B, const Epi& epi, hipStream_t s) {
  if ((N + 15) / 16 >= 512)
    hipLaunchKernelGGL((gemv_chunk_kernel<16, MB, P, Stage, Epi>), dim3((N + 15) / 16), dim3(256), 0, s, sg, W.p,
                       W.nblk, N, K, B, epi);
  else
    hipLaunchKernelGGL((gemv_chunk_kernel<8, MB, P, Stage, Epi>), dim3((N + 7) / 8), dim3(256), 0, s, sg, W.p, W.nblk,
                       N, K, B, epi);
  return hipGetLastError();
}

inline bool gemv_args_ok(const WOperand& W, int N, int K, int B) {
  return B > 0 && B <= GV_MB && K % 64 == 0 && N > 0 && W.nblk * SLAB_N >= (N + 15) / 16 * 16;
}

// parts = 1: one bf16 row per sequence (up to 4 staged rows); parts = 2: hi
// and lo rows (up to 8)
template <class Stage, class Epi>
hipError_t gemv(const Stage& sg, const WOperand& W, int N, int K, int B, int parts, const Epi& epi, hipStream_t s) {
  if (!gemv_args_ok(W, N, K, B) || parts < 1 || parts > 2) return hipErrorInvalidValue;
  if (parts == 2)
    return use_stream(K, 2 * B) ? gemv_stream<2 * GV_MB, 2>(sg, W, N, K, B, epi, s)
                                : gemv_chunk<2 * GV_MB, 2>(sg, W, N, K, B, epi, s);
  return use_stream(K, B) ? gemv_stream<GV_MB, 1>(sg, W, N, K, B, epi, s) : gemv_chunk<GV_MB, 1>(sg, W, N, K, B, epi, s);
}

// packed QKV row of true dimension d of a head (the packing keeps every
// rotary pair (d, d + dh/2) in one 64-row group, 32 rows apart)
__device__ __forceinline__ int packed_row_of_dim(int d, int dh) {
  const int half = dh / 2;
  return d < half ? (d / 32) * 64 + d % 32 : ((d - half) / 32) * 64 + 32 + (d - half) % 32;
}

// One (b, h, split): keys [split*ATT_KC, min(pos+1, (split+1)*ATT_KC)).
// qkv [B][qkv_n] fp32 in the packed row order; caches [B][Hkv][L_cap][DH].
template <int DH>
__global__ __launch_bounds__(256) void attn_decode_kernel(const float* __restrict__ qkv, int qkv_n,
                                                          const float* __restrict__ rope_cos,
                                                          const float* __restrict__ rope_sin, bf16_t* kc, bf16_t* vc,
                                                          int L_cap, int pos, int B, int H, int Hkv, float scale_log2,
                                                          int nsplit, float* __restrict__ part) {
  constexpr int DL = DH / 8;  // dims per lane (8 lanes per key)
  __shared__ float sq[DH];
  __shared__ __attribute__((aligned(16))) bf16_t knew[DH], vnew[DH];
  __shared__ float wm[4], wl[4];
  __shared__ float wo[4][DH];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x % nsplit, bh = blockIdx.x / nsplit, h = bh % H, b = bh / H;
  const int hk = h / (H / Hkv);
  const int half = DH / 2;
  const float* row = qkv + (size_t)b * qkv_n;
  const bool last = (split + 1) * ATT_KC > pos;
  // q (and for the split holding pos, the new key and value) after RoPE, bf16-rounded as the prefill stores them
  if (tid < DH) {
    const int d = tid;
    const float* qh = row + (size_t)h * DH;
    const float* kh = row + (size_t)(H + hk) * DH;
    const float* vh = row + (size_t)(H + Hkv + hk) * DH;
    const int dp = d < half ? d + half : d - half;
    float qv = qh[packed_row_of_dim(d, DH)], kv = kh[packed_row_of_dim(d, DH)];
    if (rope_cos) {
      const int i = d < half ? d : d - half;
      const float c = rope_cos[(size_t)pos * half + i], s = rope_sin[(size_t)pos * half + i];
      const float qp = qh[packed_row_of_dim(dp, DH)], kp = kh[packed_row_of_dim(dp, DH)];
      qv = d < half ? qv * c - qp * s : qv * c + qp * s;
      kv = d < half ? kv * c - kp * s : kv * c + kp * s;
    }
    sq[d] = bf2f(f2bf(qv)) * scale_log2;
    if (last) {
      knew[d] = f2bf(kv);
      vnew[d] = f2bf(vh[packed_row_of_dim(d, DH)]);
      // one writer per KV head appends the token to the cache
      if (h % (H / Hkv) == 0) {
        kc[(((size_t)b * Hkv + hk) * L_cap + pos) * DH + d] = knew[d];
        vc[(((size_t)b * Hkv + hk) * L_cap + pos) * DH + d] = vnew[d];
      }
    }
  }
  __syncthreads();
  const int g = lane >> 3, i8 = lane & 7;
  float q[DL];
#pragma unroll
  for (int e = 0; e < DL; ++e) q[e] = sq[i8 * DL + e];
  // rounds of 32 keys (8 per wave, 8 lanes per key); every key of this
  // lane's rounds is loaded before any is used -- one round trip to memory,
  // not one per round.  Keys past the split's end load its last key (in
  // bounds) and are masked.  In the split holding pos, every lane whose key
  // index is pos or beyond takes the token's own key and value from LDS: the
  // workgroup appending them to the cache may not have run yet, and the
  // masked lanes' weight of zero must multiply a finite value (the cache
  // rows from pos on may hold anything, NaN included).
  constexpr int R = ATT_KC / 32, C = DL / 8;
  const int kbeg = split * ATT_KC, kend = min(pos + 1, kbeg + ATT_KC);
  const bf16_t* kb = kc + ((size_t)b * Hkv + hk) * L_cap * DH;
  const bf16_t* vb = vc + ((size_t)b * Hkv + hk) * L_cap * DH;
  u32x4 kw[R][C], vw[R][C];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = min(kbeg + r * 32 + wave * 8 + g, kend - 1);
#pragma unroll
    for (int c = 0; c < C; ++c) {
      kw[r][c] = *(const u32x4*)(kb + (size_t)j * DH + i8 * DL + c * 8);
      vw[r][c] = *(const u32x4*)(vb + (size_t)j * DH + i8 * DL + c * 8);
    }
  }
  float sd[R];
  float m = -INFINITY;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = kbeg + r * 32 + wave * 8 + g;
    if (last && j >= pos) {
#pragma unroll
      for (int c = 0; c < C; ++c) {
        kw[r][c] = *(const u32x4*)(knew + i8 * DL + c * 8);
        vw[r][c] = *(const u32x4*)(vnew + i8 * DL + c * 8);
      }
    }
    float sdot = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        sdot = fmaf(q[c * 8 + 2 * t], bf_lo(kw[r][c][t]), sdot);
        sdot = fmaf(q[c * 8 + 2 * t + 1], bf_hi(kw[r][c][t]), sdot);
      }
    sdot += __shfl_xor(sdot, 1);
    sdot += __shfl_xor(sdot, 2);
    sdot += __shfl_xor(sdot, 4);
    sd[r] = j < kend ? sdot : -INFINITY;
    m = fmaxf(m, sd[r]);
  }
  // this lane group's keys against their own maximum (none valid: l = o = 0)
  const float mu = m == -INFINITY ? 0.f : m;
  float l = 0.f, o[DL];
#pragma unroll
  for (int e = 0; e < DL; ++e) o[e] = 0.f;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const float p = exp2f(sd[r] - mu);
    l += p;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        o[c * 8 + 2 * t] = fmaf(p, bf_lo(vw[r][c][t]), o[c * 8 + 2 * t]);
        o[c * 8 + 2 * t + 1] = fmaf(p, bf_hi(vw[r][c][t]), o[c * 8 + 2 * t + 1]);
      }
  }
  // combine the 8 key groups of the wave (lanes 8 apart share dims)
#pragma unroll
  for (int off = 8; off < 64; off <<= 1) {
    const float mo = __shfl_xor(m, off), lo = __shfl_xor(l, off);
    const float mn = fmaxf(m, mo);
    const float a = (m == -INFINITY) ? 0.f : exp2f(m - mn), ao = (mo == -INFINITY) ? 0.f : exp2f(mo - mn);
    l = l * a + lo * ao;
#pragma unroll
    for (int e = 0; e < DL; ++e) o[e] = o[e] * a + __shfl_xor(o[e], off) * ao;
    m = mn;
  }
  if (lane < 8) {
#pragma unroll
    for (int e = 0; e < DL; ++e) wo[wave][i8 * DL + e] = o[e];
    if (lane == 0) {
      wm[wave] = m;
      wl[wave] = l;
    }
  }
  __syncthreads();
  float* out = part + (((size_t)b * H + h) * nsplit + split) * (2 + DH);
  if (tid < DH) {
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) mx = fmaxf(mx, wm[w]);
    float lsum = 0.f, osum = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float a = wm[w] == -INFINITY ? 0.f : exp2f(wm[w] - mx);
      lsum += a * wl[w];
      osum += a * wo[w][tid];
    }
    out[2 + tid] = osum;
    if (tid == 0) {
      out[0] = mx;
      out[1] = lsum;
    }
  }
}

// o[b][h*dh + d] = bf16(sum_s 2^(m_s - m) o_s[d] / sum_s 2^(m_s - m) l_s) over
// the split-key partials part[B][H][nsplit][2 + dh]: one workgroup per
// (b, h), one thread per dimension.  Every split's values are loaded before
// any is combined, without branches (indices past the last split repeat it
// and get weight zero): per-element branches around the loads made the
// compiler wait for each load in turn.
template <int DH>
__global__ __launch_bounds__(DH) void combine_kernel(const float* __restrict__ part, int nsplit,
                                                     bf16_t* __restrict__ o) {
  constexpr int MAXS = 16;
  const int bh = blockIdx.x, d = threadIdx.x, stride = 2 + DH;
  const float* p = part + (size_t)bh * nsplit * stride;
  float m = -INFINITY, l = 0.f, acc = 0.f;
  for (int s0 = 0; s0 < nsplit; s0 += MAXS) {
    float ms[MAXS], ls[MAXS], os[MAXS];
#pragma unroll
    for (int s = 0; s < MAXS; ++s) {
      const int si = min(s0 + s, nsplit - 1);
      ms[s] = p[si * stride];
      ls[s] = p[si * stride + 1];
      os[s] = p[si * stride + 2 + d];
    }
#pragma unroll
    for (int s = 0; s < MAXS; ++s)
      if (s0 + s >= nsplit) ms[s] = -INFINITY;
    float mn = m;
#pragma unroll
    for (int s = 0; s < MAXS; ++s) mn = fmaxf(mn, ms[s]);
    const float r = m == -INFINITY ? 0.f : exp2f(m - mn);
    l *= r;
    acc *= r;
#pragma unroll
    for (int s = 0; s < MAXS; ++s) {
      const float w = ms[s] == -INFINITY ? 0.f : exp2f(ms[s] - mn);
      l += w * ls[s];
      acc += w * os[s];
    }
    m = mn;
  }
  o[(size_t)bh * DH + d] = f2bf(acc / l);
}

}  // namespace

hipError_t decode_qkv(const float* h, const float* g, float eps, const WOperand& W, float* raw, int B, int N, int K,
                      hipStream_t s, int parts) {
  return gemv(StageNorm{h, g, eps}, W, N, K, B, parts, EpiRaw{raw, N}, s);
}

size_t decode_attention_scratch(int B, int H, int dh, int pos) {
  return (size_t)B * H * (pos / ATT_KC + 1) * (2 + dh) * sizeof(float);
}

hipError_t decode_attention(const float* qkv, int qkv_n, const float* rope_cos, const float* rope_sin, bf16_t* kc,
                            bf16_t* vc, int L_cap, int pos, int B, int H, int Hkv, int dh, float* part, bf16_t* o,
                            hipStream_t s) {
  if (B <= 0 || H % Hkv || pos < 0 || pos >= L_cap) return hipErrorInvalidValue;
  const int ns = pos / ATT_KC + 1;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)dh);
  if (dh == 128)
    hipLaunchKernelGGL((attn_decode_kernel<128>), dim3(B * H * ns), dim3(256), 0, s, qkv, qkv_n, rope_cos, rope_sin,
                       kc, vc, L_cap, pos, B, H, Hkv, scale_log2, ns, part);
  else if (dh == 64)
    hipLaunchKernelGGL((attn_decode_kernel<64>), dim3(B * H * ns), dim3(256), 0, s, qkv, qkv_n, rope_cos, rope_sin,
                       kc, vc, L_cap, pos, B, H, Hkv, scale_log2, ns, part);
  else
    return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (dh == 128)
    hipLaunchKernelGGL((combine_kernel<128>), dim3(B * H), dim3(128), 0, s, part, ns, o);
  else
    hipLaunchKernelGGL((combine_kernel<64>), dim3(B * H), dim3(64), 0, s, part, ns, o);
  return hipGetLastError();
}

hipError_t decode_oproj(const bf16_t* o, int K, const WOperand& W, float* h, int B, int N, hipStream_t s) {
  return gemv(StageCopy{o, K, 0}, W, N, K, B, 1, EpiAdd{h, N}, s);
}

namespace {
// the gate/up product with SwiGLU: B logical rows staged P times each; the
// gated activation row b at a + b * P * fpad, its remainder (P = 2) fpad on
template <int MB, int P>
hipError_t decode_up_impl(const float* h, const float* g, float eps, const WOperand& W, int fpad, float* gu, bf16_t* a,
                          int B, int K, hipStream_t s) {
  const int N = 2 * fpad;
  const EpiGated epi{a, P * fpad, (P - 1) * fpad};
  if (use_stream(K, B * P)) {
    // SwiGLU in the product's epilogue, 16 features per workgroup
    const int Kp = stream_kp(K);
    if (!stream_offsets_ok(W, Kp)) return hipErrorInvalidValue;
    const size_t lds = (size_t)B * P * Kp * 2;
    hipError_t e = allow_lds(gemv_stream_kernel<32, true, MB, P, StageNorm, EpiGated>, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((gemv_stream_kernel<32, true, MB, P, StageNorm, EpiGated>), dim3(fpad / 16), dim3(256), lds, s,
                       StageNorm{h, g, eps}, W.p, W.nblk, N, K, B, Kp, epi);
    return hipGetLastError();
  }
  hipError_t e = gemv_chunk<MB, P>(StageNorm{h, g, eps}, W, N, K, B, EpiRaw{gu, N}, s);
  if (e != hipSuccess) return e;
  const int n = B * fpad;
  hipLaunchKernelGGL(swiglu_kernel, dim3((n + 255) / 256), dim3(256), 0, s, gu, fpad, B, a, epi.ld, epi.lo);
  return hipGetLastError();
}
}  // namespace

hipError_t decode_up(const float* h, const float* g, float eps, const WOperand& W, int fpad, float* gu, bf16_t* a,
                     int B, int K, hipStream_t s, int parts) {
  if (!gemv_args_ok(W, 2 * fpad, K, B) || fpad % 64 || parts < 1 || parts > 2) return hipErrorInvalidValue;
  return parts == 2 ? decode_up_impl<2 * GV_MB, 2>(h, g, eps, W, fpad, gu, a, B, K, s)
                    : decode_up_impl<GV_MB, 1>(h, g, eps, W, fpad, gu, a, B, K, s);
}

hipError_t decode_down(const bf16_t* a, int fpad, const WOperand& W, float* h, int B, int N, hipStream_t s,
                       int parts) {
  if (parts < 1 || parts > 2) return hipErrorInvalidValue;
  return gemv(StageCopy{a, parts * fpad, (parts - 1) * fpad}, W, N, fpad, B, parts, EpiAdd{h, N}, s);
}

}  // namespace vla
