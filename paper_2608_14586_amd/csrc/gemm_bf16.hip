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

#include <type_traits>

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
//
// Epilogue paths.
//  * Direct: every lane writes its accumulators straight to memory (4-byte
//    stores); used by the fp32-out operator.
//  * SwiGLU forms its activation in the accumulators (a wave's columns are
//    whole (gate, up) groups) and parks only the activation, in one phase.
//  * The fp32 residual epilogue adds the residual in the accumulators and
//    stores from them (EpiResidual).
//  * Through LDS: once the K loop is done the slab buffers are free, so the
//    waves add the bias to their accumulators and park the fp32 tile in LDS
//    row-major, half of the wave rows (half the tile's rows) at a time, and
//    256-thread groups then walk it in 16-byte chunks: 16-byte bf16 stores,
//    and the rotary embedding plus the q / K / V / V^T scatter done
//    row-contiguously per head.
// drain<R, NC>() is the second half of the LDS path: T is an R x NC fp32
// piece of the parked tile (row stride NC), (m0, n0) its origin, tid the
// thread index in its 256-thread group.

__device__ __forceinline__ u32x4 pack8(const f32x4& a, const f32x4& b) {
  return u32x4{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]), pack_bf2(b[0], b[1]), pack_bf2(b[2], b[3])};
}

__device__ __forceinline__ f32x4 ld4(const float* p) { return *(const f32x4*)p; }

// the four bf16 values of words (w, w+1) of a packed chunk, widened
__device__ __forceinline__ f32x4 unpack_lo4(const u32x4& v, int w) {
  return f32x4{__uint_as_float(v[w] << 16), __uint_as_float(v[w] & 0xFFFF0000u), __uint_as_float(v[w + 1] << 16),
               __uint_as_float(v[w + 1] & 0xFFFF0000u)};
}

// Exact GELU z * Phi(z) with Phi(z) = erfc(-z / sqrt 2) / 2, erfc from the
// rational approximation of Abramowitz & Stegun 7.1.26 (|error| <= 1.5e-7,
// far below bf16 resolution); erfc of |x| is formed directly, so the negative
// tail does not cancel.  Arithmetic folded for the epilogue, which no MFMA
// work overlaps: t = 1 / (1 + p |z| / sqrt 2) is one FMA and the hardware
// reciprocal (1 ulp; an IEEE divide costs ten VALU instructions), the 1/2 of
// Phi sits in the polynomial's coefficients, and e^(-z^2 / 2) is one exp2.
__device__ __forceinline__ float gelu_as(float z) {
  const float t = __builtin_amdgcn_rcpf(fmaf(fabsf(z), 0.3275911f * 0.70710678118654752f, 1.f));
  // (a1 t + a2 t^2 + ... + a5 t^5) / 2
  const float hp =
      t * (0.127414796f + t * (-0.142248368f + t * (0.7107068705f + t * (-0.7265760135f + t * 0.5307027145f))));
  const float h = hp * __builtin_amdgcn_exp2f(z * (z * -0.72134752044448170f));  // erfc(|z| / sqrt 2) / 2
  return z * (z >= 0.f ? 1.f - h : h);
}

// silu(g) = g / (1 + e^-g), the division by the hardware reciprocal (1 ulp),
// as in the GELU: an IEEE divide costs ten VALU instructions per element of
// an epilogue that no MFMA work overlaps.  Large negative g: e^-g overflows
// to inf, whose reciprocal is 0, so the result is -0 as with the divide.
__device__ __forceinline__ float silu(float g) { return g * __builtin_amdgcn_rcpf(1.f + __expf(-g)); }

struct EpiStoreF32 {
  static constexpr bool kViaLds = false, kBig = true, kActInRegs = false, kDirect = false;
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

// C (bf16) = acc + bias, or gelu(acc + bias) when GELU (the bias is added to
// the accumulators before the tile is parked).
template <bool GELU>
struct EpiBF16 {
  static constexpr bool kViaLds = true, kBig = true, kActInRegs = false, kDirect = false;
  bf16_t* C;
  const float* bias;
  int ldc, M, N;
  __device__ __forceinline__ const float* park_bias() const { return bias; }
  __device__ __forceinline__ float op(float z) const { return GELU ? gelu_as(z) : z; }
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>&, int, int, int) const {}  // LDS path only
  // T: R x NC fp32 tile (row stride NC) at (m0, n0); 256 threads.
  template <int R, int NC>
  __device__ void drain(const float* T, int m0, int n0, int tid) const {
    constexpr int CH = NC / 8;  // 16-byte output chunks per row
    static_assert((R * CH) % 256 == 0 && 256 % CH == 0, "tile must split evenly over the workgroup");
    // a thread's columns are the same in every chunk it drains
    const int c8 = (tid % CH) * 8, gc = n0 + c8;
    if (gc >= N) return;
#pragma unroll 4
    for (int j = 0; j < R * CH / 256; ++j) {
      const int row = (tid + 256 * j) / CH, gr = m0 + row;
      if (gr >= M) continue;
      f32x4 x0 = ld4(T + row * NC + c8), x1 = ld4(T + row * NC + c8 + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x0[e] = op(x0[e]);
        x1[e] = op(x1[e]);
      }
      *(u32x4*)(C + (size_t)gr * ldc + gc) = pack8(x0, x1);
    }
  }
};
using EpiStoreBF16 = EpiBF16<false>;
using EpiGelu = EpiBF16<true>;

// H (fp32 residual) += acc + bias, with no park: each lane loads the
// residual of its accumulators behind the last K slab (the accumulator
// layout: 32 columns per lane half-row), adds it (the bias is already in the
// accumulators) and stores its values back.  4-byte accesses, whole 128-byte
// rows per instruction; no LDS round trip and no barriers.
struct EpiResidual {
  static constexpr bool kViaLds = true, kBig = false, kActInRegs = false, kDirect = true;
  float* H;
  const float* bias;
  int ldh, M, N;
  __device__ __forceinline__ const float* park_bias() const { return bias; }
  // One buffer resource over the wave's rows from r0 (rows past M read as
  // zero, stores to them are dropped), one lane offset; rows step by a scalar
  // offset and 32-column blocks by the immediate offset.  The row count goes
  // through readfirstlane: the clamp compiles to a vector med3, and a
  // descriptor word in a VGPR would make every access a per-lane (waterfall)
  // loop.
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_from(int r0, int nrows) const {
    const int rows = __builtin_amdgcn_readfirstlane(min(max(M - r0, 0), nrows));
    return __builtin_amdgcn_make_buffer_rsrc((void*)(H + (size_t)min(r0, M) * ldh), (short)0, rows * ldh * 4,
                                             0x00020000);
  }
  template <int TM, int TN>
  __device__ void load_acc(f32x16 (&hv)[TM][TN], int r0, int c0, int lane) const {
    const __amdgpu_buffer_rsrc_t rh = rows_from(r0, TM * 32);
    const int voff = (((lane >> 5) * 4) * ldh + c0 + (lane & 31)) * 4;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          hv[tm][tn][r] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
              rh, voff + tn * 128, (tm * 32 + (r >> 2) * 8 + (r & 3)) * ldh * 4, 0));
  }
  template <int TM, int TN>
  __device__ void store_acc(const f32x16 (&v)[TM][TN], int r0, int c0, int lane) const {
    const __amdgpu_buffer_rsrc_t rh = rows_from(r0, TM * 32);
    const int voff = (((lane >> 5) * 4) * ldh + c0 + (lane & 31)) * 4;
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      // columns past N would land in the next row: not stored
      if (c0 + tn * 32 + (lane & 31) >= N) continue;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // through a scalar: clang's bit cast of a vector element reads element 0
          const float x = v[tm][tn][r];
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), rh, voff + tn * 128,
                                                (tm * 32 + (r >> 2) * 8 + (r & 3)) * ldh * 4, 0);
        }
    }
  }
  template <int R, int NC>
  __device__ void drain(const float*, int, int, int) const {}
};

// Pairs tiles (2p, 2p+1) = (gate, up) of the same 32 features: out[M][N/2].
// lo > 0: the activation is also written as its bf16 remainder
// bf16(y - bf16(y)) at column lo + c, so that hi + lo carries y to 16
// significant bits into the down projection.
struct EpiSwiGLU {
  // the activation is formed in the accumulators: a wave's 64 columns are
  // one (gate, up) group, so a lane holds the gate and the up value of the
  // same feature, and only the activation (half the columns) is parked
  static constexpr bool kViaLds = true, kBig = true, kActInRegs = true, kDirect = false;
  __device__ __forceinline__ const float* park_bias() const { return nullptr; }
  bf16_t* out;
  int ldo, M, N, lo;
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>&, int, int, int) const {}  // LDS path only
  template <int R, int NC>
  __device__ void drain(const float* T, int m0, int n0, int tid) const {
    // R rows x NC/16 chunks of 8 output features (4 chunks per 64-column group)
    constexpr int CH = NC / 16;
    static_assert((R * CH) % 256 == 0, "tile must split evenly over the workgroup");
#pragma unroll
    for (int j = 0; j < R * CH / 256; ++j) {
      const int f = tid + 256 * j, row = f / CH, c = f % CH;
      const int gsel = c >> 2, w = (c & 3) * 8;  // 64-column group, offset inside its 32
      const int gr = m0 + row;
      if (gr >= M || n0 + gsel * 64 >= N) continue;
      const float* tr = T + row * NC + gsel * 64 + w;
      f32x4 g0 = ld4(tr), g1 = ld4(tr + 4), u0 = ld4(tr + 32), u1 = ld4(tr + 36);
      f32x4 y0, y1;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y0[e] = silu(g0[e]) * u0[e];
        y1[e] = silu(g1[e]) * u1[e];
      }
      bf16_t* dst = out + (size_t)gr * ldo + (n0 >> 1) + gsel * 32 + w;
      const u32x4 hi = pack8(y0, y1);
      *(u32x4*)dst = hi;
      if (lo) *(u32x4*)(dst + lo) = pack8(y0 - unpack_lo4(hi, 0), y1 - unpack_lo4(hi, 2));
    }
  }
  // Y: R x NC fp32 activations (row stride NC) of the tile at (m0, feature
  // n0 / 2); 256 threads, chunks of 8 features.
  template <int R, int NC>
  __device__ void drain_act(const float* Y, int m0, int n0, int tid) const {
    constexpr int CH = NC / 8;
    static_assert((R * CH) % 256 == 0 && 256 % CH == 0, "tile must split evenly over the workgroup");
    // a thread's features are the same in every chunk it drains
    const int c8 = (tid % CH) * 8, gc = (n0 >> 1) + c8;
    if (2 * gc >= N) return;
#pragma unroll 4
    for (int j = 0; j < R * CH / 256; ++j) {
      const int row = (tid + 256 * j) / CH, gr = m0 + row;
      if (gr >= M) continue;
      const f32x4 y0 = ld4(Y + row * NC + c8), y1 = ld4(Y + row * NC + c8 + 4);
      bf16_t* dst = out + (size_t)gr * ldo + gc;
      const u32x4 hi = pack8(y0, y1);
      *(u32x4*)dst = hi;
      if (lo) *(u32x4*)(dst + lo) = pack8(y0 - unpack_lo4(hi, 0), y1 - unpack_lo4(hi, 2));
    }
  }
};

// QKV projection: bias, rotary embedding of q and k (each 64-column group
// holds 32 first-half dims and their 32 second-half partners, see QkvArgs),
// scatter to q / K / V rows and to V^T.
struct EpiQKV {
  static constexpr bool kViaLds = true, kBig = false, kActInRegs = false, kDirect = false;
  QkvArgs q;
  int M;
  __device__ __forceinline__ const float* park_bias() const { return q.bias; }
  // column group p (multiple of 64) -> kind (0 q, 1 k, 2 v, 3 none), head, dim offset
  __device__ __forceinline__ void classify(int p, int& kind, int& head, int& r) const {
    const int dh = q.dh;
    if (p < q.H * dh) {
      kind = 0; head = p / dh; r = p % dh;
    } else if (p < (q.H + q.Hkv) * dh) {
      kind = 1; head = (p - q.H * dh) / dh; r = (p - q.H * dh) % dh;
    } else if (p < (q.H + 2 * q.Hkv) * dh) {
      kind = 2; head = (p - (q.H + q.Hkv) * dh) / dh; r = (p - (q.H + q.Hkv) * dh) % dh;
    } else {
      kind = 3; head = 0; r = 0;
    }
  }
  template <int TM, int TN>
  __device__ void operator()(const Acc<TM, TN>&, int, int, int) const {}  // LDS path only
  template <int R, int NC>
  __device__ void drain(const float* T, int m0, int n0, int tid) const {
    const int dh = q.dh, L = q.L;
    // R tokens x NC/64 column groups x 4 chunks of 8 dims
    constexpr int CH = NC / 16;
    static_assert(R % 16 == 0, "whole 16-token V^T chunks");
#pragma unroll 2
    for (int j = 0; j < (R * CH + 255) / 256; ++j) {
      const int f = tid + 256 * j, row = f / CH, gsel = (f % CH) >> 2, w = (f & 3) * 8;
      if ((R * CH) % 256 && f >= R * CH) break;
      const int gr = m0 + row, p = n0 + gsel * 64;
      int kind, head, r;
      classify(p, kind, head, r);
      if (gr >= M || kind == 3 || (kind == 2 && !q.v)) continue;
      const int c = r / 64;
      const int d1 = c * 32 + w, d2 = dh / 2 + c * 32 + w;
      const float* tr = T + row * NC + gsel * 64 + w;
      f32x4 x10 = ld4(tr), x11 = ld4(tr + 4), x20 = ld4(tr + 32), x21 = ld4(tr + 36);
      const int b = gr / L, pos = gr - b * L;
      if (kind < 2 && q.rope_cos) {
        const float* cp = q.rope_cos + (size_t)pos * (dh / 2) + d1;
        const float* sp = q.rope_sin + (size_t)pos * (dh / 2) + d1;
        const f32x4 c0 = ld4(cp), c1 = ld4(cp + 4), s0 = ld4(sp), s1 = ld4(sp + 4);
        const f32x4 y10 = x10 * c0 - x20 * s0, y11 = x11 * c1 - x21 * s1;
        const f32x4 y20 = x20 * c0 + x10 * s0, y21 = x21 * c1 + x11 * s1;
        x10 = y10; x11 = y11; x20 = y20; x21 = y21;
      }
      const int nh = kind == 0 ? q.H : q.Hkv;
      bf16_t* dst = (kind == 0 ? q.q : (kind == 1 ? q.k : q.v)) + (((size_t)b * nh + head) * L + pos) * dh;
      *(u32x4*)(dst + d1) = pack8(x10, x11);
      *(u32x4*)(dst + d2) = pack8(x20, x21);
    }
    // V^T: one (dim, 16 consecutive tokens) chunk per item.  Inside every
    // 16-token group the columns hold the keys in the order
    // [0-3, 8-11, 4-7, 12-15] (bits 2 and 3 of the key index swapped), the
    // order in which the attention's PV product consumes them.
    for (int gsel = 0; gsel < NC / 64; ++gsel) {
      int kind, head, r;
      const int p = n0 + gsel * 64;
      classify(p, kind, head, r);
      if (kind != 2) continue;
      const int c = r / 64;
      // R / 16 token chunks x 64 columns, strided over the 256 threads
#pragma unroll
      for (int f = tid; f < R * 4; f += 256) {
        const int col = f & 63, t16 = (f >> 6) * 16;
        const int gr0 = m0 + t16;
        if (gr0 >= M) continue;
        const int d = (col < 32) ? c * 32 + col : dh / 2 + c * 32 + (col - 32);
        float v[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = T[(t16 + e) * NC + gsel * 64 + col];
        const int b0 = gr0 / L, pos0 = gr0 - b0 * L;
        bf16_t* row = q.vt + (((size_t)b0 * q.Hkv + head) * dh + d) * q.ldvt;
        if (gr0 + 15 < M && pos0 + 15 < L && (pos0 & 15) == 0 && (q.ldvt & 15) == 0) {
          *(u32x4*)(row + pos0) = u32x4{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[8], v[9]), pack_bf2(v[10], v[11])};
          *(u32x4*)(row + pos0 + 8) = u32x4{pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]), pack_bf2(v[12], v[13]), pack_bf2(v[14], v[15])};
        } else {
          int bb = b0, pp = pos0;
          for (int e = 0; e < 16 && gr0 + e < M; ++e) {
            const int sw = (pp & ~12) | ((pp & 4) << 1) | ((pp & 8) >> 1);
            q.vt[(((size_t)bb * q.Hkv + head) * dh + d) * q.ldvt + sw] = f2bf(v[e]);
            if (++pp == L) {
              pp = 0;
              ++bb;
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
// With three weight slots (WS = 3) W runs two slabs ahead of A: the per-slab
// wait leaves the newest W slab in flight across the barrier (vmcnt(B_INST)
// and s_barrier; __syncthreads would wait for every load), and past the last
// slab the W issue repeats the last slab into a free slot, so that every
// issue is unconditional.

__device__ __forceinline__ void buffer_load_lds16(__amdgpu_buffer_rsrc_t r, void* lds, unsigned voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, 0, 0, 0);
}

// K is the k extent of A, Kw that of W (K = Kw or 2 Kw): A's column blocks
// [0, Kw) and [Kw, 2 Kw) multiply the same W, so an operand carried as
// a hi + lo pair of bf16 values side by side ([M][2 Kw]) yields
// hi * W^T + lo * W^T in one accumulator.
template <int BM, int BN, int WM, int WN, int NW, bool WT, class Epi, int WS = 2>
__global__ __launch_bounds__(64 * NW) void gemm_bf16_dma_kernel(const bf16_t* __restrict__ A, int lda, WOperand W,
                                                                int M, int N, int K, int Kw, Epi epi) {
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int WAVES_N = BN / WN;
  static_assert((BM / WM) * (BN / WN) == NW, "wave grid must cover the tile");
  constexpr int ROWB = BK * 2;                             // bytes per LDS row (128)
  constexpr int A_INST = BM / (8 * NW), B_INST = BN / (8 * NW);  // 1 KB loads per wave per slab
  static_assert(A_INST >= 1 && B_INST >= 1, "tile too small for the wave count");
  // WS = 2: two slabs of A and W side by side; WS = 3: two A slots, then
  // three W slots, so that W runs two slabs ahead
  static_assert(WS == 2 || WS == 3, "two or three weight slots");
  __shared__ __attribute__((aligned(1024))) char smem[(2 * BM + WS * BN) * ROWB];
  auto a_slot = [&](int i) -> char* { return WS == 2 ? smem + i * (BM + BN) * ROWB : smem + i * BM * ROWB; };
  auto w_slot = [&](int i) -> char* {
    return WS == 2 ? smem + i * (BM + BN) * ROWB + BM * ROWB : smem + (2 * BM + i * BN) * ROWB;
  };

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index through a scalar register: the LDS DMA destinations (M0)
  // and the wave's fragment row offsets stay scalar arithmetic (fewer VGPRs
  // and VALU instructions).  A/B, us: SwiGLU 332.1 -> 327.7, residual 80.6
  // -> 79.9; with three weight slots also QKV 200.4 -> 198.9 and GELU 72.2
  // -> 70.7.
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  // W: row-major rows from n0 on, or the whole packed matrix (every block of
  // a tile lies inside it: the packing pads N to whole 256-row pairs)
  const int ldw = W.ld, nblk = W.nblk;
  const __amdgpu_buffer_rsrc_t rb =
      WT ? __builtin_amdgcn_make_buffer_rsrc((void*)W.p, (short)0, (int)((size_t)nblk * SLAB_N * Kw * 2), 0x00020000)
         : __builtin_amdgcn_make_buffer_rsrc((void*)(W.p + (size_t)n0 * ldw), (short)0,
                                             (int)((size_t)(N - n0) * ldw * 2), 0x00020000);

  // this lane's slot in each 1 KB load: row (lane / 8) of the 8-row group,
  // LDS chunk (lane % 8) holding global chunk (lane % 8) ^ key(tile row)
  const int lrow = lane >> 3, lslot = lane & 7;
  auto issue_a = [&](int k0, int ai) {
    char* base = a_slot(ai);
#pragma unroll
    for (int j = 0; j < A_INST; ++j) {
      const int row = (wave * A_INST + j) * 8 + lrow;
      const int ch = lslot ^ ((row >> 1) & 7);
      buffer_load_lds16(ra, base + (wave * A_INST + j) * 1024, (unsigned)((row * lda + k0 + ch * 8) * 2));
    }
  };
  auto issue_w = [&](int k0, int wi) {
    char* base = w_slot(wi);
    const int kw0 = k0 >= Kw ? k0 - Kw : k0;  // the same W slab for both column blocks of A
#pragma unroll
    for (int j = 0; j < B_INST; ++j) {
      const int row = (wave * B_INST + j) * 8 + lrow;
      const int ch = lslot ^ ((row >> 1) & 7);
      // packed: the slab of 128 rows x 64 k is one contiguous 16 KB block
      const int grow = n0 + row;  // tiles need not start on a 128-row block
      const unsigned off =
          WT ? (unsigned)((((kw0 / BK) * nblk + grow / SLAB_N) * SLAB_N + grow % SLAB_N) * ROWB + ch * 16)
             : (unsigned)((row * ldw + kw0 + ch * 8) * 2);
      buffer_load_lds16(rb, base + (wave * B_INST + j) * 1024, off);
    }
  };
  auto issue = [&](int k0, int buf) {
    issue_a(k0, buf);
    issue_w(k0, buf);
  };

  Acc<TM, TN> acc;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc.v[tm][tn][r] = 0.f;

  const int fi = lane & 31, fh = lane >> 5;
  const int a_row0 = (wm * WM + fi) * ROWB, b_row0 = (wn * WN + fi) * ROWB;
  const int key = (fi >> 1) & 7;
  bf16x8 fa[2][TM], fb[2][TN];
  // fragments of k16 step ks of slab s (buffer s & 1) into register slot `slot`
  // (W slab s lies in W slot ws: s & 1 for two slots, s % 3 for three)
  auto frags = [&](int s, int ws, int ks, int slot) {
    const char* abase = a_slot(s & 1);
    const char* wbase = w_slot(ws);
    const int off = (((2 * ks + fh) ^ key) << 4);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) fa[slot][tm] = *(const bf16x8*)(abase + a_row0 + tm * 32 * ROWB + off);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) fb[slot][tn] = *(const bf16x8*)(wbase + b_row0 + tn * 32 * ROWB + off);
  };

  constexpr int GROUPS = NW / 4, RG = BM / 2 / GROUPS;
  // the 256-thread group (0 in a 4-wave workgroup)
  const int grp = NW > 4 ? tid >> 8 : 0, t = tid & 255;

  const int nk = K / BK;
  // the MFMAs of one k16 step from fragment slot `cur`
  auto step = [&](int cur) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        acc.v[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][tm], fb[cur][tn], acc.v[tm][tn], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  // the k16 steps of slab kt but its last (W slot ws; fragments of the first
  // step already loaded), each reading the next step's fragments before its
  // MFMAs (left alone, the scheduler sinks each read onto its first use)
  constexpr int KS = BK / 16, LAST = (KS - 1) & 1;
  auto head = [&](int kt, int ws) {
#pragma unroll
    for (int ks = 0; ks + 1 < KS; ++ks) {
      frags(kt, ws, ks + 1, (ks & 1) ^ 1);
      step(ks & 1);
    }
  };
  auto slab = [&](int kt, int ws) {
    head(kt, ws);
    step(LAST);
  };
  int wl = 0;  // W slot of the last slab
  if constexpr (WS == 2) {
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    frags(0, 0, 0, 0);
    for (int kt = 0; kt + 1 < nk; ++kt) {
      // the other buffer was last read before the previous slab's barrier
      issue((kt + 1) * BK, (kt + 1) & 1);
      slab(kt, kt & 1);
      // the next slab's loads; this wave's fragment reads are consumed
      __builtin_amdgcn_s_waitcnt(0x0F70);
      __syncthreads();
      frags(kt + 1, (kt + 1) & 1, 0, 0);
    }
    wl = (nk - 1) & 1;
  } else {
    // W slabs 0 and 1 ahead of A slab 0; past the last slab, W loads repeat
    // the last one (in bounds, into a free slot, never read).  The last k16
    // step of each slab runs after the slab barrier, from fragments read
    // before it, and so covers the latency of the next slab's first
    // fragment reads.
    issue_a(0, 0);
    issue_w(0, 0);
    issue_w(min(1, nk - 1) * BK, 1);
    __builtin_amdgcn_s_waitcnt((B_INST & 15) | ((B_INST >> 4) << 14) | 0x0070);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    frags(0, 0, 0, 0);
    int ws = 0;  // W slot of slab kt
    for (int kt = 0; kt + 1 < nk; ++kt) {
      // A slot (kt+1)&1 and W slot (kt+2)%3 (slab kt-1) were last read
      // before the previous barrier
      const int wn2 = ws == 0 ? 2 : ws - 1;
      issue_a((kt + 1) * BK, (kt + 1) & 1);
      issue_w(min(kt + 2, nk - 1) * BK, wn2);
      head(kt, ws);
      // A(kt+1) and W(kt+1) landed; W(kt+2) may stay in flight across the
      // barrier; every wave's reads of slab kt are done
      __builtin_amdgcn_s_waitcnt((B_INST & 15) | ((B_INST >> 4) << 14) | 0x0070);
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      ws = ws == 2 ? 0 : ws + 1;
      frags(kt + 1, ws, 0, 0);
      step(LAST);  // slab kt's last step
    }
    wl = ws;
  }
  // the last slab, peeled so that loads issued behind it are straight-line
  // code the compiler's wait counting can follow
  // the direct epilogue's residual, read behind the last slab's MFMAs
  f32x16 hv[Epi::kDirect ? TM : 1][Epi::kDirect ? TN : 1];
  if constexpr (Epi::kDirect) epi.template load_acc<TM, TN>(hv, m0 + wm * WM, n0 + wn * WN, lane);
  // the bias of this lane's accumulator columns, added before the tile is parked
  float pb[TN];
  const float* bias = nullptr;
  if constexpr (Epi::kViaLds) {
    bias = epi.park_bias();
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col = n0 + wn * WN + tn * 32 + (lane & 31);
      pb[tn] = (bias && col < N) ? bias[col] : 0.f;
    }
  }
  slab(nk - 1, wl);
  __builtin_amdgcn_s_waitcnt(0);
  if constexpr (Epi::kViaLds) {
    if (bias) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc.v[tm][tn][r] += pb[tn];
    }
  }

  if constexpr (Epi::kDirect) {
    // residual added in the accumulators and stored from them: no park
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc.v[tm][tn][r] = hv[tm][tn][r] + acc.v[tm][tn][r];
    epi.template store_acc<TM, TN>(acc.v, m0 + wm * WM, n0 + wn * WN, lane);
  } else if constexpr (Epi::kActInRegs) {
    // gate (tn even) and up (tn odd) of the same 32 features: park silu(g) u,
    // BM x BN/2 fp32, in one phase
    constexpr int YN = BN / 2, RY = BM / GROUPS;
    static_assert(WN % 64 == 0, "a wave's columns must be whole (gate, up) groups");
    static_assert(BM * YN * 4 <= sizeof(smem), "the activation tile must fit the slab buffers");
    float* Y = (float*)smem;
    __syncthreads();
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tp = 0; tp < TN / 2; ++tp)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          Y[(wm * WM + tm * 32 + acc_row(r, lane)) * YN + wn * (WN / 2) + tp * 32 + (lane & 31)] =
              silu(acc.v[tm][2 * tp][r]) * acc.v[tm][2 * tp + 1][r];
    __syncthreads();
    epi.template drain_act<RY, YN>(Y + grp * RY * YN, m0 + grp * RY, n0, t);
  } else if constexpr (Epi::kViaLds) {
    // Park one wave row (BM/2 x BN fp32) at a time in the idle slab buffers;
    // 256-thread groups then drain BM/4 (8 waves) or BM/2 (4 waves) rows each.
    constexpr int WR = BM / WM, HR = WR / 2;  // wave rows, parked per half
    static_assert(WR % 2 == 0, "an even number of wave rows");
    static_assert((BM / 2) * BN * 4 <= sizeof(smem), "half tile must fit the slab buffers");
    float* T = (float*)smem;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      __syncthreads();
      if (wm / HR == h) {
        const int r0 = (wm % HR) * WM;
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              T[(r0 + tm * 32 + acc_row(r, lane)) * BN + wn * WN + tn * 32 + (lane & 31)] = acc.v[tm][tn][r];
      }
      __syncthreads();
      epi.template drain<RG, BN>(T + grp * RG * BN, m0 + h * (BM / 2) + grp * RG, n0, t);
    }
  } else {
    epi(acc, m0 + wm * WM, n0 + wn * WN, lane);
  }
}

// A [M][a_parts * K]: a_parts column blocks of K, each multiplied by the
// same W [N][K] into one accumulator (2: a hi + lo operand pair).
template <bool WT, class Epi>
hipError_t launch(const bf16_t* A, int lda, const WOperand& W, int M, int N, int K, const Epi& epi, hipStream_t s,
                  int a_parts = 1) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % BK != 0 || lda % 8 != 0 || a_parts < 1 || a_parts > 2 || lda < a_parts * K) return hipErrorInvalidValue;
  if (WT) {
    // every 256-column tile inside the packing, 32-bit byte offsets
    if (W.nblk <= 0 || W.nblk % 2 || W.nblk * SLAB_N < N || (size_t)W.nblk * SLAB_N * K * 2 >= (1u << 31))
      return hipErrorInvalidValue;
  } else {
    if (W.ld % 8 != 0 || W.ld < K || (size_t)256 * W.ld * 2 >= (1u << 31)) return hipErrorInvalidValue;
  }
  // byte offsets inside a tile's buffer resource are 32-bit
  if ((size_t)256 * lda * 2 >= (1u << 31)) return hipErrorInvalidValue;
  // 256x256 tiles (8 waves of 128x64) once they fill the chip at least twice;
  // 64x128 tiles (4 waves of 32x64, 48 KB of LDS, up to three workgroups per
  // CU) when 128x128 tiles would fill at most half of one round of workgroup
  // slots (two per CU; measured: O-projection and down at M = 1024 4-6%
  // faster, a 288-tile grid 7% slower); otherwise 128x128 tiles (4 waves of
  // 64x64, two workgroups per CU)
  // 8-wave tiles at one workgroup per CU where they fill whole rounds: QKV
  // 256x192 (waves of 64x96) or 192x384 (96x96), GELU 192x256 (96x64).
  // The 256x256, 192x256 and 256x192 tiles keep three weight slabs in LDS (W
  // two slabs ahead, 160, 144 and 136 KB), and so do the 128x128 residual
  // tiles (80 KB, still two workgroups per CU).  A/B, us: gate/up 330.5 ->
  // 328.4, ViT fc1 71.1 -> 69.4; with each slab's last k16 step after the
  // barrier also QKV 196.6 -> 190.7, O-projection 79.8 -> 77.3, down 193.9 ->
  // 184.9, ViT fc2 68.7 -> 64.9.
  auto rounds_of = [&](int bm, int bn) -> long {
    if (N % bn) return 0;
    const long t = (long)((M + bm - 1) / bm) * (N / bn);
    return t >= 256 && t % 256 == 0 ? t : 0;
  };
  if constexpr (std::is_same<Epi, EpiQKV>::value) {
    if (const long t = rounds_of(256, 192)) {
      hipLaunchKernelGGL((gemm_bf16_dma_kernel<256, 192, 64, 96, 8, WT, Epi, 3>), dim3((unsigned)t), dim3(512), 0, s,
                         A, lda, W, M, N, a_parts * K, K, epi);
      return hipGetLastError();
    }
    if (const long t = rounds_of(192, 384)) {
      hipLaunchKernelGGL((gemm_bf16_dma_kernel<192, 384, 96, 96, 8, WT, Epi>), dim3((unsigned)t), dim3(512), 0, s,
                         A, lda, W, M, N, a_parts * K, K, epi);
      return hipGetLastError();
    }
  }
  if constexpr (std::is_same<Epi, EpiGelu>::value) {
    if (const long t = rounds_of(192, 256)) {
      hipLaunchKernelGGL((gemm_bf16_dma_kernel<192, 256, 96, 64, 8, WT, Epi, 3>), dim3((unsigned)t), dim3(512), 0, s,
                         A, lda, W, M, N, a_parts * K, K, epi);
      return hipGetLastError();
    }
  }
  const long tiles256 = (long)((M + 255) / 256) * ((N + 255) / 256);
  const long tiles128 = (long)((M + 127) / 128) * ((N + 127) / 128);
  bool big = false;
  if constexpr (Epi::kBig) {
    if (tiles256 >= 512) {
      big = true;
      int grid = ((M + 255) / 256) * ((N + 255) / 256);
      hipLaunchKernelGGL((gemm_bf16_dma_kernel<256, 256, 128, 64, 8, WT, Epi, 3>), dim3(grid), dim3(512), 0, s, A, lda,
                         W, M, N, a_parts * K, K, epi);
    }
  }
  if (!big && 2 * tiles128 <= 512) {
    big = true;
    int grid = ((M + 63) / 64) * ((N + 127) / 128);
    hipLaunchKernelGGL((gemm_bf16_dma_kernel<64, 128, 32, 64, 4, WT, Epi>), dim3(grid), dim3(256), 0, s, A, lda, W,
                       M, N, a_parts * K, K, epi);
  }
  if (!big) {
    int grid = ((M + 127) / 128) * ((N + 127) / 128);
    if constexpr (std::is_same<Epi, EpiResidual>::value)
      hipLaunchKernelGGL((gemm_bf16_dma_kernel<128, 128, 64, 64, 4, WT, Epi, 3>), dim3(grid), dim3(256), 0, s, A, lda,
                         W, M, N, a_parts * K, K, epi);
    else
      hipLaunchKernelGGL((gemm_bf16_dma_kernel<128, 128, 64, 64, 4, WT, Epi>), dim3(grid), dim3(256), 0, s, A, lda, W,
                         M, N, a_parts * K, K, epi);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_bf16_store_f32(const bf16_t* A, int lda, const bf16_t* W, int ldw, float* C, int ldc, int M, int N,
                               int K, hipStream_t s) {
  return launch<false>(A, lda, WOperand{W, ldw, 0}, M, N, K, EpiStoreF32{C, ldc, M, N}, s);
}

hipError_t gemm_bf16_residual(const bf16_t* A, int lda, const WOperand& W, float* H, int ldh, const float* bias, int M,
                              int N, int K, hipStream_t s, int a_parts) {
  // the residual epilogue addresses a wave's rows with 32-bit byte offsets
  if (N % 4 || ldh % 4 || (size_t)256 * ldh * 4 >= (1u << 31)) return hipErrorInvalidValue;
  return launch<true>(A, lda, W, M, N, K, EpiResidual{H, bias, ldh, M, N}, s, a_parts);
}

hipError_t gemm_bf16_swiglu(const bf16_t* A, int lda, const WOperand& W, bf16_t* out, int ldo, int M, int N, int K,
                            hipStream_t s, int a_parts, int lo_col) {
  if (N % 64 != 0) return hipErrorInvalidValue;
  if (ldo % 8 || lo_col % 8 || lo_col < 0 || (lo_col > 0 && (lo_col < N / 2 || ldo < lo_col + N / 2)))
    return hipErrorInvalidValue;
  return launch<true>(A, lda, W, M, N, K, EpiSwiGLU{out, ldo, M, N, lo_col}, s, a_parts);
}

hipError_t gemm_bf16_gelu(const bf16_t* A, int lda, const WOperand& W, bf16_t* out, int ldo, const float* bias, int M,
                          int N, int K, hipStream_t s) {
  if (N % 8 || ldo % 8) return hipErrorInvalidValue;
  return launch<true>(A, lda, W, M, N, K, EpiGelu{out, bias, ldo, M, N}, s);
}

hipError_t gemm_bf16_bias(const bf16_t* A, int lda, const WOperand& W, bf16_t* out, int ldo, const float* bias, int M,
                          int N, int K, hipStream_t s) {
  if (N % 8 || ldo % 8) return hipErrorInvalidValue;
  return launch<true>(A, lda, W, M, N, K, EpiStoreBF16{out, bias, ldo, M, N}, s);
}

hipError_t gemm_bf16_qkv(const bf16_t* A, int lda, const WOperand& W, const QkvArgs& qa, int M, int N, int K,
                         hipStream_t s, int a_parts) {
  if (qa.dh % 64 != 0 || N % 64 != 0) return hipErrorInvalidValue;
  return launch<true>(A, lda, W, M, N, K, EpiQKV{qa, M}, s, a_parts);
}

}  // namespace vla
