// Flash-style attention for gfx950 (bf16 MFMA, fp32 online softmax).
//
// One workgroup = 4 waves = 128 queries of one (batch, head); each wave owns
// 32 queries.  Keys advance in tiles of 64 staged in LDS: K as [key][dh] and
// V transposed as [dh][key], so every MFMA operand is a contiguous LDS read.
// The tiles move global -> LDS with buffer_load ... lds (no VGPRs, no
// ds_write) into a ring of stages, the 16-byte chunks of each row
// XOR-swizzled so that fragment reads hit every bank once per 16-lane phase;
// a barrier waits only for the tile about to be read (vmcnt(N)), so later
// tiles stay in flight across it.  Each stage is an LDS array of its own and
// the tile loop is unrolled over the stages, so the compiler can tell a
// stage's fragment reads from the DMA writes into the next stage and never
// drains the ring before them.  Key rows past L read as zero through the
// buffer resource; V^T columns past L are zeroed in LDS in the last tile.
//
// The scores are formed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16
// (A = K tile from LDS, B = the wave's Q held in registers).  In the 32x32
// accumulator layout each lane then holds 16 keys of ONE query, so a query's
// running max/sum needs a single cross-half exchange (lane ^ 32) instead of a
// 32-lane reduction, and the probabilities already sit where the PV product
// O^T = V^T P^T wants its B operand: a lane's 8 bf16 values for keys
// {16s + 4h + j, 16s + 8 + 4h + j : j < 4} feed k-step s directly.  V^T is
// stored with the keys of every 16-key group in the order
// [0-3, 8-11, 4-7, 12-15] (bits 2 and 3 of the key index swapped), so the A
// fragment of those same keys is one contiguous 16-byte read.  The softmax
// runs in base 2 with log2(e)/sqrt(dh) folded into one FMA per score.
//
// Causal tiles are masked per element only on the diagonal; a wave skips the
// MFMAs of key tiles entirely beyond its last query.  Causal query blocks are
// issued so that co-resident workgroups carry complementary amounts of work.

#include <math.h>

#include <type_traits>

#include "kernels.h"

namespace vla {
namespace {

constexpr int BQ = 128, BKV = 64;

// key index <-> stored V^T column: bits 2 and 3 swapped (an involution)
__device__ __forceinline__ int swap23(int t) { return (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1); }

__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t r, void* lds, unsigned voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, 0, 0, 0);
}
// wait until at most N of this wave's global->LDS loads are outstanding and
// every LDS access has completed, then barrier (no vmcnt(0) drain)
template <int N>
__device__ __forceinline__ void wait_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0070);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// wait until at most N of this wave's global loads are outstanding
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

template <int DH, bool CAUSAL, int NS>
__global__ __launch_bounds__(256) void attn_bf16_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ k,
                                                       const bf16_t* __restrict__ vt, int ldvt,
                                                       bf16_t* __restrict__ o, int B, int H, int Hkv, int L,
                                                       float scale_log2) {
  constexpr int KROWB = DH * 2;                  // bytes per K row
  constexpr int KT = BKV * KROWB, VT = DH * BKV * 2;   // bytes per K / V^T tile
  constexpr int STAGE = KT + VT;
  constexpr int KI = KT / 1024 / 4, VI = VT / 1024 / 4;  // 1 KB loads per wave per tile
  constexpr int ND = DH / 32;
  // one array per stage: every access names its stage's array, so the
  // compiler can tell a stage's fragment reads from another stage's DMA writes
  __shared__ __attribute__((aligned(1024))) char sm0[STAGE];
  __shared__ __attribute__((aligned(1024))) char sm1[STAGE];
  __shared__ __attribute__((aligned(1024))) char sm2[NS > 2 ? STAGE : 16];

  // the wave index is uniform: from a scalar register, the DMA destinations
  // (M0) are scalar arithmetic and take no VGPRs
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, li = lane & 31;
  const int nqb = (L + BQ - 1) / BQ;
  const int id = blockIdx.x;
  const int rest = id % (H * B);
  const int qb_r = id / (H * B);
  const int heavy = (nqb + 1) / 2;
  const int qb = !CAUSAL ? qb_r : (qb_r < heavy ? nqb - 1 - qb_r : qb_r - heavy);
  const int h = rest % H, b = rest / H;
  const int hk = h / (H / Hkv);
  const int q0 = qb * BQ;
  const int qw0 = q0 + wave * 32;
  const int qi = qw0 + li;

  const bf16_t* qh = q + ((size_t)b * H + h) * L * DH;
  const bf16_t* kh = k + ((size_t)b * Hkv + hk) * L * DH;
  const bf16_t* vh = vt + ((size_t)b * Hkv + hk) * DH * (size_t)ldvt;
  // rows past L read as zero
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)kh, (short)0, L * DH * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)vh, (short)0, DH * ldvt * 2, 0x00020000);

  // the wave's queries as MFMA B fragments, loaded without branches: lanes
  // past L load row L-1 (their scores and outputs are never stored)
  bf16x8 fq[DH / 16];
  const int qrow = min(qi, L - 1);
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) fq[ks] = *(const bf16x8*)(qh + (size_t)qrow * DH + ks * 16 + half * 8);

  const int kend = CAUSAL ? min(L, q0 + BQ) : L;
  const int ntiles = (kend + BKV - 1) / BKV;

  // K row r of a tile: 16-byte chunk c stored at chunk c ^ ksw(r); V^T row d: chunk c at c ^ ((d >> 1) & 7)
  auto ksw = [](int r) { return DH == 128 ? (r & 15) : ((r >> 1) & 7); };
  auto issue = [&](auto S_, int t) {
    constexpr int S = decltype(S_)::value;
    char* st = S == 0 ? sm0 : (S == 1 ? sm1 : sm2);
    const int kb = t * BKV;
#pragma unroll
    for (int j = 0; j < KI; ++j) {
      const int blk = wave * KI + j;
      constexpr int RPK = 1024 / KROWB;        // rows per 1 KB
      constexpr int CPR = KROWB / 16;          // chunks per row
      const int r = blk * RPK + lane / CPR, cs = lane % CPR;
      const int c = cs ^ ksw(r);
      lds_dma16(rk, st + blk * 1024, (unsigned)(((kb + r) * DH + c * 8) * 2));
    }
#pragma unroll
    for (int j = 0; j < VI; ++j) {
      const int blk = wave * VI + j;
      const int d = blk * 8 + lane / 8, cs = lane % 8;
      const int c = cs ^ ((d >> 1) & 7);
      lds_dma16(rv, st + KT + blk * 1024, (unsigned)((d * ldvt + kb + c * 8) * 2));
    }
  };

  f32x16 acc_o[ND];
#pragma unroll
  for (int t = 0; t < ND; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[t][r] = 0.f;
  float m_run = -INFINITY, l_part = 0.f;

  constexpr int PER = KI + VI;   // loads per wave per tile
  // the first NS-1 stages, issued unconditionally (a stage past the last tile
  // reads zeros through the buffer resources and is never used); then wait
  // for the query fragments only, so that their loads are known complete
  // inside the loop and never drain the ring there
  issue(std::integral_constant<int, 0>{}, 0);
  if constexpr (NS > 2) issue(std::integral_constant<int, 1>{}, 1);
  wait_vm<(NS - 1) * PER>();

  // tile it in stage S (= it % NS)
  auto body = [&](auto S_, int it) {
    constexpr int S = decltype(S_)::value;
    // tile it landed (for every wave), and every wave is done with the stage the next issue overwrites
    if (it + NS - 2 < ntiles) wait_barrier<(NS - 2) * PER>(); else wait_barrier<0>();
    const int kb = it * BKV;
    char* st = S == 0 ? sm0 : (S == 1 ? sm1 : sm2);
    if (kb + BKV > L) {
      // ragged last tile: V^T columns of keys >= L hold whatever lies past the
      // keys; zero them (their probabilities are zero, but 0 * NaN is not)
      for (int e = tid; e < DH * BKV; e += 256) {
        const int d = e / BKV, s = e % BKV;
        const int key = kb + swap23(s);
        if (key >= L) *(bf16_t*)(st + KT + d * 128 + (((s / 8) ^ ((d >> 1) & 7)) * 16) + (s % 8) * 2) = 0;
      }
      wait_barrier<0>();
    }
    if (it + NS - 1 < ntiles) issue(std::integral_constant<int, (S + NS - 1) % NS>{}, it + NS - 1);
    const bool active = !CAUSAL || kb <= qw0 + 31;
    if (active && qw0 < L) {
      f32x16 s[2];
      const f32x16 zero = {};
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int r = t * 32 + li;
        const char* krow = st + r * KROWB;
#pragma unroll
        for (int ks = 0; ks < DH / 16; ++ks) {
          const int c = ks * 2 + half;
          bf16x8 fk = *(const bf16x8*)(krow + ((c ^ ksw(r)) * 16));
          s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fk, fq[ks], ks == 0 ? zero : s[t], 0, 0, 0);
        }
      }
      const bool need_mask = (kb + BKV > L) || (CAUSAL && kb + BKV - 1 > qw0);
      if (need_mask) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            int key = kb + t * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
            bool ok = key < L && (!CAUSAL || key <= qi);
            s[t][r] = ok ? s[t][r] : -INFINITY;
          }
      }
      float mt = -INFINITY;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[t][r]);
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64)) * scale_log2;
      if (__any((mt > m_run + 8.f) ? 1 : 0)) {
        const float m_new = fmaxf(m_run, mt);
        const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
        l_part *= alpha;
#pragma unroll
        for (int t = 0; t < ND; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc_o[t][r] *= alpha;
        m_run = m_new;
      }
      const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
      float psum = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float p = __builtin_amdgcn_exp2f(fmaf(s[t][r], scale_log2, -m_use));
          s[t][r] = p;
          psum += p;
        }
      l_part += psum;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int ih = 0; ih < 2; ++ih) {
          bf16x8 fp;
          {
            union {
              uint32_t u[4];
              bf16x8 v;
            } cv;
            cv.u[0] = pack_bf2(s[t][(2 * ih) * 4 + 0], s[t][(2 * ih) * 4 + 1]);
            cv.u[1] = pack_bf2(s[t][(2 * ih) * 4 + 2], s[t][(2 * ih) * 4 + 3]);
            cv.u[2] = pack_bf2(s[t][(2 * ih + 1) * 4 + 0], s[t][(2 * ih + 1) * 4 + 1]);
            cv.u[3] = pack_bf2(s[t][(2 * ih + 1) * 4 + 2], s[t][(2 * ih + 1) * 4 + 3]);
            fp = cv.v;
          }
          const int c = t * 4 + ih * 2 + half;
#pragma unroll
          for (int dt = 0; dt < ND; ++dt) {
            const int d = dt * 32 + li;
            const bf16x8 fv = *(const bf16x8*)(st + KT + d * 128 + ((c ^ ((d >> 1) & 7)) * 16));
            acc_o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fv, fp, acc_o[dt], 0, 0, 0);
          }
        }
    }
  };
  for (int base = 0; base < ntiles; base += NS) {
    body(std::integral_constant<int, 0>{}, base);
    if (base + 1 < ntiles) body(std::integral_constant<int, 1>{}, base + 1);
    if constexpr (NS > 2)
      if (base + 2 < ntiles) body(std::integral_constant<int, 2>{}, base + 2);
  }

  const float l_tot = l_part + __shfl_xor(l_part, 32, 64);
  if (qi < L) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    bf16_t* orow = o + ((size_t)b * L + qi) * (size_t)(H * DH) + h * DH;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int d = dt * 32 + g * 8 + half * 4;
        u32x2 w = {pack_bf2(acc_o[dt][g * 4 + 0] * inv, acc_o[dt][g * 4 + 1] * inv),
                   pack_bf2(acc_o[dt][g * 4 + 2] * inv, acc_o[dt][g * 4 + 3] * inv)};
        *(u32x2*)(orow + d) = w;
      }
  }
}

template <int DH, bool CAUSAL>
hipError_t launch_attn(const bf16_t* q, const bf16_t* k, const bf16_t* vt, int ldvt, bf16_t* o, int B, int H, int Hkv,
                       int L, hipStream_t s) {
  const int nqb = (L + BQ - 1) / BQ;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)DH);
  // three stages of 16 KB for dh = 64 (three workgroups per CU), two of 32 KB
  // for dh = 128 (a third would leave one workgroup per CU)
  constexpr int NS = DH == 64 ? 3 : 2;
  hipLaunchKernelGGL((attn_bf16_kernel<DH, CAUSAL, NS>), dim3(nqb * H * B), dim3(256), 0, s, q, k, vt, ldvt, o, B, H,
                     Hkv, L, scale_log2);
  return hipGetLastError();
}

}  // namespace

hipError_t attention_bf16(const bf16_t* q, const bf16_t* k, const bf16_t* vt, int ldvt, bf16_t* o, int B, int H,
                          int Hkv, int L, int dh, bool causal, hipStream_t s) {
  if (B <= 0 || L <= 0 || H <= 0) return hipSuccess;
  if (Hkv <= 0 || H % Hkv != 0 || ldvt < (L + 15) / 16 * 16 || ldvt % 16 != 0)
    return hipErrorInvalidValue;
  if (dh == 128) return causal ? launch_attn<128, true>(q, k, vt, ldvt, o, B, H, Hkv, L, s)
                               : launch_attn<128, false>(q, k, vt, ldvt, o, B, H, Hkv, L, s);
  if (dh == 64) return causal ? launch_attn<64, true>(q, k, vt, ldvt, o, B, H, Hkv, L, s)
                              : launch_attn<64, false>(q, k, vt, ldvt, o, B, H, Hkv, L, s);
  return hipErrorInvalidValue;
}

}  // namespace vla
