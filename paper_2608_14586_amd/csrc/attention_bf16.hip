// Flash-style attention for gfx950 (bf16 MFMA, fp32 online softmax).
//
// One workgroup = 4 waves = 128 queries of one (batch, head); each wave owns
// 32 queries.  Keys advance in tiles of 64 staged in LDS (double buffered):
// K as [key][dh] and V transposed as [dh][key], so every MFMA operand is a
// contiguous LDS read.
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

#include "kernels.h"

namespace vla {
namespace {

constexpr int BQ = 128, BKV = 64, PADK = 8, PADV = 8;

// key index <-> stored V^T column: bits 2 and 3 swapped (an involution)
__device__ __forceinline__ int swap23(int t) { return (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1); }

template <int DH, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_bf16_kernel(const bf16_t* __restrict__ q, const bf16_t* __restrict__ k,
                                                        const bf16_t* __restrict__ vt, int ldvt,
                                                        bf16_t* __restrict__ o, int B, int H, int Hkv, int L,
                                                        float scale_log2) {
  constexpr int LDK = DH + PADK, LDV = BKV + PADV;
  constexpr int KCH = BKV * DH / 8 / 256;  // 16-byte chunks per thread, K tile
  constexpr int VCH = DH * BKV / 8 / 256;  // V^T tile
  constexpr int ND = DH / 32;
  __shared__ __attribute__((aligned(16))) bf16_t sK[2][BKV * LDK];
  __shared__ __attribute__((aligned(16))) bf16_t sV[2][DH * LDV];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, li = lane & 31;
  const int nqb = (L + BQ - 1) / BQ;
  const int id = blockIdx.x;
  const int rest = id % (H * B);
  const int qb_r = id / (H * B);
  // causal: the first half of the grid takes the heavy query blocks in
  // descending order, the second half the light ones ascending, so the two
  // workgroups that share a CU (ids i and i + half the grid) sum to the same
  // number of key tiles
  const int heavy = (nqb + 1) / 2;
  const int qb = !CAUSAL ? qb_r : (qb_r < heavy ? nqb - 1 - qb_r : qb_r - heavy);
  const int h = rest % H, b = rest / H;
  const int hk = h / (H / Hkv);
  const int q0 = qb * BQ;
  const int qw0 = q0 + wave * 32;
  const int qi = qw0 + li;  // this lane's query

  const bf16_t* qh = q + ((size_t)b * H + h) * L * DH;
  const bf16_t* kh = k + ((size_t)b * Hkv + hk) * L * DH;
  const bf16_t* vh = vt + ((size_t)b * Hkv + hk) * DH * (size_t)ldvt;

  // Q fragments (B operand of S^T): query qi, dims ks*16 + half*8 .. +8
  bf16x8 fq[DH / 16];
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) {
    if (qi < L)
      fq[ks] = *(const bf16x8*)(qh + (size_t)qi * DH + ks * 16 + half * 8);
    else
      fq[ks] = bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
  }

  const int kend = CAUSAL ? min(L, q0 + BQ) : L;
  const int ntiles = (kend + BKV - 1) / BKV;

  u32x4 rk[KCH], rv[VCH];
  auto gload = [&](int kb) {
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      int idx = tid + c * 256;
      int row = idx / (DH / 8), cc = idx % (DH / 8);
      int key = kb + row;
      rk[c] = key < L ? *(const u32x4*)(kh + (size_t)key * DH + cc * 8) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int c = 0; c < VCH; ++c) {
      int idx = tid + c * 256;
      int d = idx / (BKV / 8), cc = idx % (BKV / 8);
      int pos = kb + cc * 8;  // stored column; it holds key pos ^ swap23
      const bf16_t* src = vh + (size_t)d * ldvt + pos;
      if ((pos & ~15) + 16 <= L) {
        rv[c] = *(const u32x4*)src;
      } else {
        // columns of keys >= L are zero (their probabilities are zero too)
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int k0 = swap23(pos + 2 * e), k1 = swap23(pos + 2 * e + 1);
          uint32_t lo = k0 < L ? src[2 * e] : 0u;
          uint32_t hi = k1 < L ? src[2 * e + 1] : 0u;
          w[e] = lo | (hi << 16);
        }
        rv[c] = u32x4{w[0], w[1], w[2], w[3]};
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      int idx = tid + c * 256;
      int row = idx / (DH / 8), cc = idx % (DH / 8);
      *(u32x4*)(&sK[buf][row * LDK + cc * 8]) = rk[c];
    }
#pragma unroll
    for (int c = 0; c < VCH; ++c) {
      int idx = tid + c * 256;
      int d = idx / (BKV / 8), cc = idx % (BKV / 8);
      *(u32x4*)(&sV[buf][d * LDV + cc * 8]) = rv[c];
    }
  };

  f32x16 acc_o[ND];
#pragma unroll
  for (int t = 0; t < ND; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[t][r] = 0.f;
  float m_run = -INFINITY, l_part = 0.f;

  gload(0);
  lstore(0);
  __syncthreads();

  for (int it = 0; it < ntiles; ++it) {
    const int buf = it & 1;
    const int kb = it * BKV;
    if (it + 1 < ntiles) gload(kb + BKV);
    const bool active = !CAUSAL || kb <= qw0 + 31;
    if (active && qw0 < L) {
      // S^T for two 32-key tiles (the first k-step starts from a zero accumulator)
      f32x16 s[2];
      const f32x16 zero = {};
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bf16_t* kbase = &sK[buf][(t * 32 + li) * LDK + half * 8];
#pragma unroll
        for (int ks = 0; ks < DH / 16; ++ks) {
          bf16x8 fk = *(const bf16x8*)(kbase + ks * 16);
          s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fk, fq[ks], ks == 0 ? zero : s[t], 0, 0, 0);
        }
      }
      // tile max of the raw scores (the scale is positive, so it commutes
      // with the max); masked entries become -inf
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
      // Lazy rescaling: the running max m_run only moves (and O, l are only
      // rescaled) when some query of the wave sees its max grow by more than
      // 2^8; otherwise the probabilities are taken against the stale max and
      // stay below 256, exactly representable in the same relative precision.
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
          // p = 2^(s * scale - m), one FMA and one v_exp_f32 per score
          // (results below 2^-126 flush to zero, which a softmax can ignore)
          float p = __builtin_amdgcn_exp2f(fmaf(s[t][r], scale_log2, -m_use));
          s[t][r] = p;
          psum += p;
        }
      l_part += psum;
      // O^T += V^T P^T over 4 k-steps of 16 keys
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
          // stored columns 16 (2t + ih) + 8 half .. + 7 hold this lane's 8 keys
          const int col = t * 32 + ih * 16 + half * 8;
#pragma unroll
          for (int dt = 0; dt < ND; ++dt) {
            const bf16x8 fv = *(const bf16x8*)&sV[buf][(dt * 32 + li) * LDV + col];
            acc_o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fv, fp, acc_o[dt], 0, 0, 0);
          }
        }
    }
    if (it + 1 < ntiles) lstore(buf ^ 1);
    __syncthreads();
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
  hipLaunchKernelGGL((attn_bf16_kernel<DH, CAUSAL>), dim3(nqb * H * B), dim3(256), 0, s, q, k, vt, ldvt, o, B, H, Hkv,
                     L, scale_log2);
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
