// Host (CPU) executor of the decoder suffix B_{k+1..N} (the paper's Eq. (6)):
// the blocks after the partition point run on the host from the boundary
// hidden state the GPU prefix handed over, and a consumer thread pairs every
// boundary with its frame (the cross-frame pipeline of Sec. IV-C).
//
// Arithmetic mirrors the GPU blocks: bf16 matrix-product operands with fp32
// accumulation (AVX-512 BF16 vdpbf16ps), an fp32 residual stream, fp32 norm
// reductions and softmax, bf16 rounding wherever the GPU path rounds (normed
// activations, q/k/v after RoPE, softmax probabilities, attention output,
// gated activation).
//
// This file is compiled with AVX-512 (F, BW, VL, BF16) enabled; its entry
// points are reached only through host_suffix_api.cpp, which checks that the
// CPU has those extensions before calling in.

#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <functional>
#include <memory>
#include <mutex>
#include <thread>
#include <vector>

#include "host_pool.h"
#include "host_suffix.h"

namespace vla {
namespace host {

// ------------------------------------------------------------------ helpers

static inline float bf2f(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// round to nearest even; NaN stays NaN
static inline uint16_t f2bf(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// 16 floats -> 16 bf16 (round to nearest even) with the hardware conversion
static inline __m256i cvt16(__m512 v) { return (__m256i)_mm512_cvtneps_pbh(v); }

// e^x for a vector: e^x = 2^t, t = x log2(e) = n + f with n = round(t),
// |f| <= 1/2; 2^f = e^(f ln 2) by its Taylor series to degree 7 (truncation
// below 2e-8 relative for |f ln 2| <= 0.347), then scaled by 2^n with
// vscalefps.  Inputs below -87 give 0 (callers only need the softmax range).
static inline __m512 exp512(__m512 x) {
  const __m512 t = _mm512_mul_ps(x, _mm512_set1_ps(1.4426950408889634f));
  const __m512 n = _mm512_roundscale_ps(t, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC);
  const __m512 y = _mm512_mul_ps(_mm512_sub_ps(t, n), _mm512_set1_ps(0.6931471805599453f));
  // Horner form of sum_{i<=7} y^i / i!
  __m512 p = _mm512_set1_ps(1.f / 5040.f);
  p = _mm512_fmadd_ps(p, y, _mm512_set1_ps(1.f / 720.f));
  p = _mm512_fmadd_ps(p, y, _mm512_set1_ps(1.f / 120.f));
  p = _mm512_fmadd_ps(p, y, _mm512_set1_ps(1.f / 24.f));
  p = _mm512_fmadd_ps(p, y, _mm512_set1_ps(1.f / 6.f));
  p = _mm512_fmadd_ps(p, y, _mm512_set1_ps(0.5f));
  p = _mm512_fmadd_ps(p, y, _mm512_set1_ps(1.f));
  p = _mm512_fmadd_ps(p, y, _mm512_set1_ps(1.f));
  const __m512 r = _mm512_scalef_ps(p, n);
  return _mm512_maskz_mov_ps(_mm512_cmp_ps_mask(x, _mm512_set1_ps(-87.f), _CMP_GT_OQ), r);
}

// ------------------------------------------------------------------ packed operand
//
// B operand of C = A B^T with B[N][K] bf16, stored for vdpbf16ps: panels of
// 16 rows of B; inside a panel, k-pairs outermost, then the 16 rows, then the
// pair: element (n, k) at ((n/16) * KP + k/2) * 32 + (n%16) * 2 + k%2, with
// KP = K rounded up to even / 2.  N is padded to whole groups of 64 rows and
// K to even with zeros.

struct Packed {
  std::vector<uint16_t> v;
  int N = 0, K = 0, KP = 0, NP = 0;  // NP: rows after padding
  const uint16_t* panel(int n16) const { return v.data() + (size_t)n16 * KP * 32; }
};

template <class At>
static void pack_rows(Packed& P, int N, int K, const At& at) {
  P.N = N;
  P.K = K;
  P.KP = (K + 1) / 2;
  P.NP = (N + 63) / 64 * 64;
  P.v.assign((size_t)P.NP * P.KP * 2, 0);
  for (int n = 0; n < N; ++n) {
    uint16_t* base = P.v.data() + (size_t)(n / 16) * P.KP * 32 + (n % 16) * 2;
    for (int k = 0; k < K; ++k) base[(size_t)(k / 2) * 32 + (k & 1)] = at(n, k);
  }
}

// C[MR][64] (+)= A[MR][kp0*2 .. kp1*2) . B-panels[4][...]^T.  A rows are
// bf16 with stride lda (elements); C fp32 with stride ldc.
template <int MR>
static inline void micro(const uint16_t* A, int lda, const uint16_t* W, size_t pstride, int kp0, int kp1, float* C,
                         int ldc, bool accumulate) {
  __m512 c[MR][4];
  for (int r = 0; r < MR; ++r)
    for (int j = 0; j < 4; ++j) c[r][j] = accumulate ? _mm512_loadu_ps(C + (size_t)r * ldc + 16 * j) : _mm512_setzero_ps();
  for (int kp = kp0; kp < kp1; ++kp) {
    const uint16_t* w = W + (size_t)kp * 32;
    const __m512bh w0 = (__m512bh)_mm512_loadu_si512(w);
    const __m512bh w1 = (__m512bh)_mm512_loadu_si512(w + pstride);
    const __m512bh w2 = (__m512bh)_mm512_loadu_si512(w + 2 * pstride);
    const __m512bh w3 = (__m512bh)_mm512_loadu_si512(w + 3 * pstride);
    for (int r = 0; r < MR; ++r) {
      int32_t pair;
      std::memcpy(&pair, A + (size_t)r * lda + 2 * kp, 4);
      const __m512bh a = (__m512bh)_mm512_set1_epi32(pair);
      c[r][0] = _mm512_dpbf16_ps(c[r][0], a, w0);
      c[r][1] = _mm512_dpbf16_ps(c[r][1], a, w1);
      c[r][2] = _mm512_dpbf16_ps(c[r][2], a, w2);
      c[r][3] = _mm512_dpbf16_ps(c[r][3], a, w3);
    }
  }
  for (int r = 0; r < MR; ++r)
    for (int j = 0; j < 4; ++j) _mm512_storeu_ps(C + (size_t)r * ldc + 16 * j, c[r][j]);
}

static void micro_any(int mr, const uint16_t* A, int lda, const uint16_t* W, size_t pstride, int kp0, int kp1, float* C,
                      int ldc, bool acc) {
  switch (mr) {
    case 6: micro<6>(A, lda, W, pstride, kp0, kp1, C, ldc, acc); break;
    case 5: micro<5>(A, lda, W, pstride, kp0, kp1, C, ldc, acc); break;
    case 4: micro<4>(A, lda, W, pstride, kp0, kp1, C, ldc, acc); break;
    case 3: micro<3>(A, lda, W, pstride, kp0, kp1, C, ldc, acc); break;
    case 2: micro<2>(A, lda, W, pstride, kp0, kp1, C, ldc, acc); break;
    default: micro<1>(A, lda, W, pstride, kp0, kp1, C, ldc, acc); break;
  }
}

constexpr int KC = 256;  // k-pairs per cache block
constexpr int MB = 48;   // rows per task

// One MB x 64 tile of C = A B^T: rows [m0, m0+mb), columns [n0, n0+64) of the
// padded operand, over all of K, into tile T[mb][64] (fp32, stride 64).
// A must have every row readable for 2 * KP elements (pad columns zero).
static void tile(const uint16_t* A, int lda, const Packed& B, int m0, int mb, int n0, float* T) {
  const uint16_t* W = B.panel(n0 / 16);
  const size_t ps = (size_t)B.KP * 32;
  for (int kp0 = 0; kp0 < B.KP; kp0 += KC) {
    const int kp1 = std::min(B.KP, kp0 + KC);
    for (int r = 0; r < mb; r += 6) {
      const int mr = std::min(6, mb - r);
      micro_any(mr, A + (size_t)(m0 + r) * lda, lda, W, ps, kp0, kp1, T + (size_t)r * 64, 64, kp0 > 0);
    }
  }
}

// C[M][N] = A[M][K] B^T over the pool; epi(row, col0, vals, n) receives each
// row segment of a 64-column tile (n valid columns).
template <class Epi>
static void gemm(Pool& pool, const uint16_t* A, int lda, const Packed& B, int M, const Epi& epi) {
  const int tm = (M + MB - 1) / MB, tn = B.NP / 64;
  pool.run(tm * tn, [&](int t) {
    alignas(64) float T[MB * 64];
    const int m0 = (t / tn) * MB, n0 = (t % tn) * 64;
    const int mb = std::min(MB, M - m0);
    tile(A, lda, B, m0, mb, n0, T);
    const int nv = std::min(64, B.N - n0);
    if (nv <= 0) return;
    for (int r = 0; r < mb; ++r) epi(m0 + r, n0, T + r * 64, nv);
  });
}

// ------------------------------------------------------------------ executor

struct Block {
  Packed wqkv, wo, wgu, wd;  // wgu: gate and up rows interleaved by 64-row groups
  std::vector<float> g1, g2;
};

struct Suffix {
  Cfg c;
  int k_begin = 0, k_end = 0;
  std::unique_ptr<Pool> pool;
  std::vector<Block> blocks;
  std::vector<bool> loaded;
  // workspace (grown on demand)
  std::vector<float> h, qkv, gu;
  std::vector<uint16_t> x, q, kk, vv, o, act;
  std::vector<float> rope_cos, rope_sin;
  int rope_L = 0;
  // KV caches of the blocks for decode steps: [block][B][Hkv][cache_L][dh] bf16
  int cache_B = 0, cache_L = 0;
  std::vector<std::vector<uint16_t>> kc, vc;
};

Suffix* create(const Cfg& c, int k_begin, int k_end, int n_threads) {
  auto* s = new Suffix;
  s->c = c;
  s->k_begin = k_begin;
  s->k_end = k_end;
  if (n_threads <= 0) n_threads = (int)std::max(1u, std::thread::hardware_concurrency());
  s->pool = std::make_unique<Pool>(n_threads);
  s->blocks.resize(k_end - k_begin);
  s->loaded.assign(k_end - k_begin, false);
  return s;
}

void destroy(Suffix* s) { delete s; }

int threads(const Suffix* s) { return s->pool->size(); }

bool load_block(Suffix* s, int block, const Weights& w) {
  const Cfg& c = s->c;
  const int d = c.d, hd = c.H * c.dh, kvd = c.Hkv * c.dh, F = c.F;
  Block& b = s->blocks[block - s->k_begin];
  // fused QKV operand: rows [q | k | v]
  pack_rows(b.wqkv, hd + 2 * kvd, d, [&](int n, int k) {
    if (n < hd) return w.wq[(size_t)n * d + k];
    if (n < hd + kvd) return w.wk[(size_t)(n - hd) * d + k];
    return w.wv[(size_t)(n - hd - kvd) * d + k];
  });
  pack_rows(b.wo, d, hd, [&](int n, int k) { return w.wo[(size_t)n * hd + k]; });
  // gate/up: 64-row group 2j holds gate rows [64j, 64j+64), group 2j+1 the up rows
  const int Fp = (F + 63) / 64 * 64;
  pack_rows(b.wgu, 2 * Fp, d, [&](int n, int k) -> uint16_t {
    const int grp = n / 64, r = (grp / 2) * 64 + n % 64;
    if (r >= F) return 0;
    return (grp & 1) ? w.wu[(size_t)r * d + k] : w.wg[(size_t)r * d + k];
  });
  pack_rows(b.wd, d, F, [&](int n, int k) { return w.wd[(size_t)n * F + k]; });
  b.g1.resize(d);
  b.g2.resize(d);
  for (int i = 0; i < d; ++i) {
    b.g1[i] = bf2f(w.g1[i]);
    b.g2[i] = bf2f(w.g2[i]);
  }
  s->loaded[block - s->k_begin] = true;
  return true;
}

bool all_loaded(const Suffix* s) {
  for (bool b : s->loaded)
    if (!b) return false;
  return true;
}

// y = bf16(x * rsqrt(mean(x^2) + eps) * g), one row per task batch
static void rms_rows(Pool& pool, const float* h, uint16_t* y, int ldy, int M, int d, const float* g, float eps) {
  pool.run((M + 15) / 16, [&](int t) {
    for (int m = t * 16; m < std::min(M, t * 16 + 16); ++m) {
      const float* r = h + (size_t)m * d;
      __m512 acc = _mm512_setzero_ps();
      int i = 0;
      for (; i + 16 <= d; i += 16) {
        const __m512 v = _mm512_loadu_ps(r + i);
        acc = _mm512_fmadd_ps(v, v, acc);
      }
      float ss = _mm512_reduce_add_ps(acc);
      for (; i < d; ++i) ss += r[i] * r[i];
      const float sc = 1.f / std::sqrt(ss / (float)d + eps);
      uint16_t* out = y + (size_t)m * ldy;
      i = 0;
      for (; i + 16 <= d; i += 16)
        _mm256_storeu_si256((__m256i*)(out + i),
                            cvt16(_mm512_mul_ps(_mm512_mul_ps(_mm512_loadu_ps(r + i), _mm512_set1_ps(sc)),
                                                _mm512_loadu_ps(g + i))));
      for (; i < d; ++i) out[i] = f2bf(r[i] * sc * g[i]);
    }
  });
}

static void rope_tables(Suffix* s, int L) {
  if (s->rope_L >= L) return;
  const int half = s->c.dh / 2;
  s->rope_cos.resize((size_t)L * half);
  s->rope_sin.resize((size_t)L * half);
  for (int p = 0; p < L; ++p)
    for (int i = 0; i < half; ++i) {
      const double inv = std::pow((double)s->c.rope_base, -2.0 * i / (double)s->c.dh);
      const double a = (double)p * inv;
      s->rope_cos[(size_t)p * half + i] = (float)std::cos(a);
      s->rope_sin[(size_t)p * half + i] = (float)std::sin(a);
    }
  s->rope_L = L;
}

// Causal attention of one (batch, head) query block of 64 over keys [0, q0+64).
// q [L][dh] bf16 rows of this head (stride ldq), K and V^T packed per KV head.
static void attn_block(const Cfg& c, const uint16_t* q, int ldq, const Packed& Kp, const Packed& Vtp, int L, int q0,
                       uint16_t* o, int ldo, float scale, std::vector<float>& S, std::vector<uint16_t>& P) {
  const int nq = std::min(64, L - q0);
  const int kend = c.causal ? q0 + nq : L;
  const int kpad = (kend + 63) / 64 * 64;
  S.resize((size_t)64 * kpad);
  P.assign((size_t)64 * (kpad + 2), 0);
  const int ldp = kpad + 2;  // room for the odd-length pad pair
  // scores: rows q0.., columns in 64-key tiles
  const size_t ps = (size_t)Kp.KP * 32;
  for (int n0 = 0; n0 < kend; n0 += 64)
    for (int r = 0; r < nq; r += 6) {
      const int mr = std::min(6, nq - r);
      micro_any(mr, q + (size_t)(q0 + r) * ldq, ldq, Kp.panel(n0 / 16), ps, 0, Kp.KP, S.data() + (size_t)r * kpad + n0,
                kpad, false);
    }
  // softmax per row in fp32, probabilities rounded to bf16 (as the GPU's PV operand)
  std::vector<float> inv(nq);
  for (int r = 0; r < nq; ++r) {
    const int qi = q0 + r;
    const int nk = c.causal ? qi + 1 : L;
    float* sr = S.data() + (size_t)r * kpad;
    float mx = -INFINITY;
    for (int j = 0; j < nk; ++j) mx = std::max(mx, sr[j]);
    const __m512 vs = _mm512_set1_ps(scale), vm = _mm512_set1_ps(mx * scale);
    float sum = 0.f;
    uint16_t* pr = P.data() + (size_t)r * ldp;
    int j = 0;
    for (; j + 16 <= nk; j += 16) {
      const __m512 e = exp512(_mm512_fmsub_ps(_mm512_loadu_ps(sr + j), vs, vm));
      sum += _mm512_reduce_add_ps(e);
      _mm256_storeu_si256((__m256i*)(pr + j), cvt16(e));
    }
    if (j < nk) {
      const __mmask16 m = (__mmask16)((1u << (nk - j)) - 1u);
      const __m512 e = _mm512_maskz_mov_ps(m, exp512(_mm512_fmsub_ps(_mm512_maskz_loadu_ps(m, sr + j), vs, vm)));
      sum += _mm512_reduce_add_ps(e);
      _mm256_mask_storeu_epi16(pr + j, m, cvt16(e));
    }
    inv[r] = 1.f / sum;
  }
  // O = P V: A = P rows (keys as the reduction), B = V^T packed [dh][keys]
  alignas(64) float Ot[6 * 128];
  const size_t vs2 = (size_t)Vtp.KP * 32;
  const int kp1 = (kend + 1) / 2;
  for (int r = 0; r < nq; r += 6) {
    const int mr = std::min(6, nq - r);
    for (int n0 = 0; n0 < c.dh; n0 += 64)
      micro_any(mr, P.data() + (size_t)r * ldp, ldp, Vtp.panel(n0 / 16), vs2, 0, kp1, Ot + n0, c.dh, false);
    for (int i = 0; i < mr; ++i) {
      uint16_t* orow = o + (size_t)(q0 + r + i) * ldo;
      for (int e = 0; e < c.dh; ++e) orow[e] = f2bf(Ot[i * c.dh + e] * inv[r + i]);
    }
  }
}

// q, k, v of rows m = b * L + r at positions pos0 + r, RoPE applied, to
// [B][heads][L][dh] bf16 (q, kk, vv workspaces)
static void qkv_rope(Suffix* s, const Block& w, int B, int L, int pos0) {
  const Cfg& c = s->c;
  Pool& pool = *s->pool;
  const int M = B * L, d = c.d, H = c.H, Hkv = c.Hkv, dh = c.dh, hd = H * dh, kvd = Hkv * dh;
  const int dpad = (d + 1) / 2 * 2;
  const int half = dh / 2;
  float* h = s->h.data();
  uint16_t* x = s->x.data();
  rms_rows(pool, h, x, dpad, M, d, w.g1.data(), c.eps);
  uint16_t *q = s->q.data(), *kk = s->kk.data(), *vv = s->vv.data();
  const float* cs = s->rope_cos.data();
  const float* sn = s->rope_sin.data();
  gemm(pool, x, dpad, w.wqkv, M, [&](int m, int n0, const float* v, int nv) {
    const int b = m / L, r = m % L, p = pos0 + r;
    // a 64-column tile never straddles a head (dh is 64 or a multiple of 64)
    const int kind = n0 < hd ? 0 : (n0 < hd + kvd ? 1 : 2);
    const int base = kind == 0 ? 0 : (kind == 1 ? hd : hd + kvd);
    const int head = (n0 - base) / dh, d0 = (n0 - base) % dh;
    const int nh = kind == 0 ? H : Hkv;
    uint16_t* dst = (kind == 0 ? q : (kind == 1 ? kk : vv)) + (((size_t)b * nh + head) * L + r) * dh + d0;
    if (kind < 2 && c.use_rope) {
      // rotate-half pairs (i, i + dh/2) live in the same head; handle a
      // 64-column tile by reading its partner from the tile when dh == 64,
      // else from the tile pair held in the workspace row
      if (dh == 64) {
        for (int i = 0; i < 32; ++i) {
          const float c0 = cs[(size_t)p * half + i], s0 = sn[(size_t)p * half + i];
          const float a = v[i], bb = v[i + 32];
          dst[i] = f2bf(a * c0 - bb * s0);
          dst[i + 32] = f2bf(bb * c0 + a * s0);
        }
      } else {
        // dh >= 128: stash the raw fp32 values; rotated in a second pass
        float* raw = s->qkv.data() + (size_t)m * (hd + 2 * kvd) + n0;
        std::memcpy(raw, v, sizeof(float) * nv);
      }
    } else {
      for (int i = 0; i < nv; ++i) dst[i] = f2bf(v[i]);
    }
  });
  if (c.use_rope && dh > 64) {
    pool.run(M, [&](int m) {
      const int b = m / L, r = m % L, p = pos0 + r;
      const float* raw = s->qkv.data() + (size_t)m * (hd + 2 * kvd);
      for (int head = 0; head < H + Hkv; ++head) {
        const bool isq = head < H;
        const float* rr = raw + (isq ? head * dh : hd + (head - H) * dh);
        uint16_t* dst = isq ? q + (((size_t)b * H + head) * L + r) * dh : kk + (((size_t)b * Hkv + head - H) * L + r) * dh;
        for (int i = 0; i < half; ++i) {
          const float c0 = cs[(size_t)p * half + i], s0 = sn[(size_t)p * half + i];
          const float a = rr[i], bb = rr[i + half];
          dst[i] = f2bf(a * c0 - bb * s0);
          dst[i + half] = f2bf(bb * c0 + a * s0);
        }
      }
    });
  }
}

// h += o Wo^T over M rows
static void oproj(Suffix* s, const Block& w, int M) {
  const Cfg& c = s->c;
  const int d = c.d, hdpad = (c.H * c.dh + 1) / 2 * 2;
  float* h = s->h.data();
  gemm(*s->pool, s->o.data(), hdpad, w.wo, M, [&](int m, int n0, const float* v, int nv) {
    float* hr = h + (size_t)m * d + n0;
    for (int i = 0; i < nv; ++i) hr[i] += v[i];
  });
}

// h += swiglu(RMSNorm(h) Wgu^T) Wd^T over M rows
static void mlp_half(Suffix* s, const Block& w, int M) {
  const Cfg& c = s->c;
  Pool& pool = *s->pool;
  const int d = c.d, dpad = (d + 1) / 2 * 2;
  const int Fp = (c.F + 63) / 64 * 64;
  float* h = s->h.data();
  uint16_t* x = s->x.data();
  rms_rows(pool, h, x, dpad, M, d, w.g2.data(), c.eps);
  uint16_t* act = s->act.data();
  const int ldact = (Fp + 1) / 2 * 2;
  float* gu = s->gu.data();
  // even 64-column tiles are gate rows, odd ones the matching up rows; the two
  // come from different tasks, so both land in fp32 first and combine below
  gemm(pool, x, dpad, w.wgu, M, [&](int m, int n0, const float* v, int nv) {
    std::memcpy(gu + (size_t)m * 2 * Fp + n0, v, sizeof(float) * nv);
  });
  pool.run(M, [&](int m) {
    const float* r = gu + (size_t)m * 2 * Fp;
    uint16_t* ar = act + (size_t)m * ldact;
    for (int j = 0; j < Fp; j += 64) {
      const float* g = r + 2 * j;
      const float* u = g + 64;
      for (int i = 0; i < 64; i += 16) {
        const __m512 gv = _mm512_loadu_ps(g + i), uv = _mm512_loadu_ps(u + i);
        const __m512 sg = _mm512_div_ps(gv, _mm512_add_ps(_mm512_set1_ps(1.f), exp512(_mm512_sub_ps(_mm512_setzero_ps(), gv))));
        _mm256_storeu_si256((__m256i*)(ar + j + i), cvt16(_mm512_mul_ps(sg, uv)));
      }
    }
  });
  gemm(pool, act, ldact, w.wd, M, [&](int m, int n0, const float* v, int nv) {
    float* hr = h + (size_t)m * d + n0;
    for (int i = 0; i < nv; ++i) hr[i] += v[i];
  });
}

static void block_fwd(Suffix* s, int bi, int B, int L) {
  const Block& w = s->blocks[bi];
  const Cfg& c = s->c;
  Pool& pool = *s->pool;
  const int M = B * L, H = c.H, Hkv = c.Hkv, dh = c.dh, hd = H * dh;
  const int hdpad = (hd + 1) / 2 * 2;
  qkv_rope(s, w, B, L, 0);
  uint16_t *q = s->q.data(), *kk = s->kk.data(), *vv = s->vv.data();
  // keep this block's keys and values for later decode steps
  if (s->cache_B == B && s->cache_L >= L) {
    pool.run(B * Hkv, [&](int t) {
      std::memcpy(s->kc[bi].data() + (size_t)t * s->cache_L * dh, kk + (size_t)t * L * dh, sizeof(uint16_t) * L * dh);
      std::memcpy(s->vc[bi].data() + (size_t)t * s->cache_L * dh, vv + (size_t)t * L * dh, sizeof(uint16_t) * L * dh);
    });
  }
  // pack K and V^T per (batch, KV head)
  std::vector<Packed> Kp(B * Hkv), Vp(B * Hkv);
  pool.run(B * Hkv, [&](int t) {
    const uint16_t* kh = kk + (size_t)t * L * dh;
    const uint16_t* vh = vv + (size_t)t * L * dh;
    pack_rows(Kp[t], L, dh, [&](int n, int k) { return kh[(size_t)n * dh + k]; });
    pack_rows(Vp[t], dh, L, [&](int n, int k) { return vh[(size_t)k * dh + n]; });
  });
  const int nqb = (L + 63) / 64;
  const float scale = 1.f / std::sqrt((float)dh);
  uint16_t* o = s->o.data();
  // heaviest query blocks first
  pool.run(B * H * nqb, [&](int t) {
    thread_local std::vector<float> S;
    thread_local std::vector<uint16_t> P;
    const int qb = nqb - 1 - t / (B * H), bh = t % (B * H), b = bh / H, head = bh % H;
    const int kvh = head / (H / Hkv);
    attn_block(c, q + ((size_t)b * H + head) * L * dh, dh, Kp[b * Hkv + kvh], Vp[b * Hkv + kvh], L, qb * 64,
               o + (size_t)b * L * hdpad + head * dh, hdpad, scale, S, P);
  });
  oproj(s, w, M);
  mlp_half(s, w, M);
}

// Attention of one new token per sequence at position pos over cache rows
// [0, pos] (the token's own key and value already appended): fp32 scores,
// softmax and accumulation, bf16 output.
static void decode_attention(Suffix* s, int bi, int B, int pos) {
  const Cfg& c = s->c;
  const int H = c.H, Hkv = c.Hkv, dh = c.dh, hdpad = (H * dh + 1) / 2 * 2;
  const float scale = 1.f / std::sqrt((float)dh);
  const uint16_t* q = s->q.data();
  uint16_t* o = s->o.data();
  s->pool->run(B * H, [&](int t) {
    thread_local std::vector<float> sc;
    sc.resize(pos + 1 + 16);
    const int b = t / H, head = t % H, kvh = head / (H / Hkv);
    const uint16_t* kb = s->kc[bi].data() + ((size_t)b * Hkv + kvh) * s->cache_L * dh;
    const uint16_t* vb = s->vc[bi].data() + ((size_t)b * Hkv + kvh) * s->cache_L * dh;
    const uint16_t* qh = q + ((size_t)b * H + head) * dh;
    // q in fp32 vectors (dh is a multiple of 64)
    __m512 qv[8];
    for (int i = 0; i < dh / 16; ++i)
      qv[i] = _mm512_mul_ps(_mm512_castsi512_ps(_mm512_slli_epi32(
                                _mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i*)(qh + 16 * i))), 16)),
                            _mm512_set1_ps(scale));
    float mx = -INFINITY;
    for (int j = 0; j <= pos; ++j) {
      const uint16_t* kr = kb + (size_t)j * dh;
      __m512 acc = _mm512_setzero_ps();
      for (int i = 0; i < dh / 16; ++i) {
        const __m512 kf = _mm512_castsi512_ps(
            _mm512_slli_epi32(_mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i*)(kr + 16 * i))), 16));
        acc = _mm512_fmadd_ps(qv[i], kf, acc);
      }
      sc[j] = _mm512_reduce_add_ps(acc);
      mx = std::max(mx, sc[j]);
    }
    float sum = 0.f;
    int j = 0;
    const __m512 vm = _mm512_set1_ps(mx);
    for (; j + 16 <= pos + 1; j += 16) {
      const __m512 e = exp512(_mm512_sub_ps(_mm512_loadu_ps(&sc[j]), vm));
      _mm512_storeu_ps(&sc[j], e);
      sum += _mm512_reduce_add_ps(e);
    }
    for (; j <= pos; ++j) {
      const __m512 e = exp512(_mm512_set1_ps(sc[j] - mx));
      sc[j] = _mm_cvtss_f32(_mm512_castps512_ps128(e));
      sum += sc[j];
    }
    __m512 ov[8];
    for (int i = 0; i < dh / 16; ++i) ov[i] = _mm512_setzero_ps();
    for (int jj = 0; jj <= pos; ++jj) {
      const uint16_t* vr = vb + (size_t)jj * dh;
      const __m512 pj = _mm512_set1_ps(sc[jj]);
      for (int i = 0; i < dh / 16; ++i) {
        const __m512 vf = _mm512_castsi512_ps(
            _mm512_slli_epi32(_mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i*)(vr + 16 * i))), 16));
        ov[i] = _mm512_fmadd_ps(pj, vf, ov[i]);
      }
    }
    uint16_t* orow = o + (size_t)b * hdpad + head * dh;
    const __m512 inv = _mm512_set1_ps(1.f / sum);
    for (int i = 0; i < dh / 16; ++i) _mm256_storeu_si256((__m256i*)(orow + 16 * i), cvt16(_mm512_mul_ps(ov[i], inv)));
  });
}

static void block_decode(Suffix* s, int bi, int B, int pos) {
  const Block& w = s->blocks[bi];
  const Cfg& c = s->c;
  const int Hkv = c.Hkv, dh = c.dh;
  qkv_rope(s, w, B, 1, pos);
  // append the token's key and value at pos
  for (int t = 0; t < B * Hkv; ++t) {
    std::memcpy(s->kc[bi].data() + ((size_t)t * s->cache_L + pos) * dh, s->kk.data() + (size_t)t * dh,
                sizeof(uint16_t) * dh);
    std::memcpy(s->vc[bi].data() + ((size_t)t * s->cache_L + pos) * dh, s->vv.data() + (size_t)t * dh,
                sizeof(uint16_t) * dh);
  }
  decode_attention(s, bi, B, pos);
  oproj(s, w, B);
  mlp_half(s, w, B);
}

void set_cache(Suffix* s, int B, int L_cap) {
  const size_t n = (size_t)B * s->c.Hkv * L_cap * s->c.dh;
  s->cache_B = B;
  s->cache_L = L_cap;
  s->kc.assign(s->blocks.size(), std::vector<uint16_t>());
  s->vc.assign(s->blocks.size(), std::vector<uint16_t>());
  if (B <= 0 || L_cap <= 0) {
    s->cache_B = s->cache_L = 0;
    return;
  }
  for (size_t i = 0; i < s->blocks.size(); ++i) {
    s->kc[i].assign(n, 0);
    s->vc[i].assign(n, 0);
  }
}

int cache_batch(const Suffix* s) { return s->cache_B; }
int cache_len(const Suffix* s) { return s->cache_L; }

// workspaces for M rows of B sequences of L tokens
static void reserve(Suffix* s, int B, int L) {
  const Cfg& c = s->c;
  const int M = B * L, d = c.d, hd = c.H * c.dh, kvd = c.Hkv * c.dh;
  const int dpad = (d + 1) / 2 * 2, hdpad = (hd + 1) / 2 * 2;
  const int Fp = (c.F + 63) / 64 * 64;
  s->h.resize((size_t)M * d);
  s->x.assign((size_t)M * dpad, 0);
  s->q.resize((size_t)B * c.H * L * c.dh);
  s->kk.resize((size_t)B * c.Hkv * L * c.dh);
  s->vv.resize((size_t)B * c.Hkv * L * c.dh);
  s->o.assign((size_t)M * hdpad, 0);
  s->act.assign((size_t)M * ((Fp + 1) / 2 * 2), 0);
  s->gu.resize((size_t)M * 2 * Fp);
  if (c.use_rope && c.dh > 64) s->qkv.resize((size_t)M * (hd + 2 * kvd));
}

static void load_input(Suffix* s, const void* in, bool in_f32, size_t n) {
  if (in_f32) {
    std::memcpy(s->h.data(), in, sizeof(float) * n);
  } else {
    const uint16_t* hb = (const uint16_t*)in;
    for (size_t i = 0; i < n; ++i) s->h[i] = bf2f(hb[i]);
  }
}

bool decode(Suffix* s, int k, const void* in, bool in_f32, int B, int pos, float* out) {
  const size_t n = (size_t)B * s->c.d;
  reserve(s, B, 1);
  rope_tables(s, std::max(pos + 1, s->cache_L));
  load_input(s, in, in_f32, n);
  for (int l = k; l < s->k_end; ++l) block_decode(s, l - s->k_begin, B, pos);
  std::memcpy(out, s->h.data(), sizeof(float) * n);
  return true;
}

bool run(Suffix* s, int k, const void* in, bool in_f32, int B, int L, float* out) {
  const size_t n = (size_t)B * L * s->c.d;
  reserve(s, B, L);
  rope_tables(s, std::max(L, s->cache_L));
  load_input(s, in, in_f32, n);
  for (int l = k; l < s->k_end; ++l) block_fwd(s, l - s->k_begin, B, L);
  std::memcpy(out, s->h.data(), sizeof(float) * n);
  return true;
}

}  // namespace host
}  // namespace vla
