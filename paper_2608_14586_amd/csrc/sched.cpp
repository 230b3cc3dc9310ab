// Boundary-adaptive partition controller Phi (the paper's Sec. IV-D,
// Eq. (15)-(17)): picks the partition point of the next frame from the
// runtime state z_t = [u_gpu, u_cpu, q_t] and a stage model fitted online.
// Implements the vla_sched_* calls of include/vla_suffix.h.
//
// Stage model (Eq. (8)-(10), linear in the number of blocks on each side):
//   T_G(k) = a + b k      (encoder and fixed GPU work a, b per GPU block)
//   T_X    = x            (boundary transfer, independent of k)
//   T_C(k) = c (N - k)    (c per host block)
// a and b come from a running least-squares fit over the (k, T_G) samples,
// held to the caller's prior until two distinct k have been seen; c is the
// running mean of T_C / (N - k).  Contention scales a stage by 1 / (1 - u):
// a processor other modules use a fraction u of gives the pipeline the rest.
// The decision minimises the predicted stream interval of Eq. (13),
//   max(T_G(k) / (1 - u_gpu), x + T_C(k) / (1 - u_cpu)),
// over k in the dynamic zone [k_lo, k_hi], subject to an optional GPU-time
// budget (over it, the step towards it), moving at most one block per frame
// (layers migrate only across the boundary, one at a time) and never towards
// the host while the consumer queue is backed up.

#include <algorithm>
#include <cmath>
#include <memory>

#include "../../include/vla_suffix.h"

struct vla_sched {
  int N = 0, k_lo = 0, k_hi = 0, k = 0, backlog_hi = 0;
  double a = 0, b = 0, c = 0, x = 0;
  // least squares over (k, T_G): sums of 1, k, k^2, T, k T (exponentially forgotten)
  double s0 = 0, s1 = 0, s2 = 0, sy = 0, sky = 0;
  double c_num = 0, c_den = 0, x_sum = 0, x_n = 0;
  double forget = 0.9;
};

namespace {

bool finite_nonneg(float v) { return std::isfinite(v) && v >= 0.f; }

}  // namespace

extern "C" {

vla_status vla_sched_create(int n_blocks, int k_lo, int k_hi, int k_init, float a_ms, float b_ms, float c_ms,
                            float x_ms, int backlog_hi, vla_sched** out) {
  if (!out) return VLA_ERR_INVALID_ARG;
  *out = nullptr;
  if (n_blocks <= 0 || k_lo < 0 || k_hi < k_lo || k_hi > n_blocks || k_init < k_lo || k_init > k_hi ||
      backlog_hi < 1)
    return VLA_ERR_INVALID_ARG;
  if (!finite_nonneg(a_ms) || !finite_nonneg(b_ms) || !finite_nonneg(c_ms) || !finite_nonneg(x_ms))
    return VLA_ERR_INVALID_ARG;
  try {
    auto s = std::make_unique<vla_sched>();
    s->N = n_blocks;
    s->k_lo = k_lo;
    s->k_hi = k_hi;
    s->k = k_init;
    s->backlog_hi = backlog_hi;
    s->a = a_ms;
    s->b = b_ms;
    s->c = c_ms;
    s->x = x_ms;
    *out = s.release();
    return VLA_OK;
  } catch (...) {
    return VLA_ERR_OOM;
  }
}

vla_status vla_sched_observe(vla_sched* s, int k, float t_g_ms, float t_x_ms, float t_c_ms) {
  if (!s || k < 0 || k > s->N) return VLA_ERR_INVALID_ARG;
  if (!finite_nonneg(t_g_ms) || !finite_nonneg(t_x_ms) || !finite_nonneg(t_c_ms)) return VLA_ERR_INVALID_ARG;
  const double f = s->forget;
  s->s0 = f * s->s0 + 1.0;
  s->s1 = f * s->s1 + k;
  s->s2 = f * s->s2 + (double)k * k;
  s->sy = f * s->sy + t_g_ms;
  s->sky = f * s->sky + (double)k * t_g_ms;
  const double det = s->s0 * s->s2 - s->s1 * s->s1;
  if (det > 1e-6 * s->s0 * s->s0) {
    // two or more distinct k: the least-squares line through the samples
    const double b = (s->s0 * s->sky - s->s1 * s->sy) / det;
    if (b >= 0.0) {
      s->b = b;
      s->a = std::max(0.0, (s->sy - b * s->s1) / s->s0);
    }
  } else {
    // one k so far: keep the per-block slope, move the intercept
    s->a = std::max(0.0, s->sy / s->s0 - s->b * (s->s1 / s->s0));
  }
  if (k < s->N) {
    s->c_num = f * s->c_num + t_c_ms;
    s->c_den = f * s->c_den + (s->N - k);
    s->c = s->c_num / s->c_den;
  }
  s->x_sum = f * s->x_sum + t_x_ms;
  s->x_n = f * s->x_n + 1.0;
  s->x = s->x_sum / s->x_n;
  return VLA_OK;
}

vla_status vla_sched_predict(const vla_sched* s, int k, float u_gpu, float u_cpu, float* t_g_ms, float* t_c_ms,
                             float* t_stream_ms) {
  if (!s || k < 0 || k > s->N || !(u_gpu >= 0.f && u_gpu < 1.f) || !(u_cpu >= 0.f && u_cpu < 1.f))
    return VLA_ERR_INVALID_ARG;
  const double g = (s->a + s->b * k) / (1.0 - u_gpu);
  const double c = s->c * (s->N - k) / (1.0 - u_cpu);
  if (t_g_ms) *t_g_ms = (float)g;
  if (t_c_ms) *t_c_ms = (float)c;
  if (t_stream_ms) *t_stream_ms = (float)std::max(g, (k < s->N ? s->x : 0.0) + c);
  return VLA_OK;
}

vla_status vla_sched_decide(vla_sched* s, float u_gpu, float u_cpu, int backlog, float gpu_budget_ms, int* k_out) {
  if (!s || !k_out || backlog < 0 || !(u_gpu >= 0.f && u_gpu < 1.f) || !(u_cpu >= 0.f && u_cpu < 1.f))
    return VLA_ERR_INVALID_ARG;
  // candidates: one block either way inside the dynamic zone; no move towards
  // the host while the consumer's queue is at or above its limit
  const int lo = std::max(s->k_lo, backlog >= s->backlog_hi ? s->k : s->k - 1);
  const int hi = std::min(s->k_hi, s->k + 1);
  int best = s->k;
  float best_t = INFINITY;
  bool best_fits = false;
  for (int k = lo; k <= hi; ++k) {
    float tg, ts;
    vla_sched_predict(s, k, u_gpu, u_cpu, &tg, nullptr, &ts);
    const bool fits = !(gpu_budget_ms > 0.f) || tg <= gpu_budget_ms;
    // a candidate within the GPU budget beats one outside it; among those
    // within, the shorter interval wins, among those outside, the shorter GPU
    // stage (moving towards the budget); ties keep fewer blocks on the GPU
    const float t = fits ? ts : tg;
    if ((fits && !best_fits) || (fits == best_fits && t < best_t)) {
      best = k;
      best_t = t;
      best_fits = fits;
    }
  }
  s->k = best;
  *k_out = best;
  return VLA_OK;
}

vla_status vla_sched_model(const vla_sched* s, float* a_ms, float* b_ms, float* c_ms, float* x_ms) {
  if (!s) return VLA_ERR_INVALID_ARG;
  if (a_ms) *a_ms = (float)s->a;
  if (b_ms) *b_ms = (float)s->b;
  if (c_ms) *c_ms = (float)s->c;
  if (x_ms) *x_ms = (float)s->x;
  return VLA_OK;
}

void vla_sched_destroy(vla_sched* s) { delete s; }

}  // extern "C"
