// C ABI of the host suffix executor and the cross-frame pipeline consumer
// (include/vla_suffix.h).  This file is built without AVX-512 so that the
// CPU check runs before any AVX-512 code does.

#include <hip/hip_runtime.h>

#include <chrono>
#include <condition_variable>
#include <deque>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/vla_suffix.h"
#include "host_suffix.h"

namespace vla {
int ctx_device(const vla_ctx* c);
hipStream_t ctx_copy_stream(const vla_ctx* c);
}  // namespace vla

struct vla_suffix {
  vla::host::Suffix* impl = nullptr;
  vla::host::Cfg cfg{};
  int k_begin = 0, k_end = 0;
};

namespace {

bool cpu_ok() {
  __builtin_cpu_init();
  return __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") &&
         __builtin_cpu_supports("avx512vl") && __builtin_cpu_supports("avx512bf16");
}

double ms_since(std::chrono::steady_clock::time_point t0) {
  return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
}

}  // namespace

extern "C" {

vla_status vla_suffix_create(const vla_stack_cfg* llm, int k_begin, int k_end, int n_threads, vla_suffix** out) {
  if (!llm || !out) return VLA_ERR_INVALID_ARG;
  *out = nullptr;
  if (k_begin < 0 || k_end <= k_begin) return VLA_ERR_INVALID_ARG;
  if (llm->dtype != VLA_BF16 || llm->norm_is_layernorm || llm->mlp_is_gelu || llm->has_bias) return VLA_ERR_UNSUPPORTED;
  const int d = llm->d_model, H = llm->n_heads, Hkv = llm->n_kv_heads, dh = llm->head_dim, F = llm->d_ff;
  if (d <= 0 || H <= 0 || Hkv <= 0 || dh <= 0 || F <= 0 || H % Hkv) return VLA_ERR_INVALID_ARG;
  // 64-column output tiles must not straddle a head, and d a whole number of 16-float vectors
  if (dh % 64 || d % 16 || F % 2) return VLA_ERR_UNSUPPORTED;
  if (!cpu_ok()) return VLA_ERR_UNSUPPORTED;
  try {
    auto s = std::make_unique<vla_suffix>();
    s->cfg = vla::host::Cfg{d, H, Hkv, dh, F, llm->causal, llm->use_rope, llm->norm_eps, llm->rope_base};
    s->k_begin = k_begin;
    s->k_end = k_end;
    s->impl = vla::host::create(s->cfg, k_begin, k_end, n_threads);
    *out = s.release();
    return VLA_OK;
  } catch (...) {
    return VLA_ERR_OOM;
  }
}

vla_status vla_suffix_load_block_weights(vla_suffix* s, int block, const vla_block_weights* w) {
  if (!s || !w) return VLA_ERR_INVALID_ARG;
  if (block < s->k_begin || block >= s->k_end) return VLA_ERR_INVALID_ARG;
  if (!w->w_q || !w->w_k || !w->w_v || !w->w_o || !w->w_gate || !w->w_up || !w->w_down || !w->norm1_g || !w->norm2_g)
    return VLA_ERR_INVALID_ARG;
  try {
    vla::host::Weights hw{(const uint16_t*)w->w_q,    (const uint16_t*)w->w_k,  (const uint16_t*)w->w_v,
                          (const uint16_t*)w->w_o,    (const uint16_t*)w->w_gate, (const uint16_t*)w->w_up,
                          (const uint16_t*)w->w_down, (const uint16_t*)w->norm1_g, (const uint16_t*)w->norm2_g};
    vla::host::load_block(s->impl, block, hw);
    return VLA_OK;
  } catch (...) {
    return VLA_ERR_OOM;
  }
}

vla_status vla_suffix_run_from(vla_suffix* s, int k, const void* h, vla_dtype in_dtype, int B, int L, float* out) {
  if (!s || !h || !out || B <= 0 || L <= 0) return VLA_ERR_INVALID_ARG;
  if (in_dtype != VLA_BF16 && in_dtype != VLA_F32) return VLA_ERR_INVALID_ARG;
  if (k < s->k_begin || k > s->k_end) return VLA_ERR_INVALID_ARG;
  if (!vla::host::all_loaded(s->impl)) return VLA_ERR_NOT_LOADED;
  try {
    vla::host::run(s->impl, k, h, in_dtype == VLA_F32, B, L, out);
    return VLA_OK;
  } catch (...) {
    return VLA_ERR_OOM;
  }
}

vla_status vla_suffix_run(vla_suffix* s, const void* h, vla_dtype in_dtype, int B, int L, float* out) {
  if (!s) return VLA_ERR_INVALID_ARG;
  return vla_suffix_run_from(s, s->k_begin, h, in_dtype, B, L, out);
}

vla_status vla_suffix_set_cache(vla_suffix* s, int B, int L_cap) {
  if (!s || B < 0 || L_cap < 0) return VLA_ERR_INVALID_ARG;
  try {
    vla::host::set_cache(s->impl, B, L_cap);
    return VLA_OK;
  } catch (...) {
    vla::host::set_cache(s->impl, 0, 0);
    return VLA_ERR_OOM;
  }
}

vla_status vla_suffix_decode_step(vla_suffix* s, int k, const void* h, vla_dtype in_dtype, int B, int pos,
                                  float* out) {
  if (!s || !h || !out || B <= 0) return VLA_ERR_INVALID_ARG;
  if (in_dtype != VLA_BF16 && in_dtype != VLA_F32) return VLA_ERR_INVALID_ARG;
  if (k < s->k_begin || k > s->k_end) return VLA_ERR_INVALID_ARG;
  if (B != vla::host::cache_batch(s->impl) || pos < 0 || pos >= vla::host::cache_len(s->impl)) return VLA_ERR_SHAPE;
  if (!vla::host::all_loaded(s->impl)) return VLA_ERR_NOT_LOADED;
  try {
    vla::host::decode(s->impl, k, h, in_dtype == VLA_F32, B, pos, out);
    return VLA_OK;
  } catch (...) {
    return VLA_ERR_OOM;
  }
}

vla_status vla_suffix_threads(const vla_suffix* s, int* n) {
  if (!s || !n) return VLA_ERR_INVALID_ARG;
  *n = vla::host::threads(s->impl);
  return VLA_OK;
}

void vla_suffix_destroy(vla_suffix* s) {
  if (!s) return;
  vla::host::destroy(s->impl);
  delete s;
}

}  // extern "C"

// ------------------------------------------------------------------ pipeline

struct vla_pipeline {
  struct Job {
    uint64_t id = 0;
    hipEvent_t ev = nullptr;
    const void* h = nullptr;
    vla_dtype dt = VLA_BF16;
    int B = 0, L = 0, k = 0;
    float* out = nullptr;
    bool done = false;
    vla_status st = VLA_OK;
    float t_wait = 0.f, t_cpu = 0.f;
  };
  vla_suffix* s = nullptr;
  int device = 0, depth = 1;
  hipStream_t copy = nullptr;
  std::mutex mu;
  std::condition_variable cv_work, cv_done, cv_space;
  std::deque<std::shared_ptr<Job>> all, todo;  // all: pushed, not popped (oldest first)
  std::vector<hipEvent_t> free_ev;
  bool stop = false;
  std::thread th;

  void work() {
    if (hipSetDevice(device) != hipSuccess) {
      std::lock_guard<std::mutex> g(mu);
      stop = true;
    }
    for (;;) {
      std::shared_ptr<Job> j;
      {
        std::unique_lock<std::mutex> lk(mu);
        cv_work.wait(lk, [&] { return stop || !todo.empty(); });
        if (todo.empty()) return;
        j = todo.front();
        todo.pop_front();
      }
      auto t0 = std::chrono::steady_clock::now();
      vla_status st = hipEventSynchronize(j->ev) == hipSuccess ? VLA_OK : VLA_ERR_HIP;
      const float tw = (float)ms_since(t0);
      auto t1 = std::chrono::steady_clock::now();
      if (st == VLA_OK) st = vla_suffix_run_from(s, j->k, j->h, j->dt, j->B, j->L, j->out);
      const float tc = (float)ms_since(t1);
      {
        std::lock_guard<std::mutex> g(mu);
        j->st = st;
        j->t_wait = tw;
        j->t_cpu = tc;
        j->done = true;
      }
      cv_done.notify_all();
    }
  }
};

extern "C" {

vla_status vla_pipeline_create(vla_ctx* ctx, vla_suffix* s, int depth, vla_pipeline** out) {
  if (!ctx || !s || !out || depth <= 0) return VLA_ERR_INVALID_ARG;
  *out = nullptr;
  try {
    auto p = std::make_unique<vla_pipeline>();
    p->s = s;
    p->depth = depth;
    p->device = vla::ctx_device(ctx);
    p->copy = vla::ctx_copy_stream(ctx);
    if (hipSetDevice(p->device) != hipSuccess) return VLA_ERR_HIP;
    for (int i = 0; i < depth; ++i) {
      hipEvent_t e;
      if (hipEventCreateWithFlags(&e, hipEventDisableTiming | hipEventBlockingSync) != hipSuccess) {
        for (hipEvent_t x : p->free_ev) (void)hipEventDestroy(x);
        return VLA_ERR_HIP;
      }
      p->free_ev.push_back(e);
    }
    vla_pipeline* raw = p.get();
    p->th = std::thread([raw] { raw->work(); });
    *out = p.release();
    return VLA_OK;
  } catch (...) {
    return VLA_ERR_OOM;
  }
}

vla_status vla_pipeline_push(vla_pipeline* p, uint64_t frame_id, const vla_boundary* b, int B, int L, int k,
                             float* out) {
  if (!p || !b || !b->hidden || !out || B <= 0 || L <= 0) return VLA_ERR_INVALID_ARG;
  if (k < p->s->k_begin || k > p->s->k_end) return VLA_ERR_INVALID_ARG;
  const size_t need = (size_t)B * L * p->s->cfg.d * (b->out_dtype == VLA_F32 ? 4 : 2);
  if (b->hidden_bytes < need) return VLA_ERR_SHAPE;
  auto j = std::make_shared<vla_pipeline::Job>();
  j->id = frame_id;
  j->h = b->hidden;
  j->dt = b->out_dtype;
  j->B = B;
  j->L = L;
  j->k = k;
  j->out = out;
  std::unique_lock<std::mutex> lk(p->mu);
  p->cv_space.wait(lk, [&] { return (int)p->all.size() < p->depth; });
  j->ev = p->free_ev.back();
  if (hipSetDevice(p->device) != hipSuccess || hipEventRecord(j->ev, p->copy) != hipSuccess) return VLA_ERR_HIP;
  p->free_ev.pop_back();
  p->all.push_back(j);
  p->todo.push_back(j);
  lk.unlock();
  p->cv_work.notify_one();
  return VLA_OK;
}

vla_status vla_pipeline_pop(vla_pipeline* p, uint64_t* frame_id, float* t_wait_ms, float* t_cpu_ms, int timeout_ms) {
  if (!p) return VLA_ERR_INVALID_ARG;
  std::unique_lock<std::mutex> lk(p->mu);
  if (p->all.empty()) return VLA_ERR_UNKNOWN_FRAME;
  auto ready = [&] { return p->all.front()->done; };
  if (timeout_ms < 0)
    p->cv_done.wait(lk, ready);
  else if (!p->cv_done.wait_for(lk, std::chrono::milliseconds(timeout_ms), ready))
    return VLA_ERR_TIMEOUT;
  auto j = p->all.front();
  p->all.pop_front();
  p->free_ev.push_back(j->ev);
  lk.unlock();
  p->cv_space.notify_one();
  if (frame_id) *frame_id = j->id;
  if (t_wait_ms) *t_wait_ms = j->t_wait;
  if (t_cpu_ms) *t_cpu_ms = j->t_cpu;
  return j->st;
}

vla_status vla_pipeline_backlog(vla_pipeline* p, int* n) {
  if (!p || !n) return VLA_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> g(p->mu);
  *n = (int)p->all.size();
  return VLA_OK;
}

void vla_pipeline_destroy(vla_pipeline* p) {
  if (!p) return;
  {
    std::lock_guard<std::mutex> g(p->mu);
    p->stop = true;
  }
  p->cv_work.notify_all();
  if (p->th.joinable()) p->th.join();
  (void)hipSetDevice(p->device);
  for (hipEvent_t e : p->free_ev) (void)hipEventDestroy(e);
  for (auto& j : p->all) (void)hipEventDestroy(j->ev);
  delete p;
}

}  // extern "C"
