// Runtime of the VLA prefix library: context, arena sub-allocation, weight
// packing, block sequencing on the compute stream and the frame handoff on the
// copy stream.  Implements include/vla_prefix.h.

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <memory>
#include <string>
#include <thread>
#include <vector>

#include "../../include/vla_prefix.h"
#include "kernels.h"

namespace {

thread_local std::string g_last_error;

constexpr int NSLOT = 3;          // frames that may be in flight at once
constexpr size_t ALIGN = 256;     // arena sub-allocation alignment
constexpr size_t HISTORY = 256;   // finished frames whose times are kept

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int round_up(int x, int a) { return (x + a - 1) / a * a; }

struct Status {
  vla_status code;
  std::string msg;
};

[[gnu::format(printf, 2, 3)]] Status fail(vla_status c, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return Status{c, buf};
}
const Status OK{VLA_OK, ""};

#define HIPTRY(expr)                                                                         \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(VLA_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

size_t dtype_size(vla_dtype t) { return t == VLA_BF16 ? 2 : 4; }

// Derived, validated view of one stack.
struct Stack {
  bool present = false;
  vla_stack_cfg c{};
  size_t esz = 0;
  int hd = 0, kvd = 0, qkv_n = 0, f_pad = 0, ldvt = 0;
  size_t m_max = 0;  // max_batch * max_tokens

  struct Block {
    void *w_qkv = nullptr, *w_o = nullptr, *w_up = nullptr, *w_down = nullptr;  // w_up: gate/up or fc1
    float *b_qkv = nullptr, *b_o = nullptr, *b_up = nullptr, *b_down = nullptr;
    float *n1g = nullptr, *n1b = nullptr, *n2g = nullptr, *n2b = nullptr;
    bool loaded = false;
  };
  std::vector<Block> blocks;

  // activation operands of the QKV, gate/up and down GEMMs: bf16, or split
  // into a hi + lo pair of bf16 values (bf16 decoder stacks)
  vla_precision prec = VLA_PREC_BF16;
  bool bf16() const { return c.dtype == VLA_BF16; }
  bool llm() const { return !c.norm_is_layernorm; }
  // the operand buffers hold a split pair (bf16 decoder stacks), so either
  // precision can run without a new arena
  bool split_room() const { return bf16() && llm(); }
  int parts() const { return prec == VLA_PREC_SPLIT ? 2 : 1; }
  // rows of the up projection: interleaved gate/up (LLM) or fc1 (encoder)
  int up_rows() const { return llm() ? 2 * f_pad : f_pad; }
  // arena bytes of a weight matrix [N][K]: bf16 stacks hold it packed
  // slab-major over slab_blocks(N) blocks, fp32 stacks row-major
  size_t weight_bytes(int N, int K) const {
    return bf16() ? (size_t)vla::slab_blocks(N) * vla::SLAB_N * K * esz : (size_t)N * K * esz;
  }
  // the GEMM operand of a resident bf16 weight matrix with N rows
  static vla::WOperand packed(const void* p, int N) { return vla::WOperand{(const bf16_t*)p, 0, vla::slab_blocks(N)}; }
};

Status validate_stack(const vla_stack_cfg* c, bool is_llm, Stack* s) {
  s->present = false;
  if (!c) return OK;
  const char* w = is_llm ? "llm" : "enc";
  if (c->dtype != VLA_BF16 && c->dtype != VLA_F32) return fail(VLA_ERR_INVALID_ARG, "%s: bad dtype", w);
  if (c->n_blocks < 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->d_ff <= 0 || c->max_tokens <= 0 || c->max_batch <= 0)
    return fail(VLA_ERR_INVALID_ARG, "%s: non-positive dimension", w);
  if (c->n_heads % c->n_kv_heads) return fail(VLA_ERR_INVALID_ARG, "%s: n_heads %% n_kv_heads != 0", w);
  if (is_llm) {
    if (c->norm_is_layernorm || c->mlp_is_gelu || c->has_bias)
      return fail(VLA_ERR_UNSUPPORTED, "llm stack must be RMSNorm / SwiGLU / no bias");
  } else {
    if (!c->norm_is_layernorm || !c->mlp_is_gelu || !c->has_bias || c->use_rope || c->causal)
      return fail(VLA_ERR_UNSUPPORTED, "encoder stack must be LayerNorm / GELU / biases / no rope / bidirectional");
    if (c->n_kv_heads != c->n_heads) return fail(VLA_ERR_UNSUPPORTED, "encoder stack needs n_kv_heads == n_heads");
  }
  if (c->d_model % 4) return fail(VLA_ERR_UNSUPPORTED, "%s: d_model must be a multiple of 4", w);
  if (c->d_model > 8192) return fail(VLA_ERR_UNSUPPORTED, "%s: d_model > 8192", w);
  if (c->head_dim % 2 || c->head_dim > 128) return fail(VLA_ERR_UNSUPPORTED, "%s: head_dim must be even, <= 128", w);
  if (c->dtype == VLA_BF16) {
    if (c->head_dim != 64 && c->head_dim != 128)
      return fail(VLA_ERR_UNSUPPORTED, "%s: bf16 path needs head_dim 64 or 128", w);
    if (c->d_model % 64 || (c->n_heads * c->head_dim) % 64)
      return fail(VLA_ERR_UNSUPPORTED, "%s: bf16 path needs d_model and n_heads*head_dim multiples of 64", w);
  }
  if (!(c->norm_eps >= 0.f)) return fail(VLA_ERR_INVALID_ARG, "%s: norm_eps < 0", w);
  if (c->use_rope && !(c->rope_base > 0.f)) return fail(VLA_ERR_INVALID_ARG, "%s: rope_base <= 0", w);
  s->present = true;
  s->c = *c;
  s->esz = dtype_size(c->dtype);
  s->hd = c->n_heads * c->head_dim;
  s->kvd = c->n_kv_heads * c->head_dim;
  s->qkv_n = s->hd + 2 * s->kvd;
  s->f_pad = c->dtype == VLA_BF16 ? round_up(c->d_ff, 64) : c->d_ff;
  s->ldvt = round_up(c->max_tokens, 64);
  s->m_max = (size_t)c->max_batch * c->max_tokens;
  s->blocks.assign(c->n_blocks, Stack::Block{});
  return OK;
}

// Stem and connector around the encoder stack (vla_attach_vision): weights
// and scratch in a device block the caller hands over.
struct Vision {
  bool present = false, loaded = false, bf16 = true;
  vla_vision_cfg c{};
  size_t esz = 2;
  int d = 0, gh = 0, gw = 0, L_img = 0, tpi = 0, K = 0, Kp = 0, md = 0, max_img = 0;
  void *w_patch = nullptr, *w_c1 = nullptr, *w_c2 = nullptr;
  float *b_patch = nullptr, *pos = nullptr, *post_g = nullptr, *post_b = nullptr, *b_c1 = nullptr, *b_c2 = nullptr;
  void *img = nullptr, *A = nullptr, *merged = nullptr, *hid = nullptr;
  size_t bytes = 0;
};

Status validate_vision(const Stack& enc, const vla_vision_cfg* v, Vision* out) {
  if (!v) return fail(VLA_ERR_INVALID_ARG, "NULL vision config");
  if (!enc.present) return fail(VLA_ERR_INVALID_ARG, "the vision front needs an encoder stack");
  if (v->channels <= 0 || v->img_h <= 0 || v->img_w <= 0 || v->patch <= 0 || v->merge <= 0 || v->d_hidden <= 0 ||
      v->d_out <= 0)
    return fail(VLA_ERR_INVALID_ARG, "vision: non-positive dimension");
  if (!(v->norm_eps >= 0.f)) return fail(VLA_ERR_INVALID_ARG, "vision: norm_eps < 0");
  if (v->img_h % v->patch || v->img_w % v->patch)
    return fail(VLA_ERR_UNSUPPORTED, "vision: image sides must be multiples of the patch");
  const int gh = v->img_h / v->patch, gw = v->img_w / v->patch;
  if (gh % v->merge || gw % v->merge)
    return fail(VLA_ERR_UNSUPPORTED, "vision: patch grid %dx%d is not a multiple of merge %d", gh, gw, v->merge);
  if (gh * gw > enc.c.max_tokens)
    return fail(VLA_ERR_SHAPE, "vision: %d patches per image exceed the encoder's max_tokens %d", gh * gw,
                enc.c.max_tokens);
  const bool b = enc.bf16();
  if (b && (v->d_hidden % 64 || v->d_out % 64))
    return fail(VLA_ERR_UNSUPPORTED, "vision: bf16 path needs d_hidden and d_out multiples of 64");
  if (!b && v->d_out % 4) return fail(VLA_ERR_UNSUPPORTED, "vision: d_out must be a multiple of 4");
  const long K = (long)v->channels * v->patch * v->patch;
  if (K > (1 << 20) || (long)v->merge * v->merge * enc.c.d_model > (1 << 20) || v->d_hidden > (1 << 20) ||
      v->d_out > (1 << 20))
    return fail(VLA_ERR_UNSUPPORTED, "vision: dimension above 2^20");
  Vision& o = *out;
  o = Vision{};
  o.present = true;
  o.bf16 = b;
  o.c = *v;
  o.esz = enc.esz;
  o.d = enc.c.d_model;
  o.gh = gh;
  o.gw = gw;
  o.L_img = gh * gw;
  o.tpi = (gh / v->merge) * (gw / v->merge);
  o.K = (int)K;
  o.Kp = b ? round_up((int)K, 64) : (int)K;
  o.md = v->merge * v->merge * o.d;
  o.max_img = enc.c.max_batch;
  return OK;
}

struct Slot {
  uint64_t frame_id = 0;
  bool used = false;
  bool has_kv = false;
  void* kv = nullptr;   // device [n_blocks][2][B][Hkv][L][dh]
  void* hid = nullptr;  // device staging of the boundary
  hipEvent_t ev_start = nullptr, ev_done = nullptr, ev_hid = nullptr, ev_copied = nullptr;
  std::vector<hipEvent_t> ev_kv;
};

struct FrameTimes {
  float gpu, xfer, total;
};

// Times of the last HISTORY finished frames, in a fixed ring (recording a
// frame allocates nothing).
struct History {
  struct Entry {
    uint64_t id = 0;
    bool used = false;
    FrameTimes t{};
  };
  Entry e[HISTORY];
  size_t next = 0;
  const FrameTimes* find(uint64_t id) const {
    for (const Entry& x : e)
      if (x.used && x.id == id) return &x.t;
    return nullptr;
  }
  void erase(uint64_t id) {
    for (Entry& x : e)
      if (x.used && x.id == id) x.used = false;
  }
  void put(uint64_t id, const FrameTimes& t) {
    erase(id);
    e[next] = Entry{id, true, t};
    next = (next + 1) % HISTORY;
  }
};

// Scratch of one stack.  The encoder and the decoder run on streams of their
// own and overlap, so each stack owns its workspace.
struct Workspace {
  float* h = nullptr;        // fp32 residual
  void* x = nullptr;         // normalised activations
  void* q = nullptr;         // [B][H][L][dh]
  void* ek = nullptr;        // encoder K / V (the decoder writes into the slot cache)
  void* ev = nullptr;
  void* vt = nullptr;        // V^T
  void* o = nullptr;         // attention output [M][H*dh]
  void* act = nullptr;       // MLP activation
  float* qkv_raw = nullptr;  // fp32 path only
  void* tok = nullptr;       // staging of host-resident inputs
};

}  // namespace

struct vla_ctx {
  int device = 0;
  Stack llm, enc;
  char* arena = nullptr;
  size_t arena_bytes = 0, used = 0;
  // compute: decoder blocks; encs: encoder blocks; copy: the handoff
  hipStream_t compute = nullptr, encs = nullptr, copy = nullptr;
  bool own_compute = false, own_copy = false;
  std::string last_error;

  Workspace ws[2];  // by vla_stack
  Vision vis;
  float *rope_cos = nullptr, *rope_sin = nullptr;
  // cross-stream order: a prefix waits for the latest encoder run (whose
  // output it may read); an encoder's output write waits for the latest
  // prefix intake (which may read the buffer being overwritten)
  hipEvent_t ev_enc_done = nullptr, ev_intake = nullptr;
  bool enc_recorded = false, intake_recorded = false;
  Slot slots[NSLOT];
  int next_slot = 0;
  History history;
  // the fixed decode scratch of this device (vla_decode_step_static), and an
  // event marking the copy stream's tail when such a step starts
  void* sscratch = nullptr;
  hipEvent_t ev_copy_tail = nullptr;

  // kernel profiler: event pairs around each launch on the compute stream
  struct ProfRec {
    int idx;
    hipEvent_t a, b;
  };
  // launches left before an injected failure (vla_inject_fault); < 0: none
  long fault_after = -1;
  bool prof_on = false;
  std::vector<hipEvent_t> prof_pool;
  size_t prof_used = 0;
  std::vector<ProfRec> prof_recs;
  double prof_ms[2][VLA_K_COUNT] = {};
  int prof_n[2][VLA_K_COUNT] = {};
};

// Device and copy stream of a context, for the host pipeline consumer
// (host_suffix_api.cpp), which marks the end of a frame's copies there.
namespace vla {
int ctx_device(const vla_ctx* c) { return c->device; }
hipStream_t ctx_copy_stream(const vla_ctx* c) { return c->copy; }
}  // namespace vla

namespace {

// Arena layout, shared by vla_query_sizes and vla_create: a bump allocator
// that only counts when base == nullptr.
struct Bump {
  char* base;
  size_t off = 0;
  void* take(size_t bytes) {
    off = align_up(off, ALIGN);
    void* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  }
};

void layout(vla_ctx* c, Bump& a) {
  Stack* stacks[2] = {&c->llm, &c->enc};
  for (Stack* s : stacks) {
    if (!s->present) continue;
    const size_t d = s->c.d_model;
    for (auto& b : s->blocks) {
      b.w_qkv = a.take(s->weight_bytes(s->qkv_n, (int)d));
      b.w_o = a.take(s->weight_bytes((int)d, s->hd));
      b.w_up = a.take(s->weight_bytes(s->up_rows(), (int)d));
      b.w_down = a.take(s->weight_bytes((int)d, s->f_pad));
      b.n1g = (float*)a.take(d * 4);
      b.n2g = (float*)a.take(d * 4);
      if (s->c.has_bias) {
        b.b_qkv = (float*)a.take((size_t)s->qkv_n * 4);
        b.b_o = (float*)a.take(d * 4);
        b.b_up = (float*)a.take((size_t)s->f_pad * 4);
        b.b_down = (float*)a.take(d * 4);
      }
      if (s->c.norm_is_layernorm) {
        b.n1b = (float*)a.take(d * 4);
        b.n2b = (float*)a.take(d * 4);
      }
    }
  }
  for (int si = 0; si < 2; ++si) {
    Stack* s = stacks[si];
    if (!s->present) continue;
    Workspace& w = c->ws[si];
    const size_t M = s->m_max, d = s->c.d_model, e = s->esz;
    const size_t pairs = s->split_room() ? 2 : 1;
    w.h = (float*)a.take(M * d * 4);
    w.x = a.take(pairs * M * d * e);
    w.q = a.take(M * s->hd * e);
    if (!s->llm()) {
      w.ek = a.take(M * s->kvd * e);
      // the bf16 encoder's attention reads V^T only: no V rows
      if (!s->bf16()) w.ev = a.take(M * s->kvd * e);
    }
    w.vt = a.take((size_t)s->c.max_batch * s->kvd * s->ldvt * e);
    w.o = a.take(M * s->hd * e);
    w.act = a.take(s->bf16() ? pairs * M * s->f_pad * e : M * (size_t)s->c.d_ff * (s->llm() ? 3 : 1) * 4);
    if (!s->bf16()) w.qkv_raw = (float*)a.take(M * s->qkv_n * 4);
    w.tok = a.take(M * d * e);
  }
  int rope_len = 0, rope_half = 0;
  if (c->llm.present && c->llm.c.use_rope) rope_len = c->llm.c.max_tokens, rope_half = c->llm.c.head_dim / 2;
  c->rope_cos = (float*)a.take((size_t)rope_len * rope_half * 4);
  c->rope_sin = (float*)a.take((size_t)rope_len * rope_half * 4);
  if (c->llm.present) {
    const Stack& s = c->llm;
    for (auto& sl : c->slots) {
      sl.kv = a.take((size_t)s.c.n_blocks * 2 * s.m_max * s.kvd * s.esz);
      sl.hid = a.take(s.m_max * s.c.d_model * 4);
    }
  }
  a.off = align_up(a.off, ALIGN);
}

// The vision block: weights (packed like the blocks' for bf16), then the
// image staging, patch rows, merged rows and the connector's hidden rows.
void layout_vision(Vision& v, Bump& a) {
  const auto wbytes = [&](int N, int K) {
    return v.bf16 ? (size_t)vla::slab_blocks(N) * vla::SLAB_N * K * 2 : (size_t)N * K * 4;
  };
  const vla_vision_cfg& c = v.c;
  v.w_patch = a.take(wbytes(v.d, v.Kp));
  v.b_patch = (float*)a.take((size_t)v.d * 4);
  v.pos = (float*)a.take((size_t)v.L_img * v.d * 4);
  v.post_g = (float*)a.take((size_t)v.d * 4);
  v.post_b = (float*)a.take((size_t)v.d * 4);
  v.w_c1 = a.take(wbytes(c.d_hidden, v.md));
  v.b_c1 = (float*)a.take((size_t)c.d_hidden * 4);
  v.w_c2 = a.take(wbytes(c.d_out, c.d_hidden));
  v.b_c2 = (float*)a.take((size_t)c.d_out * 4);
  const size_t rows = (size_t)v.max_img * v.L_img;
  v.img = a.take((size_t)v.max_img * c.channels * c.img_h * c.img_w * v.esz);
  v.A = a.take(rows * v.Kp * v.esz);
  v.merged = a.take(rows * v.d * v.esz);
  v.hid = a.take((size_t)v.max_img * v.tpi * c.d_hidden * v.esz);
  a.off = align_up(a.off, ALIGN);
}

// ------------------------------------------------------------ weight packing

// bf16 QKV rows: per head, 64-row groups [32 first-half dims | their 32
// second-half partners].  fp32: natural order.
int qkv_packed_to_true_dim(int r, int dh) {
  int c = r / 64, w = r % 64;
  return w < 32 ? c * 32 + w : dh / 2 + c * 32 + (w - 32);
}

float to_f32(const void* p, size_t i, vla_dtype t) {
  if (t == VLA_F32) return ((const float*)p)[i];
  uint32_t u = (uint32_t)((const uint16_t*)p)[i] << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

std::vector<float> vec_f32(const void* p, size_t n, vla_dtype t) {
  std::vector<float> v(n);
  for (size_t i = 0; i < n; ++i) v[i] = to_f32(p, i, t);
  return v;
}

Status copy_h2d(void* dst, const void* src, size_t bytes) {
  HIPTRY(hipMemcpy(dst, src, bytes, hipMemcpyHostToDevice));
  return OK;
}

// Row-major weight rows [N][K] -> the arena: packed slab-major for bf16
// stacks (the layout the GEMMs read, kernels.h), as-is for fp32 stacks.
Status put_matrix(bool bf16, void* dst, const void* rm, int N, int K) {
  if (!bf16) return copy_h2d(dst, rm, (size_t)N * K * 4);
  std::vector<uint16_t> t((size_t)vla::slab_blocks(N) * vla::SLAB_N * K);
  vla::pack_slabs((const uint16_t*)rm, t.data(), N, K);
  return copy_h2d(dst, t.data(), t.size() * 2);
}

Status put_weight(const Stack& s, void* dst, const void* rm, int N, int K) { return put_matrix(s.bf16(), dst, rm, N, K); }

Status load_vision(Vision& v, vla_dtype dt, const vla_vision_weights* w) {
  if (!w->w_patch || !w->b_patch || !w->pos || !w->post_g || !w->post_b || !w->w_c1 || !w->b_c1 || !w->w_c2 ||
      !w->b_c2)
    return fail(VLA_ERR_INVALID_ARG, "vision weights: every field is required");
  v.loaded = false;
  const vla_vision_cfg& c = v.c;
  // stem rows [d][K], zero columns up to Kp
  std::vector<char> buf((size_t)v.d * v.Kp * v.esz, 0);
  for (int r = 0; r < v.d; ++r)
    memcpy(&buf[(size_t)r * v.Kp * v.esz], (const char*)w->w_patch + (size_t)r * v.K * v.esz, (size_t)v.K * v.esz);
  Status st = put_matrix(v.bf16, v.w_patch, buf.data(), v.d, v.Kp);
  if (st.code) return st;
  if ((st = put_matrix(v.bf16, v.w_c1, w->w_c1, c.d_hidden, v.md)).code) return st;
  if ((st = put_matrix(v.bf16, v.w_c2, w->w_c2, c.d_out, c.d_hidden)).code) return st;
  auto put = [&](float* dst, const void* src, size_t n) -> Status {
    std::vector<float> f = vec_f32(src, n, dt);
    return copy_h2d(dst, f.data(), n * 4);
  };
  if ((st = put(v.b_patch, w->b_patch, v.d)).code) return st;
  if ((st = put(v.pos, w->pos, (size_t)v.L_img * v.d)).code) return st;
  if ((st = put(v.post_g, w->post_g, v.d)).code) return st;
  if ((st = put(v.post_b, w->post_b, v.d)).code) return st;
  if ((st = put(v.b_c1, w->b_c1, c.d_hidden)).code) return st;
  if ((st = put(v.b_c2, w->b_c2, c.d_out)).code) return st;
  v.loaded = true;
  return OK;
}

Status load_block(vla_ctx* c, Stack& s, int bi, const vla_block_weights* w) {
  const vla_stack_cfg& k = s.c;
  const bool llm = s.llm();
  const size_t d = k.d_model, e = s.esz, dh = k.head_dim;
  // required / forbidden pointers
  if (!w->w_q || !w->w_k || !w->w_v || !w->w_o || !w->norm1_g || !w->norm2_g)
    return fail(VLA_ERR_INVALID_ARG, "block %d: missing attention weights or norm gains", bi);
  if (llm) {
    if (!w->w_gate || !w->w_up || !w->w_down) return fail(VLA_ERR_INVALID_ARG, "block %d: missing SwiGLU weights", bi);
    if (w->w_fc1 || w->w_fc2 || w->b_fc1 || w->b_fc2 || w->b_qkv || w->b_o || w->norm1_b || w->norm2_b)
      return fail(VLA_ERR_INVALID_ARG, "block %d: decoder blocks take no biases / fc weights / norm shifts", bi);
  } else {
    if (!w->w_fc1 || !w->w_fc2 || !w->b_fc1 || !w->b_fc2 || !w->b_qkv || !w->b_o || !w->norm1_b || !w->norm2_b)
      return fail(VLA_ERR_INVALID_ARG, "block %d: missing encoder weights, biases or norm shifts", bi);
    if (w->w_gate || w->w_up || w->w_down)
      return fail(VLA_ERR_INVALID_ARG, "block %d: encoder blocks take no SwiGLU weights", bi);
  }
  Stack::Block& b = s.blocks[bi];
  b.loaded = false;
  // QKV
  {
    std::vector<char> buf((size_t)s.qkv_n * d * e);
    const void* src[3] = {w->w_q, w->w_k, w->w_v};
    const int heads[3] = {k.n_heads, k.n_kv_heads, k.n_kv_heads};
    size_t prow = 0;
    for (int part = 0; part < 3; ++part)
      for (int hh = 0; hh < heads[part]; ++hh)
        for (size_t r = 0; r < dh; ++r, ++prow) {
          size_t tr = hh * dh + (s.bf16() ? qkv_packed_to_true_dim((int)r, (int)dh) : r);
          memcpy(&buf[prow * d * e], (const char*)src[part] + tr * d * e, d * e);
        }
    Status st = put_weight(s, b.w_qkv, buf.data(), s.qkv_n, (int)d);
    if (st.code) return st;
    if (k.has_bias) {
      std::vector<float> bias(s.qkv_n);
      const size_t offs[3] = {0, (size_t)s.hd, (size_t)(s.hd + s.kvd)};
      prow = 0;
      for (int part = 0; part < 3; ++part)
        for (int hh = 0; hh < heads[part]; ++hh)
          for (size_t r = 0; r < dh; ++r, ++prow) {
            size_t tr = hh * dh + (s.bf16() ? qkv_packed_to_true_dim((int)r, (int)dh) : r);
            bias[prow] = to_f32(w->b_qkv, offs[part] + tr, k.dtype);
          }
      if ((st = copy_h2d(b.b_qkv, bias.data(), bias.size() * 4)).code) return st;
    }
  }
  Status st = put_weight(s, b.w_o, w->w_o, (int)d, s.hd);
  if (st.code) return st;
  // up projection: interleaved gate/up (bf16), [gate; up] (fp32), or fc1
  {
    const size_t F = k.d_ff;
    std::vector<char> buf((size_t)s.up_rows() * d * e, 0);
    if (llm) {
      for (int p = 0; p < s.up_rows(); ++p) {
        size_t f;
        const void* src;
        if (s.bf16()) {
          int g = p / 64, wi = p % 64;
          f = g * 32 + (wi % 32);
          src = wi < 32 ? w->w_gate : w->w_up;
        } else {
          f = p < (int)F ? p : p - F;
          src = p < (int)F ? w->w_gate : w->w_up;
        }
        if (f < F) memcpy(&buf[(size_t)p * d * e], (const char*)src + f * d * e, d * e);
      }
    } else {
      memcpy(buf.data(), w->w_fc1, F * d * e);
    }
    if ((st = put_weight(s, b.w_up, buf.data(), s.up_rows(), (int)d)).code) return st;
  }
  // down projection [d][f_pad] with zero pad columns
  {
    const size_t F = k.d_ff, FP = s.f_pad;
    const void* src = llm ? w->w_down : w->w_fc2;
    std::vector<char> buf(d * FP * e, 0);
    for (size_t r = 0; r < d; ++r) memcpy(&buf[r * FP * e], (const char*)src + r * F * e, F * e);
    if ((st = put_weight(s, b.w_down, buf.data(), (int)d, (int)FP)).code) return st;
  }
  auto put = [&](float* dst, const void* src, size_t n, size_t npad) -> Status {
    std::vector<float> v = vec_f32(src, n, k.dtype);
    v.resize(npad, 0.f);
    return copy_h2d(dst, v.data(), npad * 4);
  };
  if ((st = put(b.n1g, w->norm1_g, d, d)).code) return st;
  if ((st = put(b.n2g, w->norm2_g, d, d)).code) return st;
  if (k.norm_is_layernorm) {
    if ((st = put(b.n1b, w->norm1_b, d, d)).code) return st;
    if ((st = put(b.n2b, w->norm2_b, d, d)).code) return st;
  }
  if (k.has_bias) {
    if ((st = put(b.b_o, w->b_o, d, d)).code) return st;
    if ((st = put(b.b_up, w->b_fc1, k.d_ff, s.f_pad)).code) return st;
    if ((st = put(b.b_down, w->b_fc2, d, d)).code) return st;
  }
  b.loaded = true;
  return OK;
}

// ------------------------------------------------------------- execution

bool is_pinned_host(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeHost;
}

bool is_device(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged;
}

Status prof_event(vla_ctx* c, hipEvent_t* e) {
  if (c->prof_used == c->prof_pool.size()) {
    hipEvent_t ev;
    HIPTRY(hipEventCreate(&ev));
    c->prof_pool.push_back(ev);
  }
  *e = c->prof_pool[c->prof_used++];
  return OK;
}

hipStream_t stream_of(const vla_ctx* c, int stk) { return stk == VLA_STACK_ENC ? c->encs : c->compute; }

Status prof_drain(vla_ctx* c) {
  HIPTRY(hipStreamSynchronize(c->compute));
  if (c->encs != c->compute) HIPTRY(hipStreamSynchronize(c->encs));
  for (const auto& r : c->prof_recs) {
    float ms = 0.f;
    HIPTRY(hipEventElapsedTime(&ms, r.a, r.b));
    c->prof_ms[r.idx / VLA_K_COUNT][r.idx % VLA_K_COUNT] += ms;
    c->prof_n[r.idx / VLA_K_COUNT][r.idx % VLA_K_COUNT] += 1;
  }
  c->prof_recs.clear();
  c->prof_used = 0;
  return OK;
}

#define KTRY(expr)                                                                                   \
  do {                                                                                               \
    hipError_t e_ = (expr);                                                                          \
    if (e_ != hipSuccess) return fail(VLA_ERR_HIP, "launch %s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// Launch `expr` (on the stack's stream); with the profiler on, bracket it
// with a pair of events on that stream attributed to (stack, class).
#define PLAUNCH(c, stk, cls, expr)                                                          \
  do {                                                                                      \
    if ((c)->fault_after >= 0 && (c)->fault_after-- == 0)                                   \
      return fail(VLA_ERR_HIP, "injected failure before launch %s", #expr);                 \
    hipEvent_t a_ = nullptr, b_ = nullptr;                                                  \
    if ((c)->prof_on) {                                                                     \
      Status s_ = prof_event((c), &a_);                                                     \
      if (s_.code) return s_;                                                               \
      HIPTRY(hipEventRecord(a_, stream_of((c), (stk))));                                    \
    }                                                                                       \
    KTRY(expr);                                                                             \
    if ((c)->prof_on) {                                                                     \
      Status s_ = prof_event((c), &b_);                                                     \
      if (s_.code) return s_;                                                               \
      HIPTRY(hipEventRecord(b_, stream_of((c), (stk))));                                    \
      (c)->prof_recs.push_back(vla_ctx::ProfRec{(stk) * VLA_K_COUNT + (cls), a_, b_});      \
      if ((c)->prof_recs.size() >= (1u << 16)) {                                            \
        Status d_ = prof_drain(c);                                                          \
        if (d_.code) return d_;                                                             \
      }                                                                                     \
    }                                                                                       \
  } while (0)

// input[B*L][d] (host or device, element type in_dt) -> the fp32 residual h,
// through the staging buffer tok for host bf16 input
Status intake_to(vla_ctx* c, int stk, vla_dtype in_dt, const void* in, size_t n, float* h, void* tok) {
  const hipStream_t st = stream_of(c, stk);
  const void* src = in;
  if (!is_device(in)) {
    // host input: fp32 goes straight into the residual, bf16 through the
    // input staging buffer
    if (in_dt == VLA_F32) {
      HIPTRY(hipMemcpyAsync(h, in, n * 4, hipMemcpyHostToDevice, st));
      return OK;
    }
    HIPTRY(hipMemcpyAsync(tok, in, n * 2, hipMemcpyHostToDevice, st));
    src = tok;
  }
  if (in_dt == VLA_BF16)
    PLAUNCH(c, stk, VLA_K_OTHER, vla::bf16_to_f32((const bf16_t*)src, h, n, st));
  else
    HIPTRY(hipMemcpyAsync(h, src, n * 4, hipMemcpyDeviceToDevice, st));
  return OK;
}

// ... into the stack's own workspace
Status intake(vla_ctx* c, int stk, vla_dtype in_dt, const void* in, size_t n) {
  return intake_to(c, stk, in_dt, in, n, c->ws[stk].h, c->ws[stk].tok);
}

Status llm_block_bf16(vla_ctx* c, const Stack::Block& w, int B, int L, bf16_t* kdst, bf16_t* vdst) {
  const Stack& s = c->llm;
  const vla_stack_cfg& k = s.c;
  const int M = B * L, d = k.d_model;
  hipStream_t st = c->compute;
  Workspace& ws = c->ws[VLA_STACK_LLM];
  const int P = s.parts();
  if (P == 2)
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_NORM, vla::rmsnorm_bf16_split(ws.h, w.n1g, k.norm_eps, (bf16_t*)ws.x, M, d, st));
  else
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_NORM, vla::rmsnorm_bf16(ws.h, w.n1g, k.norm_eps, (bf16_t*)ws.x, M, d, st));
  vla::QkvArgs qa{nullptr, k.use_rope ? c->rope_cos : nullptr, k.use_rope ? c->rope_sin : nullptr,
                  (bf16_t*)ws.q, kdst, vdst, (bf16_t*)ws.vt, round_up(L, 64), L, k.n_heads, k.n_kv_heads,
                  k.head_dim};
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_QKV, vla::gemm_bf16_qkv((const bf16_t*)ws.x, P * d, Stack::packed(w.w_qkv, s.qkv_n), qa, M, s.qkv_n, d, st, P));
  return OK;
}

Status llm_block_bf16_rest(vla_ctx* c, const Stack::Block& w, int B, int L, const bf16_t* kdst) {
  const Stack& s = c->llm;
  const vla_stack_cfg& k = s.c;
  const int M = B * L, d = k.d_model;
  hipStream_t st = c->compute;
  Workspace& ws = c->ws[VLA_STACK_LLM];
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_ATTN, vla::attention_bf16((const bf16_t*)ws.q, kdst, (const bf16_t*)ws.vt, round_up(L, 64), (bf16_t*)ws.o, B,
                           k.n_heads, k.n_kv_heads, L, k.head_dim, k.causal != 0, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_OPROJ, vla::gemm_bf16_residual((const bf16_t*)ws.o, s.hd, Stack::packed(w.w_o, d), ws.h, d, nullptr, M, d, s.hd, st));
  const int P = s.parts(), F = s.f_pad;
  if (P == 2)
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_NORM, vla::rmsnorm_bf16_split(ws.h, w.n2g, k.norm_eps, (bf16_t*)ws.x, M, d, st));
  else
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_NORM, vla::rmsnorm_bf16(ws.h, w.n2g, k.norm_eps, (bf16_t*)ws.x, M, d, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_MLP_UP, vla::gemm_bf16_swiglu((const bf16_t*)ws.x, P * d, Stack::packed(w.w_up, 2 * F), (bf16_t*)ws.act,
                                                                P * F, M, 2 * F, d, st, P, P == 2 ? F : 0));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_MLP_DOWN, vla::gemm_bf16_residual((const bf16_t*)ws.act, P * F, Stack::packed(w.w_down, d), ws.h, d, nullptr,
                                                                    M, d, F, st, P));
  return OK;
}

Status llm_block_f32(vla_ctx* c, const Stack::Block& w, int B, int L, float* kdst, float* vdst) {
  const Stack& s = c->llm;
  const vla_stack_cfg& k = s.c;
  const int M = B * L, d = k.d_model;
  hipStream_t st = c->compute;
  Workspace& ws = c->ws[VLA_STACK_LLM];
  float* x = (float*)ws.x;
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_NORM, vla::rmsnorm_f32(ws.h, w.n1g, k.norm_eps, x, M, d, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_QKV, vla::gemm_f32(x, d, (const float*)w.w_qkv, d, ws.qkv_raw, s.qkv_n, nullptr, 0, M, s.qkv_n, d, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_QKV, vla::qkv_split_f32(ws.qkv_raw, k.use_rope ? c->rope_cos : nullptr, k.use_rope ? c->rope_sin : nullptr,
                          (float*)ws.q, kdst, vdst, nullptr, 0, B, L, k.n_heads, k.n_kv_heads, k.head_dim, st));
  return OK;
}

Status llm_block_f32_rest(vla_ctx* c, const Stack::Block& w, int B, int L, const float* kdst, const float* vdst) {
  const Stack& s = c->llm;
  const vla_stack_cfg& k = s.c;
  const int M = B * L, d = k.d_model, F = k.d_ff;
  hipStream_t st = c->compute;
  Workspace& ws = c->ws[VLA_STACK_LLM];
  float* x = (float*)ws.x;
  float* gu = (float*)ws.act;
  float* a = gu + (size_t)M * 2 * F;
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_ATTN, vla::attention_f32((const float*)ws.q, kdst, vdst, (float*)ws.o, B, k.n_heads, k.n_kv_heads, L, k.head_dim,
                          k.causal != 0, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_OPROJ, vla::gemm_f32((const float*)ws.o, s.hd, (const float*)w.w_o, s.hd, ws.h, d, nullptr, 1, M, d, s.hd, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_NORM, vla::rmsnorm_f32(ws.h, w.n2g, k.norm_eps, x, M, d, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_MLP_UP, vla::gemm_f32(x, d, (const float*)w.w_up, d, gu, 2 * F, nullptr, 0, M, 2 * F, d, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_MLP_UP, vla::swiglu_f32(gu, a, M, F, st));
  PLAUNCH(c, VLA_STACK_LLM, VLA_K_MLP_DOWN, vla::gemm_f32(a, F, (const float*)w.w_down, F, ws.h, d, nullptr, 1, M, d, F, st));
  return OK;
}

Status enc_block(vla_ctx* c, const Stack::Block& w, int n_img, int L) {
  const Stack& s = c->enc;
  const vla_stack_cfg& k = s.c;
  const int M = n_img * L, d = k.d_model;
  hipStream_t st = c->encs;
  Workspace& ws = c->ws[VLA_STACK_ENC];
  if (s.bf16()) {
    bf16_t* x = (bf16_t*)ws.x;
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_NORM, vla::layernorm_bf16(ws.h, w.n1g, w.n1b, k.norm_eps, x, M, d, st));
    vla::QkvArgs qa{w.b_qkv, nullptr, nullptr, (bf16_t*)ws.q, (bf16_t*)ws.ek, nullptr, (bf16_t*)ws.vt,
                    round_up(L, 64), L, k.n_heads, k.n_kv_heads, k.head_dim};
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_QKV, vla::gemm_bf16_qkv(x, d, Stack::packed(w.w_qkv, s.qkv_n), qa, M, s.qkv_n, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_ATTN, vla::attention_bf16((const bf16_t*)ws.q, (const bf16_t*)ws.ek, (const bf16_t*)ws.vt, round_up(L, 64),
                             (bf16_t*)ws.o, n_img, k.n_heads, k.n_kv_heads, L, k.head_dim, false, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_OPROJ, vla::gemm_bf16_residual((const bf16_t*)ws.o, s.hd, Stack::packed(w.w_o, d), ws.h, d, w.b_o, M, d,
                                                            s.hd, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_NORM, vla::layernorm_bf16(ws.h, w.n2g, w.n2b, k.norm_eps, x, M, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_MLP_UP, vla::gemm_bf16_gelu(x, d, Stack::packed(w.w_up, s.f_pad), (bf16_t*)ws.act, s.f_pad, w.b_up, M, s.f_pad,
                                                       d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_MLP_DOWN, vla::gemm_bf16_residual((const bf16_t*)ws.act, s.f_pad, Stack::packed(w.w_down, d), ws.h, d,
                                                               w.b_down, M, d, s.f_pad, st));
  } else {
    float* x = (float*)ws.x;
    const int F = k.d_ff;
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_NORM, vla::layernorm_f32(ws.h, w.n1g, w.n1b, k.norm_eps, x, M, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_QKV, vla::gemm_f32(x, d, (const float*)w.w_qkv, d, ws.qkv_raw, s.qkv_n, w.b_qkv, 0, M, s.qkv_n, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_QKV, vla::qkv_split_f32(ws.qkv_raw, nullptr, nullptr, (float*)ws.q, (float*)ws.ek, (float*)ws.ev, nullptr, 0,
                            n_img, L, k.n_heads, k.n_kv_heads, k.head_dim, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_ATTN, vla::attention_f32((const float*)ws.q, (const float*)ws.ek, (const float*)ws.ev, (float*)ws.o, n_img,
                            k.n_heads, k.n_kv_heads, L, k.head_dim, false, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_OPROJ, vla::gemm_f32((const float*)ws.o, s.hd, (const float*)w.w_o, s.hd, ws.h, d, w.b_o, 1, M, d, s.hd, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_NORM, vla::layernorm_f32(ws.h, w.n2g, w.n2b, k.norm_eps, x, M, d, st));
    float* a = (float*)ws.act;
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_MLP_UP, vla::gemm_f32(x, d, (const float*)w.w_up, d, a, F, w.b_up, 0, M, F, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_MLP_UP, vla::gelu_f32(a, (size_t)M * F, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_MLP_DOWN, vla::gemm_f32(a, F, (const float*)w.w_down, F, ws.h, d, w.b_down, 1, M, d, F, st));
  }
  return OK;
}

Status retire_slot(vla_ctx* c, Slot& sl) {
  if (!sl.used) return OK;
  HIPTRY(hipEventSynchronize(sl.ev_copied));
  FrameTimes t{};
  HIPTRY(hipEventElapsedTime(&t.gpu, sl.ev_start, sl.ev_done));
  HIPTRY(hipEventElapsedTime(&t.xfer, sl.ev_hid, sl.ev_copied));
  HIPTRY(hipEventElapsedTime(&t.total, sl.ev_start, sl.ev_copied));
  c->history.put(sl.frame_id, t);
  sl.used = false;
  return OK;
}

// A frame whose enqueueing failed part-way: wait for what was enqueued (the
// copies into the caller's buffers included), then free its slot and forget
// the frame, so the context runs the next frames as before and
// vla_wait_boundary reports the id as unknown.
Status abandon_frame(vla_ctx* c, Slot& sl, const Status& why) {
  (void)hipStreamSynchronize(c->compute);
  if (c->encs != c->compute) (void)hipStreamSynchronize(c->encs);
  (void)hipStreamSynchronize(c->copy);
  sl.used = false;
  c->history.erase(sl.frame_id);
  return why;
}

// Device buffers of one decode step: from the prefill workspace, or carved
// out of the device's fixed scratch (vla_decode_step_static).
struct DecodeBufs {
  float* h = nullptr;       // residual [B][d]
  void* tok = nullptr;      // staging of host input [B][d] bf16
  float* raw = nullptr;     // QKV rows [B][qkv_n]
  float* part = nullptr;    // split-key attention partials
  float* gu = nullptr;      // gate/up rows [B][2 f_pad] (inputs too wide to stage whole)
  bf16_t* obuf = nullptr;   // attention output [B][H*dh]
  bf16_t* abuf = nullptr;   // gated activation [B][parts * f_pad] (split operands: hi, then lo)
  void* hid = nullptr;      // boundary staging [B][d] (f32 at most)
};

// The fixed-scratch layout of a decode step at batch B, position pos;
// returns its bytes, and fills `b` when base is not NULL.
size_t static_decode_layout(const Stack& s, int B, int pos, char* base, DecodeBufs* b) {
  const size_t d = s.c.d_model;
  Bump a{base};
  DecodeBufs t;
  t.h = (float*)a.take((size_t)B * d * 4);
  t.tok = a.take((size_t)B * d * 2);
  t.raw = (float*)a.take((size_t)B * s.qkv_n * 4);
  t.part = (float*)a.take(vla::decode_attention_scratch(B, s.c.n_heads, s.c.head_dim, pos));
  t.gu = (float*)a.take((size_t)B * 2 * s.f_pad * 4);
  t.obuf = (bf16_t*)a.take((size_t)B * s.hd * 2);
  t.abuf = (bf16_t*)a.take((size_t)B * s.parts() * s.f_pad * 2);
  t.hid = a.take((size_t)B * d * 4);
  if (b) *b = t;
  return align_up(a.off, ALIGN);
}

Status enqueue_blocks(vla_ctx* c, Slot& sl, const void* tokens, vla_dtype in_dt, int B, int L, int k0, int k1,
                      vla_boundary* out);
Status enqueue_decode(vla_ctx* c, Slot& sl, const void* x, int B, int pos, int k, void* kv_cache, int L_cap,
                      vla_boundary* out, const DecodeBufs& buf, bool fixed);

Status run_blocks(vla_ctx* c, uint64_t frame_id, const void* tokens, vla_dtype in_dt, int B, int L, int k0,
                  int k1, vla_boundary* out) {
  if (!c->llm.present) return fail(VLA_ERR_INVALID_ARG, "context has no decoder stack");
  const Stack& s = c->llm;
  if (!tokens || !out || !out->hidden) return fail(VLA_ERR_INVALID_ARG, "NULL tokens / boundary / hidden buffer");
  if (out->out_dtype != VLA_BF16 && out->out_dtype != VLA_F32) return fail(VLA_ERR_INVALID_ARG, "bad out_dtype");
  if (in_dt != VLA_BF16 && in_dt != VLA_F32) return fail(VLA_ERR_INVALID_ARG, "bad in_dtype");
  if (k0 < 0 || k1 < k0) return fail(VLA_ERR_INVALID_ARG, "need 0 <= k_begin <= k_end (got %d, %d)", k0, k1);
  if (k1 > s.c.n_blocks) return fail(VLA_ERR_SHAPE, "k_end %d > resident blocks %d", k1, s.c.n_blocks);
  if (B <= 0 || L <= 0) return fail(VLA_ERR_SHAPE, "B and L must be positive");
  if (B > s.c.max_batch || L > s.c.max_tokens)
    return fail(VLA_ERR_SHAPE, "B=%d L=%d exceed max_batch=%d max_tokens=%d", B, L, s.c.max_batch, s.c.max_tokens);
  for (int l = k0; l < k1; ++l)
    if (!s.blocks[l].loaded) return fail(VLA_ERR_NOT_LOADED, "decoder block %d has no weights", l);
  const size_t n = (size_t)B * L * s.c.d_model;
  const size_t hid_bytes = n * dtype_size(out->out_dtype);
  const size_t layer_elems = (size_t)2 * B * s.kvd * L;
  const size_t kv_bytes = (size_t)(k1 - k0) * layer_elems * s.esz;
  if (out->hidden_bytes < hid_bytes)
    return fail(VLA_ERR_SHAPE, "hidden buffer %zu bytes < %zu", out->hidden_bytes, hid_bytes);
  if (out->kv && out->kv_bytes < kv_bytes) return fail(VLA_ERR_SHAPE, "kv buffer %zu bytes < %zu", out->kv_bytes, kv_bytes);
  if (!is_pinned_host(out->hidden)) return fail(VLA_ERR_NOT_PINNED, "hidden buffer is not pinned host memory");
  if (out->kv && !is_pinned_host(out->kv)) return fail(VLA_ERR_NOT_PINNED, "kv buffer is not pinned host memory");
  for (auto& sl : c->slots)
    if (sl.used && sl.frame_id == frame_id) return fail(VLA_ERR_INVALID_ARG, "frame %llu is already in flight",
                                                        (unsigned long long)frame_id);

  Slot& sl = c->slots[c->next_slot];
  c->next_slot = (c->next_slot + 1) % NSLOT;
  Status st = retire_slot(c, sl);
  if (st.code) return st;
  c->history.erase(frame_id);
  sl.frame_id = frame_id;
  sl.used = true;
  out->frame_id = frame_id;
  st = enqueue_blocks(c, sl, tokens, in_dt, B, L, k0, k1, out);
  return st.code ? abandon_frame(c, sl, st) : OK;
}

Status enqueue_blocks(vla_ctx* c, Slot& sl, const void* tokens, vla_dtype in_dt, int B, int L, int k0, int k1,
                      vla_boundary* out) {
  const Stack& s = c->llm;
  const size_t n = (size_t)B * L * s.c.d_model;
  const size_t hid_bytes = n * dtype_size(out->out_dtype);
  const size_t layer_elems = (size_t)2 * B * s.kvd * L;
  const size_t kv_bytes = (size_t)(k1 - k0) * layer_elems * s.esz;
  const bool want_kv = out->kv != nullptr && kv_bytes > 0;
  Status st;
  // the tokens may be the output of an encoder run enqueued before this call
  const bool split = c->encs != c->compute;
  if (split && c->enc_recorded) HIPTRY(hipStreamWaitEvent(c->compute, c->ev_enc_done, 0));
  HIPTRY(hipEventRecord(sl.ev_start, c->compute));
  if ((st = intake(c, VLA_STACK_LLM, in_dt, tokens, n)).code) return st;
  if (split) {
    HIPTRY(hipEventRecord(c->ev_intake, c->compute));
    c->intake_recorded = true;
  }
  float* h = c->ws[VLA_STACK_LLM].h;
  for (int l = k0; l < k1; ++l) {
    const Stack::Block& w = s.blocks[l];
    char* kvl = (char*)sl.kv + (size_t)(l - k0) * layer_elems * s.esz;
    void* kd = kvl;
    void* vd = kvl + layer_elems / 2 * s.esz;
    if (s.bf16())
      st = llm_block_bf16(c, w, B, L, (bf16_t*)kd, (bf16_t*)vd);
    else
      st = llm_block_f32(c, w, B, L, (float*)kd, (float*)vd);
    if (st.code) return st;
    if (want_kv) {
      HIPTRY(hipEventRecord(sl.ev_kv[l - k0], c->compute));
      HIPTRY(hipStreamWaitEvent(c->copy, sl.ev_kv[l - k0], 0));
      HIPTRY(hipMemcpyAsync((char*)out->kv + (size_t)(l - k0) * layer_elems * s.esz, kvl, layer_elems * s.esz,
                            hipMemcpyDeviceToHost, c->copy));
    }
    if (s.bf16())
      st = llm_block_bf16_rest(c, w, B, L, (const bf16_t*)kd);
    else
      st = llm_block_f32_rest(c, w, B, L, (const float*)kd, (const float*)vd);
    if (st.code) return st;
  }
  if (out->out_dtype == VLA_BF16)
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_OTHER, vla::f32_to_bf16(h, (bf16_t*)sl.hid, n, c->compute));
  else
    HIPTRY(hipMemcpyAsync(sl.hid, h, n * 4, hipMemcpyDeviceToDevice, c->compute));
  HIPTRY(hipEventRecord(sl.ev_done, c->compute));
  HIPTRY(hipStreamWaitEvent(c->copy, sl.ev_done, 0));
  HIPTRY(hipEventRecord(sl.ev_hid, c->copy));
  HIPTRY(hipMemcpyAsync(out->hidden, sl.hid, hid_bytes, hipMemcpyDeviceToHost, c->copy));
  HIPTRY(hipEventRecord(sl.ev_copied, c->copy));
  // the next frame may not overwrite this slot's KV before the copies finished:
  // retire_slot() synchronises on ev_copied before a slot is reused.
  return OK;
}

// One decode step of decoder blocks [0, k): B sequences, one token each at
// position pos, over the caller's device KV cache [k][2][B][Hkv][L_cap][dh].
// fixed: the step's scratch comes from the device's fixed array instead of
// the prefill workspace.
Status decode_step(vla_ctx* c, uint64_t frame_id, const void* x, int B, int pos, int k, void* kv_cache, int L_cap,
                   vla_boundary* out, bool fixed) {
  if (!c->llm.present) return fail(VLA_ERR_INVALID_ARG, "context has no decoder stack");
  const Stack& s = c->llm;
  const vla_stack_cfg& cf = s.c;
  if (!x || !out || !out->hidden || !kv_cache) return fail(VLA_ERR_INVALID_ARG, "NULL token / boundary / cache");
  if (!s.bf16()) return fail(VLA_ERR_UNSUPPORTED, "decode steps run on bf16 stacks");
  if (out->out_dtype != VLA_BF16 && out->out_dtype != VLA_F32) return fail(VLA_ERR_INVALID_ARG, "bad out_dtype");
  if (out->kv) return fail(VLA_ERR_INVALID_ARG, "a decode step appends to the device cache; boundary kv must be NULL");
  if (k < 0 || k > cf.n_blocks) return fail(VLA_ERR_SHAPE, "k=%d outside [0, %d]", k, cf.n_blocks);
  if (B <= 0 || B > 4 || B > cf.max_batch) return fail(VLA_ERR_SHAPE, "decode batch %d outside [1, min(4, max_batch)]", B);
  if (pos < 0 || pos >= L_cap) return fail(VLA_ERR_SHAPE, "position %d outside the cache [0, %d)", pos, L_cap);
  if (cf.use_rope && pos >= cf.max_tokens)
    return fail(VLA_ERR_SHAPE, "position %d beyond the rotary tables (max_tokens %d)", pos, cf.max_tokens);
  for (int l = 0; l < k; ++l)
    if (!s.blocks[l].loaded) return fail(VLA_ERR_NOT_LOADED, "decoder block %d has no weights", l);
  if (!is_device(kv_cache)) return fail(VLA_ERR_INVALID_ARG, "the KV cache must be device memory");
  const int d = cf.d_model, H = cf.n_heads, dh = cf.head_dim;
  const size_t hid_bytes = (size_t)B * d * dtype_size(out->out_dtype);
  if (out->hidden_bytes < hid_bytes) return fail(VLA_ERR_SHAPE, "hidden buffer %zu bytes < %zu", out->hidden_bytes, hid_bytes);
  if (!is_pinned_host(out->hidden)) return fail(VLA_ERR_NOT_PINNED, "hidden buffer is not pinned host memory");
  DecodeBufs buf;
  if (fixed) {
    const size_t need = static_decode_layout(s, B, pos, nullptr, nullptr);
    if (need > vla::static_scratch_bytes())
      return fail(VLA_ERR_SHAPE, "decode step at B=%d, position %d needs %zu bytes of fixed scratch, above its %zu",
                  B, pos, need, vla::static_scratch_bytes());
    if (!c->sscratch) return fail(VLA_ERR_HIP, "no fixed scratch on device %d", c->device);
    static_decode_layout(s, B, pos, (char*)c->sscratch, &buf);
  } else {
    // scratch borrowed from the prefill workspace
    const size_t M = s.m_max;
    if ((size_t)B * s.qkv_n * 4 > M * s.hd * 2 || vla::decode_attention_scratch(B, H, dh, pos) > M * s.hd * 2 ||
        (size_t)B * 2 * s.f_pad * 4 > M * s.f_pad * 2 || (size_t)B * s.hd > M * d ||
        (size_t)B * s.parts() * s.f_pad > M * d)
      return fail(VLA_ERR_SHAPE, "workspace too small for a decode step at position %d (raise max_tokens)", pos);
    Workspace& ws = c->ws[VLA_STACK_LLM];
    buf.h = ws.h;
    buf.tok = ws.tok;
    buf.raw = (float*)ws.q;
    buf.part = (float*)ws.o;
    buf.gu = (float*)ws.act;
    buf.obuf = (bf16_t*)ws.x;
    buf.abuf = (bf16_t*)ws.tok;  // the intake is done with it
  }
  for (auto& sl : c->slots)
    if (sl.used && sl.frame_id == frame_id)
      return fail(VLA_ERR_INVALID_ARG, "frame %llu is already in flight", (unsigned long long)frame_id);

  Slot& sl = c->slots[c->next_slot];
  c->next_slot = (c->next_slot + 1) % NSLOT;
  Status st = retire_slot(c, sl);
  if (st.code) return st;
  c->history.erase(frame_id);
  sl.frame_id = frame_id;
  sl.used = true;
  out->frame_id = frame_id;
  if (!buf.hid) buf.hid = sl.hid;
  st = enqueue_decode(c, sl, x, B, pos, k, kv_cache, L_cap, out, buf, fixed);
  return st.code ? abandon_frame(c, sl, st) : OK;
}

Status enqueue_decode(vla_ctx* c, Slot& sl, const void* x, int B, int pos, int k, void* kv_cache, int L_cap,
                      vla_boundary* out, const DecodeBufs& buf, bool fixed) {
  const Stack& s = c->llm;
  const vla_stack_cfg& cf = s.c;
  const int d = cf.d_model, H = cf.n_heads, Hkv = cf.n_kv_heads, dh = cf.head_dim;
  const size_t n = (size_t)B * d;
  const size_t hid_bytes = n * dtype_size(out->out_dtype);
  Status st;
  hipStream_t cs = c->compute;
  if (fixed) {
    // the fixed scratch also stages the boundary: an earlier step's copy out
    // of it (on the copy stream) must finish before this step writes it
    HIPTRY(hipEventRecord(c->ev_copy_tail, c->copy));
    HIPTRY(hipStreamWaitEvent(cs, c->ev_copy_tail, 0));
  }
  HIPTRY(hipEventRecord(sl.ev_start, cs));
  if ((st = intake_to(c, VLA_STACK_LLM, VLA_BF16, x, n, buf.h, buf.tok)).code) return st;
  float* h = buf.h;
  float* raw = buf.raw;
  float* part = buf.part;
  float* gu = buf.gu;
  bf16_t* obuf = buf.obuf;
  bf16_t* abuf = buf.abuf;
  const size_t layer = (size_t)B * Hkv * L_cap * dh;
  const int P = s.parts();  // split operands (hi + lo) under VLA_PREC_SPLIT
  for (int l = 0; l < k; ++l) {
    const Stack::Block& w = s.blocks[l];
    bf16_t* kc = (bf16_t*)kv_cache + (size_t)l * 2 * layer;
    bf16_t* vc = kc + layer;
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_QKV, vla::decode_qkv(h, w.n1g, cf.norm_eps, Stack::packed(w.w_qkv, s.qkv_n), raw, B, s.qkv_n, d, cs, P));
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_ATTN, vla::decode_attention(raw, s.qkv_n, cf.use_rope ? c->rope_cos : nullptr,
                                                             cf.use_rope ? c->rope_sin : nullptr, kc, vc, L_cap, pos, B,
                                                             H, Hkv, dh, part, obuf, cs));
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_OPROJ, vla::decode_oproj(obuf, s.hd, Stack::packed(w.w_o, d), h, B, d, cs));
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_MLP_UP, vla::decode_up(h, w.n2g, cf.norm_eps, Stack::packed(w.w_up, 2 * s.f_pad), s.f_pad, gu, abuf, B, d, cs, P));
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_MLP_DOWN, vla::decode_down(abuf, s.f_pad, Stack::packed(w.w_down, d), h, B, d, cs, P));
  }
  if (out->out_dtype == VLA_BF16)
    PLAUNCH(c, VLA_STACK_LLM, VLA_K_OTHER, vla::f32_to_bf16(h, (bf16_t*)buf.hid, n, cs));
  else
    HIPTRY(hipMemcpyAsync(buf.hid, h, n * 4, hipMemcpyDeviceToDevice, cs));
  HIPTRY(hipEventRecord(sl.ev_done, cs));
  HIPTRY(hipStreamWaitEvent(c->copy, sl.ev_done, 0));
  HIPTRY(hipEventRecord(sl.ev_hid, c->copy));
  HIPTRY(hipMemcpyAsync(out->hidden, buf.hid, hid_bytes, hipMemcpyDeviceToHost, c->copy));
  HIPTRY(hipEventRecord(sl.ev_copied, c->copy));
  return OK;
}

Status run_encoder(vla_ctx* c, const void* patches, int n_img, int L, void* out_dev) {
  if (!c->enc.present) return fail(VLA_ERR_INVALID_ARG, "context has no encoder stack");
  const Stack& s = c->enc;
  if (!patches || !out_dev) return fail(VLA_ERR_INVALID_ARG, "NULL patches / output");
  if (n_img <= 0 || L <= 0) return fail(VLA_ERR_SHAPE, "n_img and L_img must be positive");
  if (n_img > s.c.max_batch || L > s.c.max_tokens)
    return fail(VLA_ERR_SHAPE, "n_img=%d L_img=%d exceed max_batch=%d max_tokens=%d", n_img, L, s.c.max_batch,
                s.c.max_tokens);
  for (int l = 0; l < s.c.n_blocks; ++l)
    if (!s.blocks[l].loaded) return fail(VLA_ERR_NOT_LOADED, "encoder block %d has no weights", l);
  if (!is_device(out_dev)) return fail(VLA_ERR_INVALID_ARG, "encoder output must be device memory");
  const size_t n = (size_t)n_img * L * s.c.d_model;
  Status st = intake(c, VLA_STACK_ENC, s.c.dtype, patches, n);
  if (st.code) return st;
  for (int l = 0; l < s.c.n_blocks; ++l)
    if ((st = enc_block(c, s.blocks[l], n_img, L)).code) return st;
  // out_dev may still be the input of the latest prefix
  const bool split = c->encs != c->compute;
  if (split && c->intake_recorded) HIPTRY(hipStreamWaitEvent(c->encs, c->ev_intake, 0));
  const float* h = c->ws[VLA_STACK_ENC].h;
  if (s.bf16())
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_OTHER, vla::f32_to_bf16(h, (bf16_t*)out_dev, n, c->encs));
  else
    HIPTRY(hipMemcpyAsync(out_dev, h, n * 4, hipMemcpyDeviceToDevice, c->encs));
  if (split) {
    HIPTRY(hipEventRecord(c->ev_enc_done, c->encs));
    c->enc_recorded = true;
  }
  return OK;
}

// images -> stem -> encoder blocks -> final norm + merge -> connector MLP ->
// tokens[0, V); text -> tokens[V, V + L_text)
Status run_vision(vla_ctx* c, const void* images, int n_img, const void* text, int L_text, void* tokens,
                  size_t tokens_bytes) {
  if (!c->enc.present) return fail(VLA_ERR_INVALID_ARG, "context has no encoder stack");
  Vision& v = c->vis;
  if (!v.present) return fail(VLA_ERR_INVALID_ARG, "no vision front attached (vla_attach_vision)");
  if (!v.loaded) return fail(VLA_ERR_NOT_LOADED, "vision weights not loaded");
  const Stack& s = c->enc;
  for (int l = 0; l < s.c.n_blocks; ++l)
    if (!s.blocks[l].loaded) return fail(VLA_ERR_NOT_LOADED, "encoder block %d has no weights", l);
  if (!images || !tokens) return fail(VLA_ERR_INVALID_ARG, "NULL images / tokens");
  if (n_img <= 0 || n_img > v.max_img)
    return fail(VLA_ERR_SHAPE, "n_img=%d outside [1, %d]", n_img, v.max_img);
  if (L_text < 0) return fail(VLA_ERR_SHAPE, "negative L_text");
  if (L_text > 0 && !text) return fail(VLA_ERR_INVALID_ARG, "NULL text with L_text > 0");
  const vla_vision_cfg& vc = v.c;
  const int nv = n_img * v.tpi, M = n_img * v.L_img, d = v.d;
  const size_t need = ((size_t)nv + L_text) * vc.d_out * v.esz;
  if (tokens_bytes < need) return fail(VLA_ERR_SHAPE, "tokens buffer of %zu bytes < %zu", tokens_bytes, need);
  if (!is_device(tokens)) return fail(VLA_ERR_INVALID_ARG, "tokens must be device memory");
  if ((uintptr_t)tokens % 16) return fail(VLA_ERR_INVALID_ARG, "tokens must be 16-byte aligned");
  hipStream_t st = c->encs;
  Workspace& ws = c->ws[VLA_STACK_ENC];
  const void* img = images;
  if (!is_device(images)) {
    HIPTRY(hipMemcpyAsync(v.img, images, (size_t)n_img * vc.channels * vc.img_h * vc.img_w * v.esz,
                          hipMemcpyHostToDevice, st));
    img = v.img;
  }
  const int C = vc.channels, H = vc.img_h, W = vc.img_w, p = vc.patch, m = vc.merge, dh = vc.d_hidden;
  if (v.bf16) {
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_STEM, vla::patchify_bf16((const bf16_t*)img, n_img, C, H, W, p, (bf16_t*)v.A,
                                                             v.Kp, v.pos, ws.h, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_STEM, vla::gemm_bf16_residual((const bf16_t*)v.A, v.Kp, Stack::packed(v.w_patch, d),
                                                                  ws.h, d, v.b_patch, M, d, v.Kp, st));
  } else {
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_STEM, vla::patchify_f32((const float*)img, n_img, C, H, W, p, (float*)v.A, v.Kp,
                                                            v.pos, ws.h, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_STEM, vla::gemm_f32((const float*)v.A, v.K, (const float*)v.w_patch, v.K, ws.h, d,
                                                        v.b_patch, 1, M, d, v.K, st));
  }
  Status rs;
  for (int l = 0; l < s.c.n_blocks; ++l)
    if ((rs = enc_block(c, s.blocks[l], n_img, v.L_img)).code) return rs;
  // tokens may still be the input of the latest prefix
  const bool split = c->encs != c->compute;
  if (split && c->intake_recorded) HIPTRY(hipStreamWaitEvent(st, c->ev_intake, 0));
  if (v.bf16) {
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_CONNECTOR, vla::layernorm_merge_bf16(ws.h, v.post_g, v.post_b, vc.norm_eps,
                                                                         (bf16_t*)v.merged, n_img, v.gh, v.gw, m, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_CONNECTOR, vla::gemm_bf16_gelu((const bf16_t*)v.merged, v.md, Stack::packed(v.w_c1, dh),
                                                                   (bf16_t*)v.hid, dh, v.b_c1, nv, dh, v.md, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_CONNECTOR, vla::gemm_bf16_bias((const bf16_t*)v.hid, dh, Stack::packed(v.w_c2, vc.d_out),
                                                                   (bf16_t*)tokens, vc.d_out, v.b_c2, nv, vc.d_out, dh, st));
  } else {
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_CONNECTOR, vla::layernorm_merge_f32(ws.h, v.post_g, v.post_b, vc.norm_eps,
                                                                        (float*)v.merged, n_img, v.gh, v.gw, m, d, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_CONNECTOR, vla::gemm_f32((const float*)v.merged, v.md, (const float*)v.w_c1, v.md,
                                                             (float*)v.hid, dh, v.b_c1, 0, nv, dh, v.md, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_CONNECTOR, vla::gelu_f32((float*)v.hid, (size_t)nv * dh, st));
    PLAUNCH(c, VLA_STACK_ENC, VLA_K_CONNECTOR, vla::gemm_f32((const float*)v.hid, dh, (const float*)v.w_c2, dh,
                                                             (float*)tokens, vc.d_out, v.b_c2, 0, nv, vc.d_out, dh, st));
  }
  if (L_text > 0)
    HIPTRY(hipMemcpyAsync((char*)tokens + (size_t)nv * vc.d_out * v.esz, text, (size_t)L_text * vc.d_out * v.esz,
                          hipMemcpyDefault, st));
  if (split) {
    HIPTRY(hipEventRecord(c->ev_enc_done, st));
    c->enc_recorded = true;
  }
  return OK;
}

Status attach_vision(vla_ctx* c, const vla_vision_cfg* vc, void* mem, size_t bytes) {
  Vision v;
  Status st = validate_vision(c->enc, vc, &v);
  if (st.code) return st;
  Bump dry{nullptr};
  layout_vision(v, dry);
  if (!mem) return fail(VLA_ERR_INVALID_ARG, "NULL vision memory");
  if (dry.off > bytes) return fail(VLA_ERR_OOM, "vision block of %zu bytes < %zu required", bytes, dry.off);
  if (((uintptr_t)mem) % ALIGN) return fail(VLA_ERR_INVALID_ARG, "vision memory must be %zu-byte aligned", ALIGN);
  if (!is_device(mem)) return fail(VLA_ERR_INVALID_ARG, "vision memory is not device memory");
  // a previous block may still be read by work in flight
  HIPTRY(hipStreamSynchronize(c->compute));
  HIPTRY(hipStreamSynchronize(c->encs));
  Bump real{(char*)mem};
  layout_vision(v, real);
  v.bytes = real.off;
  // weight padding (pad rows and the stem's pad columns) must be zero
  HIPTRY(hipMemset(mem, 0, real.off));
  c->vis = v;
  return OK;
}

vla_status finish(vla_ctx* c, const Status& st) {
  if (c) c->last_error = st.msg;
  if (st.code != VLA_OK) g_last_error = st.msg;
  return st.code;
}

Status build_rope(vla_ctx* c) {
  const Stack& s = c->llm;
  if (!s.present || !s.c.use_rope) return OK;
  const int L = s.c.max_tokens, half = s.c.head_dim / 2;
  std::vector<float> cs((size_t)L * half), sn((size_t)L * half);
  for (int i = 0; i < half; ++i) {
    // theta_i = base^(-2i/dh), angles formed in double precision
    double theta = pow((double)s.c.rope_base, -2.0 * i / s.c.head_dim);
    for (int p = 0; p < L; ++p) {
      double phi = (double)p * theta;
      cs[(size_t)p * half + i] = (float)cos(phi);
      sn[(size_t)p * half + i] = (float)sin(phi);
    }
  }
  Status st = copy_h2d(c->rope_cos, cs.data(), cs.size() * 4);
  if (st.code) return st;
  return copy_h2d(c->rope_sin, sn.data(), sn.size() * 4);
}

Status create(const vla_stack_cfg* llm, const vla_stack_cfg* enc, int device, void* arena, size_t arena_bytes,
              void* compute, void* encoder, void* copy, vla_ctx** out) {
  if (!out) return fail(VLA_ERR_INVALID_ARG, "NULL out");
  *out = nullptr;
  if (!llm && !enc) return fail(VLA_ERR_INVALID_ARG, "need at least one stack");
  if (!arena) return fail(VLA_ERR_INVALID_ARG, "NULL arena");
  std::unique_ptr<vla_ctx> c(new vla_ctx());
  Status st = validate_stack(llm, true, &c->llm);
  if (st.code) return st;
  if ((st = validate_stack(enc, false, &c->enc)).code) return st;
  Bump dry{nullptr};
  layout(c.get(), dry);
  if (dry.off > arena_bytes)
    return fail(VLA_ERR_OOM, "arena of %zu bytes < %zu required", arena_bytes, dry.off);
  if (((uintptr_t)arena) % ALIGN) return fail(VLA_ERR_INVALID_ARG, "arena must be %zu-byte aligned", ALIGN);
  HIPTRY(hipSetDevice(device));
  if (!is_device(arena)) return fail(VLA_ERR_INVALID_ARG, "arena is not device memory");
  c->device = device;
  c->arena = (char*)arena;
  c->arena_bytes = arena_bytes;
  Bump real{c->arena};
  layout(c.get(), real);
  c->used = real.off;
  // zero the weight region so padding rows/columns are exact zeros
  HIPTRY(hipMemset(c->arena, 0, c->used));
  if (compute) {
    c->compute = (hipStream_t)compute;
  } else {
    HIPTRY(hipStreamCreateWithFlags(&c->compute, hipStreamNonBlocking));
    c->own_compute = true;
  }
  // no encoder stream of its own: the encoder runs on the compute stream
  c->encs = encoder ? (hipStream_t)encoder : c->compute;
  if (copy) {
    c->copy = (hipStream_t)copy;
  } else {
    HIPTRY(hipStreamCreateWithFlags(&c->copy, hipStreamNonBlocking));
    c->own_copy = true;
  }
  HIPTRY(hipEventCreateWithFlags(&c->ev_enc_done, hipEventDisableTiming));
  HIPTRY(hipEventCreateWithFlags(&c->ev_intake, hipEventDisableTiming));
  HIPTRY(hipEventCreateWithFlags(&c->ev_copy_tail, hipEventDisableTiming));
  // the device's fixed decode scratch, resolved with the device current
  HIPTRY(vla::static_scratch_resolve(device, &c->sscratch));
  int nkv = c->llm.present ? c->llm.c.n_blocks : 0;
  for (auto& sl : c->slots) {
    HIPTRY(hipEventCreate(&sl.ev_start));
    HIPTRY(hipEventCreate(&sl.ev_done));
    HIPTRY(hipEventCreate(&sl.ev_hid));
    HIPTRY(hipEventCreate(&sl.ev_copied));
    sl.ev_kv.resize(nkv);
    for (auto& e : sl.ev_kv) HIPTRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  if ((st = build_rope(c.get())).code) return st;
  HIPTRY(hipDeviceSynchronize());
  *out = c.release();
  return OK;
}

void destroy(vla_ctx* c) {
  if (!c) return;
  (void)hipSetDevice(c->device);
  if (c->compute) (void)hipStreamSynchronize(c->compute);
  if (c->encs && c->encs != c->compute) (void)hipStreamSynchronize(c->encs);
  if (c->copy) (void)hipStreamSynchronize(c->copy);
  for (auto& sl : c->slots) {
    for (hipEvent_t e : {sl.ev_start, sl.ev_done, sl.ev_hid, sl.ev_copied})
      if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : sl.ev_kv)
      if (e) (void)hipEventDestroy(e);
  }
  for (hipEvent_t e : c->prof_pool) (void)hipEventDestroy(e);
  for (hipEvent_t e : {c->ev_enc_done, c->ev_intake, c->ev_copy_tail})
    if (e) (void)hipEventDestroy(e);
  if (c->own_compute) (void)hipStreamDestroy(c->compute);
  if (c->own_copy) (void)hipStreamDestroy(c->copy);
  delete c;
}

}  // namespace

// ===================================================================== C ABI

extern "C" {

vla_status vla_query_sizes(const vla_stack_cfg* llm, const vla_stack_cfg* enc, int B, int L, int k,
                           size_t* arena_bytes, size_t* hidden_bytes, size_t* kv_bytes) {
  try {
    vla_ctx tmp;
    Status st = validate_stack(llm, true, &tmp.llm);
    if (!st.code) st = validate_stack(enc, false, &tmp.enc);
    if (!st.code && !llm && !enc) st = fail(VLA_ERR_INVALID_ARG, "need at least one stack");
    if (st.code) return finish(nullptr, st);
    Bump dry{nullptr};
    layout(&tmp, dry);
    if (arena_bytes) *arena_bytes = dry.off;
    if (llm) {
      if (B < 0 || L < 0 || k < 0) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "negative B, L or k"));
      if (hidden_bytes) *hidden_bytes = (size_t)B * L * llm->d_model * dtype_size(llm->dtype);
      if (kv_bytes)
        *kv_bytes = (size_t)k * 2 * B * llm->n_kv_heads * L * llm->head_dim * dtype_size(llm->dtype);
    } else {
      if (hidden_bytes) *hidden_bytes = 0;
      if (kv_bytes) *kv_bytes = 0;
    }
    return VLA_OK;
  } catch (...) {
    return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_create(const vla_stack_cfg* llm, const vla_stack_cfg* enc, int device, void* dev_arena,
                      size_t arena_bytes, void* compute_stream, void* encoder_stream, void* copy_stream,
                      vla_ctx** out) {
  try {
    return finish(nullptr, create(llm, enc, device, dev_arena, arena_bytes, compute_stream, encoder_stream,
                                  copy_stream, out));
  } catch (const std::bad_alloc&) {
    return finish(nullptr, fail(VLA_ERR_OOM, "host allocation failed"));
  } catch (...) {
    return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_load_block_weights(vla_ctx* ctx, vla_stack which, int block, const vla_block_weights* w) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (!w) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "NULL weights"));
    if (which != VLA_STACK_LLM && which != VLA_STACK_ENC) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "bad stack"));
    Stack& s = which == VLA_STACK_LLM ? ctx->llm : ctx->enc;
    if (!s.present) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "context has no such stack"));
    if (block < 0 || block >= s.c.n_blocks)
      return finish(ctx, fail(VLA_ERR_SHAPE, "block %d outside [0, %d)", block, s.c.n_blocks));
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    // weights may still be read by in-flight work of either stack
    if (hipStreamSynchronize(ctx->compute) != hipSuccess || hipStreamSynchronize(ctx->encs) != hipSuccess)
      return finish(ctx, fail(VLA_ERR_HIP, "hipStreamSynchronize failed"));
    return finish(ctx, load_block(ctx, s, block, w));
  } catch (const std::bad_alloc&) {
    return finish(ctx, fail(VLA_ERR_OOM, "host allocation failed"));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_run_encoder(vla_ctx* ctx, uint64_t frame_id, const void* patches, int n_img, int L_img,
                           void* out_dev) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  (void)frame_id;
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    return finish(ctx, run_encoder(ctx, patches, n_img, L_img, out_dev));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_query_vision_sizes(const vla_stack_cfg* enc, const vla_vision_cfg* vis, size_t* bytes) {
  try {
    vla_ctx tmp;
    Status st = validate_stack(enc, false, &tmp.enc);
    if (!st.code && !enc) st = fail(VLA_ERR_INVALID_ARG, "NULL encoder config");
    Vision v;
    if (!st.code) st = validate_vision(tmp.enc, vis, &v);
    if (st.code) return finish(nullptr, st);
    Bump dry{nullptr};
    layout_vision(v, dry);
    if (bytes) *bytes = dry.off;
    return VLA_OK;
  } catch (...) {
    return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_attach_vision(vla_ctx* ctx, const vla_vision_cfg* vis, void* dev_mem, size_t bytes) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    return finish(ctx, attach_vision(ctx, vis, dev_mem, bytes));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_load_vision_weights(vla_ctx* ctx, const vla_vision_weights* w) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (!w) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "NULL weights"));
    if (!ctx->vis.present) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "no vision front attached"));
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    if (hipStreamSynchronize(ctx->compute) != hipSuccess || hipStreamSynchronize(ctx->encs) != hipSuccess)
      return finish(ctx, fail(VLA_ERR_HIP, "hipStreamSynchronize failed"));
    return finish(ctx, load_vision(ctx->vis, ctx->enc.c.dtype, w));
  } catch (const std::bad_alloc&) {
    return finish(ctx, fail(VLA_ERR_OOM, "host allocation failed"));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_run_vision(vla_ctx* ctx, uint64_t frame_id, const void* images, int n_img, const void* text,
                          int L_text, void* tokens_dev, size_t tokens_bytes) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  (void)frame_id;
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    return finish(ctx, run_vision(ctx, images, n_img, text, L_text, tokens_dev, tokens_bytes));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_run_blocks(vla_ctx* ctx, uint64_t frame_id, const void* tokens, vla_dtype in_dtype, int B, int L,
                          int k_begin, int k_end, vla_boundary* out) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    return finish(ctx, run_blocks(ctx, frame_id, tokens, in_dtype, B, L, k_begin, k_end, out));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_decode_step(vla_ctx* ctx, uint64_t frame_id, const void* x, int B, int pos, int k, void* kv_cache,
                           int L_cap, vla_boundary* out) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    return finish(ctx, decode_step(ctx, frame_id, x, B, pos, k, kv_cache, L_cap, out, false));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_decode_step_static(vla_ctx* ctx, uint64_t frame_id, const void* x, int B, int pos, int k,
                                  void* kv_cache, int L_cap, vla_boundary* out) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    return finish(ctx, decode_step(ctx, frame_id, x, B, pos, k, kv_cache, L_cap, out, true));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_run_prefix(vla_ctx* ctx, uint64_t frame_id, const void* tokens, int B, int L, int k,
                          vla_boundary* out) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  if (!ctx->llm.present) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "context has no decoder stack"));
  return vla_run_blocks(ctx, frame_id, tokens, ctx->llm.c.dtype, B, L, 0, k, out);
}

vla_status vla_wait_boundary(vla_ctx* ctx, uint64_t frame_id, int timeout_ms) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    for (auto& sl : ctx->slots) {
      if (!sl.used || sl.frame_id != frame_id) continue;
      auto t0 = std::chrono::steady_clock::now();
      for (;;) {
        hipError_t e = hipEventQuery(sl.ev_copied);
        if (e == hipSuccess) return finish(ctx, retire_slot(ctx, sl));
        if (e != hipErrorNotReady) return finish(ctx, fail(VLA_ERR_HIP, "hipEventQuery: %s", hipGetErrorString(e)));
        if (timeout_ms >= 0) {
          auto ms = std::chrono::duration_cast<std::chrono::milliseconds>(std::chrono::steady_clock::now() - t0);
          if (ms.count() >= timeout_ms)
            return finish(ctx, fail(VLA_ERR_TIMEOUT, "frame %llu not done after %d ms", (unsigned long long)frame_id,
                                    timeout_ms));
        }
        std::this_thread::sleep_for(std::chrono::microseconds(20));
      }
    }
    if (ctx->history.find(frame_id)) return finish(ctx, OK);
    return finish(ctx, fail(VLA_ERR_UNKNOWN_FRAME, "no frame %llu", (unsigned long long)frame_id));
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_frame_times(vla_ctx* ctx, uint64_t frame_id, float* t_gpu_ms, float* t_xfer_ms, float* t_total_ms) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  const FrameTimes* ft = ctx->history.find(frame_id);
  if (!ft)
    return finish(ctx, fail(VLA_ERR_UNKNOWN_FRAME, "frame %llu has not been waited for", (unsigned long long)frame_id));
  if (t_gpu_ms) *t_gpu_ms = ft->gpu;
  if (t_xfer_ms) *t_xfer_ms = ft->xfer;
  if (t_total_ms) *t_total_ms = ft->total;
  return finish(ctx, OK);
}

vla_status vla_profile(vla_ctx* ctx, int enable) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    if (enable) {
      Status st = prof_drain(ctx);
      if (st.code) return finish(ctx, st);
      for (auto& row : ctx->prof_ms)
        for (double& v : row) v = 0.0;
      for (auto& row : ctx->prof_n)
        for (int& v : row) v = 0;
    }
    ctx->prof_on = enable != 0;
    return finish(ctx, OK);
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_profile_read(vla_ctx* ctx, vla_stack which, vla_kernel_class cls, double* ms_total, int* launches) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  if ((which != VLA_STACK_LLM && which != VLA_STACK_ENC) || cls < 0 || cls >= VLA_K_COUNT)
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "bad stack or kernel class"));
  try {
    if (hipSetDevice(ctx->device) != hipSuccess) return finish(ctx, fail(VLA_ERR_HIP, "hipSetDevice failed"));
    Status st = prof_drain(ctx);
    if (st.code) return finish(ctx, st);
    if (ms_total) *ms_total = ctx->prof_ms[which][cls];
    if (launches) *launches = ctx->prof_n[which][cls];
    return finish(ctx, OK);
  } catch (...) {
    return finish(ctx, fail(VLA_ERR_INVALID_ARG, "internal error"));
  }
}

vla_status vla_set_precision(vla_ctx* ctx, vla_stack which, vla_precision prec) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  if (which != VLA_STACK_LLM && which != VLA_STACK_ENC) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "bad stack"));
  if (prec != VLA_PREC_BF16 && prec != VLA_PREC_SPLIT) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "bad precision"));
  Stack& s = which == VLA_STACK_LLM ? ctx->llm : ctx->enc;
  if (!s.present) return finish(ctx, fail(VLA_ERR_INVALID_ARG, "context has no such stack"));
  if (prec == VLA_PREC_SPLIT && !s.split_room())
    return finish(ctx, fail(VLA_ERR_UNSUPPORTED, "split operands are implemented for bf16 decoder stacks"));
  // launches already enqueued keep the precision they were enqueued with
  s.prec = prec;
  return finish(ctx, OK);
}

vla_status vla_inject_fault(vla_ctx* ctx, long launches) {
  if (!ctx) return finish(nullptr, fail(VLA_ERR_INVALID_ARG, "NULL context"));
  ctx->fault_after = launches < 0 ? -1 : launches;
  return finish(ctx, OK);
}

vla_status vla_arena_used(const vla_ctx* ctx, size_t* bytes) {
  if (!ctx || !bytes) return VLA_ERR_INVALID_ARG;
  *bytes = ctx->used;
  return VLA_OK;
}

const char* vla_status_string(vla_status s) {
  switch (s) {
    case VLA_OK: return "ok";
    case VLA_ERR_INVALID_ARG: return "invalid argument";
    case VLA_ERR_SHAPE: return "shape outside the context's limits";
    case VLA_ERR_NOT_LOADED: return "block weights not loaded";
    case VLA_ERR_NOT_PINNED: return "host buffer not pinned";
    case VLA_ERR_OOM: return "device arena too small";
    case VLA_ERR_TIMEOUT: return "timed out";
    case VLA_ERR_HIP: return "HIP runtime error";
    case VLA_ERR_UNSUPPORTED: return "unsupported shape";
    case VLA_ERR_UNKNOWN_FRAME: return "unknown frame id";
  }
  return "unknown status";
}

const char* vla_last_error(const vla_ctx* ctx) { return ctx ? ctx->last_error.c_str() : g_last_error.c_str(); }

void vla_destroy(vla_ctx* ctx) {
  try {
    destroy(ctx);
  } catch (...) {
  }
}

}  // extern "C"
