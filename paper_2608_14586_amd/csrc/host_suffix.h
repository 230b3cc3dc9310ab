// Internal interface of the host suffix executor (host_suffix.cpp, built with
// AVX-512 BF16).  Only host_suffix_api.cpp calls it, after checking the CPU.
#pragma once

#include <cstdint>

namespace vla {
namespace host {

struct Cfg {
  int d, H, Hkv, dh, F;
  int causal, use_rope;
  float eps, rope_base;
};

// bf16 host weights of one decoder block, nn.Linear layout W[out][in]
struct Weights {
  const uint16_t *wq, *wk, *wv, *wo, *wg, *wu, *wd, *g1, *g2;
};

struct Suffix;

Suffix* create(const Cfg& c, int k_begin, int k_end, int n_threads);
void destroy(Suffix* s);
int threads(const Suffix* s);
bool load_block(Suffix* s, int block, const Weights& w);
bool all_loaded(const Suffix* s);
// blocks [k, k_end) over h (bf16, or f32 when in_f32) [B][L][d] -> out f32 [B][L][d];
// k_begin <= k <= k_end
bool run(Suffix* s, int k, const void* in, bool in_f32, int B, int L, float* out);
// host KV caches for decode steps ([block][B][Hkv][L_cap][dh]); a later run()
// with this B and L <= L_cap records its keys and values; B or L_cap <= 0 frees
void set_cache(Suffix* s, int B, int L_cap);
int cache_batch(const Suffix* s);
int cache_len(const Suffix* s);
// one new token per sequence at position pos through blocks [k, k_end) over
// the caches (rows [0, pos) filled), appending its keys and values
bool decode(Suffix* s, int k, const void* in, bool in_f32, int B, int pos, float* out);

}  // namespace host
}  // namespace vla
