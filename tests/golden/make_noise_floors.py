"""Write tests/golden/bf16_noise_floor.json: the relative-L2 error, against the
float32 oracle, of an exact bf16-activation computation of the d=4096 decoder
stack (every matrix-product input, the attention inputs/outputs and the gated
activation rounded to bf16, boundary cast to bf16), after each block; and the
same for each block's KV cache entries (K after RoPE and V, as the bf16 cache
holds them).

Calls only oracle/ and synth/.  Run:  python tests/golden/make_noise_floors.py
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402


def _rel(a, b):
    a = a.astype(np.float64)
    b = b.astype(np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def floors(name, L, k):
    wl = synth.CONFIGS[name]
    t = synth.as_f32(synth.tokens(wl, frame=0, L=L))
    ref_h, emu_h, ref_kv, emu_kv = [], [], [], []
    cache = {}

    def W(l):
        if l not in cache:
            cache.clear()
            cache[l] = {n: synth.as_f32(a) for n, a in synth.llm_block_weights(wl, l).items()}
        return cache[l]

    def keep(hs, kvs):
        def f(l, h, K, V):
            hs.append(h.copy())
            kvs.append(np.stack([K, V]))
        return f

    oracle.run_prefix(t, W, wl.llm, k, keep_kv=False, on_layer=keep(ref_h, ref_kv))
    oracle.run_prefix(t, W, wl.llm, k, keep_kv=False, act_round=oracle.round_bf16, on_layer=keep(emu_h, emu_kv))
    hidden = [_rel(oracle.round_bf16(a), b) for a, b in zip(emu_h, ref_h)]
    kv = [_rel(a, b) for a, b in zip(emu_kv, ref_kv)]
    return hidden, kv


def main():
    res = {"description": __doc__.strip().splitlines()[0] + " ...", "inputs": "frame 0 tokens, unperturbed weights"}
    for name, L, k in (("llm7b", 1024, 16), ("sweep7b", 2048, 32)):
        t0 = time.time()
        key = "%s_L%d" % (name, L)
        res[key], res[key + "_kv"] = floors(name, L, k)
        print(name, L, k, "%.0fs" % (time.time() - t0), res[key][-1], max(res[key + "_kv"]), flush=True)
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "bf16_noise_floor.json"), "w") as f:
        json.dump(res, f, indent=1)


if __name__ == "__main__":
    main()
