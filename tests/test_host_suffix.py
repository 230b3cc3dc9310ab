"""Host suffix executor (include/vla_suffix.h) against the oracle, on the CPU.

The suffix applies decoder blocks [k_begin, k_end) to a boundary state
(Eq. (6)); the oracle is its own prefix routine started from that state with
the later blocks' weights (positions restart at 0, as on the GPU)."""
import numpy as np
import pytest

import oracle
import synth
from synth.configs import llama_like, Workload

from paper_2608_14586_amd import binding as vb


def _cpu_has_bf16_avx512():
    try:
        flags = open("/proc/cpuinfo").read()
    except OSError:
        return False
    return all(f in flags for f in ("avx512f", "avx512bw", "avx512vl", "avx512_bf16"))


pytestmark = pytest.mark.skipif(not _cpu_has_bf16_avx512(), reason="host suffix needs AVX-512 BF16")


def _case(name, n_blocks, d, H, Hkv, dh, F, perturbed=True):
    wl = Workload(name, "bf16", llama_like(n_blocks, d, H, Hkv, dh, F), None)
    W = [synth.llm_block_weights(wl, l, perturbed=perturbed) for l in range(n_blocks)]
    return wl, W


def _suffix(wl, W, k0, k1, threads=0):
    s = vb.Suffix(vb.stack_cfg(wl.llm, "bf16", max_tokens=1), k0, k1, threads)
    for l in range(k0, k1):
        s.vla_suffix_load_block_weights(l, W[l])
    return s


def _oracle(wl, W, h, k0, k1):
    Wf = [{n: synth.as_f32(a).astype(np.float64) for n, a in w.items()} for w in W]
    out, _ = oracle.run_prefix(h.astype(np.float64), lambda j: Wf[k0 + j], wl.llm, k1 - k0, dtype=np.float64,
                               keep_kv=False)
    return out


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.mark.parametrize("n_blocks,d,H,Hkv,dh,F,B,L,k0,k1,in_f32", [
    (3, 256, 4, 2, 64, 704, 2, 77, 1, 3, False),   # GQA, ragged L, bf16 boundary
    (2, 256, 2, 1, 128, 512, 1, 130, 0, 2, True),  # dh = 128, f32 boundary (fp32 residual continued)
    (2, 128, 2, 2, 64, 320, 3, 1, 0, 2, False),    # one token
    (2, 192, 3, 1, 64, 448, 1, 64, 1, 2, False),   # one whole query tile
    (2, 192, 3, 3, 64, 448, 1, 65, 0, 1, True),    # one past a tile
])
def test_suffix_matches_oracle(n_blocks, d, H, Hkv, dh, F, B, L, k0, k1, in_f32):
    wl, W = _case("sfx_%d_%d_%d" % (d, dh, L), n_blocks, d, H, Hkv, dh, F)
    h = synth.normal_f32(synth.seed_of("sfx_h", d, L, B), (B, L, d))
    if not in_f32:
        h = synth.f32_to_bf16(h)
    s = _suffix(wl, W, k0, k1)
    out = np.empty((B, L, d), np.float32)
    s.vla_suffix_run(h, vb.VLA_F32 if in_f32 else vb.VLA_BF16, B, L, out)
    hf = synth.as_f32(h)
    ref = _oracle(wl, W, hf, k0, k1)
    for b in range(B):
        # bf16 operands with fp32 accumulation, as the GPU blocks: the same 1e-2
        # bar, on the blocks' update of the residual (the residual itself would
        # hide an error in the update)
        e = _rel(out[b] - hf[b], ref[b] - hf[b])
        assert e < 1e-2, (b, e)


def test_suffix_deterministic_across_thread_counts():
    wl, W = _case("sfx_det", 2, 256, 4, 2, 64, 704)
    h = synth.f32_to_bf16(synth.normal_f32(synth.seed_of("sfx_det_h"), (2, 96, 256)))
    outs = []
    for threads in (1, 3, 8):
        s = _suffix(wl, W, 0, 2, threads)
        assert s.vla_suffix_threads() == threads
        o = np.empty((2, 96, 256), np.float32)
        s.vla_suffix_run(h, vb.VLA_BF16, 2, 96, o)
        outs.append(o)
    # every output element is one tile's fixed-order reduction
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_suffix_run_from_inner_partition_point():
    # a frame whose partition point moved inside the dynamic zone runs only
    # the blocks after it: equal to a suffix built for that range
    wl, W = _case("sfx_from", 4, 128, 2, 1, 64, 320)
    h = synth.f32_to_bf16(synth.normal_f32(synth.seed_of("sfx_from_h"), (1, 50, 128)))
    wide = _suffix(wl, W, 1, 4)
    narrow = _suffix(wl, W, 3, 4)
    a = np.empty((1, 50, 128), np.float32)
    b = np.empty((1, 50, 128), np.float32)
    wide.vla_suffix_run_from(3, h, vb.VLA_BF16, 1, 50, a)
    narrow.vla_suffix_run(h, vb.VLA_BF16, 1, 50, b)
    assert np.array_equal(a, b)
    wide.vla_suffix_run_from(4, h, vb.VLA_BF16, 1, 50, a)   # k = k_end: the boundary itself
    assert np.array_equal(a, synth.as_f32(h))
    with pytest.raises(vb.VlaError) as e:
        wide.vla_suffix_run_from(0, h, vb.VLA_BF16, 1, 50, a)
    assert e.value.name == "VLA_ERR_INVALID_ARG"


def test_suffix_gain_matters():
    # a dropped or swapped norm gain must not pass the parity bar
    wl, W = _case("sfx_gain", 1, 128, 2, 2, 64, 320)
    h = synth.f32_to_bf16(synth.normal_f32(synth.seed_of("sfx_gain_h"), (1, 40, 128)))
    s = _suffix(wl, W, 0, 1)
    out = np.empty((1, 40, 128), np.float32)
    s.vla_suffix_run(h, vb.VLA_BF16, 1, 40, out)
    W2 = [dict(W[0], norm2_g=W[0]["norm1_g"])]
    hf = synth.as_f32(h)
    assert _rel(out[0] - hf[0], _oracle(wl, W, hf, 0, 1)[0] - hf[0]) < 1e-2
    assert _rel(out[0] - hf[0], _oracle(wl, W2, hf, 0, 1)[0] - hf[0]) > 5e-2


def test_suffix_errors():
    wl, W = _case("sfx_err", 2, 128, 2, 2, 64, 320)
    cfg = vb.stack_cfg(wl.llm, "bf16", max_tokens=1)
    with pytest.raises(vb.VlaError) as e:
        vb.Suffix(cfg, 1, 1)
    assert e.value.name == "VLA_ERR_INVALID_ARG"
    with pytest.raises(vb.VlaError) as e:
        vb.Suffix(vb.stack_cfg(wl.llm, "f32", max_tokens=1), 0, 1)
    assert e.value.name == "VLA_ERR_UNSUPPORTED"
    odd = Workload("sfx_odd", "bf16", llama_like(1, 128, 4, 4, 32, 320), None)
    with pytest.raises(vb.VlaError) as e:
        vb.Suffix(vb.stack_cfg(odd.llm, "bf16", max_tokens=1), 0, 1)
    assert e.value.name == "VLA_ERR_UNSUPPORTED"
    s = vb.Suffix(cfg, 0, 2)
    s.vla_suffix_load_block_weights(0, W[0])
    with pytest.raises(vb.VlaError) as e:
        s.vla_suffix_load_block_weights(2, W[1])
    assert e.value.name == "VLA_ERR_INVALID_ARG"
    h = np.zeros((1, 8, 128), np.uint16)
    out = np.empty((1, 8, 128), np.float32)
    with pytest.raises(vb.VlaError) as e:
        s.vla_suffix_run(h, vb.VLA_BF16, 1, 8, out)
    assert e.value.name == "VLA_ERR_NOT_LOADED"


@pytest.mark.parametrize("n_blocks,d,H,Hkv,dh,F,B,L,k0,steps", [
    (3, 256, 4, 2, 64, 704, 2, 77, 1, 3),    # GQA, two sequences
    (2, 256, 2, 1, 128, 512, 1, 40, 0, 2),   # dh = 128 (RoPE in the second pass)
    (2, 128, 2, 2, 64, 320, 1, 1, 0, 3),     # a one-token prefix
])
def test_suffix_decode_steps_match_oracle(n_blocks, d, H, Hkv, dh, F, B, L, k0, steps):
    # the prefill records its keys and values; each decode step at position p
    # must equal row p of a prefill over the p + 1 boundary states
    wl, W = _case("sfx_dec_%d_%d" % (d, L), n_blocks, d, H, Hkv, dh, F)
    seq = synth.f32_to_bf16(synth.normal_f32(synth.seed_of("sfx_dec_seq", d, L), (B, L + steps, d)))
    s = _suffix(wl, W, k0, n_blocks)
    s.vla_suffix_set_cache(B, L + steps + 2)
    out = np.empty((B, L, d), np.float32)
    s.vla_suffix_run(np.ascontiguousarray(seq[:, :L]), vb.VLA_BF16, B, L, out)
    hf = synth.as_f32(seq)
    ref = _oracle(wl, W, hf, k0, n_blocks)
    for t in range(steps):
        o = np.empty((B, d), np.float32)
        s.vla_suffix_decode_step(k0, np.ascontiguousarray(seq[:, L + t]), vb.VLA_BF16, B, L + t, o)
        for b in range(B):
            e = _rel(o[b] - hf[b, L + t], ref[b, L + t] - hf[b, L + t])
            assert e < 1e-2, (t, b, e)


def test_suffix_decode_errors():
    wl, W = _case("sfx_dec_err", 1, 128, 2, 2, 64, 320)
    s = _suffix(wl, W, 0, 1)
    h = np.zeros((1, 128), np.uint16)
    o = np.empty((1, 128), np.float32)
    with pytest.raises(vb.VlaError) as e:     # no cache
        s.vla_suffix_decode_step(0, h, vb.VLA_BF16, 1, 0, o)
    assert e.value.name == "VLA_ERR_SHAPE"
    s.vla_suffix_set_cache(1, 8)
    with pytest.raises(vb.VlaError) as e:     # past the cache
        s.vla_suffix_decode_step(0, h, vb.VLA_BF16, 1, 8, o)
    assert e.value.name == "VLA_ERR_SHAPE"
    with pytest.raises(vb.VlaError) as e:     # batch differs from the cache's
        s.vla_suffix_decode_step(0, np.zeros((2, 128), np.uint16), vb.VLA_BF16, 2, 3, np.empty((2, 128), np.float32))
    assert e.value.name == "VLA_ERR_SHAPE"
