"""Parity at the workloads' full sizes (the bench's shapes and launch
configuration), through the C ABI, against the CPU oracle.

* d=896 decoder (L=4096, k=12) and ViT-L encoder (6 x 1024, 24 blocks): whole
  boundary and every KV layer within relative L2 1e-2.
* d=4096 decoder (L=1024, k=16; L=2048, k=32 as benched):
  - with split activation operands (VLA_PREC_SPLIT: the RMSNorm outputs and
    the gated activation enter the QKV, gate/up and down GEMMs as hi + lo
    bf16 pairs), whole boundary and every KV layer within 1e-2;
  - with plain bf16 operands, exact bf16 arithmetic itself drifts past 1e-2
    with depth (tests/golden/bf16_noise_floor.json, written by
    make_noise_floors.py from the oracle alone): the boundary and every KV
    layer within 1.1x that floor, and every block, fed the GPU's own bf16
    boundary, within 1e-2 of the oracle's block on that input;
  - the fp32 debug path over the same stack within 1e-4.
"""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from prefix_cases import EncCase, LlmCase, f32_weights, log, rel_l2, to_f32

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def floor_of(key, block):
    """bf16 noise floor after `block` + 1 blocks, or of block `block`'s KV
    entries for a key ending in "_kv" (tests/golden/bf16_noise_floor.json)."""
    with open(os.path.join(HERE, "golden", "bf16_noise_floor.json")) as f:
        return json.load(f)[key][block]


def _both_precisions(c, tok, ref, kv, key, n):
    """The same frame with bf16 and with split activation operands against the
    oracle's boundary `ref` (and KV `kv` unless None), n blocks."""
    from paper_2608_14586_amd import binding as vb
    res = {}
    for name, prec in (("bf16", vb.VLA_PREC_BF16), ("split", vb.VLA_PREC_SPLIT)):
        c.ctx.vla_set_precision(vb.VLA_STACK_LLM, prec)
        bnd = c.run(tok, frame=prec + 1)
        e_h = rel_l2(to_f32(bnd.hidden), ref)
        e_kv = [rel_l2(to_f32(bnd.kv[l]), kv[l]) for l in range(n)] if kv is not None else []
        res[name] = (e_h, e_kv)
        floor = floor_of(key, n - 1)
        log("  %s, %s operands: boundary %.2e (bf16 floor %.2e, ratio %.2f)%s"
            % (key, name, e_h, floor, e_h / floor,
               ", kv max %.2e" % max(e_kv) if e_kv else ""))
    c.ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_BF16)
    return res


def test_small_llm_full():
    c = LlmCase("small_llm", 4096, 12)
    tok = c.tokens(frame=0)
    bnd = c.run(tok, frame=0)
    ref, kv = c.oracle(tok)
    e_h = rel_l2(to_f32(bnd.hidden), ref)
    e_kv = [rel_l2(to_f32(bnd.kv[l]), kv[l]) for l in range(12)]
    log("  small_llm L=4096 k=12: boundary %.2e, kv max %.2e" % (e_h, max(e_kv)))
    assert e_h <= 1e-2 and max(e_kv) <= 1e-2
    c.close()


def test_vit_l_full():
    c = EncCase("vit_l", 6, 1024)
    p = c.patches(frame=0)
    got = to_f32(c.run(p))
    ref = c.oracle(p)
    e = rel_l2(got, ref)
    log("  vit_l 6x1024 24 blocks: %.2e" % e)
    assert e <= 1e-2
    c.close()


def test_wide_tiles_with_ragged_rows():
    """The 8-wave tiles that fill whole rounds also take row counts that are
    not multiples of their height: 7B-shaped blocks at L=2000 (QKV in 256x192
    tiles, gate/up in 256x256, the last row tile 208 rows tall) and ViT-L
    blocks over 6 x 1000 patches (QKV in 192x384, fc1 in 192x256 tiles, the
    last 48 rows tall, tiles straddling images).  Two blocks each against the
    oracle, boundary and every KV layer within 1e-2."""
    c = LlmCase("llm7b", 2000, 2, perturbed=True)
    tok = c.tokens(frame=3)
    bnd = c.run(tok, frame=0)
    ref, kv = c.oracle(tok)
    e_h = rel_l2(to_f32(bnd.hidden), ref)
    e_kv = [rel_l2(to_f32(bnd.kv[l]), kv[l]) for l in range(2)]
    log("  llm7b L=2000 k=2: boundary %.2e, kv max %.2e" % (e_h, max(e_kv)))
    assert e_h <= 1e-2 and max(e_kv) <= 1e-2
    c.close()
    e = EncCase("vit_l", 6, 1000, n_blocks=2, perturbed=True)
    p = e.patches(frame=3)
    got = to_f32(e.run(p))
    ref = e.oracle(p)
    err = rel_l2(got, ref)
    log("  vit_l 6x1000, 2 blocks: %.2e" % err)
    assert err <= 1e-2
    e.close()


def _per_block(c, blocks, tok):
    """Chain the GPU block by block through bf16 boundaries; each block is
    compared with the oracle's block on the very same bf16 input."""
    import torch
    h = tok
    errs = []
    for l in range(max(blocks) + 1):
        bnd = c.run(h, frame=100 + l, k0=l, k1=l + 1)
        if l in blocks:
            ref, kv = oracle.run_prefix(synth.as_f32(h), lambda i: f32_weights(c.W[l]), c.s, 1)
            e_h = rel_l2(to_f32(bnd.hidden) - synth.as_f32(h), ref - synth.as_f32(h))
            e_b = rel_l2(to_f32(bnd.hidden), ref)
            e_kv = rel_l2(to_f32(bnd.kv[0]), kv[0])
            errs.append((l, e_b, e_h, e_kv))
            log("  block %2d: boundary %.2e, block output %.2e, kv %.2e" % (l, e_b, e_h, e_kv))
        h = bnd.hidden.view(torch.int16).numpy().view(np.uint16).copy()
    return errs


def test_llm7b_full():
    c = LlmCase("llm7b", 1024, 16)
    tok = c.tokens(frame=0)
    ref, kv = c.oracle(tok)
    res = _both_precisions(c, tok, ref, kv, "llm7b_L1024", 16)
    # split operands: the plain bar
    e_h, e_kv = res["split"]
    assert e_h <= 1e-2 and max(e_kv) <= 1e-2, (e_h, e_kv)
    # bf16 operands: on the floor of exact bf16 arithmetic
    e_h, e_kv = res["bf16"]
    assert e_h <= 1.1 * floor_of("llm7b_L1024", 15)
    for l in range(16):
        assert e_kv[l] <= 1.1 * floor_of("llm7b_L1024_kv", l), (l, e_kv[l])
    errs = _per_block(c, list(range(16)), tok)
    for l, e_b, e_h, e_kv in errs:
        assert e_b <= 1e-2 and e_kv <= 1e-2, (l, e_b, e_kv)
    c.close()


def test_llm7b_fp32_debug_full():
    """The fp32 debug path over the same 16 blocks at L=1024: 1e-4."""
    import dataclasses
    from paper_2608_14586_amd import binding as vb
    wl = synth.CONFIGS["llm7b"]
    c = LlmCase.__new__(LlmCase)
    c.wl = dataclasses.replace(wl, dtype="f32")
    c.s, c.L, c.k, c.B, c.perturbed = wl.llm, 1024, 16, 1, False
    W16 = [synth.llm_block_weights(wl, l) for l in range(16)]
    c.W = [f32_weights(w) for w in W16]
    c.ctx = vb.Context(llm=vb.stack_cfg(wl.llm, "f32", max_tokens=1024, max_batch=1, n_blocks=16))
    for l in range(16):
        c.ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, c.W[l])
    tok = synth.as_f32(synth.tokens(wl, frame=0))
    bnd = c.run(tok, frame=0, out_dtype="f32")
    ref, kv = c.oracle(tok)
    e_h, e_kv = rel_l2(bnd.hidden.numpy(), ref), rel_l2(bnd.kv.numpy(), kv)
    log("  llm7b fp32 L=1024 k=16: boundary %.2e kv %.2e" % (e_h, e_kv))
    assert e_h <= 1e-4 and e_kv <= 1e-4
    c.close()


def test_sweep7b_bench_configuration():
    """The benched configuration: 32 resident blocks, L=2048.  Whole boundary
    at k=32 within 1e-2 with split operands and within 1.1x the bf16 floor
    with bf16 operands; blocks 0, 15 and 31 per block."""
    c = LlmCase("sweep7b", 2048, 32)
    tok = c.tokens(frame=0)
    ref, _ = c.oracle(tok, keep_kv=False)
    res = _both_precisions(c, tok, ref, None, "sweep7b_L2048", 32)
    assert res["split"][0] <= 1e-2
    assert res["bf16"][0] <= 1.1 * floor_of("sweep7b_L2048", 31)
    for l, e_b, e_blk, e_kv in _per_block(c, [0, 15, 31], tok):
        assert e_b <= 1e-2 and e_kv <= 1e-2, (l, e_b, e_kv)
    c.close()
