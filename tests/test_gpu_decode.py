"""Decode steps across the boundary (vla_decode_step): decoder blocks [0, k) for
one new token per sequence over the KV cache a prefix handed over.

Pin: by causality, the step at position p equals row p of a prefill over the
p + 1 tokens, so the oracle is its own prefill of the longer sequence."""
import numpy as np
import pytest

import oracle
import synth
from synth.configs import llama_like, Workload

from paper_2608_14586_amd import binding as vb
from prefix_cases import f32_weights, log, rel_l2

pytestmark = pytest.mark.gpu


def _run(shape, B, L, k, steps, name, out_dtype="f32", nan_tail=False, prec=None, prec_decode=None):
    import torch
    wl = Workload(name, "bf16", shape, None)
    W = [synth.llm_block_weights(wl, l, perturbed=True) for l in range(k)]
    d, Hkv, dh = shape.d_model, shape.n_kv_heads, shape.head_dim
    L_cap = L + steps + 5
    ctx = vb.Context(llm=vb.stack_cfg(shape, "bf16", max_tokens=L_cap, max_batch=B, n_blocks=k))
    for l in range(k):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, W[l])
    if prec is not None:
        ctx.vla_set_precision(vb.VLA_STACK_LLM, prec)
    toks = synth.normal_bf16(synth.seed_of(name, "tok"), (B, L + steps, d))
    bnd = vb.Boundary(B, L, d, k, Hkv, dh)
    ctx.vla_run_prefix(1, np.ascontiguousarray(toks[:, :L]), B, L, k, bnd)
    ctx.vla_wait_boundary(1, 60000)
    cache = torch.zeros((k, 2, B, Hkv, L_cap, dh), dtype=torch.bfloat16, device="cuda")
    if nan_tail:
        # rows past the prefix hold bf16 NaN (0x7FC0): the interface asks only for rows [0, pos)
        cache.view(torch.int16).fill_(0x7FC0)
    cache[:, :, :, :, :L] = bnd.kv.cuda()
    if prec_decode is not None:
        ctx.vla_set_precision(vb.VLA_STACK_LLM, prec_decode)
    outs = []
    for t in range(steps):
        ob = vb.Boundary(B, 1, d, 0, Hkv, dh, out_dtype=out_dtype, with_kv=False)
        ctx.vla_decode_step(10 + t, np.ascontiguousarray(toks[:, L + t]), B, L + t, k, cache, L_cap, ob)
        ctx.vla_wait_boundary(10 + t, 60000)
        outs.append(ob.hidden.float().numpy().reshape(B, d))
    return wl, W, toks, outs, cache, ctx


def _oracle_rows(wl, W, toks, L, steps, k):
    Wf = [{n: synth.as_f32(a).astype(np.float64) for n, a in w.items()} for w in W]
    x = synth.as_f32(toks).astype(np.float64)
    h, _ = oracle.run_prefix(x, lambda l: Wf[l], wl.llm, k, dtype=np.float64, keep_kv=False)
    return x[:, L:L + steps], h[:, L:L + steps]


@pytest.mark.parametrize("name,shape,B,L,k", [
    ("dec_gqa", llama_like(2, 256, 4, 2, 64, 704), 2, 77, 2),
    ("dec_dh128", llama_like(2, 256, 2, 1, 128, 512), 1, 130, 2),
    ("dec_split", llama_like(1, 192, 3, 3, 64, 448), 2, 300, 1),   # keys cross two 128-key splits
    ("dec_short", llama_like(3, 128, 2, 2, 64, 320), 1, 1, 3),     # a one-token prefix
    # d = 1024 and d_ff = 2816: every product takes the streaming GEMV (input
    # rows staged whole in LDS), with three and four sequences
    ("dec_stream4", llama_like(2, 1024, 8, 2, 128, 2816), 4, 100, 2),
    ("dec_stream3", llama_like(1, 1024, 16, 4, 64, 2816), 3, 257, 1),
    # d_ff = 11008 with four sequences: the down product stages 96 KB of input
    # rows (one workgroup per CU)
    ("dec_stream_big", llama_like(1, 512, 8, 2, 64, 11008), 4, 60, 1),
])
def test_decode_steps_match_oracle(name, shape, B, L, k):
    steps = 3
    wl, W, toks, outs, _, _ = _run(shape, B, L, k, steps, name)
    x, ref = _oracle_rows(wl, W, toks, L, steps, k)
    for t in range(steps):
        for b in range(B):
            # the blocks' update of the residual, at the prefix's 1e-2 bar
            e = rel_l2(outs[t][b] - x[b, t], ref[b, t] - x[b, t])
            log("%s step %d seq %d: update rel L2 %.2e" % (name, t, b, e))
            assert e < 1e-2, (name, t, b, e)


@pytest.mark.parametrize("name,shape,B,L,k", [
    ("decs_gqa", llama_like(2, 256, 4, 2, 64, 704), 2, 77, 2),
    ("decs_short", llama_like(3, 128, 2, 2, 64, 320), 1, 1, 3),
    # eight staged rows (four sequences, hi and lo) in the streaming GEMV
    ("decs_stream4", llama_like(2, 1024, 8, 2, 128, 2816), 4, 100, 2),
    ("decs_stream3", llama_like(1, 1024, 16, 4, 64, 2816), 3, 257, 1),
    # d_ff = 11008: the down product's hi and lo rows of four sequences exceed
    # the streaming kernel's LDS and take the chunked GEMV
    ("decs_chunk", llama_like(1, 512, 8, 2, 64, 11008), 4, 60, 1),
])
def test_split_decode_steps_match_oracle(name, shape, B, L, k):
    # VLA_PREC_SPLIT also carries the decode step's normalised rows and gated
    # activation as hi + lo bf16 pairs; the prefill before it runs split too
    steps = 2
    wl, W, toks, outs, _, _ = _run(shape, B, L, k, steps, name, prec=vb.VLA_PREC_SPLIT)
    # the same split prefill, then bf16 decode steps
    _, _, _, outs_bf16, _, _ = _run(shape, B, L, k, steps, name, prec=vb.VLA_PREC_SPLIT,
                                    prec_decode=vb.VLA_PREC_BF16)
    x, ref = _oracle_rows(wl, W, toks, L, steps, k)
    for t in range(steps):
        # the mode reaches the step: its products differ from the bf16 ones
        assert not np.array_equal(outs[t], outs_bf16[t]), (name, t)
        for b in range(B):
            e = rel_l2(outs[t][b] - x[b, t], ref[b, t] - x[b, t])
            e16 = rel_l2(outs_bf16[t][b] - x[b, t], ref[b, t] - x[b, t])
            log("%s step %d seq %d: update rel L2 %.2e split, %.2e bf16" % (name, t, b, e, e16))
            assert e < 1e-2, (name, t, b, e)


def test_decode_ignores_cache_rows_past_pos():
    # GQA 14/2: the rows from pos on hold NaN before each step (the step
    # writes row pos itself); the keys past pos in the last split are masked
    # and must not reach the output
    shape = llama_like(2, 896, 14, 2, 64, 1216)
    B, L, k, steps = 2, 130, 2, 3
    wl, W, toks, outs, cache, _ = _run(shape, B, L, k, steps, "dec_nan", nan_tail=True)
    x, ref = _oracle_rows(wl, W, toks, L, steps, k)
    for t in range(steps):
        for b in range(B):
            assert np.isfinite(outs[t][b]).all(), (t, b)
            e = rel_l2(outs[t][b] - x[b, t], ref[b, t] - x[b, t])
            log("dec_nan step %d seq %d: update rel L2 %.2e" % (t, b, e))
            assert e < 1e-2, (t, b, e)
    # every appended row is finite, the rows after them still NaN
    import torch
    assert torch.isfinite(cache[:, :, :, :, :L + steps].float()).all()
    assert torch.isnan(cache[:, :, :, :, L + steps:].float()).all()


def test_decode_appends_the_prefill_keys():
    # the cache rows a decode step appends agree with what a prefill over the
    # longer sequence writes (bf16 rounding of nearly equal inputs apart)
    import torch
    shape = llama_like(2, 256, 4, 2, 64, 704)
    B, L, k, steps = 1, 40, 2, 2
    wl, W, toks, outs, cache, ctx = _run(shape, B, L, k, steps, "dec_keys")
    bnd = vb.Boundary(B, L + steps, shape.d_model, k, shape.n_kv_heads, shape.head_dim)
    ctx.vla_run_prefix(50, np.ascontiguousarray(toks), B, L + steps, k, bnd)
    ctx.vla_wait_boundary(50, 60000)
    got = cache[:, :, :, :, L:L + steps].float().cpu().numpy()
    want = bnd.kv[:, :, :, :, L:L + steps].float().numpy()
    assert rel_l2(got, want) < 1e-2
    # rows before the new positions are untouched
    assert torch.equal(cache[:, :, :, :, :L].cpu(), bnd.kv[:, :, :, :, :L])


def test_decode_k0_returns_input_and_rejects_bad_calls():
    import torch
    shape = llama_like(1, 128, 2, 2, 64, 320)
    wl = Workload("dec_err", "bf16", shape, None)
    ctx = vb.Context(llm=vb.stack_cfg(shape, "bf16", max_tokens=64, max_batch=4, n_blocks=1))
    ctx.vla_load_block_weights(vb.VLA_STACK_LLM, 0, synth.llm_block_weights(wl, 0))
    cache = torch.zeros((1, 2, 4, 2, 64, 64), dtype=torch.bfloat16, device="cuda")
    x = synth.normal_bf16(synth.seed_of("dec_err_x"), (2, 128))
    ob = vb.Boundary(2, 1, 128, 0, 2, 64, out_dtype="bf16", with_kv=False)
    ctx.vla_decode_step(1, x, 2, 5, 0, cache, 64, ob)
    ctx.vla_wait_boundary(1, 60000)
    assert np.array_equal(ob.hidden.view(torch.int16).numpy().view(np.uint16).reshape(2, 128), x)
    bad = [((1, x, 2, 64, 1, cache, 64, ob), "VLA_ERR_SHAPE"),          # pos == L_cap
           ((2, x, 5, 3, 1, cache, 64, ob), "VLA_ERR_SHAPE"),           # batch above 4
           ((3, x, 2, 3, 2, cache, 64, ob), "VLA_ERR_SHAPE"),           # k above the resident blocks
           ((4, x, 2, 3, 1, cache.cpu(), 64, ob), "VLA_ERR_INVALID_ARG"),  # host cache
           ((5, x, 2, 3, 1, cache, 64, vb.Boundary(2, 1, 128, 1, 2, 64)), "VLA_ERR_INVALID_ARG")]  # kv given
    for args, code in bad:
        with pytest.raises(vb.VlaError) as e:
            ctx.vla_decode_step(*args)
        assert e.value.name == code, (args[0], e.value.name)


def test_decode_full_size_against_oracle():
    # 7B-shaped blocks at the bench length: the step at position L against
    # row L of the oracle's prefill over L + 1 tokens (Eq. (6) applied per
    # token), and against row L of the GPU's own prefill
    import torch
    wl = synth.CONFIGS["sweep7b"]
    s = wl.llm
    L, k, B = 2048, 2, 1
    W = [synth.llm_block_weights(wl, l) for l in range(k)]
    ctx = vb.Context(llm=vb.stack_cfg(s, "bf16", max_tokens=L + 8, max_batch=B, n_blocks=k))
    for l in range(k):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, W[l])
    toks = synth.tokens(wl, frame=7, B=B, L=L + 1)
    full = vb.Boundary(B, L + 1, s.d_model, k, s.n_kv_heads, s.head_dim, out_dtype="f32")
    ctx.vla_run_prefix(1, toks, B, L + 1, k, full)
    ctx.vla_wait_boundary(1, 120000)
    cache = torch.zeros((k, 2, B, s.n_kv_heads, L + 8, s.head_dim), dtype=torch.bfloat16, device="cuda")
    cache[:, :, :, :, :L] = full.kv[:, :, :, :, :L].cuda()
    ob = vb.Boundary(B, 1, s.d_model, 0, s.n_kv_heads, s.head_dim, out_dtype="f32", with_kv=False)
    ctx.vla_decode_step(2, np.ascontiguousarray(toks[:, L]), B, L, k, cache, L + 8, ob)
    ctx.vla_wait_boundary(2, 120000)
    x = synth.as_f32(toks[:, L])
    got = ob.hidden.numpy().reshape(B, s.d_model)
    Wf = [f32_weights(w) for w in W]
    ref, kv = oracle.run_prefix(synth.as_f32(toks), lambda l: Wf[l], s, k)
    e = rel_l2(got - x, ref[:, L] - x)
    e_pf = rel_l2(got - x, full.hidden.numpy()[:, L] - x)
    # the appended key and value rows against the oracle's cache row L
    e_kv = rel_l2(cache[:, :, :, :, L].float().cpu().numpy(), kv[:, :, :, :, L])
    log("7B-shaped decode at position %d: update rel L2 vs the oracle %.2e, vs the GPU prefill %.2e, "
        "appended K/V %.2e" % (L, e, e_pf, e_kv))
    assert e < 1e-2 and e_pf < 1e-2 and e_kv < 1e-2


def test_split_decode_7b_k16_against_oracle():
    # 7B-shaped blocks [0, 16) at the bench length, where bf16 operands leave
    # the boundary beyond 1e-2 of the fp32 model: prefill and decode step with
    # split operands, the step at position L against row L of the oracle's
    # prefill over L + 1 tokens
    import torch
    wl = synth.CONFIGS["sweep7b"]
    s = wl.llm
    L, k, B = 2048, 16, 1
    W = [synth.llm_block_weights(wl, l) for l in range(k)]
    ctx = vb.Context(llm=vb.stack_cfg(s, "bf16", max_tokens=L + 8, max_batch=B, n_blocks=k))
    for l in range(k):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, W[l])
    toks = synth.tokens(wl, frame=9, B=B, L=L + 1)
    x = synth.as_f32(toks[:, L])
    got = {}
    for mode in (vb.VLA_PREC_SPLIT, vb.VLA_PREC_BF16):
        ctx.vla_set_precision(vb.VLA_STACK_LLM, mode)
        pre = vb.Boundary(B, L, s.d_model, k, s.n_kv_heads, s.head_dim, out_dtype="f32")
        ctx.vla_run_prefix(10 + mode, np.ascontiguousarray(toks[:, :L]), B, L, k, pre)
        ctx.vla_wait_boundary(10 + mode, 120000)
        cache = torch.zeros((k, 2, B, s.n_kv_heads, L + 8, s.head_dim), dtype=torch.bfloat16, device="cuda")
        cache[:, :, :, :, :L] = pre.kv.cuda()
        ob = vb.Boundary(B, 1, s.d_model, 0, s.n_kv_heads, s.head_dim, out_dtype="f32", with_kv=False)
        ctx.vla_decode_step(20 + mode, np.ascontiguousarray(toks[:, L]), B, L, k, cache, L + 8, ob)
        ctx.vla_wait_boundary(20 + mode, 120000)
        got[mode] = ob.hidden.numpy().reshape(B, s.d_model).copy()
        del cache
    Wf = [f32_weights(w) for w in W]
    ref, _ = oracle.run_prefix(synth.as_f32(toks), lambda l: Wf[l], s, k, keep_kv=False)
    e = rel_l2(got[vb.VLA_PREC_SPLIT] - x, ref[:, L] - x)
    e16 = rel_l2(got[vb.VLA_PREC_BF16] - x, ref[:, L] - x)
    log("7B-shaped decode at position %d, k=%d: update rel L2 vs the oracle %.2e split, %.2e bf16" % (L, k, e, e16))
    assert e < 1e-2


def test_decode_across_the_boundary():
    # the whole partitioned decode (Eq. (6) per token): blocks [0, 2) on the
    # GPU from the prefix's KV cache, the boundary to pinned host memory,
    # blocks [2, 4) on the host from its own cache; against the oracle's
    # prefill over all four blocks
    import torch
    shape = llama_like(4, 256, 4, 2, 64, 704)
    wl = Workload("dec_across", "bf16", shape, None)
    W = [synth.llm_block_weights(wl, l, perturbed=True) for l in range(4)]
    B, L, K, N, steps = 1, 60, 2, 4, 3
    d, Hkv, dh = shape.d_model, shape.n_kv_heads, shape.head_dim
    L_cap = L + steps + 4
    ctx = vb.Context(llm=vb.stack_cfg(shape, "bf16", max_tokens=L_cap, max_batch=B, n_blocks=K))
    for l in range(K):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, W[l])
    sfx = vb.Suffix(vb.stack_cfg(shape, "bf16", max_tokens=L_cap), K, N)
    for l in range(K, N):
        sfx.vla_suffix_load_block_weights(l, W[l])
    sfx.vla_suffix_set_cache(B, L_cap)
    toks = synth.normal_bf16(synth.seed_of("dec_across_tok"), (B, L + steps, d))
    # prefill: GPU prefix with its KV handoff, then the host suffix recording its own cache
    bnd = vb.Boundary(B, L, d, K, Hkv, dh, out_dtype="f32")
    ctx.vla_run_prefix(1, np.ascontiguousarray(toks[:, :L]), B, L, K, bnd)
    ctx.vla_wait_boundary(1, 60000)
    out = np.empty((B, L, d), np.float32)
    sfx.vla_suffix_run(bnd.hidden.numpy(), vb.VLA_F32, B, L, out)
    cache = torch.zeros((K, 2, B, Hkv, L_cap, dh), dtype=torch.bfloat16, device="cuda")
    cache[:, :, :, :, :L] = bnd.kv.cuda()
    Wf = [{n: synth.as_f32(a).astype(np.float64) for n, a in w.items()} for w in W]
    x = synth.as_f32(toks).astype(np.float64)
    ref, _ = oracle.run_prefix(x, lambda l: Wf[l], shape, N, dtype=np.float64, keep_kv=False)
    for t in range(steps):
        ob = vb.Boundary(B, 1, d, 0, Hkv, dh, out_dtype="f32", with_kv=False)
        ctx.vla_decode_step(10 + t, np.ascontiguousarray(toks[:, L + t]), B, L + t, K, cache, L_cap, ob)
        ctx.vla_wait_boundary(10 + t, 60000)
        o = np.empty((B, d), np.float32)
        sfx.vla_suffix_decode_step(K, ob.hidden.numpy().reshape(B, d), vb.VLA_F32, B, L + t, o)
        e = rel_l2(o[0] - x[0, L + t], ref[0, L + t] - x[0, L + t])
        log("decode across the boundary, step %d: update rel L2 %.2e" % (t, e))
        assert e < 1e-2, (t, e)
