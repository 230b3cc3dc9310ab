"""Parity of the HIP prefix and encoder (through the C ABI) with the CPU
oracle on the same seeded inputs, plus the handoff semantics: frame ids,
back-to-back frames, determinism, block-range composition and error paths.

Bars: relative L2 <= 1e-4 on the fp32 debug path, <= 1e-2 on bf16 stacks
(whole boundary and every KV layer), except where exact bf16 arithmetic
itself drifts past 1e-2 (the d=4096 stack deeper than a few blocks, see
test_gpu_fullsize.py)."""
import numpy as np
import pytest

from prefix_cases import EncCase, LlmCase, log, rel_l2, to_f32

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("perturbed", [False, True])
def test_tiny_fp32_debug_path(perturbed):
    c = LlmCase("tiny", 128, 2, perturbed=perturbed)
    tok = c.tokens(frame=3)
    bnd = c.run(tok, frame=3, out_dtype="f32")
    ref, kv = c.oracle(tok)
    e_h, e_kv = rel_l2(bnd.hidden.numpy(), ref), rel_l2(bnd.kv.numpy(), kv)
    e_d = rel_l2(bnd.hidden.numpy() - tok, ref - tok)
    log("  tiny fp32: boundary %.2e, block sum %.2e, kv %.2e" % (e_h, e_d, e_kv))
    assert bnd.frame_id == 3
    assert e_h <= 1e-4 and e_kv <= 1e-4 and e_d <= 1e-4
    c.close()


@pytest.mark.parametrize("name,L,k,B", [("small_llm", 300, 2, 1), ("small_llm", 128, 3, 2), ("llm7b", 256, 2, 1),
                                        ("llm7b", 200, 1, 1), ("llm7b", 2048, 1, 1)])
def test_bf16_prefix_reduced(name, L, k, B):
    c = LlmCase(name, L, k, B=B, perturbed=True)
    tok = c.tokens(frame=1)
    bnd = c.run(tok, frame=1)
    ref, kv = c.oracle(tok)
    got = to_f32(bnd.hidden)
    e_h = rel_l2(got, ref)
    t32 = to_f32_tok(tok)
    e_d = rel_l2(got - t32, ref - t32)
    e_kv = [rel_l2(to_f32(bnd.kv[l]), kv[l]) for l in range(k)]
    log("  %s L=%d k=%d B=%d: boundary %.2e, block sum %.2e, kv %s" % (name, L, k, B, e_h, e_d,
                                                                        ["%.1e" % e for e in e_kv]))
    assert e_h <= 1e-2 and max(e_kv) <= 1e-2 and e_d <= 2e-2
    c.close()


def to_f32_tok(tok):
    import synth
    return synth.as_f32(tok)


def test_fp32_prefix_gqa_ragged():
    """fp32 debug path on a GQA stack with a ragged length and batch 2."""
    import dataclasses
    import synth
    wl = synth.CONFIGS["small_llm"]
    shape = dataclasses.replace(wl.llm, n_blocks=2)
    c = LlmCase.__new__(LlmCase)
    c.wl = dataclasses.replace(wl, dtype="f32")
    c.s, c.L, c.k, c.B, c.perturbed = shape, 97, 2, 2, True
    c.W = [{n: synth.as_f32(a) for n, a in synth.llm_block_weights(wl, l, perturbed=True).items()} for l in range(2)]
    from paper_2608_14586_amd import binding as vb
    c.ctx = vb.Context(llm=vb.stack_cfg(shape, "f32", max_tokens=128, max_batch=2, n_blocks=2))
    for l in range(2):
        c.ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, c.W[l])
    tok = synth.as_f32(synth.tokens(wl, frame=2, B=2, L=97))
    bnd = c.run(tok, frame=2, out_dtype="f32")
    ref, kv = c.oracle(tok)
    e_h, e_kv = rel_l2(bnd.hidden.numpy(), ref), rel_l2(bnd.kv.numpy(), kv)
    log("  fp32 GQA ragged: boundary %.2e kv %.2e" % (e_h, e_kv))
    assert e_h <= 1e-4 and e_kv <= 1e-4
    c.close()


@pytest.mark.parametrize("n_img,L,blocks", [(2, 200, 2), (1, 1024, 1)])
def test_bf16_encoder_reduced(n_img, L, blocks):
    c = EncCase("vit_l", n_img, L, n_blocks=blocks, perturbed=True)
    p = c.patches(frame=5)
    got = to_f32(c.run(p))
    ref = c.oracle(p)
    e = rel_l2(got, ref)
    log("  vit_l %dx%d %d blocks: %.2e" % (n_img, L, blocks, e))
    assert e <= 1e-2
    c.close()


def test_fp32_encoder():
    import dataclasses
    import synth
    from paper_2608_14586_amd import binding as vb
    wl = synth.CONFIGS["vit_l"]
    s = dataclasses.replace(wl.enc, n_blocks=2, d_model=128, n_heads=2, n_kv_heads=2, d_ff=256)
    W = [{n: synth.as_f32(a) for n, a in synth.vit_block_weights(dataclasses.replace(wl, enc=s), l, perturbed=True).items()}
         for l in range(2)]
    ctx = vb.Context(enc=vb.stack_cfg(s, "f32", max_tokens=80, max_batch=3))
    for l in range(2):
        ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, W[l])
    import torch
    p = synth.normal_f32(synth.seed_of("encp32"), (3, 77, 128))
    out = torch.empty((3, 77, 128), dtype=torch.float32, device="cuda")
    ctx.vla_run_encoder(0, p, 3, 77, out)
    ctx.encoder_stream.synchronize()
    import oracle
    ref = oracle.run_encoder(p, lambda l: W[l], s)
    e = rel_l2(out.cpu().numpy(), ref)
    log("  fp32 encoder: %.2e" % e)
    assert e <= 1e-4
    ctx.vla_destroy()


def test_device_tokens_and_split_composition():
    """Blocks [0,2) then [2,3) on the GPU equal blocks [0,3) (Eq. (5)-(6));
    device-resident input equals host input bitwise."""
    c = LlmCase("small_llm", 160, 3)
    tok = c.tokens(frame=9)
    full = c.run(tok, frame=1, out_dtype="f32")
    dev = c.run(tok, frame=2, out_dtype="f32", device_tokens=True)
    assert np.array_equal(full.hidden.numpy(), dev.hidden.numpy())
    a = c.run(tok, frame=3, k0=0, k1=2, out_dtype="f32")
    # continue from the fp32 boundary: same fp32 residual, same result
    b = c.run(a.hidden.numpy().copy(), frame=4, k0=2, k1=3, out_dtype="f32")
    assert np.array_equal(b.hidden.numpy(), full.hidden.numpy())
    assert np.array_equal(to_f32(b.kv[0]), to_f32(full.kv[2]))
    # the bf16 handoff (b = 2 bytes, Eq. (11)) continued by the next stage
    # matches the oracle continued from the same bf16 state
    a16 = c.run(tok, frame=5, k0=0, k1=2)
    import torch
    h16 = a16.hidden.view(torch.int16).numpy().view(np.uint16).copy()
    b16 = c.run(h16, frame=6, k0=2, k1=3, out_dtype="f32")
    ref, _ = c.oracle(h16, k0=2, k1=3)
    assert rel_l2(b16.hidden.numpy(), ref) <= 1e-2
    c.close()


def test_back_to_back_frames_and_determinism():
    """Four frames in flight with distinct inputs: each handoff matches its
    own frame's oracle and repeated runs are bitwise identical."""
    c = LlmCase("small_llm", 256, 2)
    toks = [c.tokens(frame=f) for f in range(4)]
    bnds = [c.boundary() for _ in range(4)]
    for f in range(4):
        c.ctx.vla_run_prefix(100 + f, toks[f], 1, c.L, c.k, bnds[f])
    for f in range(4):
        c.ctx.vla_wait_boundary(100 + f, 60000)
        g, x, t = c.ctx.vla_frame_times(100 + f)
        assert 0 < g <= t and 0 <= x <= t
        assert bnds[f].frame_id == 100 + f
    for f in range(4):
        ref, kv = c.oracle(toks[f])
        assert rel_l2(to_f32(bnds[f].hidden), ref) <= 1e-2
        assert rel_l2(to_f32(bnds[f].kv), kv) <= 1e-2
    again = c.run(toks[2], frame=200)
    import torch
    bits = lambda t: t.view(torch.int16).numpy()
    assert np.array_equal(bits(again.hidden), bits(bnds[2].hidden))
    assert np.array_equal(bits(again.kv), bits(bnds[2].kv))
    c.close()


def test_encoder_feeds_prefix_across_streams():
    """The encoder of frame f+1 overlaps the prefix of frame f on its own
    stream.  Frames whose prefix reads the encoder's output, all through one
    output buffer, must each match a strictly serial run bit for bit: the
    prefix waits for its encoder, and the next encoder's output write waits
    for the prefix's intake."""
    import dataclasses
    import torch
    import synth
    from paper_2608_14586_amd import binding as vb
    ew, lw = synth.CONFIGS["vit_l"], synth.CONFIGS["small_llm"]
    es = dataclasses.replace(ew.enc, n_blocks=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ff=512)
    ls = dataclasses.replace(lw.llm, n_blocks=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=688)
    ew, lw = dataclasses.replace(ew, enc=es), dataclasses.replace(lw, llm=ls)
    EW = [synth.vit_block_weights(ew, l, perturbed=True) for l in range(2)]
    LW = [synth.llm_block_weights(lw, l, perturbed=True) for l in range(2)]
    n_img, L_img, nf = 2, 96, 5
    ecfg = vb.stack_cfg(es, "bf16", max_tokens=L_img, max_batch=n_img)
    lcfg = vb.stack_cfg(ls, "bf16", max_tokens=L_img, max_batch=n_img, n_blocks=2)
    pats = [synth.patches(ew, frame=f, n_img=n_img, L_img=L_img) for f in range(nf)]

    def load(ctx):
        for l in range(2):
            if ctx.enc is not None:
                ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, EW[l])
            if ctx.llm is not None:
                ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, LW[l])

    def bnd():
        return vb.Boundary(n_img, L_img, 256, 2, 2, 64)

    bits = lambda t: t.view(torch.int16).numpy()
    # pipelined: one context, one encoder output buffer for every frame
    ctx = vb.Context(llm=lcfg, enc=ecfg, encoder_stream=torch.cuda.Stream())
    load(ctx)
    enc_out = torch.empty((n_img, L_img, 256), dtype=torch.bfloat16, device="cuda")
    got = [bnd() for _ in range(nf)]
    for f in range(nf):
        ctx.vla_run_encoder(f, pats[f], n_img, L_img, enc_out)
        ctx.vla_run_prefix(f, enc_out, n_img, L_img, 2, got[f])
    for f in range(nf):
        ctx.vla_wait_boundary(f, 60000)
    ctx.vla_destroy()
    # serial reference: separate contexts, every step synchronised
    ectx, lctx = vb.Context(enc=ecfg), vb.Context(llm=lcfg)
    load(ectx)
    load(lctx)
    for f in range(nf):
        e = torch.empty((n_img, L_img, 256), dtype=torch.bfloat16, device="cuda")
        ectx.vla_run_encoder(f, pats[f], n_img, L_img, e)
        ectx.encoder_stream.synchronize()
        ref = bnd()
        lctx.vla_run_prefix(f, e, n_img, L_img, 2, ref)
        lctx.vla_wait_boundary(f, 60000)
        assert np.array_equal(bits(got[f].hidden), bits(ref.hidden)), "frame %d boundary" % f
        assert np.array_equal(bits(got[f].kv), bits(ref.kv)), "frame %d kv" % f
    ectx.vla_destroy()
    lctx.vla_destroy()


def test_k0_returns_input():
    c = LlmCase("small_llm", 64, 1)
    tok = c.tokens()
    bnd = c.boundary(n_layers=0)
    c.ctx.vla_run_prefix(7, tok, 1, 64, 0, bnd)
    c.ctx.vla_wait_boundary(7, 10000)
    assert np.array_equal(bnd.hidden.view(__import__("torch").int16).numpy().view(np.uint16), tok)
    c.close()


def test_error_paths():
    import torch
    from paper_2608_14586_amd import binding as vb
    c = LlmCase("small_llm", 64, 2)
    tok = c.tokens()
    bnd = c.boundary()
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_run_prefix(1, tok, 1, 64, 3, bnd)
    assert e.value.name == "VLA_ERR_SHAPE"
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_run_prefix(1, tok, 1, 65, 2, bnd)
    assert e.value.name == "VLA_ERR_SHAPE"
    pageable = vb.Boundary(1, 64, 896, 2, 2, 64)
    pageable.hidden = torch.empty((1, 64, 896), dtype=torch.bfloat16)
    pageable.c.hidden = pageable.hidden.data_ptr()
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_run_prefix(1, tok, 1, 64, 2, pageable)
    assert e.value.name == "VLA_ERR_NOT_PINNED"
    small = c.boundary()
    small.c.kv_bytes -= 2
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_run_prefix(1, tok, 1, 64, 2, small)
    assert e.value.name == "VLA_ERR_SHAPE"
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_wait_boundary(12345, 10)
    assert e.value.name == "VLA_ERR_UNKNOWN_FRAME"
    # an unloaded block is refused before any launch
    cfg = vb.stack_cfg(c.s, "bf16", max_tokens=64, max_batch=1, n_blocks=2)
    ctx2 = vb.Context(llm=cfg)
    ctx2.vla_load_block_weights(vb.VLA_STACK_LLM, 0, c.W[0])
    with pytest.raises(vb.VlaError) as e:
        ctx2.vla_run_prefix(1, tok, 1, 64, 2, bnd)
    assert e.value.name == "VLA_ERR_NOT_LOADED"
    ctx2.vla_run_prefix(1, tok, 1, 64, 1, c.boundary(n_layers=1))
    ctx2.vla_wait_boundary(1, 10000)
    ctx2.vla_destroy()
    c.close()
