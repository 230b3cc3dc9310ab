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
    # the fp32 debug path has no reduced-precision operand to split
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_SPLIT)
    assert e.value.name == "VLA_ERR_UNSUPPORTED"
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


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
def test_split_invariance_against_oracle(k):
    """Eq. (5)-(6): the GPU prefix [0, k) handed over as the bf16 boundary
    (b = 2, Eq. (11)) and continued by the oracle over [k, N) equals the
    oracle over the whole stack, for every partition point of an N = 4 stack."""
    import synth
    import oracle
    from prefix_cases import f32_weights
    N, L = 4, 256
    c = LlmCase("small_llm", L, N, perturbed=True)
    tok = c.tokens(frame=11)
    full, _ = c.oracle(tok, k0=0, k1=N, keep_kv=False)
    bnd = c.boundary(n_layers=k)
    c.ctx.vla_run_prefix(20 + k, tok, 1, L, k, bnd)
    c.ctx.vla_wait_boundary(20 + k, 60000)
    h = to_f32(bnd.hidden)
    rest, _ = oracle.run_prefix(h, lambda l: f32_weights(c.W[k + l]), c.s, N - k, keep_kv=False)
    e = rel_l2(rest, full)
    log("  split at k=%d of N=%d: GPU [0,k) + oracle [k,N) vs oracle [0,N): %.2e" % (k, N, e))
    assert e <= 1e-2
    if k == 0:
        assert np.array_equal(bnd.hidden.view(__import__("torch").int16).numpy().view(np.uint16), tok)
    c.close()


def test_wait_boundary_times_out_then_collects():
    """vla_wait_boundary with a zero budget right after a long prefix is
    enqueued reports VLA_ERR_TIMEOUT and leaves the frame in flight; an
    unbounded wait then collects it, identical to an undisturbed run."""
    import torch
    from paper_2608_14586_amd import binding as vb
    c = LlmCase("small_llm", 4096, 12)
    tok = c.tokens(frame=0)
    ref = c.run(tok, frame=1)
    bnd = c.boundary()
    c.ctx.vla_run_prefix(2, tok, 1, c.L, c.k, bnd)
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_wait_boundary(2, 0)
    assert e.value.name == "VLA_ERR_TIMEOUT"
    c.ctx.vla_wait_boundary(2, -1)
    bits = lambda t: t.view(torch.int16).numpy()
    assert np.array_equal(bits(bnd.hidden), bits(ref.hidden))
    assert np.array_equal(bits(bnd.kv), bits(ref.kv))
    g, x, t = c.ctx.vla_frame_times(2)
    assert 0 < g <= t
    c.close()


# a 3-block prefix makes 23 launches (intake, 7 per block, the bf16
# boundary cast), a 3-block decode step with an f32 boundary 16 (intake, 5
# per block; the boundary is a copy)
@pytest.mark.parametrize("after", [0, 1, 7, 22])
def test_failure_mid_frame_frees_its_slot(after):
    """A launch failing part-way through a frame (injected before launch
    `after` of the frame; every kernel still runs to completion) fails that
    call, forgets the frame, and leaves the context working: more frames than
    there are slots then run bit for bit as on a fresh context."""
    import torch
    from paper_2608_14586_amd import binding as vb
    c = LlmCase("small_llm", 128, 3)
    toks = [c.tokens(frame=f) for f in range(5)]
    clean = [c.run(t, frame=100 + f) for f, t in enumerate(toks)]
    c.ctx.vla_inject_fault(after)
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_run_prefix(7, toks[0], 1, c.L, c.k, c.boundary())
    assert e.value.name == "VLA_ERR_HIP" and "injected" in str(e.value)
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_wait_boundary(7, 1000)
    assert e.value.name == "VLA_ERR_UNKNOWN_FRAME"
    bnds = [c.boundary() for _ in toks]
    for f, t in enumerate(toks):
        c.ctx.vla_run_prefix(200 + f, t, 1, c.L, c.k, bnds[f])
    bits = lambda t: t.view(torch.int16).numpy()
    for f in range(len(toks)):
        c.ctx.vla_wait_boundary(200 + f, 60000)
        assert np.array_equal(bits(bnds[f].hidden), bits(clean[f].hidden)), f
        assert np.array_equal(bits(bnds[f].kv), bits(clean[f].kv)), f
    # the same for a decode step over the first frame's cache
    s, pos = c.s, 100
    cache = torch.zeros((c.k, 2, 1, s.n_kv_heads, c.L, s.head_dim), dtype=torch.bfloat16, device="cuda")
    cache[:, :, :, :, :pos] = clean[0].kv[:, :, :, :, :pos].cuda()
    x = np.ascontiguousarray(toks[1][:, pos])
    want = vb.Boundary(1, 1, s.d_model, 0, s.n_kv_heads, s.head_dim, out_dtype="f32", with_kv=False)
    c.ctx.vla_decode_step(300, x, 1, pos, c.k, cache.clone(), c.L, want)
    c.ctx.vla_wait_boundary(300, 60000)
    c.ctx.vla_inject_fault(min(after, 15))
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_decode_step(301, x, 1, pos, c.k, cache.clone(), c.L,
                              vb.Boundary(1, 1, s.d_model, 0, s.n_kv_heads, s.head_dim, out_dtype="f32", with_kv=False))
    assert e.value.name == "VLA_ERR_HIP"
    got = vb.Boundary(1, 1, s.d_model, 0, s.n_kv_heads, s.head_dim, out_dtype="f32", with_kv=False)
    c.ctx.vla_decode_step(302, x, 1, pos, c.k, cache.clone(), c.L, got)
    c.ctx.vla_wait_boundary(302, 60000)
    assert np.array_equal(got.hidden.numpy(), want.hidden.numpy())
    c.close()


def test_split_precision_small_stack():
    """VLA_PREC_SPLIT carries the products' activation operands as hi + lo
    bf16 pairs: the boundary and every KV layer move closer to the fp32
    oracle than with plain bf16 operands, on a ragged, perturbed GQA stack;
    switching back restores the bf16 result bit for bit."""
    import torch
    from paper_2608_14586_amd import binding as vb
    c = LlmCase("small_llm", 333, 6, perturbed=True)
    tok = c.tokens(frame=4)
    ref, kv = c.oracle(tok)
    plain = c.run(tok, frame=1, out_dtype="f32")
    c.ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_SPLIT)
    split = c.run(tok, frame=2, out_dtype="f32")
    c.ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_BF16)
    again = c.run(tok, frame=3, out_dtype="f32")
    e_b, e_s = rel_l2(plain.hidden.numpy(), ref), rel_l2(split.hidden.numpy(), ref)
    kv_b = [rel_l2(to_f32(plain.kv[l]), kv[l]) for l in range(6)]
    kv_s = [rel_l2(to_f32(split.kv[l]), kv[l]) for l in range(6)]
    log("  small_llm L=333 k=6: boundary bf16 %.2e, split %.2e; kv max bf16 %.2e, split %.2e"
        % (e_b, e_s, max(kv_b), max(kv_s)))
    assert e_s <= 0.7 * e_b and e_s <= 1e-2 and max(kv_s) <= 1e-2
    # the first layer's K/V see only the first RMSNorm's split operand
    assert kv_s[0] <= kv_b[0] and max(kv_s[1:]) <= 0.8 * max(kv_b[1:])
    assert np.array_equal(again.hidden.numpy(), plain.hidden.numpy())
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_set_precision(vb.VLA_STACK_ENC, vb.VLA_PREC_SPLIT)
    assert e.value.name == "VLA_ERR_INVALID_ARG"
    with pytest.raises(vb.VlaError) as e:
        c.ctx.vla_set_precision(vb.VLA_STACK_LLM, 7)
    assert e.value.name == "VLA_ERR_INVALID_ARG"
    c.close()
