"""The vision front and back on the GPU (vla_run_vision): camera images ->
patch embedding -> encoder blocks -> final norm, patch merge and connector
MLP -> the backbone's input tokens, then the decoder prefix over them.

Pins: the oracle's run_vision (oracle/vision.py, itself pinned against
torch's strided convolution, pixel_unshuffle and layer_norm / linear / gelu),
at 1e-2 relative L2 for bf16 and 1e-4 for the fp32 path; text rows and the
k = 0 boundary bit for bit; cameras permuted -> token blocks permuted bit for
bit at full size."""
import numpy as np
import pytest

import oracle
import synth
from synth.configs import VisionShape, Workload, llama_like, vit_like

from paper_2608_14586_amd import binding as vb
from prefix_cases import log, rel_l2

pytestmark = pytest.mark.gpu


def _bits(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _f32(t):
    return synth.as_f32(_bits(t))


def _f64(W):
    return {n: synth.as_f32(a).astype(np.float64) for n, a in W.items()}


class VisionCase:
    def __init__(self, name, dtype, enc, vis, n_img, T, llm=None, k=0, perturbed=True):
        import torch
        self.wl = Workload(name, dtype, llm, enc, n_img=n_img, vision=vis, text_tokens=T)
        self.dtype, self.enc, self.vis, self.n_img, self.T, self.k = dtype, enc, vis, n_img, T, k
        self.V = n_img * vis.tokens_per_image
        self.L = self.V + T
        self.EW = [synth.vit_block_weights(self.wl, l, perturbed=perturbed) for l in range(enc.n_blocks)]
        self.VW = synth.vision_weights(self.wl, perturbed=perturbed)
        self.LW = [synth.llm_block_weights(self.wl, l, perturbed=perturbed) for l in range(k)] if llm else []
        lcfg = vb.stack_cfg(llm, dtype, max_tokens=self.L, max_batch=1, n_blocks=k) if llm else None
        self.ctx = vb.Context(llm=lcfg, enc=vb.stack_cfg(enc, dtype, max_tokens=vis.L_img, max_batch=n_img))
        for l in range(enc.n_blocks):
            self.ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, self.EW[l])
        for l in range(k):
            self.ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, self.LW[l])
        self.ctx.vla_attach_vision(vb.vision_cfg(vis))
        self.ctx.vla_load_vision_weights(self.VW)
        self.tdt = torch.bfloat16 if dtype == "bf16" else torch.float32

    def inputs(self, frame=0):
        return synth.images(self.wl, frame), synth.text(self.wl, frame)

    def run_gpu(self, images, text):
        import torch
        tok = torch.empty((self.L, self.vis.d_out), dtype=self.tdt, device="cuda")
        self.ctx.vla_run_vision(1, np.ascontiguousarray(images), self.n_img, np.ascontiguousarray(text), self.T, tok)
        torch.cuda.synchronize()
        return tok

    def oracle_tokens(self, images, text):
        EW = [_f64(w) for w in self.EW]
        return oracle.run_vision(synth.as_f32(images), lambda l: EW[l], _f64(self.VW), self.enc, self.vis,
                                 synth.as_f32(text), dtype=np.float64)[0]


SMALL_ENC = vit_like(2, 128, 2, 64, 256)
CASES = [
    # 14 x 14 patches of 3 channels: K = 588, padded to 640; non-square 4 x 6 grid, 2 x 2 merge
    ("vis_pad", SMALL_ENC, VisionShape(3, 56, 84, 14, 2, 128, 192), 3, 7),
    # K = 768 (no padding), no merge, one text token
    ("vis_nomerge", SMALL_ENC, VisionShape(3, 32, 64, 16, 1, 192, 128), 2, 1),
    # one channel, K = 64, an 8 x 8 grid merged 4 x 4, no text
    ("vis_merge4", vit_like(1, 192, 3, 64, 384), VisionShape(1, 64, 64, 8, 4, 256, 64), 2, 0),
]


@pytest.mark.parametrize("name,enc,vis,n_img,T", CASES)
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_vision_tokens_match_oracle(name, enc, vis, n_img, T, dtype):
    c = VisionCase(name + "_" + dtype, dtype, enc, vis, n_img, T)
    images, text = c.inputs()
    tok = c.run_gpu(images, text)
    want = c.oracle_tokens(images, text)
    got = _f32(tok)
    e = rel_l2(got[:c.V], want[:c.V])
    bar = 1e-2 if dtype == "bf16" else 1e-4
    log("%s %s: visual tokens rel L2 %.2e (V=%d, bar %.0e)" % (name, dtype, e, c.V, bar))
    assert e < bar
    # per camera too: a camera's block mixed up with another's fails here
    tpi = vis.tokens_per_image
    for i in range(n_img):
        assert rel_l2(got[i * tpi:(i + 1) * tpi], want[i * tpi:(i + 1) * tpi]) < bar
    # text rows are copied as they are
    np.testing.assert_array_equal(_bits(tok)[c.V:], text)


def test_vision_then_prefix_matches_oracle():
    # the whole GPU stage of one frame: E(x_t) from images, then decoder blocks [0, 2)
    import torch
    llm = llama_like(2, 192, 3, 1, 64, 512)
    vis = VisionShape(3, 56, 56, 14, 2, 128, 192)
    c = VisionCase("vis_frame", "bf16", SMALL_ENC, vis, 2, 9, llm=llm, k=2)
    images, text = c.inputs(3)
    tok = c.run_gpu(images, text)
    bnd = vb.Boundary(1, c.L, llm.d_model, 2, llm.n_kv_heads, llm.head_dim, out_dtype="f32")
    c.ctx.vla_run_prefix(5, tok, 1, c.L, 2, bnd)
    c.ctx.vla_wait_boundary(5, 60000)
    x = c.oracle_tokens(images, text)
    LW = [_f64(w) for w in c.LW]
    h, kv = oracle.run_prefix(x[None], lambda l: LW[l], llm, 2, dtype=np.float64)
    e = rel_l2(bnd.hidden.numpy(), h)
    ekv = rel_l2(bnd.kv.float().numpy(), kv)
    log("images -> prefix k=2: boundary rel L2 %.2e, KV %.2e" % (e, ekv))
    assert e < 1e-2 and ekv < 1e-2


def test_dual_stack_over_one_frame():
    # two decoder stacks (a dual-expert backbone) over the same frame tokens,
    # each in a context of its own on one compute stream: the second reads
    # the first context's vision output in stream order.  k = 0 hands the
    # tokens back unchanged; k = 2 runs each stack's first two blocks.
    import torch
    llm = llama_like(2, 128, 2, 1, 64, 320)
    vis = VisionShape(3, 56, 56, 14, 2, 128, 128)
    c = VisionCase("vis_dual", "bf16", SMALL_ENC, vis, 2, 5, llm=llm, k=2)
    wl2 = Workload("vis_dual_b", "bf16", llm, None)
    LW2 = [synth.llm_block_weights(wl2, l, perturbed=True) for l in range(2)]
    ctx2 = vb.Context(llm=vb.stack_cfg(llm, "bf16", max_tokens=c.L, max_batch=1, n_blocks=2),
                      compute_stream=c.ctx.compute_stream)
    for l in range(2):
        ctx2.vla_load_block_weights(vb.VLA_STACK_LLM, l, LW2[l])
    images, text = c.inputs(1)
    tok = torch.empty((c.L, vis.d_out), dtype=torch.bfloat16, device="cuda")
    c.ctx.vla_run_vision(1, images, c.n_img, text, c.T, tok)
    outs = {}
    for k in (0, 2):
        for j, ctx in enumerate((c.ctx, ctx2)):
            b = vb.Boundary(1, c.L, llm.d_model, k, llm.n_kv_heads, llm.head_dim, out_dtype="bf16" if k == 0 else "f32")
            ctx.vla_run_prefix(10 + 10 * k + j, tok, 1, c.L, k, b)
            outs[(k, j)] = (ctx, 10 + 10 * k + j, b)
    for (k, j), (ctx, fid, b) in outs.items():
        ctx.vla_wait_boundary(fid, 60000)
    torch.cuda.synchronize()
    tb = _bits(tok)
    for j in (0, 1):
        np.testing.assert_array_equal(outs[(0, j)][2].hidden.view(torch.int16).numpy().view(np.uint16)[0], tb)
    x = synth.as_f32(tb).astype(np.float64)[None]      # both stacks read the GPU's tokens
    for j, W in enumerate((c.LW, LW2)):
        Wf = [_f64(w) for w in W]
        h, _ = oracle.run_prefix(x, lambda l: Wf[l], llm, 2, dtype=np.float64, keep_kv=False)
        e = rel_l2(outs[(2, j)][2].hidden.numpy() - x, h - x)
        log("dual stack %d, k=2: update rel L2 %.2e" % (j, e))
        assert e < 1e-2
    # the two stacks differ (their weights do)
    assert rel_l2(outs[(2, 0)][2].hidden.numpy(), outs[(2, 1)][2].hidden.numpy()) > 1e-2


def test_dual_stacks_on_two_streams_match_one_stream():
    # the two stacks on compute streams of their own, overlapping: the second
    # stream waits for each frame's vision output by an event, the token rows
    # alternate between two buffers, and the vision of frame f + 2 waits for
    # the second stack's read of frame f.  Every boundary equals that of the
    # same contexts run one step at a time, bit for bit.
    import torch
    llm = llama_like(2, 128, 2, 1, 64, 320)
    vis = VisionShape(3, 56, 56, 14, 2, 128, 128)
    c = VisionCase("vis_dual2", "bf16", SMALL_ENC, vis, 2, 5, llm=llm, k=2)
    wl2 = Workload("vis_dual2_b", "bf16", llm, None)
    ctx2 = vb.Context(llm=vb.stack_cfg(llm, "bf16", max_tokens=c.L, max_batch=1, n_blocks=2))  # own streams
    for l in range(2):
        ctx2.vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(wl2, l, perturbed=True))
    ctxs, frames = (c.ctx, ctx2), range(4)
    new_bnd = lambda: vb.Boundary(1, c.L, llm.d_model, 2, llm.n_kv_heads, llm.head_dim, out_dtype="f32")

    ref = {}
    tok = torch.empty((c.L, vis.d_out), dtype=torch.bfloat16, device="cuda")
    for f in frames:
        images, text = c.inputs(f)
        c.ctx.vla_run_vision(100 + f, images, c.n_img, text, c.T, tok)
        for j, ctx in enumerate(ctxs):
            b = new_bnd()
            ctx.vla_run_prefix(100 + f, tok, 1, c.L, 2, b)
            ctx.vla_wait_boundary(100 + f, 60000)
            torch.cuda.synchronize()
            ref[(f, j)] = b.hidden.numpy().copy()

    toks = [torch.empty_like(tok) for _ in range(2)]
    read_done = [None, None]
    got = []
    for f in frames:
        images, text = c.inputs(f)
        t = toks[f % 2]
        if read_done[f % 2] is not None:
            c.ctx.compute_stream.wait_event(read_done[f % 2])
        c.ctx.vla_run_vision(200 + f, images, c.n_img, text, c.T, t)
        ready = torch.cuda.Event()
        ready.record(c.ctx.compute_stream)
        ctx2.compute_stream.wait_event(ready)
        for j, ctx in enumerate(ctxs):
            b = new_bnd()
            ctx.vla_run_prefix(200 + f, t, 1, c.L, 2, b)
            got.append((f, j, ctx, b))
        done = torch.cuda.Event()
        done.record(ctx2.compute_stream)
        read_done[f % 2] = done
    for f, j, ctx, b in got:
        ctx.vla_wait_boundary(200 + f, 60000)
    torch.cuda.synchronize()
    for f, j, ctx, b in got:
        assert np.array_equal(b.hidden.numpy(), ref[(f, j)]), (f, j)


def test_vision_rejects_bad_calls():
    import torch
    vis = VisionShape(3, 56, 56, 14, 2, 128, 128)
    enc_cfg = vb.stack_cfg(SMALL_ENC, "bf16", max_tokens=16, max_batch=2)
    ctx = vb.Context(enc=enc_cfg)
    wl = Workload("vis_err", "bf16", None, SMALL_ENC, n_img=2, vision=vis, text_tokens=3)
    for l in range(2):
        ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, synth.vit_block_weights(wl, l))
    images, text = synth.images(wl), synth.text(wl)
    tok = torch.empty((8 + 3, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(vb.VlaError) as e:      # nothing attached
        ctx.vla_run_vision(1, images, 2, text, 3, tok)
    assert e.value.name == "VLA_ERR_INVALID_ARG"
    ctx.vla_attach_vision(vb.vision_cfg(vis))
    with pytest.raises(vb.VlaError) as e:      # weights not loaded
        ctx.vla_run_vision(1, images, 2, text, 3, tok)
    assert e.value.name == "VLA_ERR_NOT_LOADED"
    ctx.vla_load_vision_weights(synth.vision_weights(wl))
    bad = [((images, 3, text, 3, tok), "VLA_ERR_SHAPE"),                  # more images than max_batch
           ((images, 2, text, 4, tok), "VLA_ERR_SHAPE"),                  # tokens buffer too small
           ((images, 2, None, 3, tok), "VLA_ERR_INVALID_ARG"),            # text missing
           ((images, 2, text, 3, tok.cpu()), "VLA_ERR_INVALID_ARG")]      # host tokens
    for args, code in bad:
        with pytest.raises(vb.VlaError) as e:
            ctx.vla_run_vision(1, *args)
        assert e.value.name == code, (code, e.value.name)
    ctx.vla_run_vision(1, images, 2, text, 3, tok)     # and the good call still works
    torch.cuda.synchronize()
    assert np.isfinite(_f32(tok)).all()


def test_vision_full_size_camera_zero_and_permutation():
    # six 448 x 448 cameras through the ViT-L-shaped encoder and the 7B
    # connector: camera 0 against the oracle, and the cameras reversed give
    # the token blocks reversed, bit for bit
    import torch
    wl = synth.CONFIGS["sweep7b"]
    vis, enc = wl.vision, wl.enc
    ctx = vb.Context(enc=vb.stack_cfg(enc, "bf16", max_tokens=vis.L_img, max_batch=wl.n_img))
    EW = [synth.vit_block_weights(wl, l) for l in range(enc.n_blocks)]
    for l in range(enc.n_blocks):
        ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, EW[l])
    ctx.vla_attach_vision(vb.vision_cfg(vis))
    VW = synth.vision_weights(wl)
    ctx.vla_load_vision_weights(VW)
    images, text = synth.images(wl, 2), synth.text(wl, 2)
    V, T = wl.n_img * vis.tokens_per_image, wl.text_tokens
    tok = torch.empty((V + T, vis.d_out), dtype=torch.bfloat16, device="cuda")
    ctx.vla_run_vision(1, images, wl.n_img, text, T, tok)
    rev = torch.empty_like(tok)
    ctx.vla_run_vision(2, np.ascontiguousarray(images[::-1]), wl.n_img, text, T, rev)
    torch.cuda.synchronize()
    tpi = vis.tokens_per_image
    a, b = _bits(tok), _bits(rev)
    for i in range(wl.n_img):
        j = wl.n_img - 1 - i
        np.testing.assert_array_equal(a[i * tpi:(i + 1) * tpi], b[j * tpi:(j + 1) * tpi])
    EWf = [{n: synth.as_f32(x) for n, x in w.items()} for w in EW]
    want = oracle.run_vision(synth.as_f32(images[:1]), lambda l: EWf[l], {n: synth.as_f32(x) for n, x in VW.items()},
                             enc, vis, synth.as_f32(text[:0]), dtype=np.float32)[0]
    e = rel_l2(synth.as_f32(a[:tpi]), want)
    log("full-size vision, camera 0: visual tokens rel L2 %.2e" % e)
    assert e < 1e-2
