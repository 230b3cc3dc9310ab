"""vla_decode_step_static -- the decode step whose scratch lies in a fixed
device array, for callers that cannot allocate -- against vla_decode_step on
the same cache and inputs: two calls in a row, the second smaller, bit for
bit; then its size limit, refused before any launch."""
import numpy as np
import pytest

import synth
from synth.configs import Workload, llama_like

from paper_2608_14586_amd import binding as vb

pytestmark = pytest.mark.gpu


def _context(shape, B, L_cap, k, name):
    wl = Workload(name, "bf16", shape, None)
    ctx = vb.Context(llm=vb.stack_cfg(shape, "bf16", max_tokens=L_cap, max_batch=B, n_blocks=k))
    for l in range(k):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(wl, l, perturbed=True))
    return ctx


@pytest.mark.parametrize("prec", ["bf16", "split"])
def test_static_step_matches_workspace_step(prec):
    import torch
    shape = llama_like(2, 1024, 8, 2, 128, 2816)
    k, L, L_cap = 2, 300, 320
    d, Hkv, dh = shape.d_model, shape.n_kv_heads, shape.head_dim
    ctx = _context(shape, 3, L_cap, k, "noalloc")
    if prec == "split":
        # split operands: the gated activation's remainder rows also live in the fixed array
        ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_SPLIT)
    toks = synth.normal_bf16(synth.seed_of("noalloc", "tok"), (3, L + 1, d))
    bnd = vb.Boundary(3, L, d, k, Hkv, dh)
    ctx.vla_run_prefix(1, np.ascontiguousarray(toks[:, :L]), 3, L, k, bnd)
    ctx.vla_wait_boundary(1, 60000)
    cache = torch.zeros((k, 2, 3, Hkv, L_cap, dh), dtype=torch.bfloat16, device="cuda")
    cache[:, :, :, :, :L] = bnd.kv.cuda()
    fid = [10]
    # (batch, position): the second call is smaller than the first
    for B, pos in ((3, L), (1, 100)):
        x = np.ascontiguousarray(toks[:B, pos])
        c_ws, c_st = cache[:, :, :B].clone(), cache[:, :, :B].clone()
        got = {}
        for name, c, call in (("workspace", c_ws, ctx.vla_decode_step), ("static", c_st, ctx.vla_decode_step_static)):
            ob = vb.Boundary(B, 1, d, 0, Hkv, dh, out_dtype="f32", with_kv=False)
            call(fid[0], x, B, pos, k, c, L_cap, ob)
            ctx.vla_wait_boundary(fid[0], 60000)
            fid[0] += 1
            got[name] = ob.hidden.numpy().copy()
        assert np.isfinite(got["static"]).all()
        assert np.array_equal(got["static"], got["workspace"]), (B, pos)
        assert torch.equal(c_st, c_ws), (B, pos)
    ctx.vla_destroy()


def test_static_step_refuses_steps_above_its_scratch():
    import torch
    # 32 heads x 128 dims at B = 4: the split-key partials alone pass 4 MiB
    # at position 8000
    shape = llama_like(1, 512, 32, 32, 128, 512)
    B, pos, L_cap = 4, 8000, 8008
    ctx = _context(shape, B, L_cap, 1, "noalloc_big")
    cache = torch.zeros((1, 2, B, 32, L_cap, 128), dtype=torch.bfloat16, device="cuda")
    x = synth.normal_bf16(synth.seed_of("noalloc_big_x"), (B, 512))
    ob = vb.Boundary(B, 1, 512, 0, 32, 128, out_dtype="f32", with_kv=False)
    with pytest.raises(vb.VlaError) as e:
        ctx.vla_decode_step_static(1, x, B, pos, 1, cache, L_cap, ob)
    assert e.value.name == "VLA_ERR_SHAPE" and "fixed scratch" in str(e.value)
    # nothing was enqueued: the row a step would append is still zero, and a
    # step that fits runs after the refusal
    assert not cache[:, :, :, :, pos].any()
    ctx.vla_decode_step_static(2, x, B, 100, 1, cache, L_cap, ob)
    ctx.vla_wait_boundary(2, 60000)
    assert np.isfinite(ob.hidden.numpy()).all()
    ctx.vla_destroy()
