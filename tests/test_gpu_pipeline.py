"""The partitioned model end to end (Eq. (6)): decoder blocks [0, k) on the GPU,
the boundary handed to pinned host memory, blocks [k, N) on the host CPU, with
the cross-frame pipeline (Sec. IV-C) consuming boundaries in frame order."""
import numpy as np
import pytest

import oracle
import synth
from synth.configs import llama_like, Workload

from paper_2608_14586_amd import binding as vb
from prefix_cases import log, rel_l2

pytestmark = pytest.mark.gpu

N_BLOCKS, K = 4, 2
SHAPE = llama_like(N_BLOCKS, 256, 4, 2, 64, 704)
WL = Workload("pipe_small", "bf16", SHAPE, None, batch=2, seq=77)


def _setup(out_dtype):
    import torch
    W = [synth.llm_block_weights(WL, l, perturbed=True) for l in range(N_BLOCKS)]
    B, L = WL.batch, WL.seq
    ctx = vb.Context(llm=vb.stack_cfg(SHAPE, "bf16", max_tokens=L, max_batch=B, n_blocks=K))
    for l in range(K):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, W[l])
    sfx = vb.Suffix(vb.stack_cfg(SHAPE, "bf16", max_tokens=L), K, N_BLOCKS)
    for l in range(K, N_BLOCKS):
        sfx.vla_suffix_load_block_weights(l, W[l])
    bnds = [vb.Boundary(B, L, SHAPE.d_model, K, SHAPE.n_kv_heads, SHAPE.head_dim, out_dtype=out_dtype,
                        with_kv=False) for _ in range(3)]
    outs = [np.empty((B, L, SHAPE.d_model), np.float32) for _ in range(3)]
    toks = [synth.tokens(WL, frame=f) for f in range(5)]
    return W, ctx, sfx, bnds, outs, toks, torch


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_pipeline_frames_in_order_and_match_direct_suffix(out_dtype):
    W, ctx, sfx, bnds, outs, toks, torch = _setup(out_dtype)
    B, L, d = WL.batch, WL.seq, SHAPE.d_model
    log("pipeline: %d frames, prefix [0,%d) on the GPU, suffix [%d,%d) on %d host threads, boundary %s"
        % (len(toks), K, K, N_BLOCKS, sfx.vla_suffix_threads(), out_dtype))
    pipe = vb.Pipeline(ctx, sfx, depth=3)
    got = {}
    popped = []
    for f, tok in enumerate(toks):
        if f >= 3:
            fid, tw, tc = pipe.vla_pipeline_pop(60000)
            popped.append(fid)
            got[fid] = outs[(fid - 100) % 3].copy()
            assert tc > 0.0 and tw >= 0.0
        ctx.vla_run_prefix(100 + f, tok, B, L, K, bnds[f % 3])
        pipe.vla_pipeline_push(100 + f, bnds[f % 3], B, L, K, outs[f % 3])
    for _ in range(3):
        fid, _, _ = pipe.vla_pipeline_pop(60000)
        popped.append(fid)
        got[fid] = outs[(fid - 100) % 3].copy()
    pipe.vla_pipeline_destroy()
    assert popped == [100 + f for f in range(len(toks))]
    torch.cuda.synchronize()

    # every frame equals the direct suffix on that frame's boundary, bit for bit
    for f, tok in enumerate(toks):
        ctx.vla_run_prefix(200 + f, tok, B, L, K, bnds[0])
        ctx.vla_wait_boundary(200 + f, 60000)
        direct = np.empty((B, L, d), np.float32)
        hb = bnds[0].hidden
        hb = hb.view(torch.int16).numpy().view(np.uint16) if out_dtype == "bf16" else hb.numpy()
        sfx.vla_suffix_run(np.ascontiguousarray(hb), vb.VLA_BF16 if out_dtype == "bf16" else vb.VLA_F32, B, L,
                           direct)
        assert np.array_equal(got[100 + f], direct), f

    if out_dtype == "f32":
        # the fp32 handoff continues the residual exactly: GPU prefix + host
        # suffix against the oracle over all N blocks, on the blocks' update
        Wf = [{n: synth.as_f32(a).astype(np.float64) for n, a in w.items()} for w in W]
        for f in (0, 4):
            x = synth.as_f32(toks[f]).astype(np.float64)
            ref, _ = oracle.run_prefix(x, lambda l: Wf[l], SHAPE, N_BLOCKS, dtype=np.float64, keep_kv=False)
            for b in range(B):
                e = rel_l2(got[100 + f][b] - x[b], ref[b] - x[b])
                log("  frame %d batch %d: update rel L2 %.2e" % (f, b, e))
                assert e < 1e-2, (f, b, e)


def test_pipeline_rejects_bad_push():
    W, ctx, sfx, bnds, outs, toks, torch = _setup("bf16")
    pipe = vb.Pipeline(ctx, sfx, depth=1)
    small = vb.Boundary(1, 8, SHAPE.d_model, K, SHAPE.n_kv_heads, SHAPE.head_dim, with_kv=False)
    with pytest.raises(vb.VlaError) as e:
        pipe.vla_pipeline_push(1, small, WL.batch, WL.seq, K, outs[0])
    assert e.value.name == "VLA_ERR_SHAPE"
    with pytest.raises(vb.VlaError) as e:
        pipe.vla_pipeline_pop(0)
    assert e.value.name == "VLA_ERR_UNKNOWN_FRAME"
    pipe.vla_pipeline_destroy()
