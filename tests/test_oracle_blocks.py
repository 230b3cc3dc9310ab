"""Pins for the oracle's blocks and stacks (CPU only): third-party
implementations of the same block definitions (Hugging Face transformers'
LLaMA decoder layer and ViT layer, run on CPU in float64), structural
invariants, and the float32-vs-float64 and bf16-rounding error budgets."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth
from synth.configs import llama_like, vit_like, Workload

RNG = np.random.default_rng(99)


def rand_llm_weights(shape, rng, perturbed=True):
    d, H, Hkv, dh, F = shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.d_ff
    n = lambda *s: rng.standard_normal(s) * 0.05
    return {"w_q": n(H * dh, d), "w_k": n(Hkv * dh, d), "w_v": n(Hkv * dh, d), "w_o": n(d, H * dh),
            "w_gate": n(F, d), "w_up": n(F, d), "w_down": n(d, F),
            "norm1_g": rng.uniform(0.5, 1.5, d) if perturbed else np.ones(d),
            "norm2_g": rng.uniform(0.5, 1.5, d) if perturbed else np.ones(d)}


def rand_vit_weights(shape, rng):
    d, F = shape.d_model, shape.d_ff
    hd = shape.n_heads * shape.head_dim
    n = lambda *s: rng.standard_normal(s) * 0.05
    return {"w_q": n(hd, d), "w_k": n(hd, d), "w_v": n(hd, d), "b_qkv": n(3 * hd), "w_o": n(d, hd), "b_o": n(d),
            "w_fc1": n(F, d), "b_fc1": n(F), "w_fc2": n(d, F), "b_fc2": n(d),
            "norm1_g": rng.uniform(0.5, 1.5, d), "norm1_b": n(d) * 2,
            "norm2_g": rng.uniform(0.5, 1.5, d), "norm2_b": n(d) * 2}


@pytest.mark.parametrize("H,Hkv,dh", [(4, 4, 16), (8, 2, 8), (4, 1, 16)])
def test_llm_block_vs_transformers_llama(H, Hkv, dh):
    from transformers.models.llama.modeling_llama import LlamaConfig, LlamaDecoderLayer, LlamaRotaryEmbedding
    d, F, L = 64, 96, 24
    shape = llama_like(1, d, H, Hkv, dh, F)
    W = rand_llm_weights(shape, RNG)
    cfg = LlamaConfig(hidden_size=d, intermediate_size=F, num_attention_heads=H, num_key_value_heads=Hkv,
                      head_dim=dh, rms_norm_eps=shape.norm_eps, rope_theta=shape.rope_base,
                      attention_bias=False, mlp_bias=False, max_position_embeddings=256, hidden_act="silu")
    cfg._attn_implementation = "eager"
    layer = LlamaDecoderLayer(cfg, 0).double()
    sd = {"self_attn.q_proj.weight": W["w_q"], "self_attn.k_proj.weight": W["w_k"],
          "self_attn.v_proj.weight": W["w_v"], "self_attn.o_proj.weight": W["w_o"],
          "mlp.gate_proj.weight": W["w_gate"], "mlp.up_proj.weight": W["w_up"], "mlp.down_proj.weight": W["w_down"],
          "input_layernorm.weight": W["norm1_g"], "post_attention_layernorm.weight": W["norm2_g"]}
    layer.load_state_dict({k: torch.from_numpy(v) for k, v in sd.items()})
    h = RNG.standard_normal((L, d))
    x = torch.from_numpy(h)[None]
    pos = torch.arange(L)[None]
    # transformers forms its rotary angles in float32; build its (cos, sin)
    # inputs in float64 (its own duplicated-half layout) so only the block
    # arithmetic is compared
    inv = torch.tensor([shape.rope_base ** (-2.0 * i / dh) for i in range(dh // 2)], dtype=torch.float64)
    ang = torch.arange(L, dtype=torch.float64)[:, None] * inv[None, :]
    emb = torch.cat([ang, ang], dim=-1)[None]
    cos_sin = (emb.cos(), emb.sin())
    mask = torch.full((L, L), float("-inf"), dtype=torch.float64).triu(1)[None, None]
    with torch.no_grad():
        out = layer(x, attention_mask=mask, position_ids=pos, position_embeddings=cos_sin)
    out = out[0] if isinstance(out, tuple) else out
    cos, sin = oracle.rope_tables(L, dh, shape.rope_base, dtype=np.float64)
    ref, K, V = oracle.llm_block(h, W, shape, cos, sin)
    # transformers keeps its RMSNorm and softmax in float32 even for a float64
    # layer, so agreement is at float32 level; any structural slip is O(1)
    np.testing.assert_allclose(ref, out[0].numpy(), rtol=1e-6, atol=1e-6)


def test_vit_block_vs_transformers_vit():
    from transformers.models.vit.modeling_vit import ViTConfig, ViTLayer
    d, H, dh, F, L = 64, 4, 16, 128, 20
    shape = vit_like(1, d, H, dh, F)
    W = rand_vit_weights(shape, RNG)
    cfg = ViTConfig(hidden_size=d, num_attention_heads=H, intermediate_size=F, hidden_act="gelu",
                    layer_norm_eps=shape.norm_eps, qkv_bias=True, hidden_dropout_prob=0.0,
                    attention_probs_dropout_prob=0.0)
    cfg._attn_implementation = "eager"
    layer = ViTLayer(cfg).double().eval()
    hd = H * dh
    names = dict(layer.named_parameters())
    sd = {"attention.q_proj.weight": W["w_q"], "attention.q_proj.bias": W["b_qkv"][:hd],
          "attention.k_proj.weight": W["w_k"], "attention.k_proj.bias": W["b_qkv"][hd:2 * hd],
          "attention.v_proj.weight": W["w_v"], "attention.v_proj.bias": W["b_qkv"][2 * hd:],
          "attention.o_proj.weight": W["w_o"], "attention.o_proj.bias": W["b_o"],
          "mlp.fc1.weight": W["w_fc1"], "mlp.fc1.bias": W["b_fc1"],
          "mlp.fc2.weight": W["w_fc2"], "mlp.fc2.bias": W["b_fc2"],
          "layernorm_before.weight": W["norm1_g"], "layernorm_before.bias": W["norm1_b"],
          "layernorm_after.weight": W["norm2_g"], "layernorm_after.bias": W["norm2_b"]}
    assert set(sd) == set(names), sorted(names)
    layer.load_state_dict({k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()})
    h = RNG.standard_normal((L, d))
    with torch.no_grad():
        out = layer(torch.from_numpy(h)[None])
    out = out[0] if isinstance(out, tuple) else out
    # float32 softmax inside transformers' eager attention bounds the agreement
    np.testing.assert_allclose(oracle.vit_block(h, W, shape), out[0].numpy(), rtol=1e-6, atol=1e-6)


def test_zero_output_projections_give_identity_bitwise():
    shape = llama_like(1, 32, 2, 2, 16, 48)
    W = rand_llm_weights(shape, RNG)
    W["w_o"][:] = 0
    W["w_down"][:] = 0
    h = RNG.standard_normal((10, 32)).astype(np.float32)
    Wf = {k: v.astype(np.float32) for k, v in W.items()}
    cos, sin = oracle.rope_tables(10, 16, 1e4)
    out, _, _ = oracle.llm_block(h, Wf, shape, cos, sin)
    np.testing.assert_array_equal(out, h)
    vshape = vit_like(1, 32, 2, 16, 48)
    V = {k: v.astype(np.float32) for k, v in rand_vit_weights(vshape, RNG).items()}
    for n in ("w_o", "b_o", "w_fc2", "b_fc2"):
        V[n][:] = 0
    np.testing.assert_array_equal(oracle.vit_block(h, V, vshape), h)


def test_vit_permutation_equivariance():
    shape = vit_like(1, 32, 2, 16, 64)
    W = rand_vit_weights(shape, RNG)
    h = RNG.standard_normal((12, 32))
    perm = RNG.permutation(12)
    np.testing.assert_allclose(oracle.vit_block(h[perm], W, shape), oracle.vit_block(h, W, shape)[perm],
                               rtol=1e-12, atol=1e-12)


def test_batch_independence_bitwise():
    shape = vit_like(2, 32, 2, 16, 64)
    Ws = [{k: v.astype(np.float32) for k, v in rand_vit_weights(shape, RNG).items()} for _ in range(2)]
    x = RNG.standard_normal((3, 8, 32)).astype(np.float32)
    y = oracle.run_encoder(x, lambda l: Ws[l], shape)
    x2 = x.copy()
    x2[1] += 1.0
    y2 = oracle.run_encoder(x2, lambda l: Ws[l], shape)
    np.testing.assert_array_equal(y[0], y2[0])
    np.testing.assert_array_equal(y[2], y2[2])
    assert not np.array_equal(y[1], y2[1])
    lshape = llama_like(2, 32, 2, 1, 16, 48)
    Wl = [rand_llm_weights(lshape, RNG) for _ in range(2)]
    t = RNG.standard_normal((2, 6, 32)).astype(np.float32)
    a, _ = oracle.run_prefix(t, lambda l: Wl[l], lshape, 2)
    t2 = t.copy()
    t2[0] -= 0.5
    b, _ = oracle.run_prefix(t2, lambda l: Wl[l], lshape, 2)
    np.testing.assert_array_equal(a[1], b[1])


def test_prefix_split_composition_and_k0():
    """Eq. (5)-(6): the boundary after k blocks followed by blocks k..N equals
    the full stack; k = 0 returns the input itself."""
    shape = llama_like(4, 32, 4, 2, 8, 40)
    Ws = [rand_llm_weights(shape, RNG) for _ in range(4)]
    t = RNG.standard_normal((1, 9, 32)).astype(np.float32)
    full, kv_full = oracle.run_prefix(t, lambda l: Ws[l], shape, 4)
    for k in range(5):
        hk, kvk = oracle.run_prefix(t, lambda l: Ws[l], shape, k)
        rest, kv_rest = oracle.run_prefix(hk, lambda l: Ws[k + l], shape, 4 - k)
        np.testing.assert_array_equal(rest, full)
        if k:
            np.testing.assert_array_equal(kvk, kv_full[:k])
    h0, kv0 = oracle.run_prefix(t, lambda l: Ws[l], shape, 0)
    np.testing.assert_array_equal(h0, t)
    assert kv0 is None


def test_kv_cache_contents():
    """The cache holds K after RoPE and V as projected, [k][2][B][H_kv][L][dh]."""
    shape = llama_like(1, 32, 4, 2, 8, 40)
    W = rand_llm_weights(shape, RNG)
    t = RNG.standard_normal((2, 7, 32))
    _, kv = oracle.run_prefix(t, lambda l: W, shape, 1, dtype=np.float64)
    cos, sin = oracle.rope_tables(7, 8, 1e4, dtype=np.float64)
    for b in range(2):
        x = oracle.rms_norm(t[b], W["norm1_g"], shape.norm_eps)
        kk = oracle.rope_apply((x @ W["w_k"].T).reshape(7, 2, 8), cos, sin)
        vv = (x @ W["w_v"].T).reshape(7, 2, 8)
        np.testing.assert_allclose(kv[0, 0, b], kk.transpose(1, 0, 2), rtol=1e-13)
        np.testing.assert_allclose(kv[0, 1, b], vv.transpose(1, 0, 2), rtol=1e-13)


def _rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def test_tiny_fp32_oracle_vs_fp64():
    wl = synth.CONFIGS["tiny"]
    t = synth.as_f32(synth.tokens(wl))
    W = lambda l: {n: synth.as_f32(a) for n, a in synth.llm_block_weights(wl, l, perturbed=True).items()}
    h32, kv32 = oracle.run_prefix(t, W, wl.llm, wl.k, dtype=np.float32)
    h64, kv64 = oracle.run_prefix(t, W, wl.llm, wl.k, dtype=np.float64)
    assert _rel_l2(h32, h64) < 1e-6
    assert _rel_l2(h32 - t, h64 - t) < 1e-5
    assert _rel_l2(kv32, kv64) < 1e-6
    assert np.all(np.isfinite(h32))


def _floor(name, L, k, n_img=1):
    """rel-L2 of a bf16-activation computation (matrix-product inputs,
    attention inputs/outputs and gated activations rounded to bf16, boundary
    cast to bf16) against the float32 oracle, after k blocks."""
    wl = synth.CONFIGS[name]
    if name == "vit_l":
        p = synth.as_f32(synth.patches(wl, n_img=n_img, L_img=L))
        W = lambda l: {n: synth.as_f32(a) for n, a in synth.vit_block_weights(wl, l).items()}
        ref = oracle.run_encoder(p, W, wl.enc, n_blocks=k)
        emu = oracle.run_encoder(p, W, wl.enc, n_blocks=k, act_round=oracle.round_bf16)
        return _rel_l2(oracle.round_bf16(emu), ref)
    t = synth.as_f32(synth.tokens(wl, L=L))
    W = lambda l: {n: synth.as_f32(a) for n, a in synth.llm_block_weights(wl, l).items()}
    ref, _ = oracle.run_prefix(t, W, wl.llm, k, keep_kv=False)
    emu, _ = oracle.run_prefix(t, W, wl.llm, k, keep_kv=False, act_round=oracle.round_bf16)
    return _rel_l2(oracle.round_bf16(emu), ref)


@pytest.mark.parametrize("name,L,k", [("small_llm", 512, 6), ("vit_l", 256, 6)])
def test_bf16_noise_floor_within_bar(name, L, k):
    """For the d=896 decoder and the ViT-L encoder, exact bf16-activation
    arithmetic stays far inside the 1e-2 relative-L2 bar (shortened runs)."""
    assert _floor(name, L, k) < 4e-3


def test_bf16_noise_floor_d4096_grows_past_bar():
    """For the d=4096 decoder the same bf16-activation arithmetic already loses
    about 0.4% per block and crosses 1e-2 within about 8 blocks, so no bf16
    path can meet a 1e-2 whole-stack bar against the float32 oracle at k=16
    or k=32; parity there is judged per block and against this floor."""
    e1 = _floor("llm7b", 128, 1)
    e8 = _floor("llm7b", 128, 8)
    assert 2e-3 < e1 < 8e-3
    assert e8 > 9e-3
