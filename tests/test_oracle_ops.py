"""Pins for the oracle's operator definitions (CPU only).

Each operator is checked against something other than itself: brute-force
loops in float64, closed forms, invariants, and independent library routines
(torch CPU, Python's math module)."""
import math

import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(1234)


def brute_attention(q, k, v, causal):
    """Triple-loop float64 attention: for each head, query i, key j."""
    L, H, dh = q.shape
    Lk, Hkv, _ = k.shape
    g = H // Hkv
    out = np.zeros((L, H, dh))
    for h in range(H):
        kh = h // g
        for i in range(L):
            js = [j for j in range(Lk) if (not causal or j <= i)]
            s = [sum(q[i, h, t] * k[j, kh, t] for t in range(dh)) / math.sqrt(dh) for j in js]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            z = sum(w)
            for t in range(dh):
                out[i, h, t] = sum(w[n] * v[js[n], kh, t] for n in range(len(js))) / z
    return out


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("H,Hkv", [(2, 2), (4, 2), (4, 1)])
def test_attention_brute_force(causal, H, Hkv):
    L, dh = 9, 8
    q = RNG.standard_normal((L, H, dh))
    k = RNG.standard_normal((L, Hkv, dh))
    v = RNG.standard_normal((L, Hkv, dh))
    np.testing.assert_allclose(oracle.attention(q, k, v, causal), brute_attention(q, k, v, causal),
                               rtol=1e-12, atol=1e-12)


def test_attention_causal_invariant_bitwise():
    L, H, dh = 32, 4, 16
    q = RNG.standard_normal((L, H, dh)).astype(np.float32)
    k = RNG.standard_normal((L, 2, dh)).astype(np.float32)
    v = RNG.standard_normal((L, 2, dh)).astype(np.float32)
    o = oracle.attention(q, k, v, causal=True)
    for i in (0, 5, 17, 30):
        k2, v2, q2 = k.copy(), v.copy(), q.copy()
        k2[i + 1:] += 3.0
        v2[i + 1:] -= 7.0
        q2[i + 1:] *= -2.0
        o2 = oracle.attention(q2, k2, v2, causal=True)
        np.testing.assert_array_equal(o[:i + 1], o2[:i + 1])
        assert not np.array_equal(o[i + 1:], o2[i + 1:])


def test_attention_identical_keys_closed_form():
    L, H, dh = 12, 2, 4
    q = RNG.standard_normal((L, H, dh))
    k = np.tile(RNG.standard_normal((1, H, dh)), (L, 1, 1))
    v = RNG.standard_normal((L, H, dh))
    np.testing.assert_allclose(oracle.attention(q, k, v, False), np.broadcast_to(v.mean(0), (L, H, dh)),
                               rtol=1e-12, atol=1e-12)
    prefix_mean = np.cumsum(v, axis=0) / np.arange(1, L + 1)[:, None, None]
    np.testing.assert_allclose(oracle.attention(q, k, v, True), prefix_mean, rtol=1e-12, atol=1e-12)


def test_attention_gqa_equals_mha_on_repeated_kv():
    L, H, Hkv, dh = 16, 6, 2, 8
    q = RNG.standard_normal((L, H, dh))
    k = RNG.standard_normal((L, Hkv, dh))
    v = RNG.standard_normal((L, Hkv, dh))
    rep = H // Hkv
    np.testing.assert_allclose(oracle.attention(q, k, v, True),
                               oracle.attention(q, np.repeat(k, rep, axis=1), np.repeat(v, rep, axis=1), True),
                               rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("causal", [True, False])
def test_attention_vs_torch_sdpa(causal):
    L, H, Hkv, dh = 40, 8, 2, 32
    q = RNG.standard_normal((L, H, dh))
    k = RNG.standard_normal((L, Hkv, dh))
    v = RNG.standard_normal((L, Hkv, dh))
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2)[None] for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=causal, enable_gqa=True)
    np.testing.assert_allclose(oracle.attention(q, k, v, causal), ref[0].permute(1, 0, 2).numpy(),
                               rtol=1e-10, atol=1e-10)


def test_rope_identity_at_pos0_and_norm_preserving():
    dh = 16
    cos, sin = oracle.rope_tables(5, dh, 10000.0, dtype=np.float64)
    x = RNG.standard_normal((5, 3, dh))
    y = oracle.rope_apply(x, cos, sin)
    np.testing.assert_array_equal(y[0], x[0])
    half = dh // 2
    pair_x = x[..., :half] ** 2 + x[..., half:] ** 2
    pair_y = y[..., :half] ** 2 + y[..., half:] ** 2
    np.testing.assert_allclose(pair_y, pair_x, rtol=1e-12)


def test_rope_complex_form():
    L, dh, base = 20, 32, 10000.0
    cos, sin = oracle.rope_tables(L, dh, base, dtype=np.float64)
    x = RNG.standard_normal((L, 2, dh))
    half = dh // 2
    z = x[..., :half] + 1j * x[..., half:]
    ang = np.array([[p * base ** (-2.0 * i / dh) for i in range(half)] for p in range(L)])
    w = z * np.exp(1j * ang)[:, None, :]
    ref = np.concatenate([w.real, w.imag], axis=-1)
    np.testing.assert_allclose(oracle.rope_apply(x, cos, sin), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("dtype,tol", [(np.float64, 1e-10), (np.float32, 2e-4)])
def test_rope_relative_position(dtype, tol):
    dh, L, shift = 64, 50, 37
    q = RNG.standard_normal((L, 1, dh)).astype(dtype)
    k = RNG.standard_normal((L, 1, dh)).astype(dtype)
    c0, s0 = oracle.rope_tables(L, dh, 10000.0, dtype=dtype)
    c1, s1 = oracle.rope_tables(L, dh, 10000.0, dtype=dtype, pos0=shift)
    d0 = oracle.rope_apply(q, c0, s0)[:, 0] @ oracle.rope_apply(k, c0, s0)[:, 0].T
    d1 = oracle.rope_apply(q, c1, s1)[:, 0] @ oracle.rope_apply(k, c1, s1)[:, 0].T
    assert np.max(np.abs(d1 - d0)) / np.max(np.abs(d0)) < tol


def test_rmsnorm_unit_rms_and_scale_invariance():
    x = RNG.standard_normal((7, 300))
    eps = 1e-6
    y = oracle.rms_norm(x, np.ones(300), eps)
    ms = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), np.sqrt(ms / (ms + eps)), rtol=1e-12)
    np.testing.assert_allclose(oracle.rms_norm(5.0 * x, np.ones(300), 0.0), oracle.rms_norm(x, np.ones(300), 0.0),
                               rtol=1e-12)
    g = RNG.uniform(0.5, 1.5, 300)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (300,), torch.from_numpy(g), eps)
    np.testing.assert_allclose(oracle.rms_norm(x, g, eps), ref.numpy(), rtol=1e-12)


def test_layernorm_moments_shift_invariance_and_torch():
    x = RNG.standard_normal((7, 300)) * 3 + 1
    eps = 1e-6
    y = oracle.layer_norm(x, np.ones(300), np.zeros(300), eps)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-12)
    var = x.var(-1)
    np.testing.assert_allclose(y.var(-1), var / (var + eps), rtol=1e-12)
    np.testing.assert_allclose(oracle.layer_norm(x + 11.0, np.ones(300), np.zeros(300), eps), y, atol=1e-12)
    g, b = RNG.uniform(0.5, 1.5, 300), RNG.standard_normal(300)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (300,), torch.from_numpy(g), torch.from_numpy(b), eps)
    np.testing.assert_allclose(oracle.layer_norm(x, g, b, eps), ref.numpy(), rtol=1e-11, atol=1e-12)


def test_activations_on_grid():
    z = np.linspace(-12, 12, 2001)
    np.testing.assert_allclose(oracle.gelu_erf(z), [t * 0.5 * (1 + math.erf(t / math.sqrt(2))) for t in z],
                               rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(oracle.silu(z), [t / (1 + math.exp(-t)) for t in z], rtol=1e-13)
    assert oracle.gelu_erf(np.zeros(1))[0] == 0 and oracle.silu(np.zeros(1))[0] == 0
    g, u = RNG.standard_normal(50), RNG.standard_normal(50)
    np.testing.assert_allclose(oracle.swiglu(g, u), [a / (1 + math.exp(-a)) * b for a, b in zip(g, u)], rtol=1e-13)
    z32 = z.astype(np.float32)
    np.testing.assert_allclose(oracle.gelu_erf(z32), oracle.gelu_erf(z32.astype(np.float64)), rtol=2e-6, atol=1e-12)
    # torch's float32 GELU loses the far negative tail to cancellation; compare absolutely
    np.testing.assert_allclose(oracle.gelu_erf(z32), torch.nn.functional.gelu(torch.from_numpy(z32)).numpy(),
                               rtol=1e-6, atol=1e-6)


def test_round_bf16_matches_torch():
    x = (RNG.standard_normal(100000) * 10).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x), ref)


def test_transfer_bytes_eq11():
    # S_hid = B * L_p * D * b: a 1024-token, 4096-wide bf16 boundary is 8 MiB.
    assert oracle.transfer_bytes(1, 1024, 4096, 2) == 8 * 1024 * 1024
    assert oracle.transfer_bytes(2, 3, 5, 4) == 120


def test_pins_catch_planted_mistakes():
    """Plausible slips planted into copies of oracle functions (on the CPU)
    are caught by the same independent references the pins above use."""
    L, H, Hkv, dh = 10, 4, 2, 8
    q = RNG.standard_normal((L, H, dh))
    k = RNG.standard_normal((L, Hkv, dh))
    v = RNG.standard_normal((L, Hkv, dh))
    ref = brute_attention(q, k, v, True)

    def attn_off_by_one(q, k, v):          # mask j < i instead of j <= i
        o = np.empty_like(q)
        for h in range(H):
            s = q[:, h] @ k[:, h // 2].T / math.sqrt(dh)
            blocked = np.triu(np.ones((L, L), bool), k=0)
            blocked[0, 0] = False               # keep row 0 finite
            s = np.where(blocked, -np.inf, s)
            p = np.exp(s - s.max(-1, keepdims=True))
            o[:, h] = (p / p.sum(-1, keepdims=True)) @ v[:, h // 2]
        return o

    def attn_bad_group(q, k, v):            # head h -> KV head h % H_kv
        o = np.empty_like(q)
        for h in range(H):
            s = q[:, h] @ k[:, h % Hkv].T / math.sqrt(dh)
            s = np.where(np.triu(np.ones((L, L), bool), k=1), -np.inf, s)
            p = np.exp(s - s.max(-1, keepdims=True))
            o[:, h] = (p / p.sum(-1, keepdims=True)) @ v[:, h % Hkv]
        return o

    for bad in (attn_off_by_one, attn_bad_group):
        assert not np.allclose(bad(q, k, v), ref, atol=1e-6)

    cos, sin = oracle.rope_tables(L, dh, 10000.0, dtype=np.float64)
    x = RNG.standard_normal((L, 2, dh))
    half = dh // 2
    z = x[..., :half] + 1j * x[..., half:]
    ang = np.array([[p * 10000.0 ** (-2.0 * i / dh) for i in range(half)] for p in range(L)])
    w = z * np.exp(1j * ang)[:, None, :]
    rope_ref = np.concatenate([w.real, w.imag], axis=-1)
    x1, x2 = x[..., :half], x[..., half:]
    flipped = np.concatenate([x1 * cos[:, None] + x2 * sin[:, None], x2 * cos[:, None] - x1 * sin[:, None]], -1)
    adjacent = x.copy()                      # rotate interleaved pairs instead of halves
    adjacent[..., 0::2] = x[..., 0::2] * cos[:, None] - x[..., 1::2] * sin[:, None]
    adjacent[..., 1::2] = x[..., 1::2] * cos[:, None] + x[..., 0::2] * sin[:, None]
    for bad in (flipped, adjacent):
        assert not np.allclose(bad, rope_ref, atol=1e-6)

    xn = RNG.standard_normal((5, 64))
    g = RNG.uniform(0.5, 1.5, 64)
    tref = torch.nn.functional.rms_norm(torch.from_numpy(xn), (64,), torch.from_numpy(g), 1e-6).numpy()
    no_gain = xn / np.sqrt(np.mean(xn * xn, -1, keepdims=True) + 1e-6)
    sum_not_mean = xn / np.sqrt(np.sum(xn * xn, -1, keepdims=True) + 1e-6) * g
    for bad in (no_gain, sum_not_mean):
        assert not np.allclose(bad, tref, atol=1e-6)
