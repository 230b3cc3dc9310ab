"""Plain numpy definitions of the prefix's blocks (test infrastructure only).

Shapes: a sequence's residual stream is ``h[L, d]``; projections use the
nn.Linear convention ``y = x @ W.T`` with ``W[out, in]``.  Attention tensors
are ``[L, heads, head_dim]``.  The KV cache the prefix writes is
``[k][2][B][H_kv][L][head_dim]`` (K after RoPE, V as projected).
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erfc as _erfc


# ----------------------------------------------------------------------------
# elementwise and normalisation
# ----------------------------------------------------------------------------

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm (Zhang & Sennrich, 2019): x / sqrt(mean(x^2) + eps) * g, over
    the last axis.  It is the "normalized feature transformation" inside a
    decoder block (Sec. IV-B)."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + x.dtype.type(eps)) * g


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm (Ba et al., 2016) with biased variance: (x - mu) / sqrt(var +
    eps) * g + b over the last axis; the pre-norm of a ViT block."""
    mu = np.mean(x, axis=-1, keepdims=True)
    xc = x - mu
    var = np.mean(xc * xc, axis=-1, keepdims=True)
    return xc / np.sqrt(var + x.dtype.type(eps)) * g + b


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU / swish: z * sigmoid(z) = z / (1 + exp(-z))."""
    one = z.dtype.type(1)
    return z / (one + np.exp(-z))


def swiglu(gate: np.ndarray, up: np.ndarray) -> np.ndarray:
    """SwiGLU gating (Shazeer, 2020): silu(gate) * up."""
    return silu(gate) * up


def gelu_erf(z: np.ndarray) -> np.ndarray:
    """Exact GELU (Hendrycks & Gimpel, 2016): z * Phi(z) with the normal CDF
    Phi(z) = 0.5 * (1 + erf(z / sqrt 2)), evaluated as 0.5 * erfc(-z / sqrt 2)
    so the negative tail does not cancel."""
    t = z.dtype.type
    return z * t(0.5) * _erfc(-z / t(math.sqrt(2.0))).astype(z.dtype)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as
    float32.  Used only by the rounding-emulation mode that estimates the bf16
    noise floor; the plain oracle never calls it."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = (u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    return u.astype(np.uint32).view(np.float32)


# ----------------------------------------------------------------------------
# rotary position embedding
# ----------------------------------------------------------------------------

def rope_tables(L: int, head_dim: int, base: float, dtype=np.float32, pos0: int = 0):
    """Rotary angles (Su et al., RoFormer, 2021): theta_i = base^(-2i/head_dim)
    for i < head_dim/2, phi[p, i] = p * theta_i for positions p = pos0 ..
    pos0+L-1.  Angles are formed in float64 and the cos/sin tables cast to
    ``dtype``.  Returns (cos, sin), each [L, head_dim/2]."""
    half = head_dim // 2
    i = np.arange(half, dtype=np.float64)
    theta = np.power(np.float64(base), -2.0 * i / head_dim)
    pos = np.arange(pos0, pos0 + L, dtype=np.float64)
    phi = pos[:, None] * theta[None, :]
    return np.cos(phi).astype(dtype), np.sin(phi).astype(dtype)


def rope_apply(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half RoPE on x[L, heads, head_dim]: with x1 = x[..., :h/2] and
    x2 = x[..., h/2:], out = [x1 cos - x2 sin, x2 cos + x1 sin]."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# ----------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------

def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, causal: bool) -> np.ndarray:
    """Scaled dot-product attention (Vaswani et al., 2017) with grouped KV heads.

    q[L, H, dh], k/v[L, H_kv, dh].  Query head h reads KV head h // (H / H_kv)
    (contiguous groups).  Scores q.k / sqrt(dh); a causal mask gives query i
    only keys j <= i; softmax is max-subtracted.  Returns o[L, H, dh].
    """
    L, H, dh = q.shape
    Hkv = k.shape[1]
    assert H % Hkv == 0
    group = H // Hkv
    scale = q.dtype.type(1.0 / math.sqrt(dh))
    o = np.empty_like(q)
    if causal:
        future = np.triu(np.ones((L, k.shape[0]), dtype=bool), k=1)
    for h in range(H):
        g = h // group
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        if causal:
            s = np.where(future, -np.inf, s)
        s = s - np.max(s, axis=-1, keepdims=True)
        p = np.exp(s)
        p = p / np.sum(p, axis=-1, keepdims=True)
        o[:, h, :] = p @ v[:, g, :]
    return o


# ----------------------------------------------------------------------------
# blocks
# ----------------------------------------------------------------------------

def _ident(x):
    return x


def llm_block(h: np.ndarray, W: dict, shape, cos: np.ndarray, sin: np.ndarray, act_round=None):
    """One pre-norm decoder block B_l (Sec. IV-B: normalisation, projections,
    attention, feed-forward, residual connections), LLaMA-style:

        x = RMSNorm(h, g1);  q, k, v = x Wq^T, x Wk^T, x Wv^T
        q, k = RoPE(q), RoPE(k);  h = h + Attn_causal(q, k, v) Wo^T
        x = RMSNorm(h, g2);  h = h + (silu(x Wg^T) * (x Wu^T)) Wd^T

    h[L, d].  Returns (h_out, K[H_kv, L, dh], V[H_kv, L, dh]) with K after RoPE.
    ``act_round`` (noise-floor mode only) rounds every matrix-product input,
    the attention inputs and the gated activation.
    """
    r = act_round or _ident
    L, d = h.shape
    H, Hkv, dh = shape.n_heads, shape.n_kv_heads, shape.head_dim
    x = r(rms_norm(h, W["norm1_g"], shape.norm_eps))
    q = (x @ W["w_q"].T).reshape(L, H, dh)
    k = (x @ W["w_k"].T).reshape(L, Hkv, dh)
    v = (x @ W["w_v"].T).reshape(L, Hkv, dh)
    if shape.use_rope:
        q = rope_apply(q, cos, sin)
        k = rope_apply(k, cos, sin)
    q, k, v = r(q), r(k), r(v)
    o = r(attention(q, k, v, causal=shape.causal)).reshape(L, H * dh)
    h = h + o @ W["w_o"].T
    x = r(rms_norm(h, W["norm2_g"], shape.norm_eps))
    a = r(swiglu(x @ W["w_gate"].T, x @ W["w_up"].T))
    h = h + a @ W["w_down"].T
    return h, np.ascontiguousarray(k.transpose(1, 0, 2)), np.ascontiguousarray(v.transpose(1, 0, 2))


def vit_block(h: np.ndarray, W: dict, shape, act_round=None) -> np.ndarray:
    """One pre-LayerNorm ViT block (Dosovitskiy et al., 2020) on one image's
    tokens h[L, d], bidirectional attention (no mask, no position term):

        x = LN(h; g1, b1);  q|k|v = x W^T + b_qkv
        h = h + Attn(q, k, v) Wo^T + b_o
        x = LN(h; g2, b2);  h = h + GELU(x W1^T + b1) W2^T + b2
    """
    r = act_round or _ident
    L, d = h.shape
    H, dh = shape.n_heads, shape.head_dim
    hd = H * dh
    x = r(layer_norm(h, W["norm1_g"], W["norm1_b"], shape.norm_eps))
    b = W["b_qkv"]
    q = (x @ W["w_q"].T + b[:hd]).reshape(L, H, dh)
    k = (x @ W["w_k"].T + b[hd:2 * hd]).reshape(L, H, dh)
    v = (x @ W["w_v"].T + b[2 * hd:]).reshape(L, H, dh)
    q, k, v = r(q), r(k), r(v)
    o = r(attention(q, k, v, causal=False)).reshape(L, hd)
    h = h + (o @ W["w_o"].T + W["b_o"])
    x = r(layer_norm(h, W["norm2_g"], W["norm2_b"], shape.norm_eps))
    a = r(gelu_erf(x @ W["w_fc1"].T + W["b_fc1"]))
    h = h + (a @ W["w_fc2"].T + W["b_fc2"])
    return h


# ----------------------------------------------------------------------------
# stacks
# ----------------------------------------------------------------------------

def _cast_weights(W: dict, dtype) -> dict:
    return {n: np.asarray(a, dtype=dtype) for n, a in W.items()}


def run_prefix(tokens: np.ndarray, weights_of, shape, k: int, dtype=np.float32,
               keep_kv: bool = True, on_layer=None, act_round=None, pos0: int = 0):
    """The GPU-executed prefix of the partitioned backbone (Eq. (5)):
    h^(k) = B_k(...B_1(E(x))), here with E(x) given as input embeddings.

    tokens[B, L, d] (already float); ``weights_of(l)`` returns block l's
    weights as float arrays; ``k`` whole blocks are applied (the partition
    point is a block count, Sec. IV-B).  k = 0 returns the input.
    Returns (h[B, L, d], kv[k, 2, B, H_kv, L, dh] or None).
    ``on_layer(l, h, K, V)`` is called after each block with that block's
    output and cache entries (K, V as [B, H_kv, L, dh]).
    """
    h = np.array(tokens, dtype=dtype, copy=True)
    B, L, d = h.shape
    Hkv, dh = shape.n_kv_heads, shape.head_dim
    cos, sin = rope_tables(L, dh, shape.rope_base, dtype=dtype, pos0=pos0)
    kv = np.empty((k, 2, B, Hkv, L, dh), dtype=dtype) if (keep_kv and k > 0) else None
    for l in range(k):
        W = _cast_weights(weights_of(l), dtype)
        Ks, Vs = [], []
        for b in range(B):
            h[b], K, V = llm_block(h[b], W, shape, cos, sin, act_round=act_round)
            Ks.append(K)
            Vs.append(V)
        if kv is not None:
            kv[l, 0] = np.stack(Ks)
            kv[l, 1] = np.stack(Vs)
        if on_layer is not None:
            on_layer(l, h, np.stack(Ks), np.stack(Vs))
        del W
    return h, kv


def run_encoder(patches: np.ndarray, weights_of, shape, n_blocks: int = None, dtype=np.float32,
                act_round=None, on_layer=None) -> np.ndarray:
    """The visual encoder's transformer blocks applied to each image's patch
    embeddings independently (the ViT part of the GPU stage, Sec. IV-A).
    patches[n_img, L_img, d]; returns the encoder output [n_img, L_img, d]."""
    h = np.array(patches, dtype=dtype, copy=True)
    nb = shape.n_blocks if n_blocks is None else n_blocks
    for l in range(nb):
        W = _cast_weights(weights_of(l), dtype)
        for i in range(h.shape[0]):
            h[i] = vit_block(h[i], W, shape, act_round=act_round)
        if on_layer is not None:
            on_layer(l, h)
        del W
    return h


def transfer_bytes(B: int, L: int, D: int, elem_bytes: int) -> int:
    """Size of the boundary tensor moved across devices, S_hid = B * L_p * D * b
    (Eq. (11))."""
    return B * L * D * elem_bytes
