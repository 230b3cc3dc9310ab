"""Seeded synthetic inputs and random-init weights for the prefix workloads.

This package holds no arithmetic of the transformer blocks.  It fills arrays
with pseudo-random values (Philox4x32-10 + Box-Muller, see ``philox.c``) so the
oracle and the GPU path consume identical, reproducible inputs.  bf16 tensors
are returned as ``uint16`` bit patterns; ``bf16_to_f32`` widens them exactly.

Stream identity: every tensor is drawn from its own stream whose 64-bit seed is
``seed_of(workload, stack, layer, tensor_name, frame)`` (BLAKE2b of the parts),
so one layer can be generated without generating the others.
"""
from __future__ import annotations

import ctypes
import hashlib
import os
import subprocess

import numpy as np

from .configs import CONFIGS, StackShape, VisionShape, Workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``philox.c`` into ``libsynth.so`` (gcc + OpenMP)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC",
                               os.path.join(_HERE, "philox.c"), "-o", tmp, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build(force=False)
        L = ctypes.CDLL(_SO)
        u64, f32, vp = ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p
        L.synth_philox4x32_10.argtypes = [vp, vp, vp]
        L.synth_normal_f32.argtypes = [u64, u64, u64, f32, f32, vp]
        L.synth_normal_bf16.argtypes = [u64, u64, u64, f32, f32, vp]
        L.synth_uniform_f32.argtypes = [u64, u64, u64, f32, f32, vp]
        L.synth_bf16_to_f32.argtypes = [vp, u64, vp]
        L.synth_f32_to_bf16.argtypes = [vp, u64, vp]
        for fn in ("synth_philox4x32_10", "synth_normal_f32", "synth_normal_bf16",
                   "synth_uniform_f32", "synth_bf16_to_f32", "synth_f32_to_bf16"):
            getattr(L, fn).restype = None
        _lib = L
    return _lib


def seed_of(*parts) -> int:
    """64-bit stream seed from a tuple of names/ints (BLAKE2b, 8-byte digest)."""
    s = "/".join(str(p) for p in parts).encode()
    return int.from_bytes(hashlib.blake2b(s, digest_size=8).digest(), "little")


def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, dtype=np.uint32)
    lib().synth_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def normal_f32(seed: int, shape, std: float = 1.0, mean: float = 0.0, offset: int = 0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    lib().synth_normal_f32(seed, offset, out.size, mean, std, out.ctypes.data)
    return out


def normal_bf16(seed: int, shape, std: float = 1.0, mean: float = 0.0, offset: int = 0) -> np.ndarray:
    """bf16 bit patterns (uint16) of round_to_nearest_even(mean + std * z)."""
    out = np.empty(shape, dtype=np.uint16)
    lib().synth_normal_bf16(seed, offset, out.size, mean, std, out.ctypes.data)
    return out


def uniform_f32(seed: int, shape, lo: float, hi: float, offset: int = 0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    lib().synth_uniform_f32(seed, offset, out.size, lo, hi, out.ctypes.data)
    return out


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.uint16)
    out = np.empty(a.shape, dtype=np.float32)
    lib().synth_bf16_to_f32(a.ctypes.data, a.size, out.ctypes.data)
    return out


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.uint16)
    lib().synth_f32_to_bf16(a.ctypes.data, a.size, out.ctypes.data)
    return out


def _draw(seed, shape, std, dtype, mean=0.0):
    if dtype == "bf16":
        return normal_bf16(seed, shape, std, mean)
    return normal_f32(seed, shape, std, mean)


def _gain(seed, n, dtype, perturbed):
    if not perturbed:
        g = np.ones(n, dtype=np.float32)
    else:
        g = uniform_f32(seed, (n,), 0.5, 1.5)
    return f32_to_bf16(g) if dtype == "bf16" else g


def _shift(seed, n, dtype, perturbed):
    if not perturbed:
        b = np.zeros(n, dtype=np.float32)
        return f32_to_bf16(b) if dtype == "bf16" else b
    return _draw(seed, (n,), 0.1, dtype)


def llm_block_weights(wl: "Workload", layer: int, perturbed: bool = False) -> dict:
    """Weights of decoder block ``layer`` (nn.Linear convention W[out][in]).

    Projection matrices ~ N(0, 0.02).  RMSNorm gains are 1, or U(0.5, 1.5) when
    ``perturbed`` (so a dropped gain cannot pass parity).  bf16 workloads
    return uint16 bit patterns, fp32 ones float32 arrays.
    """
    s = wl.llm
    dt = wl.dtype
    tag = (wl.name, "llm", layer)
    d, dh, H, Hkv, F = s.d_model, s.head_dim, s.n_heads, s.n_kv_heads, s.d_ff
    return {
        "w_q": _draw(seed_of(*tag, "w_q"), (H * dh, d), 0.02, dt),
        "w_k": _draw(seed_of(*tag, "w_k"), (Hkv * dh, d), 0.02, dt),
        "w_v": _draw(seed_of(*tag, "w_v"), (Hkv * dh, d), 0.02, dt),
        "w_o": _draw(seed_of(*tag, "w_o"), (d, H * dh), 0.02, dt),
        "w_gate": _draw(seed_of(*tag, "w_gate"), (F, d), 0.02, dt),
        "w_up": _draw(seed_of(*tag, "w_up"), (F, d), 0.02, dt),
        "w_down": _draw(seed_of(*tag, "w_down"), (d, F), 0.02, dt),
        "norm1_g": _gain(seed_of(*tag, "norm1_g"), d, dt, perturbed),
        "norm2_g": _gain(seed_of(*tag, "norm2_g"), d, dt, perturbed),
    }


def vit_block_weights(wl: "Workload", layer: int, perturbed: bool = False) -> dict:
    """Weights of ViT block ``layer``: projections and biases ~ N(0, 0.02);
    LayerNorm gains 1 / shifts 0, or U(0.5,1.5) / N(0, 0.1) when ``perturbed``."""
    s = wl.enc
    dt = wl.dtype
    tag = (wl.name, "enc", layer)
    d, F = s.d_model, s.d_ff
    hd = s.n_heads * s.head_dim
    return {
        "w_q": _draw(seed_of(*tag, "w_q"), (hd, d), 0.02, dt),
        "w_k": _draw(seed_of(*tag, "w_k"), (hd, d), 0.02, dt),
        "w_v": _draw(seed_of(*tag, "w_v"), (hd, d), 0.02, dt),
        "b_qkv": _draw(seed_of(*tag, "b_qkv"), (3 * hd,), 0.02, dt),
        "w_o": _draw(seed_of(*tag, "w_o"), (d, hd), 0.02, dt),
        "b_o": _draw(seed_of(*tag, "b_o"), (d,), 0.02, dt),
        "w_fc1": _draw(seed_of(*tag, "w_fc1"), (F, d), 0.02, dt),
        "b_fc1": _draw(seed_of(*tag, "b_fc1"), (F,), 0.02, dt),
        "w_fc2": _draw(seed_of(*tag, "w_fc2"), (d, F), 0.02, dt),
        "b_fc2": _draw(seed_of(*tag, "b_fc2"), (d,), 0.02, dt),
        "norm1_g": _gain(seed_of(*tag, "norm1_g"), d, dt, perturbed),
        "norm1_b": _shift(seed_of(*tag, "norm1_b"), d, dt, perturbed),
        "norm2_g": _gain(seed_of(*tag, "norm2_g"), d, dt, perturbed),
        "norm2_b": _shift(seed_of(*tag, "norm2_b"), d, dt, perturbed),
    }


def tokens(wl: "Workload", frame: int = 0, B: int = None, L: int = None) -> np.ndarray:
    """LLM input embeddings [B, L, d] ~ N(0, 1) for ``frame``."""
    B = wl.batch if B is None else B
    L = wl.seq if L is None else L
    return _draw(seed_of(wl.name, "tokens", frame, B, L), (B, L, wl.llm.d_model), 1.0, wl.dtype)


def patches(wl: "Workload", frame: int = 0, n_img: int = None, L_img: int = None) -> np.ndarray:
    """Encoder input patch embeddings [n_img, L_img, d_enc] ~ N(0, 1) for ``frame``."""
    n_img = wl.n_img if n_img is None else n_img
    L_img = wl.img_tokens if L_img is None else L_img
    return _draw(seed_of(wl.name, "patches", frame, n_img, L_img), (n_img, L_img, wl.enc.d_model),
                 1.0, wl.dtype)


def vision_weights(wl: "Workload", perturbed: bool = False) -> dict:
    """Stem, final encoder norm and connector weights: projections, biases and
    the position embedding ~ N(0, 0.02); LayerNorm gain 1 / shift 0, or
    U(0.5, 1.5) / N(0, 0.1) when ``perturbed``."""
    v, e = wl.vision, wl.enc
    dt = wl.dtype
    tag = (wl.name, "vision")
    d, kin = e.d_model, v.channels * v.patch * v.patch
    return {
        "w_patch": _draw(seed_of(*tag, "w_patch"), (d, kin), 0.02, dt),
        "b_patch": _draw(seed_of(*tag, "b_patch"), (d,), 0.02, dt),
        "pos": _draw(seed_of(*tag, "pos"), (v.L_img, d), 0.02, dt),
        "post_g": _gain(seed_of(*tag, "post_g"), d, dt, perturbed),
        "post_b": _shift(seed_of(*tag, "post_b"), d, dt, perturbed),
        "w_c1": _draw(seed_of(*tag, "w_c1"), (v.d_hidden, v.merge * v.merge * d), 0.02, dt),
        "b_c1": _draw(seed_of(*tag, "b_c1"), (v.d_hidden,), 0.02, dt),
        "w_c2": _draw(seed_of(*tag, "w_c2"), (v.d_out, v.d_hidden), 0.02, dt),
        "b_c2": _draw(seed_of(*tag, "b_c2"), (v.d_out,), 0.02, dt),
    }


def images(wl: "Workload", frame: int = 0, n_img: int = None) -> np.ndarray:
    """Camera images [n_img, C, H, W] ~ N(0, 1) (pixels after the usual
    per-channel normalisation) for ``frame``."""
    v = wl.vision
    n_img = wl.n_img if n_img is None else n_img
    return _draw(seed_of(wl.name, "images", frame, n_img), (n_img, v.channels, v.img_h, v.img_w), 1.0, wl.dtype)


def text(wl: "Workload", frame: int = 0, T: int = None) -> np.ndarray:
    """Text token embeddings [T, d_out] ~ N(0, 1) that follow the visual tokens
    (d_out is the decoder's d_model)."""
    T = wl.text_tokens if T is None else T
    return _draw(seed_of(wl.name, "text", frame, T), (T, wl.vision.d_out), 1.0, wl.dtype)


def as_f32(a: np.ndarray) -> np.ndarray:
    """float32 view of a generated tensor (bf16 bits widened exactly)."""
    if a.dtype == np.uint16:
        return bf16_to_f32(a)
    return np.ascontiguousarray(a, dtype=np.float32)
