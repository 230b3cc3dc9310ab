"""Shapes of the five synthetic workloads (no arithmetic here).

tiny      : 2-block causal decoder, d=256, 4 heads x 64, SwiGLU 688, fp32,
            batch 1, seq 128, boundary k=2 (the whole stack).
small_llm : 24 decoder blocks, d=896, 14 query heads x 64, 2 KV heads (GQA),
            SwiGLU 4864, causal prefill batch 1 seq 4096, bf16, k=12.
vit_l     : 24 bidirectional pre-LayerNorm blocks, d=1024, 16 heads x 64,
            GELU 4096, 6 camera images x 1024 patch tokens, bf16.
llm7b     : 32 decoder blocks, d=4096, 32 heads x 128 (MHA), SwiGLU 11008,
            batch 1 seq 1024 (768 visual + 256 text positions), bf16, k=16.
sweep7b   : the llm7b stack at seq 2048 with k in {8, 16, 24, 32}, the vit_l
            encoder run first for every frame.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class StackShape:
    n_blocks: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    norm_is_layernorm: bool
    mlp_is_gelu: bool
    causal: bool
    use_rope: bool
    has_bias: bool
    norm_eps: float = 1e-6
    rope_base: float = 10000.0


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                       # "bf16" or "f32"
    llm: Optional[StackShape]
    enc: Optional[StackShape]
    batch: int = 1
    seq: int = 0
    k: int = 0
    ks: Tuple[int, ...] = field(default_factory=tuple)
    n_img: int = 0
    img_tokens: int = 0


def llama_like(n_blocks, d, H, Hkv, dh, F):
    return StackShape(n_blocks, d, H, Hkv, dh, F, norm_is_layernorm=False, mlp_is_gelu=False,
                      causal=True, use_rope=True, has_bias=False)


def vit_like(n_blocks, d, H, dh, F):
    return StackShape(n_blocks, d, H, H, dh, F, norm_is_layernorm=True, mlp_is_gelu=True,
                      causal=False, use_rope=False, has_bias=True)


VIT_L = vit_like(24, 1024, 16, 64, 4096)
LLM_7B = llama_like(32, 4096, 32, 32, 128, 11008)

CONFIGS = {
    "tiny": Workload("tiny", "f32", llama_like(2, 256, 4, 4, 64, 688), None, batch=1, seq=128, k=2),
    "small_llm": Workload("small_llm", "bf16", llama_like(24, 896, 14, 2, 64, 4864), None,
                          batch=1, seq=4096, k=12),
    "vit_l": Workload("vit_l", "bf16", None, VIT_L, n_img=6, img_tokens=1024),
    "llm7b": Workload("llm7b", "bf16", LLM_7B, None, batch=1, seq=1024, k=16),
    "sweep7b": Workload("sweep7b", "bf16", LLM_7B, VIT_L, batch=1, seq=2048, k=16,
                        ks=(8, 16, 24, 32), n_img=6, img_tokens=1024),
}
