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
            encoder run first for every frame.  With images: six 448 x 448
            cameras, 14 x 14 patches, 2 x 2 merged into 1536 visual tokens,
            followed by 512 text tokens.
dual05b   : two 24-block 0.5B-class stacks (the small_llm block shape) over
            the same 1536 visual + 512 text tokens, vit_l encoder, k in
            {0, 12, 24} per stack.
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
class VisionShape:
    """Front and back of the visual encoder: images [n_img][channels][img_h][img_w]
    cut into patch x patch patches; the connector merges merge x merge
    neighbouring patches and maps them through a d_hidden-wide MLP to d_out
    (the LLM's d_model)."""
    channels: int
    img_h: int
    img_w: int
    patch: int
    merge: int
    d_hidden: int
    d_out: int
    norm_eps: float = 1e-6

    @property
    def grid(self):
        return self.img_h // self.patch, self.img_w // self.patch

    @property
    def L_img(self):
        gh, gw = self.grid
        return gh * gw

    @property
    def tokens_per_image(self):
        gh, gw = self.grid
        return (gh // self.merge) * (gw // self.merge)


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
    vision: Optional[VisionShape] = None
    text_tokens: int = 0
    branches: int = 1                # decoder stacks sharing one input sequence


def llama_like(n_blocks, d, H, Hkv, dh, F):
    return StackShape(n_blocks, d, H, Hkv, dh, F, norm_is_layernorm=False, mlp_is_gelu=False,
                      causal=True, use_rope=True, has_bias=False)


def vit_like(n_blocks, d, H, dh, F):
    return StackShape(n_blocks, d, H, H, dh, F, norm_is_layernorm=True, mlp_is_gelu=True,
                      causal=False, use_rope=False, has_bias=True)


VIT_L = vit_like(24, 1024, 16, 64, 4096)
LLM_7B = llama_like(32, 4096, 32, 32, 128, 11008)
LLM_05B = llama_like(24, 896, 14, 2, 64, 4864)
# 448 x 448 cameras in 14 x 14 patches: 32 x 32 = 1024 patch tokens per image;
# 2 x 2 merging leaves 256 visual tokens per camera, 1536 for six
VISION_7B = VisionShape(3, 448, 448, 14, 2, 4096, 4096)
VISION_05B = VisionShape(3, 448, 448, 14, 2, 896, 896)

CONFIGS = {
    "tiny": Workload("tiny", "f32", llama_like(2, 256, 4, 4, 64, 688), None, batch=1, seq=128, k=2),
    "small_llm": Workload("small_llm", "bf16", llama_like(24, 896, 14, 2, 64, 4864), None,
                          batch=1, seq=4096, k=12),
    "vit_l": Workload("vit_l", "bf16", None, VIT_L, n_img=6, img_tokens=1024),
    "llm7b": Workload("llm7b", "bf16", LLM_7B, None, batch=1, seq=1024, k=16),
    "sweep7b": Workload("sweep7b", "bf16", LLM_7B, VIT_L, batch=1, seq=2048, k=16,
                        ks=(8, 16, 24, 32), n_img=6, img_tokens=1024, vision=VISION_7B, text_tokens=512),
    # two 24-block 0.5B-class decoder stacks over one frame's tokens (a
    # dual-expert VLA); k = 0 keeps only the encoder on the GPU
    "dual05b": Workload("dual05b", "bf16", LLM_05B, VIT_L, batch=1, seq=2048, k=0, ks=(0, 12, 24),
                        n_img=6, img_tokens=1024, vision=VISION_05B, text_tokens=512, branches=2),
}
