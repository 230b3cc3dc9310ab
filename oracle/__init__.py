"""CPU oracle for the GPU-resident prefix of block-layer partitioned VLA inference.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The product path (the HIP library and its Python binding) never
routes through it and shares no code with it.

It is a plain, slow, obviously-correct numpy implementation of what the prefix
computes: the boundary hidden state after the first p whole transformer blocks
(the paper's Eq. (5), Sec. IV-B), the prefix KV cache those blocks write, and
the visual-encoder blocks, and the encoder's stem and connector that turn
camera images into the backbone's input tokens.  Default precision is float32 (the precision the
prefix's parity bar is stated in); every function also runs in float64, which
the pins use.  Block internals follow the workload definitions (LLaMA-style
pre-RMSNorm decoder with RoPE and SwiGLU; pre-LayerNorm ViT with GELU), since
the paper fixes none of them; each function names the published definition it
writes out.

Parity pins: every function here is pinned by ``tests/test_oracle_*.py``
against brute force, closed forms, invariants and independent library
routines.  The whole-stack values are pinned only transitively (the paper
prints no activations).
"""
from .reference import (  # noqa: F401
    attention,
    gelu_erf,
    layer_norm,
    llm_block,
    rms_norm,
    rope_apply,
    rope_tables,
    round_bf16,
    run_encoder,
    run_prefix,
    silu,
    swiglu,
    vit_block,
    transfer_bytes,
)
from .vision import connector, merge_patches, patch_embed, run_vision  # noqa: F401
