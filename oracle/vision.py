"""Front and back of the visual encoder E(x_t) (test infrastructure only).

The paper's frame x_t holds multi-camera images (Eq. (1)); the GPU stage runs
the visual encoder (Sec. IV-A) and the backbone consumes its output as tokens
(Eq. (5)).  The paper names no stem, final norm or connector, so these follow
the common ViT / LLaVA-style definitions, each named below:

  images -> patch embedding + position embedding -> encoder blocks
         -> final LayerNorm -> r x r merge of neighbouring patches
         -> Linear -> GELU -> Linear  = visual tokens, then the text tokens.

Shapes: images [n_img, C, H, W]; patch features [n_img, L_img, d_enc] with
L_img = (H / p) * (W / p) in row-major grid order; tokens [V + T, d_out].
"""
from __future__ import annotations

import numpy as np

from .reference import _cast_weights, _ident, gelu_erf, layer_norm, run_encoder


def patch_embed(images: np.ndarray, w_patch: np.ndarray, b_patch: np.ndarray, pos: np.ndarray,
                patch: int) -> np.ndarray:
    """ViT patch embedding (Dosovitskiy et al., 2020, Sec. 3.1, Eq. 1): each
    image is cut into non-overlapping patch x patch squares, taken row by row
    over the (H/p) x (W/p) grid; a square flattened channel first, then pixel
    row, then pixel column (the element order of a convolution kernel
    w[d][C][p][p]) is projected by w_patch[d][C*p*p] plus b_patch, and the
    learned position embedding pos[l] of its grid index l is added.  The same
    map as a stride-p convolution with kernel w_patch.reshape(d, C, p, p).
    Returns [n_img, L_img, d]."""
    n, C, H, W = images.shape
    gh, gw = H // patch, W // patch
    x = images.reshape(n, C, gh, patch, gw, patch)
    x = x.transpose(0, 2, 4, 1, 3, 5).reshape(n, gh * gw, C * patch * patch)
    return x @ w_patch.T + b_patch + pos


def merge_patches(x: np.ndarray, grid_h: int, grid_w: int, r: int) -> np.ndarray:
    """Space-to-depth merge of r x r neighbouring patches (the token
    reduction in front of the connector): output token (ty, tx), row-major
    over the (grid_h/r) x (grid_w/r) grid, is the concatenation of the
    features of patches (ty*r + dy, tx*r + dx), dy outer and dx inner, so
    feature (dy*r + dx)*d + c of the token is feature c of that patch.
    x[n, grid_h*grid_w, d] -> [n, (grid_h/r)*(grid_w/r), r*r*d]."""
    n, L, d = x.shape
    y = x.reshape(n, grid_h // r, r, grid_w // r, r, d)
    y = y.transpose(0, 1, 3, 2, 4, 5)
    return y.reshape(n, (grid_h // r) * (grid_w // r), r * r * d)


def connector(feat: np.ndarray, V: dict, vis, act_round=None) -> np.ndarray:
    """Encoder output feat[n, L_img, d_enc] -> visual tokens [n*L_img/r^2, d_out]:
    the encoder's final LayerNorm (post_g, post_b), the r x r merge, then the
    two-layer GELU MLP projector of LLaVA-1.5 (Liu et al., 2023):
    t = GELU(m W1^T + b1) W2^T + b2.  Cameras follow each other in order."""
    rnd = act_round or _ident
    gh, gw = vis.img_h // vis.patch, vis.img_w // vis.patch
    x = rnd(layer_norm(feat, V["post_g"], V["post_b"], vis.norm_eps))
    m = merge_patches(x, gh, gw, vis.merge)
    a = rnd(gelu_erf(m @ V["w_c1"].T + V["b_c1"]))
    t = a @ V["w_c2"].T + V["b_c2"]
    return t.reshape(-1, vis.d_out)


def run_vision(images: np.ndarray, enc_weights_of, V: dict, enc_shape, vis, text: np.ndarray,
               dtype=np.float32, act_round=None, n_blocks: int = None) -> np.ndarray:
    """E(x_t) of one frame as the backbone's input sequence: the stem, the
    encoder blocks (each camera attends within itself), the connector; the
    visual tokens of camera 0, 1, ... followed by the text embeddings
    text[T, d_out].  Returns [1, V + T, d_out]."""
    V = _cast_weights(V, dtype)
    x = patch_embed(np.asarray(images, dtype=dtype), V["w_patch"], V["b_patch"], V["pos"], vis.patch)
    feat = run_encoder(x, enc_weights_of, enc_shape, n_blocks=n_blocks, dtype=dtype, act_round=act_round)
    vis_tok = connector(feat, V, vis, act_round=act_round)
    seq = np.concatenate([vis_tok, np.asarray(text, dtype=dtype)], axis=0)
    return seq[None]
