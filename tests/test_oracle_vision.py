"""Pins of the oracle's stem, patch merge and connector (oracle/vision.py).

Each is checked against an independent library route (torch's strided
convolution, pixel_unshuffle, layer_norm / linear / gelu, all on the CPU in
float64) or brute force over coordinates, so a transposed flatten order, a
swapped merge order, a dropped bias or gain fails."""
import numpy as np
import pytest

import oracle
from synth.configs import VisionShape, vit_like


def _rng(seed):
    return np.random.default_rng(seed)


def _vision_weights(rng, d, vis, perturbed=True):
    kin = vis.channels * vis.patch * vis.patch
    r2 = vis.merge * vis.merge
    return {
        "w_patch": rng.normal(0, 0.1, (d, kin)), "b_patch": rng.normal(0, 0.1, d),
        "pos": rng.normal(0, 0.1, (vis.L_img, d)),
        "post_g": rng.uniform(0.5, 1.5, d) if perturbed else np.ones(d),
        "post_b": rng.normal(0, 0.1, d) if perturbed else np.zeros(d),
        "w_c1": rng.normal(0, 0.1, (vis.d_hidden, r2 * d)), "b_c1": rng.normal(0, 0.1, vis.d_hidden),
        "w_c2": rng.normal(0, 0.1, (vis.d_out, vis.d_hidden)), "b_c2": rng.normal(0, 0.1, vis.d_out),
    }


@pytest.mark.parametrize("C,H,W,p,d", [(3, 28, 42, 7, 16), (1, 16, 16, 4, 8), (3, 14, 28, 14, 12)])
def test_patch_embed_is_a_strided_convolution(C, H, W, p, d):
    import torch
    import torch.nn.functional as F
    rng = _rng(1)
    n = 2
    img = rng.normal(size=(n, C, H, W))
    w = rng.normal(size=(d, C * p * p))
    b = rng.normal(size=d)
    pos = rng.normal(size=((H // p) * (W // p), d))
    got = oracle.patch_embed(img, w, b, pos, p)
    conv = F.conv2d(torch.from_numpy(img), torch.from_numpy(w.reshape(d, C, p, p)), torch.from_numpy(b), stride=p)
    want = conv.flatten(2).transpose(1, 2).numpy() + pos
    assert got.shape == (n, (H // p) * (W // p), d)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_patch_embed_one_patch_by_loops():
    rng = _rng(2)
    C, H, W, p, d = 2, 9, 12, 3, 4
    img = rng.normal(size=(1, C, H, W))
    w = rng.normal(size=(d, C * p * p))
    b = rng.normal(size=d)
    pos = rng.normal(size=((H // p) * (W // p), d))
    got = oracle.patch_embed(img, w, b, pos, p)
    gw = W // p
    for gy, gx in [(0, 0), (2, 3), (1, 2)]:
        l = gy * gw + gx
        for o in range(d):
            s = b[o] + pos[l, o]
            for c in range(C):
                for y in range(p):
                    for x in range(p):
                        s += w[o, (c * p + y) * p + x] * img[0, c, gy * p + y, gx * p + x]
            assert abs(got[0, l, o] - s) < 1e-12


@pytest.mark.parametrize("gh,gw,r", [(4, 6, 2), (6, 6, 3), (3, 5, 1), (2, 2, 2)])
def test_merge_matches_pixel_unshuffle(gh, gw, r):
    import torch
    import torch.nn.functional as F
    rng = _rng(3)
    n, d = 2, 5
    x = rng.normal(size=(n, gh * gw, d))
    got = oracle.merge_patches(x, gh, gw, r)
    grid = torch.from_numpy(x.reshape(n, gh, gw, d)).permute(0, 3, 1, 2)       # [n, d, gh, gw]
    pu = F.pixel_unshuffle(grid, r).numpy()                                     # channel c*r*r + dy*r + dx
    for dy in range(r):
        for dx in range(r):
            for c in range(d):
                want = pu[:, c * r * r + dy * r + dx].reshape(n, -1)
                np.testing.assert_array_equal(got[:, :, (dy * r + dx) * d + c], want)


def test_merge_gathers_the_right_neighbours():
    gh, gw, r, d = 4, 6, 2, 3
    x = np.zeros((1, gh * gw, d))
    for gy in range(gh):
        for gx in range(gw):
            x[0, gy * gw + gx] = (gy, gx, 100 * gy + gx)
    m = oracle.merge_patches(x, gh, gw, r)
    assert m.shape == (1, (gh // r) * (gw // r), r * r * d)
    for ty in range(gh // r):
        for tx in range(gw // r):
            row = m[0, ty * (gw // r) + tx].reshape(r * r, d)
            assert [tuple(v[:2]) for v in row] == [(ty * r + dy, tx * r + dx) for dy in range(r) for dx in range(r)]
    # r = 1 is the identity
    np.testing.assert_array_equal(oracle.merge_patches(x, gh, gw, 1), x)


@pytest.mark.parametrize("r", [1, 2])
def test_connector_matches_torch_modules(r):
    import torch
    import torch.nn.functional as F
    rng = _rng(4)
    vis = VisionShape(3, 28, 56, 7, r, 24, 20)
    d, n = 16, 3
    V = _vision_weights(rng, d, vis)
    feat = rng.normal(size=(n, vis.L_img, d))
    got = oracle.connector(feat, V, vis)
    t = {k: torch.from_numpy(np.asarray(a)) for k, a in V.items()}
    gh, gw = vis.grid
    x = F.layer_norm(torch.from_numpy(feat), (d,), t["post_g"], t["post_b"], vis.norm_eps)
    x = F.pixel_unshuffle(x.reshape(n, gh, gw, d).permute(0, 3, 1, 2), r)      # [n, d*r*r, gh/r, gw/r]
    x = x.reshape(n, d, r * r, gh // r, gw // r).permute(0, 3, 4, 2, 1).reshape(n, -1, r * r * d)
    a = F.gelu(F.linear(x, t["w_c1"], t["b_c1"]))
    want = F.linear(a, t["w_c2"], t["b_c2"]).reshape(-1, vis.d_out).numpy()
    assert got.shape == (n * vis.tokens_per_image, vis.d_out)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-10)


def test_run_vision_layout_and_camera_independence():
    rng = _rng(5)
    vis = VisionShape(3, 28, 28, 7, 2, 24, 20)
    enc = vit_like(2, 16, 2, 8, 32)
    d = enc.d_model
    V = _vision_weights(rng, d, vis)
    EW = [{
        "w_q": rng.normal(0, 0.1, (16, d)), "w_k": rng.normal(0, 0.1, (16, d)), "w_v": rng.normal(0, 0.1, (16, d)),
        "b_qkv": rng.normal(0, 0.1, 48), "w_o": rng.normal(0, 0.1, (d, 16)), "b_o": rng.normal(0, 0.1, d),
        "w_fc1": rng.normal(0, 0.1, (32, d)), "b_fc1": rng.normal(0, 0.1, 32),
        "w_fc2": rng.normal(0, 0.1, (d, 32)), "b_fc2": rng.normal(0, 0.1, d),
        "norm1_g": np.ones(d), "norm1_b": np.zeros(d), "norm2_g": np.ones(d), "norm2_b": np.zeros(d)}
        for _ in range(2)]
    img = rng.normal(size=(3, 3, 28, 28))
    text = rng.normal(size=(5, vis.d_out))
    seq = oracle.run_vision(img, lambda l: EW[l], V, enc, vis, text, dtype=np.float64)
    nv = 3 * vis.tokens_per_image
    assert seq.shape == (1, nv + 5, vis.d_out)
    np.testing.assert_array_equal(seq[0, nv:], text)
    # the visual rows are the connector over the encoder over the stem
    x = oracle.patch_embed(img, V["w_patch"], V["b_patch"], V["pos"], vis.patch)
    feat = oracle.run_encoder(x, lambda l: EW[l], enc, dtype=np.float64)
    np.testing.assert_allclose(seq[0, :nv], oracle.connector(feat, V, vis), rtol=1e-12, atol=1e-12)
    # cameras are independent: changing camera 1 leaves cameras 0 and 2 exactly as they were
    img2 = img.copy()
    img2[1] += rng.normal(size=img2[1].shape)
    seq2 = oracle.run_vision(img2, lambda l: EW[l], V, enc, vis, text, dtype=np.float64)
    tpi = vis.tokens_per_image
    np.testing.assert_array_equal(seq2[0, :tpi], seq[0, :tpi])
    np.testing.assert_array_equal(seq2[0, 2 * tpi:], seq[0, 2 * tpi:])
    assert not np.allclose(seq2[0, tpi:2 * tpi], seq[0, tpi:2 * tpi])
