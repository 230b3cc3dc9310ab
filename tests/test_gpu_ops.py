"""Per-kernel parity of the HIP operators against the oracle's definitions,
called through the C ABI (include/vla_ops.h), on ragged shapes."""
import math

import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu


def _dev_bf16(a_u16):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a_u16).view(np.int16)).cuda()


@pytest.mark.parametrize("M,N,K", [(128, 128, 64), (200, 320, 128), (77, 96, 256), (1024, 1152, 896),
                                   (33, 4096, 4096), (2048, 16384, 128), (2000, 16400, 192),
                                   (6104, 1000, 192), (1, 1, 64), (1, 8, 128), (3, 200, 64)])
def test_gemm_bf16(M, N, K):
    import torch
    from paper_2608_14586_amd import binding as vb
    A = synth.normal_bf16(synth.seed_of("gemmA", M, N, K), (M, K))
    W = synth.normal_bf16(synth.seed_of("gemmW", M, N, K), (N, K))
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    vb.vla_op_gemm_bf16(_dev_bf16(A), _dev_bf16(W), C, M, N, K)
    torch.cuda.synchronize()
    ref = synth.as_f32(A).astype(np.float64) @ synth.as_f32(W).astype(np.float64).T
    err = np.abs(C.cpu().numpy() - ref).max() / np.abs(ref).max()
    assert err < 1e-5, err


def _packed(W, N, K):
    from paper_2608_14586_amd import binding as vb
    return _dev_bf16(vb.vla_op_pack_weight_bf16(W, N, K))


# Tile choices these shapes reach: 128x128 over three quarters of a round
# (ViT proj / fc2, also over ragged rows), one round of 128x128 (decoder
# O-projection / down at L=2048), 64x128 (half a round of 128x128), 128x128
# over ragged rows and columns, single rows.
@pytest.mark.parametrize("M,N,K,bias", [(6144, 1024, 128, True), (6100, 1024, 64, True), (2048, 4096, 192, False),
                                        (1024, 4096, 128, False), (6104, 1000, 192, True), (77, 96, 64, True),
                                        (1, 4, 64, True), (130, 8, 128, False)])
def test_gemm_residual_bf16(M, N, K, bias):
    """H += A W^T + b through the fused residual epilogue (each lane's
    residual read behind the last K slab, bias and residual added in the
    accumulators): element-wise against float64, to the fp32 accumulation
    error."""
    import torch
    from paper_2608_14586_amd import binding as vb
    A = synth.normal_bf16(synth.seed_of("resA", M, N, K), (M, K))
    W = synth.normal_bf16(synth.seed_of("resW", M, N, K), (N, K))
    H0 = synth.normal_f32(synth.seed_of("resH", M, N, K), (M, N))
    b = synth.normal_f32(synth.seed_of("resb", M, N, K), (N,)) if bias else None
    H = torch.from_numpy(H0.copy()).cuda()
    vb.vla_op_gemm_residual_bf16(_dev_bf16(A), _packed(W, N, K), H, None if b is None else torch.from_numpy(b).cuda(),
                                 M, N, K)
    torch.cuda.synchronize()
    prod = synth.as_f32(A).astype(np.float64) @ synth.as_f32(W).astype(np.float64).T
    ref = H0.astype(np.float64) + prod + (0.0 if b is None else b.astype(np.float64))
    got = H.cpu().numpy().astype(np.float64)
    # fp32 accumulation of K <= 192 exact bf16 products (at most K roundings,
    # K 2^-24 <= 2^-16 of the sum of |products|) and three fp32 additions; a
    # lost or doubled bias or residual is off by O(1)
    mag = np.abs(synth.as_f32(A)).astype(np.float64) @ np.abs(synth.as_f32(W)).astype(np.float64).T
    bound = 2.0 ** -16 * mag + 2.0 ** -22 * np.abs(ref) + 1e-30
    err = np.abs(got - ref)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    assert (err <= bound).all(), (worst, err[worst], bound[worst])


# 192x256 tiles with 8 waves in whole rounds (ViT fc1), the same over ragged
# rows, 256x256 tiles (two rounds and more), 64x128 tiles, single rows.
@pytest.mark.parametrize("M,N,K,bias,gelu", [(6144, 4096, 128, True, True), (6000, 4096, 64, True, True),
                                             (2048, 16384, 64, True, False), (300, 1000, 128, True, True),
                                             (77, 96, 64, False, False), (1, 8, 64, False, True)])
def test_gemm_bias_gelu_bf16(M, N, K, bias, gelu):
    """out = f(A W^T + b) in bf16 through the fused bias / GELU epilogues (the
    bias added before the park): element-wise against float64 with the exact
    GELU, to one bf16 rounding plus the fp32 accumulation and erfc errors."""
    import torch
    from paper_2608_14586_amd import binding as vb
    A = synth.normal_bf16(synth.seed_of("geluA", M, N, K), (M, K))
    W = synth.normal_bf16(synth.seed_of("geluW", M, N, K), (N, K), std=0.1)
    b = synth.normal_f32(synth.seed_of("gelub", M, N, K), (N,)) if bias else None
    out = torch.empty((M, N), dtype=torch.int16, device="cuda")
    vb.vla_op_gemm_bias_bf16(_dev_bf16(A), _packed(W, N, K), out, None if b is None else torch.from_numpy(b).cuda(),
                             M, N, K, gelu)
    torch.cuda.synchronize()
    z = synth.as_f32(A).astype(np.float64) @ synth.as_f32(W).astype(np.float64).T
    if b is not None:
        z = z + b.astype(np.float64)
    ref = oracle.gelu_erf(z) if gelu else z
    got = synth.as_f32(out.cpu().numpy().view(np.uint16)).astype(np.float64)
    mag = np.abs(synth.as_f32(A)).astype(np.float64) @ np.abs(synth.as_f32(W)).astype(np.float64).T + np.abs(z)
    # half a bf16 ulp of the result (2^-9, with a factor 2), the fp32
    # accumulation of K <= 128 products through GELU's slope (<= 1.13), and
    # the erfc approximation (|error| <= 1.5e-7 on Phi, times |z|)
    bound = 2.0 ** -8 * np.abs(ref) + 2.0 ** -16 * mag + (2e-7 * np.abs(z) if gelu else 0.0) + 1e-30
    err = np.abs(got - ref)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    assert (err <= bound).all(), (worst, got[worst], ref[worst], bound[worst])


def _sample_rows(M, tag, n=24):
    """Tile edges plus seeded random rows of an M-row product."""
    rng = np.random.default_rng(synth.seed_of("rows", M, *tag))
    fixed = [0, 1, 127, 128, 191, 192, 255, 256, M // 2, M - 2, M - 1]
    return np.unique(np.concatenate([[r for r in fixed if 0 <= r < M], rng.integers(0, M, n)]))


# The products at their full K, in the launch configuration of the bench
# frame: decoder down (K = 11008, 172 k-slabs) and O-projection (K = 4096) on
# one round of three-slot 128x128 tiles, ViT fc2 (K = 4096) with its bias;
# sampled rows against float64.
@pytest.mark.parametrize("M,N,K,bias", [(2048, 4096, 11008, False), (2048, 4096, 4096, False),
                                        (6144, 1024, 4096, True)])
def test_gemm_residual_bf16_full_k(M, N, K, bias):
    import torch
    from paper_2608_14586_amd import binding as vb
    tag = ("resfull", M, N, K)
    A = synth.normal_bf16(synth.seed_of("A", *tag), (M, K))
    W = synth.normal_bf16(synth.seed_of("W", *tag), (N, K), std=0.02)
    H0 = synth.normal_f32(synth.seed_of("H", *tag), (M, N))
    b = synth.normal_f32(synth.seed_of("b", *tag), (N,)) if bias else None
    H = torch.from_numpy(H0.copy()).cuda()
    vb.vla_op_gemm_residual_bf16(_dev_bf16(A), _packed(W, N, K), H, None if b is None else torch.from_numpy(b).cuda(),
                                 M, N, K)
    torch.cuda.synchronize()
    rows = _sample_rows(M, tag)
    a64 = synth.as_f32(A[rows]).astype(np.float64)
    w64 = synth.as_f32(W).astype(np.float64)
    prod = a64 @ w64.T
    ref = H0[rows].astype(np.float64) + prod + (0.0 if b is None else b.astype(np.float64))
    got = H.cpu().numpy()[rows].astype(np.float64)
    # fp32 accumulation over K / 16 MFMA steps, each rounding the running sum
    # once (K/16 2^-24 <= 2^-14 of the sum of |products|), with a factor 4; a
    # dropped, doubled or misplaced k-slab is off by about sqrt(64) products,
    # several times this bound
    mag = np.abs(a64) @ np.abs(w64).T
    bound = 2.0 ** -12 * mag + 2.0 ** -22 * np.abs(ref) + 1e-30
    err = np.abs(got - ref)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    assert (err <= bound).all(), (rows[worst[0]], worst[1], err[worst], bound[worst])
    e = np.linalg.norm(got - ref) / np.linalg.norm(ref - H0[rows])
    assert e < 1e-5, e


# ViT fc1 + GELU at its full K (192x256 three-slot tiles, two whole rounds)
# and the plain bias product over a two-round 256x256 grid; sampled rows.
@pytest.mark.parametrize("M,N,K,gelu", [(6144, 4096, 1024, True), (2048, 16384, 4096, False)])
def test_gemm_bias_gelu_bf16_full_k(M, N, K, gelu):
    import torch
    from paper_2608_14586_amd import binding as vb
    tag = ("gelufull", M, N, K)
    A = synth.normal_bf16(synth.seed_of("A", *tag), (M, K))
    W = synth.normal_bf16(synth.seed_of("W", *tag), (N, K), std=0.05)
    b = synth.normal_f32(synth.seed_of("b", *tag), (N,))
    out = torch.empty((M, N), dtype=torch.int16, device="cuda")
    vb.vla_op_gemm_bias_bf16(_dev_bf16(A), _packed(W, N, K), out, torch.from_numpy(b).cuda(), M, N, K, gelu)
    torch.cuda.synchronize()
    rows = _sample_rows(M, tag)
    a64 = synth.as_f32(A[rows]).astype(np.float64)
    w64 = synth.as_f32(W).astype(np.float64)
    z = a64 @ w64.T + b.astype(np.float64)
    ref = oracle.gelu_erf(z) if gelu else z
    got = synth.as_f32(out.cpu().numpy()[rows].view(np.uint16)).astype(np.float64)
    mag = np.abs(a64) @ np.abs(w64).T + np.abs(z)
    # one bf16 rounding (2^-9, with a factor 2), the fp32 accumulation over
    # K / 16 MFMA steps (2^-14 of mag, with a factor 4) through GELU's slope,
    # and the erfc approximation
    bound = 2.0 ** -8 * np.abs(ref) + 2.0 ** -12 * mag + (2e-7 * np.abs(z) if gelu else 0.0) + 1e-30
    err = np.abs(got - ref)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    assert (err <= bound).all(), (rows[worst[0]], worst[1], got[worst], ref[worst], bound[worst])
    # over all sampled elements: the bf16 rounding alone (about 2^-9 / sqrt 3 rms)
    e = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert e < 3e-3, e


@pytest.mark.parametrize("B,H,Hkv,L,dh,causal", [
    (1, 4, 4, 128, 128, True), (1, 4, 4, 200, 128, True), (2, 6, 2, 77, 64, True), (1, 14, 2, 300, 64, True),
    (3, 4, 4, 130, 64, False), (1, 2, 2, 1024, 64, False), (1, 2, 1, 513, 128, False),
    # degenerate lengths: one token, less than one 16-key group, exactly one key tile
    (1, 2, 2, 1, 64, True), (1, 2, 1, 1, 128, False), (2, 4, 2, 15, 64, True), (1, 2, 2, 64, 128, True),
    # wide grids: the decoder's own shape (L=2048, 32 heads); ragged with GQA; an odd block count, B=2; a last
    # block one tile past its partner; one key tile and one token over 256 heads
    (1, 32, 32, 2048, 128, True), (1, 64, 8, 1000, 128, True), (2, 64, 16, 330, 128, True),
    (1, 256, 64, 138, 128, True), (1, 256, 256, 64, 128, True), (1, 256, 32, 1, 128, True)])
def test_attention_bf16(B, H, Hkv, L, dh, causal):
    import torch
    from paper_2608_14586_amd import binding as vb
    tag = (B, H, Hkv, L, dh, causal)
    q = synth.normal_bf16(synth.seed_of("q", *tag), (B, H, L, dh))
    k = synth.normal_bf16(synth.seed_of("k", *tag), (B, Hkv, L, dh))
    v = synth.normal_bf16(synth.seed_of("v", *tag), (B, Hkv, L, dh))
    ldvt = (L + 15) // 16 * 16 if L % 2 else (L + 63) // 64 * 64  # tight and padded strides
    vt = np.zeros((B, Hkv, dh, ldvt), np.uint16)
    # column c holds key c with bits 2 and 3 swapped (the layout the op documents)
    cols = np.arange(L)
    cols = (cols & ~12) | ((cols & 4) << 1) | ((cols & 8) >> 1)
    vt[..., cols] = v.transpose(0, 1, 3, 2)
    o = torch.empty((B, L, H * dh), dtype=torch.bfloat16, device="cuda")
    vb.vla_op_attention_bf16(_dev_bf16(q), _dev_bf16(k), _dev_bf16(vt), ldvt, o, B, H, Hkv, L, dh, causal)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()
    for b in range(B):
        q64, k64, v64 = (synth.as_f32(t[b]).transpose(1, 0, 2).astype(np.float64) for t in (q, k, v))
        ref = oracle.attention(q64, k64, v64, causal).reshape(L, H * dh)
        # element-wise: the kernel rounds each probability and each output to
        # bf16 once (relative error <= 2^-8 each), so |o - ref| <= 2^-8 |ref|
        # + 2^-8 sum_j p_j |v_j|, the second term being attention over |v|;
        # asserted with a factor-2 margin on every element, ragged rows and
        # heads included
        mag = oracle.attention(q64, k64, np.abs(v64), causal).reshape(L, H * dh)
        err = np.abs(got[b] - ref)
        bound = 2.0 ** -7 * (np.abs(ref) + mag) + 1e-6
        worst = np.unravel_index(np.argmax(err / bound), err.shape)
        assert (err <= bound).all(), (b, worst, err[worst], bound[worst])
        e = np.linalg.norm(got[b] - ref) / np.linalg.norm(ref)
        assert e < 1e-2, (b, e)


def test_attention_bf16_vit_shape():
    """The encoder's attention at the bench frame's shape (6 images x 16 heads
    x 1024 patches, head dim 64, bidirectional), in its launch configuration;
    sampled query rows of every image against the float64 oracle (a query's
    output depends on its own row only), element-wise."""
    import torch
    from paper_2608_14586_amd import binding as vb
    B, H, Hkv, L, dh = 6, 16, 16, 1024, 64
    tag = ("vitattn", B, H, L, dh)
    q = synth.normal_bf16(synth.seed_of("q", *tag), (B, H, L, dh))
    k = synth.normal_bf16(synth.seed_of("k", *tag), (B, Hkv, L, dh))
    v = synth.normal_bf16(synth.seed_of("v", *tag), (B, Hkv, L, dh))
    ldvt = L
    vt = np.zeros((B, Hkv, dh, ldvt), np.uint16)
    cols = np.arange(L)
    cols = (cols & ~12) | ((cols & 4) << 1) | ((cols & 8) >> 1)
    vt[..., cols] = v.transpose(0, 1, 3, 2)
    o = torch.empty((B, L, H * dh), dtype=torch.bfloat16, device="cuda")
    vb.vla_op_attention_bf16(_dev_bf16(q), _dev_bf16(k), _dev_bf16(vt), ldvt, o, B, H, Hkv, L, dh, False)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()
    for b in range(B):
        rows = _sample_rows(L, tag + (b,), n=40)
        q64, k64, v64 = (synth.as_f32(t[b]).transpose(1, 0, 2).astype(np.float64) for t in (q, k, v))
        ref = oracle.attention(q64[rows], k64, v64, False).reshape(len(rows), H * dh)
        mag = oracle.attention(q64[rows], k64, np.abs(v64), False).reshape(len(rows), H * dh)
        err = np.abs(got[b][rows] - ref)
        bound = 2.0 ** -7 * (np.abs(ref) + mag) + 1e-6
        worst = np.unravel_index(np.argmax(err / bound), err.shape)
        assert (err <= bound).all(), (b, rows[worst[0]], worst[1], err[worst], bound[worst])


@pytest.mark.parametrize("M,d,ln", [(5, 256, False), (300, 896, False), (64, 4096, False), (70, 1024, True),
                                    (9, 4096, True), (1, 4, False), (1, 4, True), (3, 36, True),
                                    # the bench frame's decoder RMSNorm and ViT LayerNorm
                                    (2048, 4096, False), (6144, 1024, True)])
def test_norms_bf16(M, d, ln):
    import torch
    from paper_2608_14586_amd import binding as vb
    x = synth.normal_f32(synth.seed_of("nx", M, d), (M, d), std=3.0, mean=0.5)
    g = synth.uniform_f32(synth.seed_of("ng", d), (d,), 0.5, 1.5)
    bta = synth.normal_f32(synth.seed_of("nb", d), (d,), std=0.1) if ln else None
    y = torch.empty((M, d), dtype=torch.bfloat16, device="cuda")
    tx, tg = torch.from_numpy(x).cuda(), torch.from_numpy(g).cuda()
    tb = torch.from_numpy(bta).cuda() if ln else None
    vb.vla_op_norm_bf16(tx, tg, tb, 1e-6, y, M, d)
    torch.cuda.synchronize()
    x64 = x.astype(np.float64)
    ref = oracle.layer_norm(x64, g, bta, 1e-6) if ln else oracle.rms_norm(x64, g, 1e-6)
    got = y.float().cpu().numpy()
    # bf16 output: within half an ulp of bf16 (relative 2^-9) plus fp32 noise
    assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-6)
