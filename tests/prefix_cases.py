"""Shared helpers for the GPU parity tests: run the HIP prefix / encoder
through the C ABI and the oracle on the same seeded inputs."""
import dataclasses
import time

import numpy as np

import oracle
import synth
from paper_2608_14586_amd import binding as vb


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def to_f32(t):
    """torch tensor (bf16 or f32, host) -> float32 numpy."""
    import torch
    return t.to(torch.float32).numpy()


def f32_weights(W):
    return {n: synth.as_f32(a) for n, a in W.items()}


def log(msg):
    print(msg, flush=True)


class LlmCase:
    """A decoder stack held on the GPU with k resident blocks."""

    def __init__(self, name, L, k, B=1, perturbed=False, shape=None, max_tokens=None):
        self.wl = synth.CONFIGS[name]
        self.s = shape or self.wl.llm
        self.L, self.k, self.B = L, k, B
        self.perturbed = perturbed
        self.W = [synth.llm_block_weights(self.wl, l, perturbed=perturbed) for l in range(k)] \
            if shape is None else None
        cfg = vb.stack_cfg(self.s, self.wl.dtype, max_tokens=max_tokens or L, max_batch=B, n_blocks=k)
        self.ctx = vb.Context(llm=cfg)
        for l in range(k):
            self.ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, self.W[l])

    def tokens(self, frame=0):
        return synth.tokens(self.wl, frame=frame, B=self.B, L=self.L)

    def boundary(self, n_layers=None, out_dtype=None, with_kv=True):
        s = self.s
        return vb.Boundary(self.B, self.L, s.d_model, self.k if n_layers is None else n_layers, s.n_kv_heads,
                           s.head_dim, stack_dtype=self.wl.dtype, out_dtype=out_dtype or self.wl.dtype,
                           with_kv=with_kv)

    def run(self, tok, frame=0, k0=0, k1=None, out_dtype=None, device_tokens=False):
        import torch
        k1 = self.k if k1 is None else k1
        bnd = self.boundary(n_layers=k1 - k0, out_dtype=out_dtype)
        src = tok
        if device_tokens:
            src = torch.from_numpy(tok.view(np.int16) if tok.dtype == np.uint16 else tok).cuda()
        in_dt = vb.VLA_BF16 if tok.dtype == np.uint16 else vb.VLA_F32
        self.ctx.vla_run_blocks(frame, src, in_dt, self.B, self.L, k0, k1, bnd)
        self.ctx.vla_wait_boundary(frame, 120000)
        return bnd

    def oracle(self, tok, k0=0, k1=None, keep_kv=True):
        k1 = self.k if k1 is None else k1
        t0 = time.time()
        h, kv = oracle.run_prefix(synth.as_f32(tok), lambda l: f32_weights(self.W[k0 + l]), self.s, k1 - k0,
                                  keep_kv=keep_kv)
        log("  oracle %s L=%d blocks [%d,%d): %.1fs" % (self.wl.name, self.L, k0, k1, time.time() - t0))
        return h, kv

    def close(self):
        self.ctx.vla_destroy()


class EncCase:
    def __init__(self, name, n_img, L, n_blocks=None, perturbed=False):
        self.wl = synth.CONFIGS[name]
        self.s = self.wl.enc if n_blocks is None else dataclasses.replace(self.wl.enc, n_blocks=n_blocks)
        self.n_img, self.L = n_img, L
        self.W = [synth.vit_block_weights(self.wl, l, perturbed=perturbed) for l in range(self.s.n_blocks)]
        cfg = vb.stack_cfg(self.s, self.wl.dtype, max_tokens=L, max_batch=n_img)
        self.ctx = vb.Context(enc=cfg)
        for l in range(self.s.n_blocks):
            self.ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, self.W[l])

    def patches(self, frame=0):
        return synth.patches(self.wl, frame=frame, n_img=self.n_img, L_img=self.L)

    def run(self, p, frame=0):
        import torch
        dt = torch.bfloat16 if self.wl.dtype == "bf16" else torch.float32
        out = torch.empty((self.n_img, self.L, self.s.d_model), dtype=dt, device="cuda")
        self.ctx.vla_run_encoder(frame, p, self.n_img, self.L, out)
        self.ctx.encoder_stream.synchronize()
        return out.cpu()

    def oracle(self, p):
        t0 = time.time()
        h = oracle.run_encoder(synth.as_f32(p), lambda l: f32_weights(self.W[l]), self.s)
        log("  oracle %s %dx%d, %d blocks: %.1fs" % (self.wl.name, self.n_img, self.L, self.s.n_blocks,
                                                     time.time() - t0))
        return h

    def close(self):
        self.ctx.vla_destroy()
