"""ctypes binding of the C ABI in include/vla_prefix.h, include/vla_ops.h and
include/vla_suffix.h.

Argument marshalling only: every step of the prefix runs in the HIP library.
PyTorch supplies the device arena, the streams and the pinned host
buffers (``torch.empty(..., pin_memory=True)``).  Functions keep the C names.
If the library has not been built this module raises at first use; there is
no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int, c_size_t, c_uint64, c_void_p

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvlaprefix.so")

VLA_OK = 0
STATUS = {0: "VLA_OK", -1: "VLA_ERR_INVALID_ARG", -2: "VLA_ERR_SHAPE", -3: "VLA_ERR_NOT_LOADED",
          -4: "VLA_ERR_NOT_PINNED", -5: "VLA_ERR_OOM", -6: "VLA_ERR_TIMEOUT", -7: "VLA_ERR_HIP",
          -8: "VLA_ERR_UNSUPPORTED", -9: "VLA_ERR_UNKNOWN_FRAME"}
VLA_BF16, VLA_F32 = 0, 1
VLA_STACK_LLM, VLA_STACK_ENC = 0, 1
VLA_PREC_BF16, VLA_PREC_SPLIT = 0, 1
KERNEL_CLASSES = ["norm", "qkv", "attn", "oproj", "mlp_up", "mlp_down", "other", "stem", "connector"]


class VlaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s: %s" % (STATUS.get(code, code), msg))
        self.code = code
        self.name = STATUS.get(code, str(code))


class vla_stack_cfg(ctypes.Structure):
    _fields_ = [("n_blocks", c_int), ("d_model", c_int), ("n_heads", c_int), ("n_kv_heads", c_int),
                ("head_dim", c_int), ("d_ff", c_int), ("max_tokens", c_int), ("max_batch", c_int),
                ("norm_is_layernorm", c_int), ("mlp_is_gelu", c_int), ("causal", c_int), ("use_rope", c_int),
                ("has_bias", c_int), ("norm_eps", c_float), ("rope_base", c_float), ("dtype", c_int)]


_WEIGHT_FIELDS = ["w_q", "w_k", "w_v", "w_o", "b_qkv", "b_o", "w_gate", "w_up", "w_down", "w_fc1", "b_fc1",
                  "w_fc2", "b_fc2", "norm1_g", "norm1_b", "norm2_g", "norm2_b"]


class vla_block_weights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in _WEIGHT_FIELDS]


class vla_boundary(ctypes.Structure):
    _fields_ = [("hidden", c_void_p), ("hidden_bytes", c_size_t), ("kv", c_void_p), ("kv_bytes", c_size_t),
                ("out_dtype", c_int), ("frame_id", c_uint64)]


class vla_vision_cfg(ctypes.Structure):
    _fields_ = [("channels", c_int), ("img_h", c_int), ("img_w", c_int), ("patch", c_int), ("merge", c_int),
                ("d_hidden", c_int), ("d_out", c_int), ("norm_eps", c_float)]


_VISION_FIELDS = ["w_patch", "b_patch", "pos", "post_g", "post_b", "w_c1", "b_c1", "w_c2", "b_c2"]


class vla_vision_weights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in _VISION_FIELDS]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("HIP library %s is missing: build it with __graft_entry__.build() "
                               "(there is no CPU fallback)" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P = POINTER
        sig = {
            "vla_query_sizes": [P(vla_stack_cfg), P(vla_stack_cfg), c_int, c_int, c_int, P(c_size_t), P(c_size_t),
                                P(c_size_t)],
            "vla_create": [P(vla_stack_cfg), P(vla_stack_cfg), c_int, c_void_p, c_size_t, c_void_p, c_void_p,
                           c_void_p, P(c_void_p)],
            "vla_load_block_weights": [c_void_p, c_int, c_int, P(vla_block_weights)],
            "vla_run_encoder": [c_void_p, c_uint64, c_void_p, c_int, c_int, c_void_p],
            "vla_run_prefix": [c_void_p, c_uint64, c_void_p, c_int, c_int, c_int, P(vla_boundary)],
            "vla_run_blocks": [c_void_p, c_uint64, c_void_p, c_int, c_int, c_int, c_int, c_int, P(vla_boundary)],
            "vla_decode_step": [c_void_p, c_uint64, c_void_p, c_int, c_int, c_int, c_void_p, c_int, P(vla_boundary)],
            "vla_decode_step_static": [c_void_p, c_uint64, c_void_p, c_int, c_int, c_int, c_void_p, c_int,
                                       P(vla_boundary)],
            "vla_query_vision_sizes": [P(vla_stack_cfg), P(vla_vision_cfg), P(c_size_t)],
            "vla_attach_vision": [c_void_p, P(vla_vision_cfg), c_void_p, c_size_t],
            "vla_load_vision_weights": [c_void_p, P(vla_vision_weights)],
            "vla_run_vision": [c_void_p, c_uint64, c_void_p, c_int, c_void_p, c_int, c_void_p, c_size_t],
            "vla_profile": [c_void_p, c_int],
            "vla_profile_read": [c_void_p, c_int, c_int, P(ctypes.c_double), P(c_int)],
            "vla_wait_boundary": [c_void_p, c_uint64, c_int],
            "vla_frame_times": [c_void_p, c_uint64, P(c_float), P(c_float), P(c_float)],
            "vla_arena_used": [c_void_p, P(c_size_t)],
            "vla_set_precision": [c_void_p, c_int, c_int],
            "vla_inject_fault": [c_void_p, ctypes.c_long],
            "vla_op_gemm_bf16": [c_void_p, c_void_p, c_void_p, c_int, c_int, c_int, c_void_p],
            "vla_op_attention_bf16": [c_void_p, c_void_p, c_void_p, c_int, c_void_p, c_int, c_int, c_int, c_int,
                                      c_int, c_int, c_void_p],
            "vla_op_norm_bf16": [c_void_p, c_void_p, c_void_p, c_float, c_void_p, c_int, c_int, c_void_p],
            "vla_op_pack_weight_bf16": [c_void_p, c_void_p, c_int, c_int],
            "vla_op_gemm_residual_bf16": [c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_int, c_int, c_void_p],
            "vla_op_gemm_bias_bf16": [c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_int, c_int, c_int, c_void_p],
            "vla_suffix_create": [P(vla_stack_cfg), c_int, c_int, c_int, P(c_void_p)],
            "vla_suffix_load_block_weights": [c_void_p, c_int, P(vla_block_weights)],
            "vla_suffix_run": [c_void_p, c_void_p, c_int, c_int, c_int, c_void_p],
            "vla_suffix_run_from": [c_void_p, c_int, c_void_p, c_int, c_int, c_int, c_void_p],
            "vla_suffix_threads": [c_void_p, P(c_int)],
            "vla_suffix_set_cache": [c_void_p, c_int, c_int],
            "vla_suffix_decode_step": [c_void_p, c_int, c_void_p, c_int, c_int, c_int, c_void_p],
            "vla_pipeline_create": [c_void_p, c_void_p, c_int, P(c_void_p)],
            "vla_pipeline_push": [c_void_p, c_uint64, P(vla_boundary), c_int, c_int, c_int, c_void_p],
            "vla_pipeline_pop": [c_void_p, P(c_uint64), P(c_float), P(c_float), c_int],
            "vla_pipeline_backlog": [c_void_p, P(c_int)],
            "vla_sched_create": [c_int, c_int, c_int, c_int, c_float, c_float, c_float, c_float, c_int, P(c_void_p)],
            "vla_sched_observe": [c_void_p, c_int, c_float, c_float, c_float],
            "vla_sched_predict": [c_void_p, c_int, c_float, c_float, P(c_float), P(c_float), P(c_float)],
            "vla_sched_decide": [c_void_p, c_float, c_float, c_int, c_float, P(c_int)],
            "vla_sched_model": [c_void_p, P(c_float), P(c_float), P(c_float), P(c_float)],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = c_int
        L.vla_op_packed_weight_elems.argtypes = [c_int, c_int]
        L.vla_op_packed_weight_elems.restype = c_size_t
        L.vla_status_string.argtypes = [c_int]
        L.vla_status_string.restype = c_char_p
        L.vla_last_error.argtypes = [c_void_p]
        L.vla_last_error.restype = c_char_p
        L.vla_destroy.argtypes = [c_void_p]
        L.vla_destroy.restype = None
        for name in ("vla_suffix_destroy", "vla_pipeline_destroy", "vla_sched_destroy"):
            getattr(L, name).argtypes = [c_void_p]
            getattr(L, name).restype = None
        _lib = L
    return _lib


def _check(code: int, ctx=None):
    if code != VLA_OK:
        msg = lib().vla_last_error(ctx)
        raise VlaError(code, msg.decode() if msg else "")


def stack_cfg(shape, dtype: str, max_tokens: int, max_batch: int = 1, n_blocks: int = None) -> vla_stack_cfg:
    """Build a vla_stack_cfg from any object with the StackShape attributes."""
    return vla_stack_cfg(
        n_blocks=shape.n_blocks if n_blocks is None else n_blocks, d_model=shape.d_model, n_heads=shape.n_heads,
        n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, d_ff=shape.d_ff, max_tokens=max_tokens,
        max_batch=max_batch, norm_is_layernorm=int(shape.norm_is_layernorm), mlp_is_gelu=int(shape.mlp_is_gelu),
        causal=int(shape.causal), use_rope=int(shape.use_rope), has_bias=int(shape.has_bias),
        norm_eps=shape.norm_eps, rope_base=shape.rope_base, dtype=VLA_BF16 if dtype == "bf16" else VLA_F32)


def vision_cfg(vis) -> vla_vision_cfg:
    """A vla_vision_cfg from any object with the VisionShape attributes."""
    return vla_vision_cfg(channels=vis.channels, img_h=vis.img_h, img_w=vis.img_w, patch=vis.patch, merge=vis.merge,
                          d_hidden=vis.d_hidden, d_out=vis.d_out, norm_eps=vis.norm_eps)


def vla_query_vision_sizes(enc, vis) -> int:
    n = c_size_t()
    _check(lib().vla_query_vision_sizes(ctypes.byref(enc) if enc else None, ctypes.byref(vis) if vis else None,
                                        ctypes.byref(n)))
    return n.value


def vla_query_sizes(llm, enc, B: int, L: int, k: int):
    """(arena_bytes, hidden_bytes, kv_bytes) for these stacks (either may be None)."""
    a, h, kv = c_size_t(), c_size_t(), c_size_t()
    _check(lib().vla_query_sizes(ctypes.byref(llm) if llm else None, ctypes.byref(enc) if enc else None, B, L, k,
                                 ctypes.byref(a), ctypes.byref(h), ctypes.byref(kv)))
    return a.value, h.value, kv.value


def _ptr(x):
    """Address of a numpy array or torch tensor (or None)."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        assert x.flags["C_CONTIGUOUS"]
        return x.ctypes.data
    assert x.is_contiguous()
    return x.data_ptr()


class Boundary:
    """Pinned host buffers of one frame's handoff: hidden [B][L][d] and KV
    [k][2][B][H_kv][L][dh] (see vla_boundary)."""

    def __init__(self, B, L, d, n_layers, n_kv_heads, head_dim, stack_dtype="bf16", out_dtype="bf16",
                 with_kv=True):
        import torch
        tdt = {"bf16": torch.bfloat16, "f32": torch.float32}
        self.hidden = torch.empty((B, L, d), dtype=tdt[out_dtype], pin_memory=True)
        kv_shape = (n_layers, 2, B, n_kv_heads, L, head_dim)
        self.kv = torch.empty(kv_shape, dtype=tdt[stack_dtype], pin_memory=True) \
            if (with_kv and n_layers > 0) else None
        self.out_dtype = out_dtype
        self.c = vla_boundary(hidden=self.hidden.data_ptr(), hidden_bytes=self.hidden.numel() * self.hidden.element_size(),
                              kv=self.kv.data_ptr() if self.kv is not None else None,
                              kv_bytes=(self.kv.numel() * self.kv.element_size()) if self.kv is not None else 0,
                              out_dtype=VLA_BF16 if out_dtype == "bf16" else VLA_F32, frame_id=0)

    @property
    def frame_id(self):
        return self.c.frame_id


def _block_weights(weights: dict):
    """A vla_block_weights over contiguous copies of the arrays (kept alive by
    the returned list)."""
    w = vla_block_weights()
    keep = []
    for name, arr in weights.items():
        if arr is None:
            continue
        if name not in _WEIGHT_FIELDS:
            raise KeyError(name)
        arr = np.ascontiguousarray(arr)
        keep.append(arr)
        setattr(w, name, arr.ctypes.data)
    return w, keep


class Context:
    """One vla_ctx over a torch-allocated device arena and torch streams for
    the decoder blocks, the encoder blocks (the decoder's stream unless one
    is given) and the handoff copies."""

    def __init__(self, llm: vla_stack_cfg = None, enc: vla_stack_cfg = None, device: int = 0,
                 compute_stream=None, copy_stream=None, encoder_stream=None):
        import torch
        self.llm, self.enc = llm, enc
        self.device = device
        arena_bytes, _, _ = vla_query_sizes(llm, enc, 0, 0, 0)
        self.arena_bytes = arena_bytes
        with torch.cuda.device(device):
            self.arena = torch.empty(max(arena_bytes, 256), dtype=torch.uint8, device="cuda:%d" % device)
            self.compute_stream = compute_stream or torch.cuda.Stream(device=device)
            # no encoder stream given: the encoder shares the compute stream
            self.encoder_stream = encoder_stream or self.compute_stream
            self.copy_stream = copy_stream or torch.cuda.Stream(device=device)
        h = c_void_p()
        _check(lib().vla_create(ctypes.byref(llm) if llm else None, ctypes.byref(enc) if enc else None, device,
                                self.arena.data_ptr(), self.arena.numel(), self.compute_stream.cuda_stream,
                                self.encoder_stream.cuda_stream, self.copy_stream.cuda_stream, ctypes.byref(h)))
        self.h = h.value

    def vla_load_block_weights(self, which: int, block: int, weights: dict):
        w, keep = _block_weights(weights)
        _check(lib().vla_load_block_weights(self.h, which, block, ctypes.byref(w)), self.h)

    def vla_run_encoder(self, frame_id: int, patches, n_img: int, L_img: int, out_dev):
        _check(lib().vla_run_encoder(self.h, frame_id, _ptr(patches), n_img, L_img, _ptr(out_dev)), self.h)

    def vla_attach_vision(self, vis: vla_vision_cfg):
        """Allocate the vision block (torch device memory kept by this object)
        and attach it."""
        import torch
        n = vla_query_vision_sizes(self.enc, vis)
        with torch.cuda.device(self.device):
            mem = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda:%d" % self.device)
        _check(lib().vla_attach_vision(self.h, ctypes.byref(vis), mem.data_ptr(), mem.numel()), self.h)
        self.vision_mem = mem
        self.vis = vis

    def vla_load_vision_weights(self, weights: dict):
        w = vla_vision_weights()
        keep = []
        for name, arr in weights.items():
            if name not in _VISION_FIELDS:
                raise KeyError(name)
            arr = np.ascontiguousarray(arr)
            keep.append(arr)
            setattr(w, name, arr.ctypes.data)
        _check(lib().vla_load_vision_weights(self.h, ctypes.byref(w)), self.h)

    def vla_run_vision(self, frame_id: int, images, n_img: int, text, L_text: int, tokens_out):
        nbytes = tokens_out.numel() * tokens_out.element_size()
        _check(lib().vla_run_vision(self.h, frame_id, _ptr(images), n_img, _ptr(text), L_text, _ptr(tokens_out),
                                    nbytes), self.h)

    def vla_run_prefix(self, frame_id: int, tokens, B: int, L: int, k: int, out: Boundary):
        _check(lib().vla_run_prefix(self.h, frame_id, _ptr(tokens), B, L, k, ctypes.byref(out.c)), self.h)

    def vla_run_blocks(self, frame_id: int, tokens, in_dtype: int, B: int, L: int, k_begin: int, k_end: int,
                       out: Boundary):
        _check(lib().vla_run_blocks(self.h, frame_id, _ptr(tokens), in_dtype, B, L, k_begin, k_end,
                                    ctypes.byref(out.c)), self.h)

    def vla_decode_step(self, frame_id: int, x, B: int, pos: int, k: int, kv_cache, L_cap: int, out: Boundary):
        _check(lib().vla_decode_step(self.h, frame_id, _ptr(x), B, pos, k, _ptr(kv_cache), L_cap, ctypes.byref(out.c)),
               self.h)

    def vla_decode_step_static(self, frame_id: int, x, B: int, pos: int, k: int, kv_cache, L_cap: int,
                               out: Boundary):
        _check(lib().vla_decode_step_static(self.h, frame_id, _ptr(x), B, pos, k, _ptr(kv_cache), L_cap,
                                            ctypes.byref(out.c)), self.h)

    def vla_profile(self, enable: bool):
        _check(lib().vla_profile(self.h, int(enable)), self.h)

    def vla_profile_read(self, which: int, cls: int):
        ms, n = ctypes.c_double(), c_int()
        _check(lib().vla_profile_read(self.h, which, cls, ctypes.byref(ms), ctypes.byref(n)), self.h)
        return ms.value, n.value

    def vla_wait_boundary(self, frame_id: int, timeout_ms: int = -1):
        _check(lib().vla_wait_boundary(self.h, frame_id, timeout_ms), self.h)

    def vla_frame_times(self, frame_id: int):
        g, x, t = c_float(), c_float(), c_float()
        _check(lib().vla_frame_times(self.h, frame_id, ctypes.byref(g), ctypes.byref(x), ctypes.byref(t)), self.h)
        return g.value, x.value, t.value

    def vla_set_precision(self, which: int, prec: int):
        _check(lib().vla_set_precision(self.h, which, prec), self.h)

    def vla_inject_fault(self, launches: int):
        _check(lib().vla_inject_fault(self.h, launches), self.h)

    def vla_arena_used(self) -> int:
        n = c_size_t()
        _check(lib().vla_arena_used(self.h, ctypes.byref(n)))
        return n.value

    def vla_destroy(self):
        if getattr(self, "h", None):
            lib().vla_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.vla_destroy()
        except Exception:
            pass


# ----------------------------------------------------------- operator calls

def vla_op_gemm_bf16(A, W, C, M, N, K, stream=None):
    _check(lib().vla_op_gemm_bf16(_ptr(A), _ptr(W), _ptr(C), M, N, K, stream))


def vla_op_attention_bf16(q, k, vt, ldvt, o, B, H, Hkv, L, dh, causal, stream=None):
    _check(lib().vla_op_attention_bf16(_ptr(q), _ptr(k), _ptr(vt), ldvt, _ptr(o), B, H, Hkv, L, dh, int(causal),
                                       stream))


def vla_op_norm_bf16(x, g, b, eps, y, M, d, stream=None):
    _check(lib().vla_op_norm_bf16(_ptr(x), _ptr(g), _ptr(b), eps, _ptr(y), M, d, stream))


def vla_op_packed_weight_elems(N, K):
    return lib().vla_op_packed_weight_elems(N, K)


def vla_op_pack_weight_bf16(W, N, K):
    """Host row-major bf16 rows W[N][K] (uint16 array) -> the packed slab-major
    host array the fused-epilogue products take."""
    out = np.zeros(vla_op_packed_weight_elems(N, K), dtype=np.uint16)
    _check(lib().vla_op_pack_weight_bf16(_ptr(np.ascontiguousarray(W)), _ptr(out), N, K))
    return out


def vla_op_gemm_residual_bf16(A, Wp, H, bias, M, N, K, stream=None):
    _check(lib().vla_op_gemm_residual_bf16(_ptr(A), _ptr(Wp), _ptr(H), _ptr(bias), M, N, K, stream))


def vla_op_gemm_bias_bf16(A, Wp, out, bias, M, N, K, gelu, stream=None):
    _check(lib().vla_op_gemm_bias_bf16(_ptr(A), _ptr(Wp), _ptr(out), _ptr(bias), M, N, K, int(gelu), stream))


def vla_status_string(code: int) -> str:
    return lib().vla_status_string(code).decode()


# ----------------------------------------------------------- host suffix

class Suffix:
    """One vla_suffix: decoder blocks [k_begin, k_end) on the host CPU."""

    def __init__(self, llm: vla_stack_cfg, k_begin: int, k_end: int, n_threads: int = 0):
        h = c_void_p()
        _check(lib().vla_suffix_create(ctypes.byref(llm), k_begin, k_end, n_threads, ctypes.byref(h)))
        self.h = h.value
        self.d = llm.d_model

    def vla_suffix_load_block_weights(self, block: int, weights: dict):
        w, keep = _block_weights(weights)
        _check(lib().vla_suffix_load_block_weights(self.h, block, ctypes.byref(w)))

    def vla_suffix_run(self, h, in_dtype: int, B: int, L: int, out):
        _check(lib().vla_suffix_run(self.h, _ptr(h), in_dtype, B, L, _ptr(out)))

    def vla_suffix_run_from(self, k: int, h, in_dtype: int, B: int, L: int, out):
        _check(lib().vla_suffix_run_from(self.h, k, _ptr(h), in_dtype, B, L, _ptr(out)))

    def vla_suffix_set_cache(self, B: int, L_cap: int):
        _check(lib().vla_suffix_set_cache(self.h, B, L_cap))

    def vla_suffix_decode_step(self, k: int, h, in_dtype: int, B: int, pos: int, out):
        _check(lib().vla_suffix_decode_step(self.h, k, _ptr(h), in_dtype, B, pos, _ptr(out)))

    def vla_suffix_threads(self) -> int:
        n = c_int()
        _check(lib().vla_suffix_threads(self.h, ctypes.byref(n)))
        return n.value

    def vla_suffix_destroy(self):
        if getattr(self, "h", None):
            lib().vla_suffix_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.vla_suffix_destroy()
        except Exception:
            pass


class Pipeline:
    """One vla_pipeline: a consumer thread running `suffix` on the boundaries
    of `ctx`, in push order."""

    def __init__(self, ctx: Context, suffix: Suffix, depth: int):
        h = c_void_p()
        _check(lib().vla_pipeline_create(ctx.h, suffix.h, depth, ctypes.byref(h)))
        self.h = h.value
        self._held = {}

    def vla_pipeline_push(self, frame_id: int, b: Boundary, B: int, L: int, k: int, out):
        _check(lib().vla_pipeline_push(self.h, frame_id, ctypes.byref(b.c), B, L, k, _ptr(out)))
        self._held[frame_id] = (b, out)

    def vla_pipeline_backlog(self) -> int:
        n = c_int()
        _check(lib().vla_pipeline_backlog(self.h, ctypes.byref(n)))
        return n.value

    def vla_pipeline_pop(self, timeout_ms: int = -1):
        """(frame_id, t_wait_ms, t_cpu_ms) of the oldest pushed frame."""
        f, tw, tc = c_uint64(), c_float(), c_float()
        code = lib().vla_pipeline_pop(self.h, ctypes.byref(f), ctypes.byref(tw), ctypes.byref(tc), timeout_ms)
        self._held.pop(f.value, None)
        _check(code)
        return f.value, tw.value, tc.value

    def vla_pipeline_destroy(self):
        if getattr(self, "h", None):
            lib().vla_pipeline_destroy(self.h)
            self.h = None
            self._held.clear()

    def __del__(self):
        try:
            self.vla_pipeline_destroy()
        except Exception:
            pass


class Sched:
    """One vla_sched: the partition controller over the dynamic zone [k_lo, k_hi]."""

    def __init__(self, n_blocks, k_lo, k_hi, k_init, a_ms, b_ms, c_ms, x_ms, backlog_hi=2):
        h = c_void_p()
        _check(lib().vla_sched_create(n_blocks, k_lo, k_hi, k_init, a_ms, b_ms, c_ms, x_ms, backlog_hi,
                                      ctypes.byref(h)))
        self.h = h.value

    def vla_sched_observe(self, k, t_g_ms, t_x_ms, t_c_ms):
        _check(lib().vla_sched_observe(self.h, k, t_g_ms, t_x_ms, t_c_ms))

    def vla_sched_predict(self, k, u_gpu=0.0, u_cpu=0.0):
        """(T_G', T_C', T_stream) predicted for partition point k."""
        g, c, t = c_float(), c_float(), c_float()
        _check(lib().vla_sched_predict(self.h, k, u_gpu, u_cpu, ctypes.byref(g), ctypes.byref(c), ctypes.byref(t)))
        return g.value, c.value, t.value

    def vla_sched_decide(self, u_gpu=0.0, u_cpu=0.0, backlog=0, gpu_budget_ms=0.0) -> int:
        k = c_int()
        _check(lib().vla_sched_decide(self.h, u_gpu, u_cpu, backlog, gpu_budget_ms, ctypes.byref(k)))
        return k.value

    def vla_sched_model(self):
        """(a, b, c, x) in ms."""
        a, b, c, x = c_float(), c_float(), c_float(), c_float()
        _check(lib().vla_sched_model(self.h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c), ctypes.byref(x)))
        return a.value, b.value, c.value, x.value

    def vla_sched_destroy(self):
        if getattr(self, "h", None):
            lib().vla_sched_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.vla_sched_destroy()
        except Exception:
            pass
