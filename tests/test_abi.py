"""The C-ABI library on the CPU: it loads, exports every symbol the headers
declare, and its host-side logic (sizes, validation, status strings) behaves;
no GPU work is launched here."""
import ctypes
import os
import re

import pytest

import synth
from paper_2608_14586_amd import binding as vb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in os.listdir(os.path.join(ROOT, "include")):
        if h.endswith(".h"):
            text = open(os.path.join(ROOT, "include", h)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(vla_[a-z0-9_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    lib = vb.lib()
    names = declared_symbols()
    assert {"vla_create", "vla_run_prefix", "vla_run_encoder", "vla_load_block_weights", "vla_wait_boundary",
            "vla_op_gemm_bf16"} <= names
    for n in sorted(names):
        assert hasattr(lib, n), n
        assert ctypes.cast(getattr(lib, n), ctypes.c_void_p).value


def test_status_strings():
    for code in vb.STATUS:
        assert vb.vla_status_string(code)
    assert vb.vla_status_string(0) == "ok"


def _cfg(name, **over):
    wl = synth.CONFIGS[name]
    s = wl.llm if wl.llm is not None else wl.enc
    c = vb.stack_cfg(s, wl.dtype, max_tokens=wl.seq or wl.img_tokens, max_batch=wl.batch if wl.llm else wl.n_img,
                     n_blocks=wl.k if wl.llm and wl.k else s.n_blocks)
    for k, v in over.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("name,k", [("tiny", 2), ("small_llm", 12), ("llm7b", 16)])
def test_query_sizes_transfer_bytes(name, k):
    """hidden bytes = B * L * D * b (Eq. (11)); KV = k * 2 * B * H_kv * L * dh * b."""
    wl = synth.CONFIGS[name]
    s = wl.llm
    c = _cfg(name)
    b = 2 if wl.dtype == "bf16" else 4
    arena, hid, kv = vb.vla_query_sizes(c, None, 1, wl.seq, k)
    assert hid == wl.seq * s.d_model * b
    assert kv == k * 2 * s.n_kv_heads * wl.seq * s.head_dim * b
    if name == "llm7b":
        assert hid == 8 * 2 ** 20 and kv == 256 * 2 ** 20


def test_arena_grows_with_resident_blocks():
    """GPU memory follows the number of prefix blocks held on the GPU."""
    a8 = vb.vla_query_sizes(_cfg("llm7b", n_blocks=8), None, 1, 1024, 8)[0]
    a16 = vb.vla_query_sizes(_cfg("llm7b", n_blocks=16), None, 1, 1024, 16)[0]
    a24 = vb.vla_query_sizes(_cfg("llm7b", n_blocks=24), None, 1, 1024, 24)[0]
    per_block = (a16 - a8) // 8
    assert a16 - a8 == a24 - a16
    wl = synth.CONFIGS["llm7b"].llm
    weights = (wl.d_model * (wl.n_heads + 2 * wl.n_kv_heads) * wl.head_dim + wl.d_model * wl.n_heads * wl.head_dim
               + 3 * wl.d_model * wl.d_ff) * 2
    # weights plus the per-slot device KV staging of one more block
    norms = 2 * wl.d_model * 4
    assert weights + norms <= per_block <= weights + norms + 3 * 2 * 1024 * 4096 * 2 + 8 * 256


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 96, "VLA_ERR_UNSUPPORTED"),
    ("n_kv_heads", 3, "VLA_ERR_INVALID_ARG"),
    ("d_model", 0, "VLA_ERR_INVALID_ARG"),
    ("norm_is_layernorm", 1, "VLA_ERR_UNSUPPORTED"),
    ("dtype", 7, "VLA_ERR_INVALID_ARG"),
])
def test_query_sizes_rejects_bad_configs(field, value, code):
    c = _cfg("small_llm", **{field: value})
    with pytest.raises(vb.VlaError) as e:
        vb.vla_query_sizes(c, None, 1, 128, 1)
    assert e.value.name == code
    assert vb.lib().vla_last_error(None)


def test_create_rejects_small_arena_before_touching_the_gpu():
    c = _cfg("tiny")
    need = vb.vla_query_sizes(c, None, 1, 128, 2)[0]
    h = ctypes.c_void_p()
    rc = vb.lib().vla_create(ctypes.byref(c), None, 0, ctypes.c_void_p(4096), need - 1, None, None, None,
                             ctypes.byref(h))
    assert vb.STATUS[rc] == "VLA_ERR_OOM" and not h.value
    rc = vb.lib().vla_create(ctypes.byref(c), None, 0, None, need, None, None, None, ctypes.byref(h))
    assert vb.STATUS[rc] == "VLA_ERR_INVALID_ARG"


def test_encoder_stack_validation():
    wl = synth.CONFIGS["vit_l"]
    enc = vb.stack_cfg(wl.enc, "bf16", max_tokens=1024, max_batch=6)
    arena, _, _ = vb.vla_query_sizes(None, enc, 0, 0, 0)
    assert arena > 24 * 12 * 1024 * 1024 * 2
    bad = vb.stack_cfg(wl.enc, "bf16", max_tokens=1024, max_batch=6)
    bad.causal = 1
    with pytest.raises(vb.VlaError):
        vb.vla_query_sizes(None, bad, 0, 0, 0)


def _vis_case(dtype="bf16"):
    from synth.configs import VisionShape, vit_like
    enc = vb.stack_cfg(vit_like(2, 128, 2, 64, 256), dtype, max_tokens=64, max_batch=3)
    return enc, VisionShape(3, 56, 84, 14, 2, 128, 192)


def test_vision_sizes_grow_with_images():
    enc, vis = _vis_case()
    n3 = vb.vla_query_vision_sizes(enc, vb.vision_cfg(vis))
    enc.max_batch = 6
    n6 = vb.vla_query_vision_sizes(enc, vb.vision_cfg(vis))
    # per image: staging 3*56*84 bf16, 24 patch rows of 640 (588 padded), 24 merged rows of 128, 6 x 128 hidden
    per_img = 3 * 56 * 84 * 2 + 24 * 640 * 2 + 24 * 128 * 2 + 6 * 128 * 2
    assert n6 - n3 >= 3 * per_img and n6 - n3 < 3 * per_img + 4 * 256


@pytest.mark.parametrize("field,value,code", [
    ("img_h", 60, "VLA_ERR_UNSUPPORTED"),      # not a multiple of the patch
    ("merge", 4, "VLA_ERR_UNSUPPORTED"),       # 4 x 6 grid not a multiple of 4
    ("d_hidden", 96, "VLA_ERR_UNSUPPORTED"),   # bf16 needs multiples of 64
    ("d_out", 100, "VLA_ERR_UNSUPPORTED"),
    ("patch", 7, "VLA_ERR_SHAPE"),             # 8 x 12 = 96 patches > max_tokens 64
    ("channels", 0, "VLA_ERR_INVALID_ARG"),
])
def test_vision_validation(field, value, code):
    enc, vis = _vis_case()
    v = vb.vision_cfg(vis)
    setattr(v, field, value)
    with pytest.raises(vb.VlaError) as e:
        vb.vla_query_vision_sizes(enc, v)
    assert e.value.name == code


def test_vision_needs_an_encoder_and_f32_relaxes_widths():
    enc, vis = _vis_case("f32")
    v = vb.vision_cfg(vis)
    v.d_hidden, v.d_out = 96, 100
    assert vb.vla_query_vision_sizes(enc, v) > 0
    with pytest.raises(vb.VlaError) as e:
        vb.vla_query_vision_sizes(None, v)
    assert e.value.name == "VLA_ERR_INVALID_ARG"


def test_pack_weight_layout():
    """The host packer puts element (n, k) of row-major W at the slab-major
    position the header documents, pads rows to whole 256-row pairs with zeros
    and rejects K % 64 != 0; no GPU work."""
    import numpy as np
    N, K = 300, 192
    rng = np.random.default_rng(7)
    W = rng.integers(1, 65535, size=(N, K), dtype=np.uint16)
    nblk = (N + 255) // 256 * 2
    assert vb.vla_op_packed_weight_elems(N, K) == nblk * 128 * K
    assert vb.vla_op_packed_weight_elems(N, 100) == 0
    P = vb.vla_op_pack_weight_bf16(W, N, K)
    n, k = np.meshgrid(np.arange(N), np.arange(K), indexing="ij")
    pos = ((k // 64 * nblk + n // 128) * 128 + n % 128) * 64 + k % 64
    assert np.array_equal(P[pos], W)
    mask = np.ones(P.size, dtype=bool)
    mask[pos.ravel()] = False
    assert not P[mask].any()
    with pytest.raises(vb.VlaError) as e:
        vb.vla_op_pack_weight_bf16(np.zeros((4, 128), np.uint16), 4, 100)
    assert e.value.name == "VLA_ERR_UNSUPPORTED"
