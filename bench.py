"""Benchmark of the GPU-resident prefix on one MI355X.

One step = one frame of the partitioned pipeline's GPU stage (Sec. IV-A/C):
the ViT-L-shaped encoder over 6 camera images x 1024 patch tokens, then the
7B-shaped decoder blocks [0, k) as a causal prefill over 2048 tokens, then the
handoff of the boundary hidden state and the k-layer KV cache to pinned host
memory on a side stream, overlapping the next frame's encoder.  The encoder
and the decoder blocks share one compute stream: overlapping them on two
streams let the per-layer KV copies fall behind the frames (measured).  The
headline is k = 16; the sweep reports k in {8, 16, 24, 32}.  Inputs and weights are
seeded synthetic tensors already resident in HBM; weights are random-init
N(0, 0.02) at the stated shapes.

Prints ONE JSON line (rank 0, N = 1 only).

``--pipeline`` measures the whole partitioned model instead (Eq. (6), Sec.
IV-C): the GPU stage (encoder + decoder blocks [0, k)), the boundary handoff
and the host suffix (blocks [k, 32) on the CPU), run frame by frame and as the
cross-frame pipeline, for each k in ``--pipeline-ks``; it prints one JSON line
of per-k stage times and stream intervals (T_G, T_X, T_C of Eq. (8)-(10), the
serial frame time of Eq. (12), the pipelined interval against Eq. (13)).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# kernel classes launched once per block; the others once per frame
PER_BLOCK = ("qkv", "attn", "oproj", "mlp_up", "mlp_down", "norm")


def class_work(wl, kind, k, images=False):
    """Algorithmic FLOPs (GEMM / attention classes) or HBM bytes (norm) of
    each kernel class of one stack, from the stack shapes:
    {class: (unit, work, launches)}, the work of `launches` consecutive
    launches (one block's, or the vision front's per frame)."""
    if kind == "llm":
        s, B, L = wl.llm, wl.batch, wl.seq
        M = B * L
        pairs = B * L * (L + 1) // 2  # causal query-key pairs per head
    else:
        s, B, L = wl.enc, wl.n_img, wl.img_tokens
        M = B * L
        pairs = B * L * L
    d, H, Hkv, dh, F = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.d_ff
    up_rows = 2 * F if kind == "llm" else F
    w = {
        "qkv": ("flop", 2.0 * M * d * (H + 2 * Hkv) * dh, 1),
        "attn": ("flop", 4.0 * pairs * dh * H, 1),
        "oproj": ("flop", 2.0 * M * H * dh * d, 1),
        "mlp_up": ("flop", 2.0 * M * d * up_rows, 1),
        "mlp_down": ("flop", 2.0 * M * F * d, 1),
        "norm": ("byte", M * d * 4.0 + M * d * 2.0 + d * 4.0 * (2 if s.norm_is_layernorm else 1), 1),
    }
    if kind == "enc" and images:
        v = wl.vision
        V = wl.n_img * v.tokens_per_image
        # patch rows + the stem GEMM (K = channels * patch^2, unpadded)
        w["stem"] = ("flop", 2.0 * M * d * v.channels * v.patch * v.patch, 2)
        # final norm + merge, then the two connector GEMMs
        w["connector"] = ("flop", 2.0 * V * v.merge * v.merge * d * v.d_hidden + 2.0 * V * v.d_hidden * v.d_out, 3)
    return w


def profiled_traffic(kernel_class):
    """HBM bytes per launch of `kernel_class` from the committed rocprofv3 PMC
    summaries in profiles/, or None when none matches or the kernel source has
    changed since the counters were taken."""
    import glob
    import hashlib
    import re
    for path in glob.glob(os.path.join(ROOT, "profiles", "*_hbm_traffic.md")):
        for line in open(path):
            m = re.match(r"machine-readable: kernel=(\S+) traffic_bytes=(\d+) sources=(\S+) sha256_16=(\w+)", line)
            if not m or m.group(1) != kernel_class:
                continue
            h = hashlib.sha256()
            for src in m.group(3).split(","):
                path = os.path.join(ROOT, src)
                if not os.path.exists(path):
                    break
                h.update(open(path, "rb").read())
            else:
                if h.hexdigest()[:16] == m.group(4):
                    return int(m.group(2))
    return None


def frame_flops(wl, k, images=False):
    tot = 0.0
    for kind, n in (("llm", k), ("enc", wl.enc.n_blocks)):
        for c, (u, v, _) in class_work(wl, kind, k, images).items():
            if u == "flop":
                tot += v * (n if c in PER_BLOCK else 1)
    return tot


def cpu_baseline(wl, k, budget_s=20.0):
    """The oracle timed on this host on a bounded sample: decoder blocks at the
    full sequence length and encoder blocks over all 6 images, timed until the
    budget is spent, scaled to one frame (k decoder + 24 encoder blocks)."""
    import numpy as np
    import oracle
    import synth
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        threads = max([i.get("num_threads", 1) for i in info] or [1])
        if info:
            blas = "%s %s (%s)" % (info[0].get("internal_api"), info[0].get("version"), info[0].get("architecture"))
    except Exception:
        threads = len(os.sched_getaffinity(0))
    tok = synth.as_f32(synth.tokens(wl, frame=0))
    pat = synth.as_f32(synth.patches(wl, frame=0))
    t_llm, n_llm, t_enc, n_enc = 0.0, 0, 0.0, 0
    t_start = time.time()
    while (n_llm == 0 or n_enc == 0 or time.time() - t_start < budget_s) and n_llm < 4:
        W = {n: synth.as_f32(a) for n, a in synth.llm_block_weights(wl, n_llm).items()}
        t0 = time.time()
        oracle.run_prefix(tok, lambda l: W, wl.llm, 1, keep_kv=False)
        t_llm += time.time() - t0
        n_llm += 1
        E = {n: synth.as_f32(a) for n, a in synth.vit_block_weights(wl, n_enc).items()}
        t0 = time.time()
        oracle.run_encoder(pat, lambda l: E, wl.enc, n_blocks=1)
        t_enc += time.time() - t0
        n_enc += 1
    per_frame = k * t_llm / n_llm + wl.enc.n_blocks * t_enc / n_enc
    return {"value": wl.seq / per_frame, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": "%d decoder block(s) at L=%d and %d ViT block(s) over %dx%d patches, numpy fp32, "
                      "scaled to %d decoder + %d encoder blocks per frame (%.1f s per frame)"
                      % (n_llm, wl.seq, n_enc, wl.n_img, wl.img_tokens, k, wl.enc.n_blocks, per_frame),
            "blas": "numpy %s, %s" % (np.__version__, blas), "affinity_cores": len(os.sched_getaffinity(0))}


def decode_bench(args):
    """Decode steps across the boundary: decoder blocks [0, k) for one new
    token per sequence after a 2048-token prefix, over the KV cache the prefix
    handed over.  A step streams the k blocks' weights once, so it is priced
    against HBM bandwidth."""
    import numpy as np
    import torch
    import synth
    from paper_2608_14586_amd import binding as vb

    wl = synth.CONFIGS["sweep7b"]
    s = wl.llm
    L, k, B, T = wl.seq, args.k, args.decode_batch, args.decode_steps
    d, Hkv, dh, H, F = s.d_model, s.n_kv_heads, s.head_dim, s.n_heads, s.d_ff
    L_cap = L + T + 8
    ctx = vb.Context(llm=vb.stack_cfg(s, "bf16", max_tokens=L_cap, max_batch=B, n_blocks=k))
    for l in range(k):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(wl, l))
    if args.decode_precision == "split":
        ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_SPLIT)
    toks = synth.tokens(wl, frame=3, B=B, L=L + T)
    bnd = vb.Boundary(B, L, d, k, Hkv, dh)
    ctx.vla_run_prefix(1, np.ascontiguousarray(toks[:, :L]), B, L, k, bnd)
    ctx.vla_wait_boundary(1, 600000)
    cache = torch.zeros((k, 2, B, Hkv, L_cap, dh), dtype=torch.bfloat16, device="cuda")
    cache[:, :, :, :, :L] = bnd.kv.cuda()
    xs = torch.from_numpy(np.ascontiguousarray(toks[:, L:]).view(np.int16)).cuda()  # [B][T][d]
    xs = [xs[:, t].contiguous() for t in range(T)]
    outs = [vb.Boundary(B, 1, d, 0, Hkv, dh, with_kv=False) for _ in range(4)]
    fid = [100]

    def steps(n, t0, profile=False):
        if profile:
            ctx.vla_profile(True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        ids = []
        for i in range(n):
            f = fid[0]
            fid[0] += 1
            ctx.vla_decode_step(f, xs[(t0 + i) % T], B, L + (t0 + i) % T, k, cache, L_cap, outs[i % 4])
            ids.append(f)
        for f in ids[-3:]:
            ctx.vla_wait_boundary(f, 600000)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t) * 1000 / n
        if profile:
            ctx.vla_profile(False)
        return dt

    steps(4, 0)
    ms = steps(T, 0)
    steps(T, 0, profile=True)
    w_bytes = k * 2 * (d * (H + 2 * Hkv) * dh + H * dh * d + d * 2 * F + F * d)
    kv_bytes = k * 2 * B * Hkv * (L + T // 2) * dh * 2  # cache rows read per step (mean position)
    kern = {}
    cls_bytes = {"qkv": d * (H + 2 * Hkv) * dh * 2, "oproj": H * dh * d * 2, "mlp_up": d * 2 * F * 2,
                 "mlp_down": F * d * 2, "attn": 2 * B * Hkv * (L + T // 2) * dh * 2}
    for ci, cname in enumerate(vb.KERNEL_CLASSES):
        tot, cnt = ctx.vla_profile_read(vb.VLA_STACK_LLM, ci)
        if cnt == 0:
            continue
        ent = {"avg_us": round(tot / cnt * 1000, 2), "launches": cnt}
        if cname in cls_bytes:
            ent["gbs"] = round(cls_bytes[cname] / (tot / cnt / 1000) / 1e9, 1)
            ent["frac"] = round(ent["gbs"] / PEAK_HBM_GBS, 4)
        kern[cname] = ent
    achieved = (w_bytes + kv_bytes) / (ms / 1000) / 1e9
    out = {"metric": "decode step time across the boundary (blocks [0,%d), %d sequence(s), after a %d-token prefix)"
                     % (k, B, L),
           "value": round(ms, 4), "unit": "ms/step", "higher_is_better": False, "n_gpus": 1, "steps": T,
           "dtype": "bf16", "data": "synthetic",
           "tokens_per_s": round(B * 1000 / ms, 1),
           "config": {"workload": "sweep7b decoder blocks (d=4096, 32x128 MHA, SwiGLU 11008) [0,k), bf16 weights "
                                  "N(0,0.02), KV cache from the prefix handoff", "k": k, "batch": B, "prefix_len": L,
                      "operands": args.decode_precision},
           "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(achieved / PEAK_HBM_GBS, 4), "bytes_per_step": w_bytes + kv_bytes},
           "kernels": kern}
    if args.decode_host_blocks > 0:
        out["across"] = decode_across(args, ctx, wl, bnd, cache, xs, outs[0], L_cap)
    ctx.vla_destroy()
    print(json.dumps(out), flush=True)


def decode_across(args, ctx, wl, bnd, cache, xs, ob, L_cap):
    """One token through the whole partitioned model (Eq. (6) per token): the
    GPU step over blocks [0, k), its boundary to pinned host memory, then the
    host decode step over blocks [k, N) from the host's own KV cache, which
    its prefill of the same prefix filled.  Tokens are serial (each needs the
    previous one), so the stages add up: T_G + T_X + T_C per token."""
    import torch
    import synth
    from paper_2608_14586_amd import binding as vb

    s = wl.llm
    L, k, B, T = wl.seq, args.k, args.decode_batch, len(xs)
    N = k + args.decode_host_blocks
    sfx = vb.Suffix(vb.stack_cfg(s, "bf16", max_tokens=L_cap), k, N, args.pipeline_threads)
    for l in range(k, N):
        sfx.vla_suffix_load_block_weights(l, synth.llm_block_weights(wl, l))
    sfx.vla_suffix_set_cache(B, L_cap)
    h = torch.empty((B, L, s.d_model), dtype=torch.float32)
    t = time.perf_counter()
    sfx.vla_suffix_run(bnd.hidden, vb.VLA_BF16, B, L, h)
    prefill_ms = (time.perf_counter() - t) * 1000
    o = torch.empty((B, s.d_model), dtype=torch.float32)
    tg, tc = [], []
    fid = 5000
    for i in range(T):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ctx.vla_decode_step(fid + i, xs[i], B, L + i, k, cache, L_cap, ob)
        ctx.vla_wait_boundary(fid + i, 600000)
        t1 = time.perf_counter()
        sfx.vla_suffix_decode_step(k, ob.hidden, vb.VLA_BF16, B, L + i, o)
        t2 = time.perf_counter()
        tg.append((t1 - t0) * 1000)
        tc.append((t2 - t1) * 1000)
    tg, tc = sorted(tg[2:]), sorted(tc[2:])
    mg, mc = tg[len(tg) // 2], tc[len(tc) // 2]
    w_block = 2 * (s.d_model * (s.n_heads + 2 * s.n_kv_heads) * s.head_dim + s.n_heads * s.head_dim * s.d_model
                   + 3 * s.d_model * s.d_ff)
    kv_block = 2 * B * s.n_kv_heads * L * s.head_dim * 2
    host_gbs = (N - k) * (w_block + kv_block) / (mc / 1000) / 1e9
    r = {"n_blocks": N, "host_blocks": N - k, "host_threads": sfx.vla_suffix_threads(),
         "gpu_step_ms": round(mg, 3), "host_step_ms": round(mc, 3), "token_ms": round(mg + mc, 3),
         "host_ms_per_block": round(mc / (N - k), 3), "host_gbs": round(host_gbs, 1),
         "host_prefill_ms": round(prefill_ms, 1), "steps": len(tc)}
    sfx.vla_suffix_destroy()
    return r


def prefix_leg(ctx, wl, L, k, steps, warmup, weights_note):
    """Decoder blocks [0, k) alone over one sequence of L device-resident
    tokens, back to back, with the boundary and k-layer KV handoff to pinned
    host memory on the copy stream: ms per frame, prefix tokens/s, T_G, T_X,
    and per-class kernel times against the algorithmic work (a pass of its own
    with per-launch events)."""
    import numpy as np
    import torch
    import synth
    from paper_2608_14586_amd import binding as vb
    s = wl.llm
    dev = torch.device("cuda:0")
    toks = [torch.from_numpy(synth.tokens(wl, frame=f, L=L).view(np.int16)).to(dev) for f in range(2)]
    bnds = [vb.Boundary(1, L, s.d_model, k, s.n_kv_heads, s.head_dim) for _ in range(3)]
    fid = [50000 + 1000 * k + L]

    def frames(n, profile=False):
        ids = []
        if profile:
            ctx.vla_profile(True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for i in range(n):
            f = fid[0]
            fid[0] += 1
            ctx.vla_run_prefix(f, toks[i % 2], 1, L, k, bnds[i % 3])
            ids.append(f)
        for f in ids[-3:]:
            ctx.vla_wait_boundary(f, 120000)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t
        if profile:
            ctx.vla_profile(False)
        return wall * 1000.0 / n, [ctx.vla_frame_times(f) for f in ids]

    frames(warmup)
    ms, times = frames(steps)
    frames(steps, profile=True)
    tg = np.array([t[0] for t in times])
    tx = np.array([t[1] for t in times])
    work = class_work(wl, "llm", k)
    classes = {}
    flops = 0.0
    for ci, cname in enumerate(vb.KERNEL_CLASSES):
        tot, cnt = ctx.vla_profile_read(vb.VLA_STACK_LLM, ci)
        if cnt == 0:
            continue
        ent = {"ms_total": round(tot, 4), "launches": cnt, "avg_us": round(tot / cnt * 1000, 2)}
        if cname in work:
            unit, per, group = work[cname]
            avg_s = tot / cnt * group / 1000.0
            if unit == "flop":
                flops += per * k
                ent["tflops"] = round(per / avg_s / 1e12, 1)
                ent["frac"] = round(per / avg_s / 1e12 / PEAK_BF16_TFLOPS, 4)
            else:
                ent["gbs"] = round(per / avg_s / 1e9, 1)
                ent["frac"] = round(per / avg_s / 1e9 / PEAK_HBM_GBS, 4)
            ent["per_launch"] = per
        classes["llm.%s" % cname] = ent
    return {"workload": "%s: %d decoder blocks (d=%d, %dx%d heads, %d KV heads, SwiGLU %d) over 1x%d tokens, "
                        "boundary + %d-layer KV to pinned host; %s"
                        % (wl.name, k, s.d_model, s.n_heads, s.head_dim, s.n_kv_heads, s.d_ff, L, k, weights_note),
            "k": k, "seq_len": L, "ms_per_frame": round(ms, 3), "prefix_tokens_per_s": round(L / (ms / 1000.0), 1),
            "t_gpu_prefix_ms": round(float(np.mean(tg)), 3), "t_gpu_prefix_ms_median": round(float(np.median(tg)), 3),
            "t_boundary_copy_ms": round(float(np.mean(tx)), 4),
            "t_prefix_plus_handoff_ms": round(float(np.mean([t[2] for t in times])), 3),
            "frame_tflops": round(flops / 1e12, 3),
            "mfma_frac_of_bf16_peak": round(flops / (ms / 1000.0) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "kernels": classes}


def norm_large():
    """RMSNorm over a 1 GiB fp32 input (65536 x 4096 -> bf16): a working set
    four times the 256 MiB Infinity Cache, so the rate is HBM's, not the
    cache's (the frame's norms read a residual the previous GEMM just wrote)."""
    import torch
    from paper_2608_14586_amd import binding as vb
    M, d = 65536, 4096
    x = torch.randn((M, d), dtype=torch.float32, device="cuda")
    g = torch.ones(d, dtype=torch.float32, device="cuda")
    y = torch.empty((M, d), dtype=torch.bfloat16, device="cuda")
    st = torch.cuda.current_stream()
    for _ in range(3):
        vb.vla_op_norm_bf16(x, g, None, 1e-6, y, M, d, st.cuda_stream)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    n = 10
    ev[0].record(st)
    for _ in range(n):
        vb.vla_op_norm_bf16(x, g, None, 1e-6, y, M, d, st.cuda_stream)
    ev[1].record(st)
    torch.cuda.synchronize()
    us = ev[0].elapsed_time(ev[1]) * 1000 / n
    nbytes = M * d * (4 + 2) + d * 4
    return {"shape": [M, d], "avg_us": round(us, 1), "gbs": round(nbytes / us / 1e3, 1),
            "frac": round(nbytes / us / 1e3 / PEAK_HBM_GBS, 4), "bytes": nbytes}


def dual_bench(args):
    """The dual-stack workload: camera images through the stem, the ViT-L
    encoder and the connector into 1536 visual + 512 text tokens, then two
    24-block 0.5B-class decoder stacks over the same tokens (a dual-expert
    backbone), each to partition point k on the GPU; the host suffix runs
    blocks [k, 24) of both.  k = 0 leaves only the encoder on the GPU."""
    import numpy as np
    import torch
    import synth
    from paper_2608_14586_amd import binding as vb

    wl = synth.CONFIGS["dual05b"]
    s, e, vis = wl.llm, wl.enc, wl.vision
    n_img, T = wl.n_img, wl.text_tokens
    L = n_img * vis.tokens_per_image + T
    N = s.n_blocks
    ks = sorted(set(int(x) for x in args.dual_ks.split(",")))
    assert all(0 <= k <= N for k in ks)
    lcfg = vb.stack_cfg(s, "bf16", max_tokens=L, max_batch=1, n_blocks=N)
    ctx = [vb.Context(llm=lcfg, enc=vb.stack_cfg(e, "bf16", max_tokens=vis.L_img, max_batch=n_img))]
    # the second stack on compute and copy streams of its own: the two
    # stacks' small GEMMs overlap instead of queueing behind each other
    ctx.append(vb.Context(llm=lcfg))
    t0 = time.time()
    for l in range(e.n_blocks):
        ctx[0].vla_load_block_weights(vb.VLA_STACK_ENC, l, synth.vit_block_weights(wl, l))
    ctx[0].vla_attach_vision(vb.vision_cfg(vis))
    ctx[0].vla_load_vision_weights(synth.vision_weights(wl))
    # stack j holds blocks j*N .. j*N + N-1 of the workload's weight sequence
    for j in range(2):
        for l in range(N):
            ctx[j].vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(wl, j * N + l))
    dev = torch.device("cuda:0")
    imgs = [torch.from_numpy(synth.images(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
    texts = [torch.from_numpy(synth.text(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
    # token rows rotate over three buffers: the vision of frame f + 3 waits for
    # the second stack's read of frame f (with its handoff behind it)
    NTOK = 3
    toks = [torch.empty((L, s.d_model), dtype=torch.bfloat16, device=dev) for _ in range(NTOK)]
    torch.cuda.synchronize()
    log("dual stack resident (%.0fs)" % (time.time() - t0))
    fid = [1]
    table = {}
    last = {}
    for k in ks:
        bnds = [[vb.Boundary(1, L, s.d_model, k, s.n_kv_heads, s.head_dim) for _ in range(3)] for _ in range(2)]

        def frames(n):
            ids = []
            ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            torch.cuda.synchronize()
            t = time.perf_counter()
            read_done = [None] * NTOK
            for i in range(n):
                f = fid[0]
                fid[0] += 1
                tok = toks[i % NTOK]
                if read_done[i % NTOK] is not None:
                    ctx[0].compute_stream.wait_event(read_done[i % NTOK])
                if i == 0:
                    ev[0].record(ctx[0].compute_stream)
                ctx[0].vla_run_vision(f, imgs[i % 2], n_img, texts[i % 2], T, tok)
                ready = torch.cuda.Event()
                ready.record(ctx[0].compute_stream)
                if i == 0:
                    ev[1].record(ctx[0].compute_stream)
                ctx[1].compute_stream.wait_event(ready)
                for j in range(2):
                    ctx[j].vla_run_prefix(f, tok, 1, L, k, bnds[j][i % 3])
                done = torch.cuda.Event()
                done.record(ctx[1].compute_stream)
                read_done[i % NTOK] = done
                ids.append((f, i % 3))
            for f, _ in ids[-3:]:
                for j in range(2):
                    ctx[j].vla_wait_boundary(f, 120000)
            torch.cuda.synchronize()
            return (time.perf_counter() - t) * 1000 / n, ev[0].elapsed_time(ev[1]), ids[-1][1]

        frames(args.warmup)
        ms, vis_ms, slot = frames(args.steps)
        table[k] = {"t_gpu_ms": round(ms, 3), "t_vision_ms": round(vis_ms, 3),
                    "handoff_mib": round(2 * (L * s.d_model * 2 + k * 2 * s.n_kv_heads * L * s.head_dim * 2) / 2 ** 20, 1)}
        last[k] = [bnds[j][slot] for j in range(2)]
        log("dual k=%d: %s" % (k, json.dumps(table[k])))
    # the host suffix of both stacks on the last frame's boundaries
    for k in [k for k in ks if k < N and k in args.dual_host_ks]:
        t_c = 0.0
        for j in range(2):
            sfx = vb.Suffix(vb.stack_cfg(s, "bf16", max_tokens=L), k, N, args.pipeline_threads)
            for l in range(k, N):
                sfx.vla_suffix_load_block_weights(l, synth.llm_block_weights(wl, j * N + l))
            out = np.empty((1, L, s.d_model), np.float32)
            sfx.vla_suffix_run(last[k][j].hidden, vb.VLA_BF16, 1, L, out)   # first touch of the packed weights
            t = time.perf_counter()
            sfx.vla_suffix_run(last[k][j].hidden, vb.VLA_BF16, 1, L, out)
            t_c += (time.perf_counter() - t) * 1000
            threads = sfx.vla_suffix_threads()
            sfx.vla_suffix_destroy()
        r = table[k]
        r["t_host_ms"] = round(t_c, 1)
        r["host_threads"] = threads
        r["host_ms_per_block"] = round(t_c / (2 * (N - k)), 2)
        r["frame_by_frame_ms"] = round(r["t_gpu_ms"] + t_c, 1)            # Eq. (12) without T_X
        r["pipelined_interval_ms"] = round(max(r["t_gpu_ms"], t_c), 1)     # Eq. (13) without T_X
        log("dual k=%d host: %.1f ms over %d blocks" % (k, t_c, 2 * (N - k)))
    out = {"metric": "dual-stack frame: GPU stage (images -> stem + ViT-L + connector -> two 0.5B-class stacks "
                     "[0,k) over 2048 tokens) per partition point k, and the host suffix of both stacks",
           "unit": "ms", "higher_is_better": False, "n_gpus": 1, "steps": args.steps, "dtype": "bf16",
           "data": "synthetic",
           "config": {"workload": "dual05b: 6 cameras 448x448, 14x14 patches, ViT-L 24 blocks, 2x2 merge, "
                                  "connector 4096->896->896; 2 x 24 decoder blocks d=896 14x64 GQA 2 KV SwiGLU "
                                  "4864; 1536 visual + 512 text tokens", "ks": ks},
           "per_k": {str(k): v for k, v in table.items()}}
    for c in ctx[::-1]:
        c.vla_destroy()
    print(json.dumps(out), flush=True)


def gpu_stage_factory(ctx, pats, toks, enc_out, n_img, L_img, L, fid):
    """gpu_stage(i, k, boundary): the GPU stage of one frame (encoder +
    decoder blocks [0, k)) enqueued, with events around it on the compute
    stream; returns (frame id, (start, end) events)."""
    import torch

    def gpu_stage(i, k, b):
        f = fid[0]
        fid[0] += 1
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record(ctx.compute_stream)
        ctx.vla_run_encoder(f, pats[i % 2], n_img, L_img, enc_out)
        ctx.vla_run_prefix(f, toks[i % 2], 1, L, k, b)
        ev[1].record(ctx.compute_stream)
        return f, ev
    return gpu_stage


def adaptive_run(args, ctx, gpu_stage, wl, N):
    """Closed loop with the partition controller (Sec. IV-D): each frame's
    partition point comes from Phi over the dynamic zone [N - 8, N], which
    learns the stage model from the frames it observes.  The first half runs
    alone; in the second half another module declares a share of the GPU
    (u_gpu), which Phi trades against the host stage."""
    import numpy as np
    import synth
    from paper_2608_14586_amd import binding as vb

    s = wl.llm
    L = wl.seq
    k_lo, k_hi, k0 = N - 8, N, N - 6
    sfx = vb.Suffix(vb.stack_cfg(s, "bf16", max_tokens=L), k_lo, N, args.pipeline_threads)
    for l in range(k_lo, N):
        sfx.vla_suffix_load_block_weights(l, synth.llm_block_weights(wl, l))
    # uninformative priors: one ms per block on each side, nothing fixed
    phi = vb.Sched(N, k_lo, k_hi, k0, 0.0, 1.0, 1.0, 0.0, backlog_hi=2)
    pipe = vb.Pipeline(ctx, sfx, depth=2)
    bnds = [vb.Boundary(1, L, s.d_model, k_hi, s.n_kv_heads, s.head_dim, with_kv=False) for _ in range(3)]
    outs = [np.empty((1, L, s.d_model), np.float32) for _ in range(3)]
    n = args.pipeline_adaptive
    pending = []  # (frame id, k, events, push index)
    trace = []
    last_pop = [None]

    def pop_one():
        f, tw, tc = pipe.vla_pipeline_pop(600000)
        fid, k, ev, i = pending.pop(0)
        assert f == fid
        ctx.vla_wait_boundary(f, 600000)  # already copied: retires the slot, records T_X
        tg = ev[0].elapsed_time(ev[1])
        tx = ctx.vla_frame_times(f)[1]
        phi.vla_sched_observe(k, tg, tx, tc)
        now = time.perf_counter()
        trace[i].update({"T_G_ms": round(tg, 2), "T_X_ms": round(tx, 3), "T_C_ms": round(tc, 1),
                         "interval_ms": None if last_pop[0] is None else round((now - last_pop[0]) * 1000, 1)})
        last_pop[0] = now

    for i in range(n):
        u_gpu = 0.0 if i < n // 2 else 0.95
        if len(pending) == 2:
            pop_one()
        k = phi.vla_sched_decide(u_gpu, 0.0, pipe.vla_pipeline_backlog(), 0.0)
        f, ev = gpu_stage(i, k, bnds[i % 3])
        pipe.vla_pipeline_push(f, bnds[i % 3], 1, L, k, outs[i % 3])
        pending.append((f, k, ev, i))
        trace.append({"frame": i, "u_gpu": u_gpu, "k": k})
    while pending:
        pop_one()
    pipe.vla_pipeline_destroy()
    a, b, c, x = phi.vla_sched_model()
    log("adaptive: k per frame %s; model a=%.1f b=%.3f c=%.1f x=%.3f ms" % ([t["k"] for t in trace], a, b, c, x))
    return {"zone": [k_lo, k_hi], "k_init": k0, "model_ms": {"a": round(a, 2), "b": round(b, 3), "c": round(c, 1),
                                                             "x": round(x, 3)}, "frames": trace}


def pipeline_bench(args):
    """Stage times and stream interval of the partitioned model per k."""
    import numpy as np
    import torch
    import synth
    from paper_2608_14586_amd import binding as vb

    wl = synth.CONFIGS["sweep7b"]
    s, e = wl.llm, wl.enc
    N = s.n_blocks
    L, n_img, L_img = wl.seq, wl.n_img, wl.img_tokens
    ks = sorted(int(k) for k in args.pipeline_ks.split(","))
    if not all(0 < k <= N for k in ks):
        raise SystemExit("--pipeline-ks must lie in (0, %d]" % N)
    kmax = max(ks)
    nf = args.pipeline_frames
    ctx = vb.Context(llm=vb.stack_cfg(s, "bf16", max_tokens=L, max_batch=1, n_blocks=kmax),
                     enc=vb.stack_cfg(e, "bf16", max_tokens=L_img, max_batch=n_img))
    for l in range(e.n_blocks):
        ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, synth.vit_block_weights(wl, l))
    for l in range(kmax):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(wl, l))
    dev = torch.device("cuda:0")
    toks = [torch.from_numpy(synth.tokens(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
    pats = [torch.from_numpy(synth.patches(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
    enc_out = torch.empty((n_img, L_img, e.d_model), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    cs = ctx.compute_stream
    fid = [5000]
    res = {}
    threads = None
    for k in ks:
        sfx = None
        if k < N:
            t0 = time.time()
            sfx = vb.Suffix(vb.stack_cfg(s, "bf16", max_tokens=L), k, N, args.pipeline_threads)
            for l in range(k, N):
                sfx.vla_suffix_load_block_weights(l, synth.llm_block_weights(wl, l))
            threads = sfx.vla_suffix_threads()
            log("k=%d: host suffix [%d,%d) loaded on %d threads (%.0fs)" % (k, k, N, threads, time.time() - t0))
        bnds = [vb.Boundary(1, L, s.d_model, k, s.n_kv_heads, s.head_dim, with_kv=False) for _ in range(3)]
        outs = [np.empty((1, L, s.d_model), np.float32) for _ in range(3)]

        def gpu_stage(i, b):
            f = fid[0]
            fid[0] += 1
            ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            ev[0].record(cs)
            ctx.vla_run_encoder(f, pats[i % 2], n_img, L_img, enc_out)
            ctx.vla_run_prefix(f, toks[i % 2], 1, L, k, b)
            ev[1].record(cs)
            return f, ev

        # frame by frame: T_G + T_X + T_C on one frame's critical path (Eq. (12))
        serial, tg, tx, tc = [], [], [], []
        for i in range(nf + 1):
            t = time.perf_counter()
            f, ev = gpu_stage(i, bnds[0])
            ctx.vla_wait_boundary(f, 600000)
            t1 = time.perf_counter()
            if sfx is not None:
                hb = bnds[0].hidden.view(torch.int16).numpy().view(np.uint16)
                sfx.vla_suffix_run(hb, vb.VLA_BF16, 1, L, outs[0])
            t2 = time.perf_counter()
            if i == 0:
                continue  # warm-up
            serial.append((t2 - t) * 1000)
            tg.append(ev[0].elapsed_time(ev[1]))
            tx.append(ctx.vla_frame_times(f)[1])
            tc.append((t2 - t1) * 1000)
        # cross-frame pipeline: the GPU runs frame i+1 while the host runs frame i
        pops = []
        if sfx is not None:
            pipe = vb.Pipeline(ctx, sfx, depth=2)
            pending = 0
            for i in range(nf + 2):
                if pending == 2:
                    pipe.vla_pipeline_pop(600000)
                    pops.append(time.perf_counter())
                    pending -= 1
                f, _ = gpu_stage(i, bnds[i % 3])
                pipe.vla_pipeline_push(f, bnds[i % 3], 1, L, k, outs[i % 3])
                pending += 1
            while pending:
                pipe.vla_pipeline_pop(600000)
                pops.append(time.perf_counter())
                pending -= 1
            pipe.vla_pipeline_destroy()
            pops = pops[2:]  # steady state
        else:
            for i in range(nf + 2):
                f, _ = gpu_stage(i, bnds[i % 3])
                if i >= 2:
                    ctx.vla_wait_boundary(f - 2, 600000)
                    pops.append(time.perf_counter())
        stream = (pops[-1] - pops[0]) * 1000 / (len(pops) - 1)
        T = {"T_G_ms": float(np.mean(tg)), "T_X_ms": float(np.mean(tx)), "T_C_ms": float(np.mean(tc))}
        res[str(k)] = {**{n: round(v, 3) for n, v in T.items()},
                       "suffix_blocks": N - k,
                       "T_frame_serial_ms": round(float(np.mean(serial)), 3),
                       "T_stream_ms": round(stream, 3),
                       "eq13_max_ms": round(max(T["T_G_ms"], T["T_X_ms"] + T["T_C_ms"]), 3),
                       "F_exec_hz": round(1000.0 / stream, 2)}
        log("k=%d: %s" % (k, res[str(k)]))
        del sfx
    adaptive = adaptive_run(args, ctx, gpu_stage_factory(ctx, pats, toks, enc_out, n_img, L_img, L, fid),
                            wl, N) if args.pipeline_adaptive > 0 else None
    best = min(res, key=lambda k: res[k]["T_stream_ms"])
    out = {"metric": "stream interval of the partitioned model (GPU encoder + blocks [0,k), host blocks [k,%d))" % N,
           "value": res[best]["T_stream_ms"], "unit": "ms", "higher_is_better": False, "best_k": int(best),
           "n_gpus": 1, "frames": nf, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": "sweep7b encoder 24x ViT-L over 6x1024 + %d 7B-shaped decoder blocks over 1x%d "
                                  "tokens, boundary bf16 to pinned host" % (N, L),
                      "host_threads": threads},
           "per_k": res}
    if adaptive is not None:
        out["adaptive"] = adaptive
    ctx.vla_destroy()
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--k", type=int, default=16)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-legs", action="store_true",
                    help="skip the extra prefix-only legs (7B at L=1024, split precision, the 0.5B GQA stack)")
    ap.add_argument("--only-leg", choices=("llm7b_L1024_k16", "small_llm_L4096_k12"), default=None,
                    help="run one prefix-only leg alone (for profiling) and print its JSON")
    ap.add_argument("--frame", choices=("embeddings", "images"), default="embeddings",
                    help="encoder input: synthetic patch embeddings, or camera images through the stem, with the "
                         "connector's tokens as the decoder's input")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (HBM counter calibration)")
    ap.add_argument("--pipeline", action="store_true",
                    help="measure the partitioned model (GPU prefix + host suffix) instead of the GPU prefix")
    ap.add_argument("--pipeline-ks", default="16,24,28,31,32")
    ap.add_argument("--encoder-stream", action="store_true",
                    help="run the encoder on a stream of its own, overlapping the previous frame's prefix")
    ap.add_argument("--decode-precision", choices=("bf16", "split"), default="bf16",
                    help="activation operands of the prefill and the decode steps (split: hi + lo bf16 pairs)")
    ap.add_argument("--decode", action="store_true",
                    help="measure decode steps of blocks [0,k) over the prefix's KV cache instead")
    ap.add_argument("--decode-steps", type=int, default=32)
    ap.add_argument("--decode-batch", type=int, default=1)
    ap.add_argument("--decode-host-blocks", type=int, default=0,
                    help="with --decode: also run blocks [k, k + n) on the host per token")
    ap.add_argument("--dual", action="store_true",
                    help="the dual 0.5B-stack workload from camera images (GPU stage per k, host suffix)")
    ap.add_argument("--dual-ks", default="0,6,12,18,24")
    ap.add_argument("--dual-host-ks", type=lambda x: [int(v) for v in x.split(",") if v], default=[0, 12, 18],
                    help="partition points whose host suffix is timed")
    ap.add_argument("--pipeline-frames", type=int, default=4)
    ap.add_argument("--pipeline-threads", type=int, default=0, help="host suffix threads (0: all)")
    ap.add_argument("--pipeline-adaptive", type=int, default=20, metavar="FRAMES",
                    help="frames of the closed loop with the partition controller (0: skip)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the prefix is a single-GPU stage (frames, cameras or block "
              "ranges would shard across GPUs). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.pipeline:
        pipeline_bench(args)
        return
    if args.decode:
        decode_bench(args)
        return
    if args.dual:
        dual_bench(args)
        return

    if args.only_leg:
        import synth
        from paper_2608_14586_amd import binding as vb
        name = args.only_leg.split("_L")[0]
        lw = synth.CONFIGS[name]
        L = 1024 if name == "llm7b" else lw.seq
        k = 16 if name == "llm7b" else lw.k
        lctx = vb.Context(llm=vb.stack_cfg(lw.llm, "bf16", max_tokens=L, max_batch=1, n_blocks=k))
        for l in range(k):
            lctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(lw, l))
        leg = prefix_leg(lctx, lw, L, k, args.steps, args.warmup, "random-init N(0,0.02) weights")
        lctx.vla_destroy()
        print(json.dumps({args.only_leg: leg}), flush=True)
        return

    if args.copy_calibration:
        n = args.copy_calibration * 2 ** 20 // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 4, "bytes_written": n * 4, "launches": 3}))
        return

    import synth
    from paper_2608_14586_amd import binding as vb

    wl = synth.CONFIGS["sweep7b"]
    ks = sorted(set(([] if args.no_sweep else list(wl.ks)) + [args.k]))
    kmax = max(ks)
    s, e = wl.llm, wl.enc
    L, n_img, L_img = wl.seq, wl.n_img, wl.img_tokens
    llm_cfg = vb.stack_cfg(s, "bf16", max_tokens=L, max_batch=1, n_blocks=kmax)
    enc_cfg = vb.stack_cfg(e, "bf16", max_tokens=L_img, max_batch=n_img)
    t0 = time.time()
    # device memory the context takes, by hipMemGetInfo before and after
    # (its arena plus whatever the runtime adds for its streams and events)
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    # --encoder-stream: the encoder of frame f+1 runs on a stream of its own,
    # beside the prefix of frame f (the default keeps one compute stream)
    ctx = vb.Context(llm=llm_cfg, enc=enc_cfg,
                     encoder_stream=torch.cuda.Stream() if args.encoder_stream else None)
    torch.cuda.synchronize()
    mem_delta = free0 - torch.cuda.mem_get_info()[0]
    log("arena %.2f GiB, hipMemGetInfo delta %.2f GiB" % (ctx.arena_bytes / 2 ** 30, mem_delta / 2 ** 30))
    for l in range(e.n_blocks):
        ctx.vla_load_block_weights(vb.VLA_STACK_ENC, l, synth.vit_block_weights(wl, l))
    for l in range(kmax):
        ctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(wl, l))
        if l % 8 == 7:
            log("loaded %d/%d decoder blocks (%.0fs)" % (l + 1, kmax, time.time() - t0))
    dev = torch.device("cuda:0")
    toks = [torch.from_numpy(synth.tokens(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
    pats = [torch.from_numpy(synth.patches(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
    enc_out = torch.empty((n_img, L_img, e.d_model), dtype=torch.bfloat16, device=dev)
    images = args.frame == "images"
    if images:
        # E(x_t) from camera images: stem, encoder, connector; the prefix reads its tokens
        vis = wl.vision
        assert n_img * vis.tokens_per_image + wl.text_tokens == L
        ctx.vla_attach_vision(vb.vision_cfg(vis))
        ctx.vla_load_vision_weights(synth.vision_weights(wl))
        imgs = [torch.from_numpy(synth.images(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
        texts = [torch.from_numpy(synth.text(wl, frame=f).view(np.int16)).to(dev) for f in range(2)]
        frame_tok = torch.empty((L, s.d_model), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    log("weights and inputs resident (%.0fs)" % (time.time() - t0))

    fid = [1000]

    def run(k, n, profile=False):
        bnds = [vb.Boundary(1, L, s.d_model, k, s.n_kv_heads, s.head_dim) for _ in range(3)]
        ids = []
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        enc_ms = []
        if profile:
            ctx.vla_profile(True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for i in range(n):
            f = fid[0]
            fid[0] += 1
            st = ctx.encoder_stream
            if i == 0:
                ev0.record(st)
            if images:
                ctx.vla_run_vision(f, imgs[i % 2], n_img, texts[i % 2], wl.text_tokens, frame_tok)
            else:
                ctx.vla_run_encoder(f, pats[i % 2], n_img, L_img, enc_out)
            if i == 0:
                ev1.record(st)
            ctx.vla_run_prefix(f, frame_tok if images else toks[i % 2], 1, L, k, bnds[i % 3])
            ids.append(f)
        for f in ids[-3:]:
            ctx.vla_wait_boundary(f, 120000)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t
        if profile:
            ctx.vla_profile(False)
        enc_ms.append(ev0.elapsed_time(ev1))
        times = [ctx.vla_frame_times(f) for f in ids]
        return wall * 1000.0 / n, times, enc_ms[0]

    results = {}
    for k in ks:
        run(k, args.warmup)
        prof = k == args.k
        ms, times, enc_ms = run(k, args.steps)
        if prof:
            # per-kernel event timing in a separate pass, so the event pairs
            # around every launch do not slow the headline frames
            run(k, args.steps, profile=True)
        foot = vb.vla_query_sizes(vb.stack_cfg(s, "bf16", max_tokens=L, max_batch=1, n_blocks=k), enc_cfg,
                                  1, L, k)
        tg = np.array([t[0] for t in times])
        tx = np.array([t[1] for t in times])
        r = {"ms_per_frame": round(ms, 3), "prefix_tokens_per_s": round(L / (ms / 1000.0), 1),
             "t_gpu_prefix_ms": round(float(np.mean(tg)), 3),
             "t_gpu_prefix_ms_median": round(float(np.median(tg)), 3),
             "t_gpu_prefix_ms_std": round(float(np.std(tg)), 3),
             "frames_timed": len(tg),
             "t_boundary_copy_ms": round(float(np.mean(tx)), 4),
             "d2h_gbs": round(L * s.d_model * 2 / (float(np.mean(tx)) / 1000) / 1e9, 1),
             "t_prefix_plus_handoff_ms": round(float(np.mean([t[2] for t in times])), 3),
             "t_encoder_ms": round(enc_ms, 3),
             "frame_tflops": round(frame_flops(wl, k, images) / 1e12, 3),
             "mfma_frac_of_bf16_peak": round(frame_flops(wl, k, images) / (ms / 1000.0) / 1e12 / PEAK_BF16_TFLOPS,
                                             4),
             "hbm_footprint_gib": round(foot[0] / 2 ** 30, 3),
             "hbm_footprint_note": "arena bytes with k resident decoder blocks (vla_query_sizes)",
             "handoff_bytes": foot[1] + foot[2]}
        if prof:
            classes = {}
            for kind, stk, nl in (("llm", vb.VLA_STACK_LLM, k), ("enc", vb.VLA_STACK_ENC, e.n_blocks)):
                work = class_work(wl, kind, k, images)
                for ci, cname in enumerate(vb.KERNEL_CLASSES):
                    tot, cnt = ctx.vla_profile_read(stk, ci)
                    if cnt == 0:
                        continue
                    ent = {"ms_total": round(tot, 4), "launches": cnt, "avg_us": round(tot / cnt * 1000, 2)}
                    if cname in work:
                        unit, per, group = work[cname]
                        avg_s = tot / cnt * group / 1000.0   # time of the launches the work covers
                        if unit == "flop":
                            ent["tflops"] = round(per / avg_s / 1e12, 1)
                            ent["frac"] = round(per / avg_s / 1e12 / PEAK_BF16_TFLOPS, 4)
                        else:
                            ent["gbs"] = round(per / avg_s / 1e9, 1)
                            ent["frac"] = round(per / avg_s / 1e9 / PEAK_HBM_GBS, 4)
                        ent["per_launch"] = per
                    classes["%s.%s" % (kind, cname)] = ent
            r["kernels"] = classes
        results[k] = r
        log("k=%d: %s" % (k, json.dumps({kk: v for kk, v in r.items() if kk != "kernels"})))

    head = results[args.k]
    kern = head["kernels"]
    dom_name = max((n for n in kern if "tflops" in kern[n] or "gbs" in kern[n]), key=lambda n: kern[n]["ms_total"])
    dom = kern[dom_name]
    roofline = {"kernel": dom_name, "bound": "mfma" if "tflops" in dom else "hbm",
                "achieved": dom.get("tflops", dom.get("gbs")), "peak": PEAK_BF16_TFLOPS if "tflops" in dom else PEAK_HBM_GBS,
                "unit": "TFLOP/s" if "tflops" in dom else "GB/s", "frac": dom["frac"],
                "traffic": profiled_traffic(dom_name),
                "per_launch": dom["per_launch"], "avg_launch_us": dom["avg_us"]}
    front = ("6 camera images 448x448 -> patch stem + ViT-L encoder + 2x2-merge MLP connector -> 1536 visual + "
             "512 text tokens" if images else "ViT-L encoder 6x1024")
    out = {
        "metric": "GPU-prefix tokens/s at boundary k=%d (frame: %s + 7B-shaped decoder blocks "
                  "[0,k) over 2048 tokens + boundary/KV handoff to pinned host)" % (args.k, front),
        "value": head["prefix_tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": head["ms_per_frame"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "sweep7b: encoder 24x ViT-L block (d=1024, 16x64, GELU 4096) over 6 images x 1024 "
                               "patches; decoder 7B-shaped blocks (d=4096, 32x128 MHA, SwiGLU 11008, RoPE) [0,k) "
                               "over 1x2048 tokens; bf16 weights N(0,0.02), inputs N(0,1)",
                   "k": args.k, "seq_len": L, "batch": 1, "n_img": n_img, "img_tokens": L_img,
                   "frame_input": args.frame},
        "mfma_frac_of_bf16_peak": head["mfma_frac_of_bf16_peak"],
        "hbm_context": {"resident_decoder_blocks": kmax, "arena_gib": round(ctx.arena_bytes / 2 ** 30, 3),
                        "hipMemGetInfo_delta_gib": round(mem_delta / 2 ** 30, 3)},
        "roofline": roofline,
        "kernels": kern,
        "sweep": {str(k): {kk: v for kk, v in r.items() if kk != "kernels"} for k, r in results.items()},
    }
    # the 7B-shaped prefix at L=1024, k=16 (the shorter causal prefill: O-proj
    # and down give 256 128x128 tiles, half the workgroup slots)
    if not args.no_legs:
        log("leg llm7b L=1024 k=16")
        out["llm7b_L1024_k16"] = prefix_leg(ctx, synth.CONFIGS["llm7b"], 1024, 16, args.steps, args.warmup,
                                            "the bench context's random-init 7B-shaped blocks")
        # what the <= 1e-2 parity mode costs at the headline shape: split
        # (hi + lo) activation operands into the QKV, gate/up and down GEMMs
        log("leg precision split, L=%d k=%d" % (L, args.k))
        ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_SPLIT)
        leg = prefix_leg(ctx, wl, L, args.k, args.steps, args.warmup,
                         "activation operands of the QKV, gate/up and down GEMMs split into hi + lo bf16")
        ctx.vla_set_precision(vb.VLA_STACK_LLM, vb.VLA_PREC_BF16)
        leg["vs_bf16_operands_ms"] = round(leg["t_gpu_prefix_ms"] / head["t_gpu_prefix_ms"], 3)
        out["precision_split_L%d_k%d" % (L, args.k)] = leg
    ctx.vla_destroy()
    if not args.no_legs:
        # the 0.5B-class GQA prefix: d=896, 14x64 heads over 2 KV heads, L=4096, k=12
        sw = synth.CONFIGS["small_llm"]
        log("leg small_llm L=%d k=%d" % (sw.seq, sw.k))
        sctx = vb.Context(llm=vb.stack_cfg(sw.llm, "bf16", max_tokens=sw.seq, max_batch=1, n_blocks=sw.k))
        for l in range(sw.k):
            sctx.vla_load_block_weights(vb.VLA_STACK_LLM, l, synth.llm_block_weights(sw, l))
        out["small_llm_L4096_k12"] = prefix_leg(sctx, sw, sw.seq, sw.k, args.steps, args.warmup,
                                                "random-init N(0,0.02) weights")
        sctx.vla_destroy()
    out["norm_large"] = norm_large()
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, args.k)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
