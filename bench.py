"""DMS decode-attention benchmark on one MI355X.

One step = one DMS decode step of every layer for the whole batch: append of
the new token (delayed release, slot recycling, page pops), the split-K
decode over the retained slots and the log-sum-exp combine, all through the
libdms C ABI.  The cache state is built beforehand through the library's own
chunk commits from seeded synthetic inputs.

Prints one JSON line.  `value` is the whole step's algorithmic retained-KV
bytes (every retained key and value row read once) divided by the step time,
in GB/s; `roofline` reports the same bytes against the decode kernel's own
duration, timed with HIP events around each launch.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# rocprofv3 summary of the decode kernel on the default workload
# rocprofv3 summaries of the decode kernel by (workload, page format)
TRAFFIC_PROFILES = {
    ("qwen-r1-32b-8x", "bf16"): "decode_kernel_qwen-r1-32b-8x.txt",
    ("qwen-r1-32b-8x", "fp8"): "decode_kernel_qwen-r1-32b-8x-fp8.txt",
    ("qwen-r1-7b-4x", "bf16"): "decode_kernel_qwen-r1-7b-4x.txt",
    ("qwen-r1-1.5b-8x", "bf16"): "decode_step_kernel_qwen-r1-1.5b-8x.txt",
}
LATENCY_STEPS = 50   # default steps timed one by one for the per-step distribution

# Synthetic stand-ins for the paper's reasoning-model shapes (Qwen-R1 family).
WORKLOADS = {
    "qwen-r1-32b-8x": dict(layers=64, batch=128, kv_heads=8, group=5, head_dim=128,
                           context=32768, window=256, p_evict=7 / 8, seed=3,
                           desc="Qwen-R1-32B-shaped DMS decode, 8 prompts x 16 chains, "
                                "context 32768, w=256, flags Bernoulli(7/8)"),
    "qwen-r1-1.5b-8x": dict(layers=28, batch=32, kv_heads=2, group=6, head_dim=128,
                            context=8192, window=256, p_evict=7 / 8, seed=1,
                            desc="Qwen-R1-1.5B-shaped DMS decode, context 8192, w=256, "
                                 "flags Bernoulli(7/8)"),
    "qwen-r1-7b-4x": dict(layers=28, batch=64, kv_heads=4, group=7, head_dim=128,
                          context=(4096, 32768), window=256, p_evict=3 / 4, seed=2,
                          desc="Qwen-R1-7B-shaped DMS decode, contexts uniform in "
                               "[4096, 32768], w=256, flags Bernoulli(3/4)"),
    # latent attention: one cached row of 512 latent + 64 rotary dims per
    # token, shared by all 16 query heads (DeepSeek-V2-Lite's attention shape)
    "deepseek-v2-lite-8x": dict(layers=27, batch=128, kv_heads=1, group=16, head_dim=576,
                                context=32768, window=256, p_evict=7 / 8, seed=4, kv_format=2,
                                desc="DeepSeek-V2-Lite-shaped latent-attention (MLA) DMS decode, "
                                     "absorbed form, 8 prompts x 16 chains, context 32768, w=256, "
                                     "flags Bernoulli(7/8)"),
    # the same rows shared by 128 query heads (DeepSeek-V2's attention shape)
    "deepseek-v2-8x": dict(layers=60, batch=128, kv_heads=1, group=128, head_dim=576,
                           context=32768, window=256, p_evict=7 / 8, seed=5, kv_format=2,
                           desc="DeepSeek-V2-shaped latent-attention (MLA) DMS decode, absorbed "
                                "form, 128 query heads, 8 prompts x 16 chains, context 32768, "
                                "w=256, flags Bernoulli(7/8)"),
}
MLA = 2            # kv_format of latent-attention pools
MLA_LATENT = 512   # output (value) dims of a latent-attention row
TRAFFIC_PROFILES_MLA = {
    "deepseek-v2-lite-8x": "decode_mla_kernel_deepseek-v2-lite-8x.txt",
    "deepseek-v2-8x": "decode_mla_kernel_deepseek-v2-8x.txt",
}
MFMA_BF16_PEAK_TFLOPS = 2500.0


def profiled_traffic(profile, sources):
    """HBM bytes per launch that a committed rocprofv3 summary measured
    (FETCH_SIZE and WRITE_SIZE, scaled by a copy kernel of known size), or
    None when the kernel's sources have changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    h = hashlib.sha256()
    for f in sources:
        with open(os.path.join(ROOT, "paper_2506_05345_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    fields = {}
    with open(path) as fh:
        for line in fh:
            key, sep, val = line.partition(": ")
            if sep:
                fields[key.strip()] = val.strip()
    if fields.get(f"source_sha256({', '.join(sources)})") != h.hexdigest():
        return None
    val = fields.get("traffic_bytes_per_launch")
    return int(val) if val else None


def decode_kernel_name(wl, quest_pages):
    """The launch that the decode kernel timing covers for this workload: the
    latent-attention kernel, the decode over Quest's selection (planned in the
    launch up to 1024 call heads), the fused small-call step (up to 128 call
    heads), or the planned decode kernel with the merge launch after it."""
    D, NH = wl["head_dim"], wl["batch"] * wl["kv_heads"]
    if wl.get("kv_format", 0) == MLA:
        return "decode_mla_kernel"
    planned = f"decode_kernel<{D}> + merge_kernel<{D}>"
    if quest_pages > 0:
        return f"decode_attended_kernel<{D}>" if NH <= 1024 else planned
    return f"decode_step_kernel<{D}>" if NH <= 128 else planned


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def row_bytes(wl):
    """Bytes read per retained token of one KV head: K and V rows in bf16,
    E4M3 codes plus one float32 scale per row in FP8 pages, or the one bf16
    row of a latent-attention cache."""
    D = wl["head_dim"]
    fmt = wl.get("kv_format", 0)
    return 2 * D + 8 if fmt == 1 else 2 * D if fmt == MLA else 2 * D * 2


def attend_flops(wl):
    """Matrix flops per retained token of one KV head in a decode step: each
    query head of the group scores the key (2 d) and adds the weighted value
    (2 d; the 512 latent dims of a latent row)."""
    D, g = wl["head_dim"], wl["group"]
    return g * (2 * D + 2 * (MLA_LATENT if wl.get("kv_format", 0) == MLA else D))


def contexts(wl, rng_seed):
    import numpy as np
    c = wl["context"]
    if isinstance(c, tuple):
        rng = np.random.default_rng(rng_seed)
        return rng.integers(c[0], c[1] + 1, size=wl["batch"]).astype(np.int64)
    return np.full(wl["batch"], c, dtype=np.int64)


def build(wl, steps_total, chunk_tokens, dev):
    """Allocate the cache and fill every layer's state with its context."""
    import numpy as np
    import torch

    import dms_synth as sy
    from paper_2506_05345_amd import dms

    B, H, g, D, w, p = (wl["batch"], wl["kv_heads"], wl["group"], wl["head_dim"],
                        wl["window"], wl["p_evict"])
    nl, seed = wl["layers"], wl["seed"]
    P = 64
    ctx = contexts(wl, seed)
    ctx_t = torch.as_tensor(ctx, device=dev)
    seqs = torch.arange(B, device=dev, dtype=torch.int64)
    heads = torch.arange(H, device=dev, dtype=torch.int64)
    # exact retained counts at decode start (flags are a pure function of the
    # coordinates), used only to size the page pool
    max_pages_head, pages_layer = 0, 0
    L0 = []
    for layer in range(nl):
        Lh = torch.zeros((B, H), dtype=torch.int64, device=dev)
        for p0 in range(0, int(ctx.max()), 8192):
            pos = torch.arange(p0, min(p0 + 8192, int(ctx.max())), device=dev)
            f = sy.flags_torch(seed, p, layer, seqs[:, None, None], heads[None, None, :],
                               pos[None, :, None], dev)
            keep = (pos[None, :, None] < (ctx_t[:, None, None] - w)) & (f == 0)
            Lh += keep.sum(dim=1)
        Lh += torch.clamp(ctx_t, max=w)[:, None]
        L0.append(Lh)
        need = torch.div(Lh + steps_total + P - 1, P, rounding_mode="floor")
        max_pages_head = max(max_pages_head, int(need.max()))
        pages_layer = max(pages_layer, int(need.sum()))
    # the state is built by chunk appends of up to 16 sequences at a time
    grp = min(B, 16)
    cfg = dms.make_config(nl, B, H, g, D, w, P, pages_layer + 8, max_pages_head + 1,
                          chunk_tokens * grp, kv_format=wl.get("kv_format", dms.DMS_KV_BF16),
                          quest_page_budget=wl.get("quest_pages", 0))
    mb, pb, wb, _ = dms.dms_layout(cfg)
    log(f"pool {pb * nl / 2**30:.1f} GiB ({pages_layer + 8} pages/layer), meta "
        f"{mb / 2**30:.2f} GiB, workspace {wb / 2**20:.1f} MiB")
    cache = dms.DmsCache(cfg, device=dev)
    gen = torch.Generator(device=dev)
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    t0 = time.perf_counter()
    for layer in range(nl):
        gen.manual_seed(seed * 1000 + layer)
        for g0 in range(0, B, grp):
            ids = np.arange(g0, min(B, g0 + grp))
            gsid, gseqs = sid[g0:g0 + len(ids)], seqs[g0:g0 + len(ids)]
            done = np.zeros(len(ids), np.int64)
            while (done < ctx[ids]).any():
                lens = np.minimum(chunk_tokens, ctx[ids] - done)
                cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
                T = int(cu[-1])
                k = torch.randn((T, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
                v = (None if wl.get("kv_format", 0) == MLA
                     else torch.randn((T, H, D), generator=gen, device=dev, dtype=torch.bfloat16))
                # flags of every sequence's next positions, varlen layout [T, H]
                lens_t = torch.as_tensor(lens, device=dev)
                seq_of = torch.repeat_interleave(gseqs, lens_t)
                start = torch.as_tensor(cu[:-1], device=dev, dtype=torch.int64)
                pos = (torch.arange(T, device=dev) - torch.repeat_interleave(start, lens_t)
                       + torch.as_tensor(done, device=dev)[seq_of - g0])
                f = sy.flags_torch(seed, p, layer, seq_of[:, None], heads[None, :], pos[:, None], dev)
                dms.dms_append_chunk(cache.ctx, layer, len(ids), gsid, torch.as_tensor(cu, device=dev),
                                     T, int(lens.max()), k, v, f)
                done += lens
        if layer % 8 == 7 or layer == nl - 1:
            torch.cuda.synchronize()
            log(f"built layers 0..{layer} ({time.perf_counter() - t0:.1f}s)")
    st = dms.dms_status(cache.ctx)
    if st != 0:
        raise RuntimeError(f"state build failed: {dms.dms_strerror(st)}")
    # the device's retained lengths must equal the closed form
    out = torch.empty((B, H), dtype=torch.int32, device=dev)
    for layer in range(nl):
        dms.dms_retained_lengths(cache.ctx, layer, B, sid, out)
        if not torch.equal(out.to(torch.int64), L0[layer]):
            raise RuntimeError(f"layer {layer}: retained lengths differ from the closed form")
    return cache, ctx, L0


class _Cycled:
    """Per-step inputs indexed [step, ...] over a smaller pool of steps."""

    def __init__(self, pool):
        self.pool, self.n = pool, pool.shape[0]

    def __getitem__(self, idx):
        return self.pool[(idx[0] % self.n, *idx[1:])]


def step_inputs(wl, ctx, steps_total, dev):
    """Per (step, layer) decode inputs and the retained length of every head
    at every step (closed form from the flags)."""
    import torch

    import dms_synth as sy
    B, H, g, D, w, p = (wl["batch"], wl["kv_heads"], wl["group"], wl["head_dim"],
                        wl["window"], wl["p_evict"])
    nl, seed = wl["layers"], wl["seed"]
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed * 7919 + 17)
    # queries: distinct for every step up to about 8 GB of them, then taken
    # again in turn (their values change neither the rows read nor the work;
    # 128-head latent queries are 1.1 GB per step)
    nq = max(1, min(steps_total, int(8e9 // (nl * B * H * g * D * 2))))
    q = _Cycled(torch.randn((nq, nl, B, H * g, D), generator=gen, device=dev, dtype=torch.bfloat16))
    k = torch.randn((steps_total, nl, B, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
    v = (None if wl.get("kv_format", 0) == MLA
         else torch.randn((steps_total, nl, B, H, D), generator=gen, device=dev, dtype=torch.bfloat16))
    ctx_t = torch.as_tensor(ctx, device=dev)
    seqs = torch.arange(B, device=dev, dtype=torch.int64)
    heads = torch.arange(H, device=dev, dtype=torch.int64)
    steps = torch.arange(steps_total, device=dev, dtype=torch.int64)
    flags = torch.empty((steps_total, nl, B, H), dtype=torch.uint8, device=dev)
    fresh = torch.empty((steps_total, nl, B, H), dtype=torch.int64, device=dev)
    for layer in range(nl):
        pos = ctx_t[None, :, None] + steps[:, None, None]          # [S, B, 1]
        flags[:, layer] = sy.flags_torch(seed, p, layer, seqs[None, :, None], heads[None, None, :],
                                         pos, dev)
        # token t takes a fresh slot unless t >= w and token t - w was flagged
        prev = sy.flags_torch(seed, p, layer, seqs[None, :, None], heads[None, None, :],
                              pos - w, dev)
        fresh[:, layer] = ((pos < w) | (prev == 0)).to(torch.int64)
    return q, k, v, flags, fresh


def cpu_baseline(wl, ctx, budget_s=12.0):
    """Time the CPU oracle's dense masked attention on sampled heads."""
    import numpy as np

    import dms_synth as sy
    from oracle import dense_dms_attention_head, fake_quantize_fp8, mla_attention
    from oracle import visible as key_visible

    B, H, g, D, w, p = (wl["batch"], wl["kv_heads"], wl["group"], wl["head_dim"],
                        wl["window"], wl["p_evict"])
    fp8 = wl.get("kv_format", 0) == 1
    mla = wl.get("kv_format", 0) == MLA
    nl, seed = wl["layers"], wl["seed"]
    rng = np.random.default_rng(12345)

    def _wide(heads, dims, width, positions):
        hh, dd = sy.wide_coords(heads, dims, width)
        return hh, positions, dd

    triples = [(int(rng.integers(nl)), int(rng.integers(B)), int(rng.integers(H))) for _ in range(6)]
    f32 = sy.bf16_bits_to_f32_np
    head_steps, bytes_equiv, elapsed = 0, 0, 0.0
    samples = []
    for (layer, s, h) in triples:
        T = int(ctx[s]) + 8
        pos = np.arange(T)
        fh = sy.flags_np(seed, p, layer, s, h, pos)
        qd = np.arange(D)[None, None, :]
        qh_ = (h * g + np.arange(g))[None, :, None]
        if mla:   # 576-wide rows and queries
            kh = f32(sy.token_vectors_np(seed, sy.STREAM_K, layer, s,
                                         *_wide(np.full((1, 1), h), np.arange(D)[None, :], D, pos[:, None])))
            vh = None
            qh = f32(sy.token_vectors_np(seed, sy.STREAM_Q, layer, s,
                                         *_wide(qh_, qd, D, pos[-8:][:, None, None])))
        else:
            kh = f32(sy.head_sequence_np(seed, sy.STREAM_K, layer, s, h, pos, D))
            vh = f32(sy.head_sequence_np(seed, sy.STREAM_V, layer, s, h, pos, D))
            if fp8:   # the stored (dequantized) rows
                kh, vh = fake_quantize_fp8(kh), fake_quantize_fp8(vh)
            qh = f32(sy.token_vectors_np(seed, sy.STREAM_Q, layer, s, qh_, pos[-8:][:, None, None], qd))
        samples.append((kh, vh, fh, qh, T))
    t_start = time.perf_counter()
    while elapsed < budget_s:
        for (kh, vh, fh, qh, T) in samples:
            for i in range(4):
                t = T - 8 + i
                t0 = time.perf_counter()
                if mla:
                    mask = np.asarray(key_visible(t, np.arange(t + 1), fh[:t + 1], w), dtype=bool)
                    mla_attention(qh[i], kh[:t + 1], np.broadcast_to(mask, (g, t + 1)), MLA_LATENT,
                                  1.0 / math.sqrt(D))
                else:
                    dense_dms_attention_head(qh[i:i + 1], kh[:t + 1], vh[:t + 1], fh[:t + 1], w, [t])
                elapsed += time.perf_counter() - t0
                head_steps += 1
                visible = min(w, t + 1) + int(np.sum(fh[: max(0, t - w + 1)] == 0))
                bytes_equiv += visible * row_bytes(wl)
        if time.perf_counter() - t_start > 4 * budget_s:
            break
    threads = os.cpu_count()
    blas = None
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        if info:
            threads = max(int(x.get("num_threads", 1)) for x in info)
            blas = ", ".join(sorted({f"{x.get('internal_api')} {x.get('version')}" for x in info
                                     if x.get("user_api") == "blas"})) or None
    except Exception:
        pass
    return {
        "value": bytes_equiv / elapsed / 1e9,
        "unit": "GB/s",
        "cores": threads,
        "host_cpus": os.cpu_count(),
        "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
        "numpy_blas": blas,
        "kind": "oracle",
        "sample": f"{head_steps} head-steps (one KV head, its {g} query heads, one decode "
                  f"position, dense float64 masked {'absorbed latent ' if mla else ''}attention over "
                  f"the full history{' of the dequantized FP8 rows' if fp8 else ''}) on "
                  f"{len(samples)} sampled (layer, sequence, KV head) triples; value = their "
                  f"retained-KV bytes / CPU time",
        "head_steps_per_s": head_steps / elapsed,
        "seconds": elapsed,
    }


def chunk_visible_counts(L0, pos, flags_back, w):
    """Keys visible to every query of a prefill chunk, per KV head.

    After a token's append the live slots of its head are exactly the keys
    visible to it, so the count at chunk token c is the head's retained count
    after appending tokens 0 .. c: the count before the chunk, L0 [n, H], plus
    one for every chunk token that took a fresh slot (position < w, or the
    token w positions earlier was kept).  pos [n, C] positions of the chunk
    tokens; flags_back [n, C, H] decisions of the tokens at pos - w (ignored
    where pos < w).  Returns int64 [n, C, H]."""
    import torch
    fresh = ((pos[..., None] < w) | (flags_back == 0)).to(torch.int64)
    return L0.to(torch.int64)[:, None, :] + torch.cumsum(fresh, dim=1)


def prefill_flops(visible_counts, group, head_dim):
    """Algorithmic flops of masked prefill: q.k and p.v over every visible
    (query, key) pair of every query head of the group, 4 d flops each."""
    return float(visible_counts.sum()) * group * 4 * head_dim


def mla_prefill_flops(visible_counts, group):
    """Algorithmic flops of latent-attention prefill: for every visible
    (query, key) pair of every query head, q . row over 576 dims and the
    weighted sum of the 512 latent dims, 2 flops per multiply-add."""
    return float(visible_counts.sum()) * group * 2 * (576 + MLA_LATENT)


def run_mla_prefill(args):
    """Latent-attention chunked prefill: a 4096-token DMS-masked chunk for each
    of 4 sequences on every layer, after 32768 tokens of context (flags
    Bernoulli(7/8), w = 256), DeepSeek-V2-Lite (16 query heads) or -V2 (128)
    shapes.  Queries and rows are random and shared by the layers of a step;
    flags are per layer and position."""
    import numpy as np
    import torch

    import dms_synth as sy
    from paper_2506_05345_amd import dms

    base = WORKLOADS[args.workload.replace("-prefill", "-8x")]
    C, B = 4096, 4
    wl = dict(base, batch=B)
    desc = (base["desc"].split(",")[0] + ": masked chunked prefill, a 4096-token chunk for each of 4 "
            "sequences on every layer after 32768 tokens of context, w=256, flags Bernoulli(7/8)")
    nl, g, w, p, seed = wl["layers"], wl["group"], wl["window"], wl["p_evict"], wl["seed"]
    dev = "cuda"
    S = args.warmup + args.steps
    cache, ctx, L0 = build(wl, S * C, C, dev)
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed * 31 + 7)
    q = torch.randn((B * C, g, 576), generator=gen, device=dev, dtype=torch.bfloat16)
    k = torch.randn((B * C, 1, 576), generator=gen, device=dev, dtype=torch.bfloat16)
    out = torch.empty((B * C, g, MLA_LATENT), dtype=torch.float32, device=dev)
    cu = torch.arange(B + 1, dtype=torch.int32, device=dev) * C
    seqs = torch.arange(B, device=dev)
    zero = torch.zeros(1, dtype=torch.int64, device=dev)
    ctx_t = torch.as_tensor(ctx, device=dev)

    def positions(st):
        return ctx_t[:, None] + st * C + torch.arange(C, device=dev)[None, :]      # [B, C]

    def flags_at(layer, pos):
        return sy.flags_torch(seed, p, layer, seqs[:, None, None], zero[None, None, :], pos[:, :, None], dev)

    flags = [[flags_at(layer, positions(st)).reshape(B * C, 1) for layer in range(nl)] for st in range(S)]
    for st in range(args.warmup):
        for layer in range(nl):
            dms.dms_prefill_chunk(cache.ctx, layer, B, sid, cu, B * C, C, q, k, None, flags[st][layer], out)
    torch.cuda.synchronize()
    log("warmup done")
    # algorithmic work of the timed steps: visible keys of every chunk query
    # (the retained count after its own append), stepping the closed form
    # from the device's retained lengths before the first timed chunk
    lens = torch.empty((B, 1), dtype=torch.int32, device=dev)
    Ls, flops = [], 0.0
    for layer in range(nl):
        dms.dms_retained_lengths(cache.ctx, layer, B, sid, lens)
        Ls.append(lens.to(torch.int64).clone())
    for st in range(args.warmup, S):
        pos = positions(st)
        for layer in range(nl):
            vis = chunk_visible_counts(Ls[layer], pos, flags_at(layer, pos - w), w)
            flops += mla_prefill_flops(vis, g)
            Ls[layer] = vis[:, -1, :]
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    dms.dms_profile_start(cache.ctx, args.steps * nl)
    torch.cuda.synchronize()
    ev0.record()
    for st in range(args.warmup, S):
        for layer in range(nl):
            dms.dms_prefill_chunk(cache.ctx, layer, B, sid, cu, B * C, C, q, k, None, flags[st][layer], out)
    ev1.record()
    torch.cuda.synchronize()
    kern_ms, launches = dms.dms_profile_stop(cache.ctx)[dms.DMS_PROFILE_PREFILL]
    st_code = dms.dms_status(cache.ctx)
    if st_code != 0:
        raise RuntimeError(f"prefill failed: {dms.dms_strerror(st_code)}")
    for layer in range(nl):
        dms.dms_retained_lengths(cache.ctx, layer, B, sid, lens)
        if not torch.equal(lens.to(torch.int64), Ls[layer]):
            raise RuntimeError(f"layer {layer}: retained lengths diverged from the closed form")
    if not torch.isfinite(out).all():
        raise RuntimeError("non-finite prefill output")
    step_ms = ev0.elapsed_time(ev1) / args.steps
    tflops = flops / args.steps / (step_ms * 1e-3) / 1e12
    call_us = 1e3 * kern_ms / max(launches, 1)
    res = {
        "metric": "DMS latent-attention chunked prefill: algorithmic TFLOP/s",
        "value": round(tflops, 1), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(step_ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": desc, "layers": nl, "batch": B, "chunk": C, "query_heads": g,
                   "row_dim": 576, "latent_dim": MLA_LATENT, "context": 32768, "window": w,
                   "p_evict": p},
        "prefill_tokens_per_s": round(B * C / (step_ms * 1e-3 / nl), 1),
        "roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "call_avg_us": round(call_us, 1),
                     "call_timing": "HIP events around each dms_prefill_chunk (list, tile copy and "
                                    "attention passes)",
                     "flops_per_call": round(flops / (args.steps * nl))},
    }
    print(json.dumps(res), flush=True)


TINY = dict(layers=1, batch=1, kv_heads=2, group=2, head_dim=64, window=16, page=64, context=512,
            decode=64, p_evict=0.5, seed=0)


def run_tiny(args):
    """The tiny configuration timed whole: one sequence (2 KV heads x group 2,
    d = 64, w = 16, flags Bernoulli(1/2)) prefilled with a 512-token masked
    chunk (dms_prefill_chunk: attention over the chunk and its commit), then
    64 decode steps (dms_decode_step), from an empty cache.  Each timed job
    starts with dms_seq_reset; HIP events around the whole job on the launch
    stream; eager launches (every call of the job is timed, host work
    included)."""
    import numpy as np
    import torch

    import dms_synth as sy
    from paper_2506_05345_amd import dms

    t = TINY
    H, g, D, w, C, ND = t["kv_heads"], t["group"], t["head_dim"], t["window"], t["context"], t["decode"]
    seed, p = t["seed"], t["p_evict"]
    T = C + ND
    pos = np.arange(T)
    flags = sy.flags_np(seed, p, 0, 0, np.arange(H)[None, :], pos[:, None]).astype(np.uint8)
    dim = np.arange(D)[None, None, :]
    pp = pos[:, None, None]
    k = sy.token_vectors_np(seed, sy.STREAM_K, 0, 0, np.arange(H)[None, :, None], pp, dim)
    v = sy.token_vectors_np(seed, sy.STREAM_V, 0, 0, np.arange(H)[None, :, None], pp, dim)
    q = sy.token_vectors_np(seed, sy.STREAM_Q, 0, 0, np.arange(H * g)[None, :, None], pp, dim)
    dev = "cuda:0"

    def bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    qd, kd, vd = bf16(q), bf16(k), bf16(v)
    fd = torch.from_numpy(flags).to(dev)
    cfg = dms.make_config(num_layers=1, max_seqs=1, num_kv_heads=H, group_size=g, head_dim=D, window=w,
                          page_size=t["page"], num_pages=32, max_pages_per_head=16, max_chunk_tokens=C)
    cache = dms.DmsCache(cfg)
    sid = torch.zeros(1, dtype=torch.int32, device=dev)
    cu = torch.tensor([0, C], dtype=torch.int32, device=dev)
    out_pf = torch.empty((C, H * g, D), dtype=torch.float32, device=dev)
    out_dc = torch.empty((ND, 1, H * g, D), dtype=torch.float32, device=dev)
    st = torch.cuda.current_stream()

    def job():
        dms.dms_seq_reset(cache.ctx, 0, 1, sid)
        dms.dms_prefill_chunk(cache.ctx, 0, 1, sid, cu, C, C, qd[:C], kd[:C], vd[:C], fd[:C], out_pf)
        for j in range(ND):
            x = C + j
            dms.dms_decode_step(cache.ctx, 0, 1, sid, qd[x:x + 1], kd[x:x + 1], vd[x:x + 1], fd[x:x + 1],
                                out_dc[j])

    for _ in range(args.warmup):
        job()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    times = []
    for _ in range(args.steps):
        e0.record(st)
        job()
        e1.record(st)
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    if dms.dms_status(cache.ctx) != 0:
        raise RuntimeError(f"device status {dms.dms_status(cache.ctx)}")
    if not (torch.isfinite(out_pf).all() and torch.isfinite(out_dc).all()):
        raise RuntimeError("non-finite outputs")
    ms = float(np.mean(times))
    res = {
        "metric": "tiny configuration timed whole: 512-token masked prefill + 64 decode steps, ms per job",
        "value": round(ms, 4), "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "tiny: 1 sequence, 2 KV heads x group 2, d=64, w=16, flags Bernoulli(1/2), "
                               "seed 0; 512-token prefill chunk then 64 decode steps", "layers": 1, "batch": 1,
                   "kv_heads": H, "query_heads": H * g, "head_dim": D, "window": w, "context": C,
                   "decode_steps": ND, "parallelism": "single GPU", "launch": "eager (every call of the job)"},
        "job_ms": {"mean": round(ms, 4), "p10": round(float(np.percentile(times, 10)), 4),
                   "p50": round(float(np.percentile(times, 50)), 4),
                   "p90": round(float(np.percentile(times, 90)), 4)},
        "decode_tok_per_s": round(ND / (ms * 1e-3), 1),
    }
    cnt = torch.zeros(H, dtype=torch.int32, device=dev)
    dms.dms_retained_lengths(cache.ctx, 0, 1, sid, cnt)
    torch.cuda.synchronize()
    res["retained_after_job"] = [int(x) for x in cnt.cpu()]
    # after token T - 1: the last w tokens plus every unflagged older one
    expect = [int(((pos > T - 1 - w) | (flags[:, h] == 0)).sum()) for h in range(H)]
    if res["retained_after_job"] != expect:
        raise RuntimeError(f"retained lengths {res['retained_after_job']} differ from the closed form {expect}")
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = tiny_cpu_baseline(q, k, v, flags, g, w, C, ND)
    print(json.dumps(res), flush=True)


def tiny_cpu_baseline(q, k, v, flags, g, w, C, ND):
    """The oracle's dense float64 masked attention for the same job: every
    chunk query, then every decode query over the full history."""
    import os
    import time

    import numpy as np

    import dms_synth as sy
    from oracle import dense_dms_attention

    f32 = sy.bf16_bits_to_f32_np
    qf, kf, vf = f32(q), f32(k), f32(v)
    t0 = time.perf_counter()
    dense_dms_attention(qf[:C], kf[:C], vf[:C], flags[:C], w, g)
    for j in range(ND):
        x = C + j
        dense_dms_attention(qf[x:x + 1], kf[:x + 1], vf[:x + 1], flags[:x + 1], w, g, t_query=np.array([x]))
    sec = time.perf_counter() - t0
    return {"value": round(1e3 * sec, 3), "unit": "ms", "cores": 1, "kind": "oracle",
            "sample": "the whole job once (512 chunk queries, then 64 decode queries over the full history)",
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


STRESS = dict(layers=64, batch=32, kv_heads=8, group=5, head_dim=128, prefill_seqs=4,
              chunk=4096, ctx_lo=1024, ctx_hi=131072)


def run_stress(args):
    """Heterogeneous 32B-shaped step: a 4096-token DMS-masked prefill chunk for
    4 sequences and a decode step for the other 28, on every layer; per-(layer,
    sequence, head) eviction rates ~ Beta(7,1), contexts log-uniform in
    [1K, 128K].  Prefill inputs (q/k/v values) are shared by the layers of a
    step; flags are per layer."""
    import numpy as np
    import torch

    import dms_synth as sy
    from paper_2506_05345_amd import dms

    cfgw = STRESS
    nl, B, H, g, D, C = (cfgw["layers"], cfgw["batch"], cfgw["kv_heads"], cfgw["group"],
                         cfgw["head_dim"], cfgw["chunk"])
    w = args.window
    seed = 4 if w == 64 else 5
    dev = "cuda:0"
    P = 64
    rng = np.random.default_rng(seed)
    ctx = np.exp(rng.uniform(np.log(cfgw["ctx_lo"]), np.log(cfgw["ctx_hi"]), size=B)).astype(np.int64)
    npf = cfgw["prefill_seqs"]
    pf = np.arange(B - npf, B)
    dc = np.arange(B - npf)
    S = args.warmup + args.steps
    final = ctx.copy()
    final[pf] += S * C
    final[dc] += S
    thr = torch.as_tensor(np.stack([sy.beta71_rates_np(seed, l, np.arange(B)[:, None],
                                                       np.arange(H)[None, :]) for l in range(nl)]),
                          device=dev)                                        # [nl, B, H]
    seqs_t = torch.arange(B, device=dev)
    heads_t = torch.arange(H, device=dev)

    def flags(layer, seq_t, pos_t):
        """flags of (seq_t[i], head h, pos_t[i]) -> [len, H] uint8"""
        return sy.flags_rate_torch(seed, thr[layer][seq_t[:, None], heads_t[None, :]], layer,
                                   seq_t[:, None], heads_t[None, :], pos_t[:, None], dev)

    # exact retained length of every head after every appended position is
    # L(t) = min(w, t+1) + #{kept j <= t - w}; size the pool for the end state
    max_pages, pages = 0, 0
    for layer in range(nl):
        need = torch.zeros((B, H), dtype=torch.int64, device=dev)
        for s in range(B):
            T = int(final[s])
            kept = 0
            for p0 in range(0, max(0, T - w), 65536):
                pos = torch.arange(p0, min(p0 + 65536, T - w), device=dev)
                kept = kept + (flags(layer, torch.full_like(pos, s), pos) == 0).sum(dim=0)
            need[s] = (min(w, T) + kept + P - 1) // P
        max_pages = max(max_pages, int(need.max()))
        pages = max(pages, int(need.sum()))
    fp8 = args.kv_format == "fp8"
    cfg = dms.make_config(nl, B, H, g, D, w, P, pages + 64, max_pages + 2, C * B,
                          kv_format=dms.DMS_KV_FP8 if fp8 else dms.DMS_KV_BF16)
    cache = dms.DmsCache(cfg, device=dev)
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    t0 = time.perf_counter()
    for layer in range(nl):
        done = np.zeros(B, np.int64)
        while (done < ctx).any():
            lens = np.minimum(C, ctx - done)
            cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
            T = int(cu[-1])
            k = torch.randn((T, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
            v = torch.randn((T, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
            seq_of = torch.as_tensor(np.repeat(np.arange(B), lens), device=dev)
            pos = torch.as_tensor(np.concatenate([np.arange(done[i], done[i] + lens[i]) for i in range(B)]),
                                  device=dev)
            dms.dms_append_chunk(cache.ctx, layer, B, sid, torch.as_tensor(cu, device=dev), T,
                                 int(lens.max()), k, v, flags(layer, seq_of, pos))
            done += lens
    torch.cuda.synchronize()
    log(f"stress state built ({time.perf_counter() - t0:.1f}s)")
    if dms.dms_status(cache.ctx) != 0:
        raise RuntimeError("state build failed")
    # step inputs: values shared by layers, flags per layer and step
    pf_sid = torch.as_tensor(pf.astype(np.int32), device=dev)
    dc_sid = torch.as_tensor(dc.astype(np.int32), device=dev)
    cu_pf = torch.arange(npf + 1, dtype=torch.int32, device=dev) * C
    qp = torch.randn((npf * C, H * g, D), generator=gen, device=dev, dtype=torch.bfloat16)
    kp = torch.randn((npf * C, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
    vp = torch.randn((npf * C, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
    qd = torch.randn((len(dc), H * g, D), generator=gen, device=dev, dtype=torch.bfloat16)
    kd = torch.randn((len(dc), H, D), generator=gen, device=dev, dtype=torch.bfloat16)
    vd = torch.randn((len(dc), H, D), generator=gen, device=dev, dtype=torch.bfloat16)
    out_p = torch.empty((npf * C, H * g, D), device=dev)
    out_d = torch.empty((len(dc), H * g, D), device=dev)
    fp, fd = {}, {}
    flops, dbytes = np.zeros(S), np.zeros(S)
    lens = torch.empty((B, H), dtype=torch.int32, device=dev)
    for layer in range(nl):
        dms.dms_retained_lengths(cache.ctx, layer, B, sid, lens)
        L = lens.to(torch.int64)
        for st in range(S):
            # prefill positions of this step and their retained counts
            ppos = torch.cat([torch.arange(int(ctx[s]) + st * C, int(ctx[s]) + (st + 1) * C, device=dev)
                              for s in pf])
            pseq = torch.as_tensor(np.repeat(pf, C), device=dev)
            fp[layer, st] = flags(layer, pseq, ppos)
            prev = flags(layer, pseq, ppos - w).view(npf, C, H)
            Lq = chunk_visible_counts(L[torch.as_tensor(pf, device=dev)], ppos.view(npf, C), prev, w)
            flops[st] += prefill_flops(Lq, g, D)
            L[torch.as_tensor(pf, device=dev)] = Lq[:, -1]
            dpos = torch.as_tensor(ctx[dc] + st, device=dev)
            dseq = torch.as_tensor(dc, device=dev)
            fd[layer, st] = flags(layer, dseq, dpos)
            prev = flags(layer, dseq, dpos - w)
            freshd = ((dpos[:, None] < w) | (prev == 0)).to(torch.int64)
            L[torch.as_tensor(dc, device=dev)] += freshd
            dbytes[st] += float(L[torch.as_tensor(dc, device=dev)].sum()) * row_bytes(
                dict(head_dim=D, kv_format=1 if fp8 else 0))

    def step(st):
        for layer in range(nl):
            dms.dms_prefill_chunk(cache.ctx, layer, npf, pf_sid, cu_pf, npf * C, C, qp, kp, vp,
                                  fp[layer, st], out_p)
            dms.dms_decode_step(cache.ctx, layer, len(dc), dc_sid, qd, kd, vd, fd[layer, st], out_d)

    for st in range(args.warmup):
        step(st)
    torch.cuda.synchronize()
    dms.dms_profile_start(cache.ctx, 2 * nl * args.steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for st in range(args.warmup, S):
        step(st)
    e1.record()
    torch.cuda.synchronize()
    prof = dms.dms_profile_stop(cache.ctx)
    if dms.dms_status(cache.ctx) != 0:
        raise RuntimeError("stress step failed")
    step_ms = e0.elapsed_time(e1) / args.steps
    dms_ms, dn = prof[dms.DMS_PROFILE_DECODE]
    pms, pn = prof[dms.DMS_PROFILE_PREFILL]
    fl = flops[args.warmup:].sum()
    db = dbytes[args.warmup:].sum()
    res = {
        "metric": "DMS heterogeneous mixed step: prefill TFLOP/s and decode KV GB/s",
        "value": round(fl / (pms * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"kv_format": args.kv_format,
                   "workload": "32B-shaped heterogeneous stress: 64 layers, 32 sequences x 8 KV "
                               "heads (group 5), per-head eviction rate ~ Beta(7,1), contexts "
                               "log-uniform in [1K, 128K]; per step a 4096-token masked prefill "
                               "for 4 sequences and a decode step for 28",
                   "window": w, "mean_context": float(ctx.mean())},
        "prefill": {"kernel_avg_us": round(1e3 * pms / pn, 1),
                    "algorithmic_tflop_per_launch": round(fl / pn / 1e12, 4),
                    "achieved_tflops": round(fl / (pms * 1e-3) / 1e12, 2),
                    "peak_tflops": 2500.0,
                    "frac": round(fl / (pms * 1e-3) / 1e12 / 2500.0, 4)},
        "decode": {"kernel_avg_us": round(1e3 * dms_ms / dn, 1),
                   "kv_gb_per_launch": round(db / dn / 1e9, 4),
                   "achieved_gbs": round(db / (dms_ms * 1e-3) / 1e9, 1),
                   "frac_of_hbm_peak": round(db / (dms_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "decode_tok_per_s": round(len(dc) / (step_ms * 1e-3), 1),
    }
    print(json.dumps(res), flush=True)


TRAIN = dict(batch=2, seq_len=8192, kv_heads=8, group=5, head_dim=128, window=256, tau=0.1,
             seed=21)


def run_train(args):
    """Training-time DMS attention of one Qwen-R1-32B-shaped layer (8 KV heads,
    group 5, d = 128) on a micro-batch of 2 sequences x 8192 tokens (the
    retrofitting context of the R1-distilled models), window 256: Gumbel-
    sigmoid decisions from synthetic logits, masked attention forward, its
    backward (dq, dk, dv, dalpha) and the Gumbel-sigmoid backward.  FLOPs are
    algorithmic over the causal (query, key) pairs: 2 products of 2 d per pair
    and query head forward, 5 backward; the mask evicts nothing during
    training, so every causal pair is computed."""
    import torch
    from paper_2506_05345_amd import dms

    c = TRAIN
    B, T, H, g, D, w = c["batch"], c["seq_len"], c["kv_heads"], c["group"], c["head_dim"], c["window"]
    Hq = H * g
    dev = "cuda:0"
    gen = torch.Generator(device=dev)
    gen.manual_seed(c["seed"])
    q = torch.randn((B, T, Hq, D), generator=gen, device=dev, dtype=torch.bfloat16)
    k = torch.randn((B, T, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
    v = torch.randn((B, T, H, D), generator=gen, device=dev, dtype=torch.bfloat16)
    dout = torch.randn((B, T, Hq, D), generator=gen, device=dev, dtype=torch.bfloat16)
    logits = torch.randn((B, T, H), generator=gen, device=dev) * 2.0
    u = torch.rand((B, T, H), generator=gen, device=dev).clamp_(1e-6, 1 - 1e-6)
    dal_in = torch.randn((B, T, H), generator=gen, device=dev)
    cfg = dms.make_train_config(B, T, H, g, D, w)
    ws = torch.empty(dms.dms_train_workspace(cfg), dtype=torch.uint8, device=dev)
    alpha = torch.empty((B, T, H), device=dev)
    out = torch.empty((B, T, Hq, D), device=dev)
    lse = torch.empty((B, Hq, T), device=dev)
    dq = torch.empty((B, T, Hq, D), device=dev)
    dk = torch.empty((B, T, H, D), device=dev)
    dv = torch.empty((B, T, H, D), device=dev)
    dal = torch.empty((B, T, H), device=dev)
    dlog = torch.empty((B, T, H), device=dev)
    n = B * T * H
    tau = c["tau"]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]

    def step(timed=None):
        if timed is not None:
            timed[0].record()
        dms.dms_gumbel_sigmoid_fwd(n, logits, u, tau, alpha)
        if timed is not None:
            timed[1].record()
        dms.dms_train_attention_fwd(cfg, q, k, v, alpha, out, lse, ws)
        if timed is not None:
            timed[2].record()
        dms.dms_train_attention_bwd(cfg, q, k, v, alpha, out, lse, dout, dq, dk, dv, dal, ws)
        if timed is not None:
            timed[3].record()
        # the decision gradient of the step plus an independent upstream term
        dms.dms_gumbel_sigmoid_bwd(n, alpha, dal, tau, dlog)
        if timed is not None:
            timed[4].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    tot = [0.0] * 4
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step(ev)
        torch.cuda.synchronize()
        for i in range(4):
            tot[i] += ev[i].elapsed_time(ev[i + 1])
    e1.record()
    torch.cuda.synchronize()
    if not (torch.isfinite(dq).all() and torch.isfinite(dal).all() and torch.isfinite(dlog).all()):
        raise RuntimeError("non-finite training gradients")
    step_ms = sum(tot) / args.steps
    pairs = B * Hq * T * (T + 1) / 2
    f_fwd, f_bwd = 4 * D * pairs, 10 * D * pairs
    fwd_ms, bwd_ms = tot[1] / args.steps, tot[2] / args.steps
    peak = MFMA_PEAK_FLOPS / 1e12
    res = {
        "metric": "DMS training attention (continuous decisions): fwd+bwd TFLOP/s",
        "value": round((f_fwd + f_bwd) / (step_ms * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "Qwen-R1-32B-shaped layer, 2 sequences x 8192 tokens, 8 KV heads "
                               "x group 5, d=128, w=256, Gumbel-sigmoid tau=0.1 over N(0, 2) logits",
                   "batch": B, "seq_len": T, "kv_heads": H, "query_heads": Hq, "window": w},
        "forward": {"ms": round(fwd_ms, 3), "algorithmic_tflop": round(f_fwd / 1e12, 4),
                    "achieved_tflops": round(f_fwd / (fwd_ms * 1e-3) / 1e12, 2),
                    "frac": round(f_fwd / (fwd_ms * 1e-3) / 1e12 / peak, 4)},
        "backward": {"ms": round(bwd_ms, 3), "algorithmic_tflop": round(f_bwd / 1e12, 4),
                     "achieved_tflops": round(f_bwd / (bwd_ms * 1e-3) / 1e12, 2),
                     "frac": round(f_bwd / (bwd_ms * 1e-3) / 1e12 / peak, 4)},
        "gumbel_us": {"fwd": round(1e3 * tot[0] / args.steps, 1),
                      "bwd": round(1e3 * tot[3] / args.steps, 1)},
        "roofline": {"bound": "mfma", "peak": peak, "unit": "TFLOP/s",
                     "achieved": round((f_fwd + f_bwd) / (step_ms * 1e-3) / 1e12, 2),
                     "frac": round((f_fwd + f_bwd) / (step_ms * 1e-3) / 1e12 / peak, 4),
                     "traffic": None,
                     "kernel_timing": "HIP events on the launch stream around each entry point"},
    }
    print(json.dumps(res), flush=True)


# Attention shapes of the paper's models (layers, KV heads, group, head dim)
# and the dense-model sizes (public model configurations) that the App. I
# latency estimate needs: hidden size d, MLP width d_ff, vocabulary V.
SWEEP_SHAPES = {
    "qwen-r1-1.5b": dict(layers=28, kv_heads=2, group=6, head_dim=128, d=1536, d_ff=8960, V=151936),
    "qwen-r1-7b": dict(layers=28, kv_heads=4, group=7, head_dim=128, d=3584, d_ff=18944, V=152064),
    "qwen-r1-32b": dict(layers=64, kv_heads=8, group=5, head_dim=128, d=5120, d_ff=27648, V=152064),
    "qwen3-8b": dict(layers=36, kv_heads=8, group=4, head_dim=128, d=4096, d_ff=12288, V=151936),
}
HBM_BYTES = 288e9
MFMA_PEAK_FLOPS = 2.5e15


def app_i_estimate(sh, B, L):
    """App. I step model with MI355X peaks: FLOPS(B, L), Reads(B, L) (the
    "4 d d_ff" read term taken as 4 d d_kv) and latency = max(compute, reads);
    returns (latency s, share of it that is KV-cache reads, weight bytes)."""
    n, d, dff, V = sh["layers"], sh["d"], sh["d_ff"], sh["V"]
    dkv = sh["kv_heads"] * sh["head_dim"]
    flops = n * B * (6 * d * dff + 4 * d * d + 4 * d * dkv + 4 * d * L) + 2 * B * d * V
    weights = n * (6 * d * dff + 4 * d * d + 4 * d * dkv) + 2 * d * V
    kv = n * 4 * B * L * dkv
    lat = max(flops / MFMA_PEAK_FLOPS, (weights + kv) / (HBM_PEAK_GBS * 1e9))
    return lat, (kv / (HBM_PEAK_GBS * 1e9)) / lat, weights


def measure_decode(wl, steps, warmup, dev):
    """Build a workload's cache, replay `steps` decode steps of every layer as
    one HIP graph; returns step ms, KV bytes per step, mean retained length."""
    import torch
    from paper_2506_05345_amd import dms
    S = warmup + steps
    cache, ctx, L0 = build(wl, S, 4096, dev)
    q, k, v, flags, fresh = step_inputs(wl, ctx, S, dev)
    B, nl, D = wl["batch"], wl["layers"], wl["head_dim"]
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    Dout = MLA_LATENT if wl.get("kv_format", 0) == MLA else D
    out = torch.empty((nl, B, wl["kv_heads"] * wl["group"], Dout), dtype=torch.float32, device=dev)

    def run_step(s):
        for layer in range(nl):
            dms.dms_decode_step(cache.ctx, layer, B, sid, q[s, layer], k[s, layer],
                                None if v is None else v[s, layer],
                                flags[s, layer], out[layer])

    for s in range(warmup):
        run_step(s)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for s in range(warmup, S):
            run_step(s)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    if dms.dms_status(cache.ctx) != 0:
        raise RuntimeError("decode failed")
    Lstep = torch.stack(L0)[None] + torch.cumsum(fresh, dim=0)
    kv = float(Lstep[warmup:].sum()) * row_bytes(wl) / steps
    mean_L = float(Lstep[warmup:].double().mean())
    ms = e0.elapsed_time(e1) / steps
    del graph, q, k, v, flags, fresh, out
    cache.close()
    torch.cuda.empty_cache()
    return ms, kv, mean_L


def run_sweep(args):
    """Attention-only sweeps on one GPU (one JSON line per point):
    fig4-r1: step latency vs context, Qwen-R1 1.5B / 7B / 32B shapes, batch 32;
    fig4-qwen3: the same for the Qwen3-8B shape at batch 32 / 64 / 128;
    maxbatch: the largest batch whose KV cache fits next to the weights in
    288 GB, at CR 1 / 4 / 8, and its decode tokens/s (attention only).
    CR c is emulated by eviction probability 1 - 1/c; points whose cache does
    not fit in HBM are reported as such."""
    import torch
    dev = "cuda:0"
    fmt = 1 if args.kv_format == "fp8" else 0
    points = []
    if args.sweep == "fig4-r1":
        for name in ("qwen-r1-1.5b", "qwen-r1-7b", "qwen-r1-32b"):
            for ctxlen in (4096, 8192, 16384, 32768):
                for cr in (1, 4, 8):
                    points.append((name, 32, ctxlen, cr, 256))
    elif args.sweep == "fig4-qwen3":
        for B in (32, 64, 128):
            for ctxlen in (4096, 8192, 16384, 32768):
                for cr in (1, 4, 8):
                    points.append(("qwen3-8b", B, ctxlen, cr, 512))
    else:
        ctxlen = 32768
        for name in SWEEP_SHAPES:
            w = 512 if name == "qwen3-8b" else 256
            sh = SWEEP_SHAPES[name]
            for cr in (1, 4, 8):
                p = 1 - 1 / cr
                Lr = min(w, ctxlen) + (1 - p) * max(0, ctxlen - w)
                per_seq = sh["layers"] * sh["kv_heads"] * Lr * row_bytes(dict(sh, kv_format=fmt)) * 1.03
                _, _, weights = app_i_estimate(sh, 1, 0)
                budget = HBM_BYTES - weights - 24e9       # weights, inputs, workspace, margin
                points.append((name, int(budget // per_seq), ctxlen, cr, w))
    for (name, B, ctxlen, cr, w) in points:
        sh = SWEEP_SHAPES[name]
        p = 1 - 1 / cr
        Lr = min(w, ctxlen) + (1 - p) * max(0, ctxlen - w)
        kv_est = sh["layers"] * B * sh["kv_heads"] * Lr * row_bytes(dict(sh, kv_format=fmt))
        lat, share, weights = app_i_estimate(sh, B, Lr)
        rec = {"sweep": args.sweep, "model_shape": name, "batch": B, "context": ctxlen, "cr": cr,
               "window": w, "kv_format": args.kv_format, "kv_cache_gb": round(kv_est / 1e9, 2),
               "app_i_latency_ms": round(1e3 * lat, 3), "app_i_kv_share": round(share, 3)}
        if kv_est + weights + 16e9 > HBM_BYTES:
            rec["status"] = "KV cache does not fit in HBM next to the weights"
            print(json.dumps(rec), flush=True)
            continue
        wl = dict(layers=sh["layers"], batch=B, kv_heads=sh["kv_heads"], group=sh["group"],
                  head_dim=sh["head_dim"], context=ctxlen, window=w, p_evict=p, seed=11,
                  kv_format=fmt)
        ms, kv, mean_L = measure_decode(wl, args.steps, args.warmup, dev)
        rec.update({"status": "measured", "attn_ms_per_step": round(ms, 3),
                    "kv_gb_per_step": round(kv / 1e9, 3),
                    "achieved_gbs": round(kv / (ms * 1e-3) / 1e9, 1),
                    "decode_tok_per_s": round(B / (ms * 1e-3), 1),
                    "mean_retained": round(mean_L, 1)})
        print(json.dumps(rec), flush=True)
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen-r1-32b-8x",
                    choices=sorted(WORKLOADS) + ["tiny", "qwen-r1-32b-stress", "qwen-r1-32b-train",
                                                 "deepseek-v2-lite-prefill", "deepseek-v2-prefill"])
    ap.add_argument("--window", type=int, default=256, choices=[64, 256],
                    help="window of the heterogeneous stress workload")
    ap.add_argument("--chunk", type=int, default=4096)
    ap.add_argument("--quest-pages", type=int, default=0,
                    help="decode workloads: attend only this many pages (64 slots) per head, chosen "
                         "by Quest's bound (page retrieval within the retained set)")
    ap.add_argument("--kv-format", choices=["bf16", "fp8"], default="bf16",
                    help="page format of the decode workloads (fp8: E4M3 rows with power-of-two scales)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--latency-steps", type=int, default=LATENCY_STEPS,
                    help="decode workloads: further steps timed one by one (own HIP graph each) for "
                         "the per-step p10/p50/p90; 0 skips them")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run a 1 GiB device copy first (reference kernel for HBM counters)")
    ap.add_argument("--eager", action="store_true",
                    help="launch the timed steps one by one instead of replaying a HIP graph")
    ap.add_argument("--sweep", choices=["fig4-r1", "fig4-qwen3", "maxbatch"],
                    help="attention-only sweeps (one JSON line per point) instead of the benchmark")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; the DMS decode path "
                                   "has no multi-GPU mode (--gpus must be 1)"}))
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2506_05345_amd import dms

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.sweep:
        run_sweep(args)
        return
    if args.calibrate_copy:
        # plain copy of known size: reads 1 GiB, writes 1 GiB
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.workload == "tiny":
        run_tiny(args)
        return
    if args.workload == "qwen-r1-32b-stress":
        run_stress(args)
        return
    if args.workload.endswith("-prefill"):
        run_mla_prefill(args)
        return
    if args.workload == "qwen-r1-32b-train":
        run_train(args)
        return
    wl = dict(WORKLOADS[args.workload])
    if wl.get("kv_format", 0) == MLA and (args.kv_format != "bf16" or args.quest_pages > 0):
        print(json.dumps({"error": "latent-attention pools hold bf16 rows and attend every "
                                   "retained row (no --kv-format fp8, no --quest-pages)"}))
        sys.exit(2)
    if args.kv_format == "fp8":
        wl["kv_format"] = dms.DMS_KV_FP8
        wl["desc"] += ", FP8 E4M3 KV pages"
    quest = args.quest_pages > 0
    if quest:
        wl["quest_pages"] = args.quest_pages
        wl["desc"] += f", Quest page retrieval: {args.quest_pages} pages of 64 slots per head"
    S = args.warmup + 2 * args.steps + args.latency_steps
    cache, ctx, L0 = build(wl, S, args.chunk, dev)
    q, k, v, flags, fresh = step_inputs(wl, ctx, S, dev)
    B, H, g, D, nl = wl["batch"], wl["kv_heads"], wl["group"], wl["head_dim"], wl["layers"]
    sid = torch.arange(B, dtype=torch.int32, device=dev)
    mla = wl.get("kv_format", 0) == MLA
    out = torch.empty((nl, B, H * g, MLA_LATENT if mla else D), dtype=torch.float32, device=dev)
    # retained length of every head when step s attends (after its append)
    Lstep = torch.stack(L0)[None] + torch.cumsum(fresh, dim=0)        # [S, nl, B, H]
    kv_bytes = Lstep.sum(dim=(1, 2, 3)).to(torch.float64) * row_bytes(wl)  # per step, all layers

    def run_step(s):
        for layer in range(nl):
            dms.dms_decode_step(cache.ctx, layer, B, sid, q[s, layer], k[s, layer],
                                None if v is None else v[s, layer],
                                flags[s, layer], out[layer])

    for s in range(args.warmup):
        run_step(s)
    torch.cuda.synchronize()
    log("warmup done")
    # The timed steps: every layer's decode step, captured once into a HIP
    # graph (as a serving loop would) and replayed once.
    t_lo, t_hi = args.warmup, args.warmup + args.steps
    graph = None
    if not args.eager:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for s in range(t_lo, t_hi):
                run_step(s)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    log("timed steps captured" if graph is not None else "timed steps: eager")
    t0 = time.perf_counter()
    ev0.record()
    if graph is not None:
        graph.replay()
    else:
        for s in range(t_lo, t_hi):
            run_step(s)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    log("timed steps done; kernel-timing pass")
    # Decode-kernel duration: HIP events recorded by the library around every
    # decode launch of an eager pass over the next `steps` steps (events inside
    # a captured graph only mark dependencies on this runtime).
    k_lo, k_hi = t_hi, t_hi + args.steps
    dms.dms_profile_start(cache.ctx, args.steps * nl)
    if quest:
        # page retrieval: the bytes a launch reads are the live slots of the
        # pages it selected, exported after every launch (outside its events)
        Bq, P = args.quest_pages, 64
        sel_p = torch.empty((nl, B * H, Bq), dtype=torch.int32, device=dev)
        sel_c = torch.empty((nl, B * H), dtype=torch.int32, device=dev)
        attended = []
        for s in range(k_lo, k_hi):
            for layer in range(nl):
                dms.dms_decode_step(cache.ctx, layer, B, sid, q[s, layer], k[s, layer],
                                None if v is None else v[s, layer],
                                    flags[s, layer], out[layer])
                dms.dms_quest_selection(cache.ctx, B, sel_p[layer], sel_c[layer])
            Ls = Lstep[s].reshape(nl, B * H)
            npg = (Ls + P - 1) // P
            cnt = sel_c.to(torch.int64)
            last = torch.gather(sel_p.to(torch.int64), 2, (cnt - 1).clamp(min=0)[..., None])[..., 0]
            lq = cnt * P - torch.where(last == npg - 1, npg * P - Ls, torch.zeros_like(Ls))
            attended.append(torch.where(npg <= Bq, Ls, lq).sum(dim=1).to(torch.float64))   # per layer
        attended = torch.stack(attended)                                                  # [steps, nl]
    else:
        for s in range(k_lo, k_hi):
            run_step(s)
    torch.cuda.synchronize()
    kern_ms, launches = dms.dms_profile_stop(cache.ctx)[dms.DMS_PROFILE_DECODE]
    log("kernel-timing pass done")
    if launches != args.steps * nl:
        raise RuntimeError(f"timing events recorded {launches} of {args.steps * nl} decode launches")
    step_ms = ev0.elapsed_time(ev1) / args.steps
    st = dms.dms_status(cache.ctx)
    if st != 0:
        raise RuntimeError(f"decode failed: {dms.dms_strerror(st)}")
    # the device bookkeeping must have followed the closed form through every step
    lens = torch.empty((B, H), dtype=torch.int32, device=dev)
    for layer in range(nl):
        dms.dms_retained_lengths(cache.ctx, layer, B, sid, lens)
        if not torch.equal(lens.to(torch.int64), Lstep[k_hi - 1, layer]):
            raise RuntimeError(f"layer {layer}: retained lengths diverged from the closed form")
    per_step_bytes = float(kv_bytes[t_lo:t_hi].sum()) / args.steps
    per_launch_bytes = float(kv_bytes[k_lo:k_hi].sum()) / (args.steps * nl)
    if quest:
        # attended bytes, measured on the eager pass that follows the timed steps
        per_launch_bytes = float(attended.mean()) * row_bytes(wl)
        per_step_bytes = per_launch_bytes * nl
    value = per_step_bytes / (step_ms * 1e-3) / 1e9
    kern_avg_ms = kern_ms / max(launches, 1)
    achieved = per_launch_bytes / (kern_avg_ms * 1e-3) / 1e9
    mean_L = float(Lstep[t_lo:t_hi].double().mean())
    # per-step latency distribution: args.latency_steps further steps, each
    # captured as its own graph and replayed once between HIP events
    lat_ms = []
    n_lat = args.latency_steps
    if not args.eager and n_lat > 0:
        l_lo = k_hi
        graphs = []
        for s in range(l_lo, l_lo + n_lat):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                run_step(s)
            graphs.append(gr)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_lat + 1)]
        torch.cuda.synchronize()
        evs[0].record()
        for i, gr in enumerate(graphs):
            gr.replay()
            evs[i + 1].record()
        torch.cuda.synchronize()
        lat_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(n_lat)]
        log(f"per-step latency of {n_lat} steps done")
        del graphs
        st = dms.dms_status(cache.ctx)
        if st != 0:
            raise RuntimeError(f"decode failed: {dms.dms_strerror(st)}")
        for layer in range(nl):
            dms.dms_retained_lengths(cache.ctx, layer, B, sid, lens)
            if not torch.equal(lens.to(torch.int64), Lstep[l_lo + n_lat - 1, layer]):
                raise RuntimeError(f"layer {layer}: retained lengths diverged from the closed form")
    traffic, traffic_profile = None, None
    if not quest and not mla and (args.workload, args.kv_format) in TRAFFIC_PROFILES:
        traffic_profile = TRAFFIC_PROFILES[(args.workload, args.kv_format)]
        traffic = profiled_traffic(traffic_profile, ["dms_common.h", "dms_fp8.h", "dms_decode.hip"])
    elif mla and args.workload in TRAFFIC_PROFILES_MLA:
        traffic_profile = TRAFFIC_PROFILES_MLA[args.workload]
        traffic = profiled_traffic(traffic_profile, ["dms_common.h", "dms_mla.hip"])
    # the same launches' matrix work (the roofline's other axis)
    launch_tflops = per_launch_bytes / row_bytes(wl) * attend_flops(wl) / (kern_avg_ms * 1e-3) / 1e12
    res = {
        "metric": "DMS decode attn: achieved KV HBM GB/s (% of peak) + decode tok/s at 8x",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if args.kv_format == "bf16" else "fp8-e4m3 kv, bf16 mfma",
        "data": "synthetic",
        "config": {
            "workload": wl["desc"],
            "kv_format": "mla (bf16 rows)" if mla else args.kv_format,
            "quest_pages": args.quest_pages,
            "layers": nl, "batch": B, "kv_heads": H, "query_heads": H * g,
            "head_dim": D, **({"latent_dim": MLA_LATENT, "rope_dim": D - MLA_LATENT} if mla else {}), "window": wl["window"], "p_evict": wl["p_evict"],
            "context": wl["context"] if not isinstance(wl["context"], tuple) else list(wl["context"]),
            "mean_retained_tokens": round(mean_L, 1),
            "effective_compression": round(float((ctx.mean() + t_lo + args.steps / 2) / mean_L), 2),
            "parallelism": "single GPU",
            "launch": "eager" if args.eager else "hip graph (all timed steps)",
        },
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 1),
        "decode_tok_per_s": round(B / (step_ms * 1e-3), 1),
        "wall_ms_per_step": round(1e3 * wall / args.steps, 4),
        "step_latency_ms": ({"steps": len(lat_ms), "how": "one HIP graph per step, HIP events between replays",
                             "p10": round(float(np.percentile(lat_ms, 10)), 4),
                             "p50": round(float(np.percentile(lat_ms, 50)), 4),
                             "p90": round(float(np.percentile(lat_ms, 90)), 4)} if lat_ms else None),
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "traffic_source": "profiles/" + traffic_profile if traffic is not None else None,
            "kernel": decode_kernel_name(wl, args.quest_pages),
            "kernel_timing": "HIP events around each decode launch, eager pass of the next "
                             f"{args.steps} steps",
            "kernel_avg_us": round(1e3 * kern_avg_ms, 2),
            "bytes_per_launch": int(per_launch_bytes),
            "flops_per_byte": round(attend_flops(wl) / row_bytes(wl), 1),
            "mfma_tflops": round(launch_tflops, 1),
            "mfma_frac": round(launch_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        },
    }
    if quest:
        res["attended_tokens_per_head"] = round(float(attended.mean()) / (B * H), 1)
    if not args.no_cpu_baseline and not quest:
        log("timing the CPU oracle")
        res["cpu_baseline"] = cpu_baseline(wl, ctx)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
