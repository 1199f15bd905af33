#!/usr/bin/env python3
"""Benchmark of the compressed-KV decode hot path on one MI355X.

One step = the whole hot path over one batch of synthetic input:
latent_append of the workload's new tokens (z = x [L_K | L_v] into the paged
cache) followed by one decode over every sequence's full context (fold,
split-K attention over the latents, fixed-order merge, up-projection).
Default workload: long-context MHA, 32 heads x 128, one sequence of 131072
tokens whose last 512 are appended in the step, 6 key groups with ranks
summing to 1536, value rank 2048, bf16 latents.

Prints one JSON line.  `value` is decode tokens/s (sequences decoded per
second of step time) with every input resident in HBM before timing starts.
`roofline` covers the dominant kernel (the split-K attention kernel, or the
value pass when a call takes the two-pass kernels), timed with HIP events
stamped by its own dispatch; `decode_call` is the whole decode call (fold,
attention, merge, up-projection) against the same peak; `copy_peak` is a
2 GiB device copy timed the same way, a measured second denominator.
`cpu_baseline` times the fp64 CPU oracle on a bounded sample of the same
workload.  Latent pools are touched in turn (`pool_copies`) so that more
than 512 MB pass between two reads of one pool: the 256 MB last-level cache
cannot serve them.  With the default workload the GQA layer (4 sequences x
32768 tokens) is timed in the same run and reported under `also`, with its
own step time, roofline, decode call and CPU baseline.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--profile-every", type=int, default=4,
                    help="record the split-kernel HIP events on every n-th timed step (an "
                         "event pair costs a few microseconds of dispatch gap)")
    ap.add_argument("--workload", default="mha_long_t128k")
    ap.add_argument("--split-tokens", type=int, default=0)
    ap.add_argument("--head-slices", type=int, default=0)
    ap.add_argument("--decode-waves", type=int, default=0)
    ap.add_argument("--decode-passes", type=int, default=0, choices=[0, 1, 2],
                    help="decode kernels: 0 chosen per call, 1 single-pass split kernel, "
                         "2 two-pass score and value kernels")
    ap.add_argument("--queries", type=int, default=1,
                    help="causal queries a sequence in each decode (speculative verification / "
                         "chunked prefill); 1 is plain decode")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--also", default="auto",
                    help="a second workload timed in the same run and reported under 'also' "
                         "(auto: the GQA layer when the default long-context layer is timed; "
                         "none: no second workload)")
    ap.add_argument("--pool-copies", type=int, default=0,
                    help="latent pool copies touched in turn (0: enough for > 512 MB a rotation, "
                         "so steps stream from HBM rather than the 256 MB last-level cache)")
    ap.add_argument("--decode-only", action="store_true",
                    help="time the decode alone (no latent append in the step)")
    ap.add_argument("--dense", action="store_true",
                    help="time the uncompressed bf16 KV decode baseline on the workload's shape")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one device copy of this many MiB before timing (a known-size "
                         "kernel for scaling hardware traffic counters)")
    ap.add_argument("--rope", type=float, default=None, metavar="BASE",
                    help="time the rotary decode (keys rebuilt per token and turned by their "
                         "position, planes at angle pos * BASE^(-2i/d_h)) instead of the "
                         "position-free one")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--offline", choices=["cka", "calib"], default=None,
                    help="time an offline compression contraction instead of the decode path: "
                         "cka = centred Gram of 32 heads x 128 activations over 2048 samples plus "
                         "the CKA head similarity; calib = calibration Gram X^T X, hidden 4096, "
                         "8192 samples")
    return ap.parse_args()


MFMA_F32_PEAK_TFLOPS = 157.3
MFMA_BF16_PEAK_TFLOPS = 2500.0


def main_offline(args, torch):
    """Offline Gram contractions (fp32 MFMA) against the fp32 MFMA peak."""
    import numpy as np
    from paper_2607_24331_amd import gram, head_similarity
    if args.offline == "cka":
        h, d, N = 32, 128, 2048
        cols, center = h * d, True
        name = "cka_h32_d128_s2048"
    else:
        h = d = None
        N, cols, center = 8192, 4096, False
        name = "calib_m4096_s8192"
    g = torch.Generator(device="cuda")
    g.manual_seed(4242)
    A = torch.randn((N, cols), generator=g, device="cuda") + 0.25
    G = torch.empty((cols, cols), dtype=torch.float32, device="cuda")
    S = torch.empty((h, h), dtype=torch.float32, device="cuda") if h else None

    def step():
        gram(A, center=center, out=G)
        if h:
            head_similarity(G, h, d, out=S)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    K = args.steps
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(K):
        step()
    t1.record()
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / K
    # the Gram tile kernel alone: an uncentred launch is that one kernel
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    for a, b in ev:
        a.record()
        gram(A, center=False, out=G)
        b.record()
    torch.cuda.synchronize()
    kern_ms = sum(a.elapsed_time(b) for a, b in ev) / K
    flops = float(N) * cols * (cols + 1)          # the n(n+1)/2 distinct entries, 2 flops a term
    rec = {
        "metric": ("offline CKA head similarity: Gram TFLOP/s" if h
                   else "offline calibration Gram TFLOP/s"),
        "value": flops / (ms_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded N(0,1) + 0.25 samples)",
        "config": {"workload": name, "samples": N, "cols": cols, "centred": center,
                   "heads": h, "head_dim": d},
        "roofline": {"kernel": "gram_tiles (fp32 MFMA)", "bound": "mfma",
                     "achieved": flops / (kern_ms * 1e-3) / 1e12, "peak": MFMA_F32_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": flops / (kern_ms * 1e-3) / 1e12 / MFMA_F32_PEAK_TFLOPS,
                     "traffic": None, "kernel_ms": kern_ms, "flops_per_launch": flops},
    }
    if not args.no_cpu_baseline:
        from oracle import calibrate as ocal
        from oracle import compress as oc
        An = A.double().cpu().numpy()
        t = time.perf_counter()
        if h:
            oc.head_similarity(An, h, d)
        else:
            ocal.gram(An)
        dt = time.perf_counter() - t
        rec["cpu_baseline"] = {
            "value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": _blas_threads(),
            "kind": "oracle",
            "sample": ("oracle head_similarity over the full input (fp64 numpy: per-pair CKA)"
                       if h else "oracle gram over the full input (fp64 numpy X^T X)"),
            "seconds": dt}
    print(json.dumps(rec), flush=True)


def _blas_threads():
    """Threads of the BLAS numpy calls into (the oracle's matrix products)."""
    try:
        import numpy  # noqa: F401  (loads the BLAS)
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()
                    if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        return len(os.sched_getaffinity(0))


def device_inputs(wl, plan, torch, Q=1):
    """Synthetic device tensors of the workload's shapes (seeded)."""
    from workloads.inputs import random_pool_fill
    dev = "cuda"
    g = torch.Generator(device=dev)
    g.manual_seed(1000 + wl.seed)
    tdt = plan.torch_dtype
    pool = random_pool_fill(wl.total_pages, plan.page_elems, wl.dtype, seed=wl.seed, device=dev)
    pages = wl.pages_per_seq
    table = torch.zeros((wl.batch, wl.max_pages), dtype=torch.int32)
    pos = 0
    for b, n in enumerate(pages):
        table[b, :n] = torch.arange(pos, pos + n, dtype=torch.int32)
        pos += n
    d = dict(
        pool=pool,
        page_table=table.to(dev),
        seq_lens=torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev),
        q=torch.randn((wl.batch, Q, wl.num_q_heads, wl.head_dim) if Q > 1
                      else (wl.batch, wl.num_q_heads, wl.head_dim), generator=g, device=dev),
        R_keys=(torch.randn(plan.key_factor_elems, generator=g, device=dev) * 0.05).to(tdt),
        R_value=(torch.randn((wl.value_rank, wl.kv_dim), generator=g, device=dev) * 0.02).to(tdt),
    )
    if wl.append_tokens:
        d["x"] = torch.randn((wl.append_tokens, wl.hidden), generator=g, device=dev).to(tdt)
        d["L_keys"] = (torch.randn((wl.key_rank_total, wl.hidden), generator=g, device=dev)
                       / math.sqrt(wl.hidden)).to(tdt)       # [out, in] layout
        d["L_value"] = (torch.randn((wl.value_rank, wl.hidden), generator=g, device=dev)
                        / math.sqrt(wl.hidden)).to(tdt)
        p0 = wl.prefill_lens[0]
        posn = torch.arange(p0, p0 + wl.append_tokens)
        d["slot"] = (table[0, posn // 64].long() * 64 + posn % 64).to(dev)
    return d


def _auto_split(plan, wl, max_ctx):
    """Split size the library picks when none is given (reported only)."""
    if plan.geometry["mfma_path"]:
        J = plan.geometry["head_slices"]
        L = -(-wl.batch * max_ctx * J // 256)
        return max(64, -(-L // 64) * 64)
    return 1024


def algorithmic_bytes(wl):
    """Bytes the method must move per step (see the design notes)."""
    s = wl.elem_bytes
    ctx = sum(wl.seq_lens)
    latent = ctx * (wl.key_rank_total + wl.value_rank) * s
    sizes = wl.group_sizes
    factors = (sum(r * h * wl.head_dim for r, h in zip(wl.group_rank, sizes))
               + wl.value_rank * wl.kv_dim) * s
    qo = 2 * wl.batch * wl.num_q_heads * wl.head_dim * 4
    append = 0
    if wl.append_tokens:
        R = wl.key_rank_total + wl.value_rank
        append = (wl.append_tokens * wl.hidden + wl.hidden * R + wl.append_tokens * R) * s
    value_latent = ctx * wl.value_rank * s
    return dict(latent=latent, value_latent=value_latent, factors=factors, q_out=qo, append=append,
                decode_total=latent + factors + qo)


KERNEL_SOURCES = ("paper_2607_24331_amd/csrc/decode_mfma.hip", "paper_2607_24331_amd/csrc/plan.cpp",
                  "paper_2607_24331_amd/csrc/internal.h")
ROPE_KERNEL_SOURCES = ("paper_2607_24331_amd/csrc/rope.hip", "paper_2607_24331_amd/csrc/plan.cpp",
                       "paper_2607_24331_amd/csrc/internal.h")
PASS_KERNEL_SOURCES = ("paper_2607_24331_amd/csrc/decode_pass.hip", "paper_2607_24331_amd/csrc/plan.cpp",
                       "paper_2607_24331_amd/csrc/internal.h")


def sources_of(kernel):
    """The sources whose hash a counter summary of `kernel` is tied to."""
    if kernel == "rope_scores":
        return ROPE_KERNEL_SOURCES
    if kernel in ("value_pages", "value_shared", "score_pages"):
        return PASS_KERNEL_SOURCES
    return KERNEL_SOURCES


def kernel_sources_sha256(sources=KERNEL_SOURCES):
    import hashlib
    h = hashlib.sha256()
    root = os.path.dirname(os.path.abspath(__file__))
    for rel in sources:
        with open(os.path.join(root, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(wl, launch, Q=1, kernel="split_mfma"):
    """HBM bytes per launch of the dominant kernel (the split kernel, or the
    rotary key rebuild) from the committed counter summary (FETCH_SIZE and
    WRITE_SIZE, each scaled by the same counter's reading for a plain device
    copy of known size), or None when there is no summary for this workload
    and launch shape, or the kernel sources changed since the counters were
    taken."""
    root = os.path.dirname(os.path.abspath(__file__))
    tag = wl.name if Q == 1 else f"{wl.name}_q{Q}"
    path = os.path.join(root, "profiles", f"{kernel}_{tag}_counters.md")
    sources = sources_of(kernel)
    if not os.path.exists(path):
        return None
    keys = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.split(":", 1)[0].strip() in (
                    "workload", "launch", "kernel_sources_sha256", "traffic_bytes_per_launch"):
                k, v = line.split(":", 1)
                keys[k.strip()] = v.strip()
    if (keys.get("workload") != wl.name or keys.get("launch") != launch
            or keys.get("kernel_sources_sha256") != kernel_sources_sha256(sources)):
        return None
    try:
        return int(keys["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(wl, budget_s, Q=1, with_append=True, rope_base=None):
    """The oracle, as it stands, on a bounded sample of the same workload:
    the append of all new tokens plus whole-context decode of as many heads
    as fit the time budget; the step time is extrapolated to every (sequence,
    query, head) row."""
    import numpy as np
    from oracle import append as oappend
    from oracle import attention as oattn
    from oracle import rope as orope
    from oracle.bookkeeping import book_for
    from workloads.inputs import make_factors
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()
                       if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    bk = book_for(wl)
    g = np.random.default_rng(wl.seed)
    L_keys, L_value, R_blocks, R_value = make_factors(wl)
    b = 0
    T = wl.seq_lens[b]
    Zk = g.standard_normal((T, wl.key_rank_total), dtype=np.float32)
    Zv = g.standard_normal((T, wl.value_rank), dtype=np.float32)
    q = g.standard_normal((wl.batch, wl.num_q_heads, wl.head_dim))
    t_app = 0.0
    if wl.append_tokens and with_append:
        x = g.standard_normal((wl.append_tokens, wl.hidden), dtype=np.float32)
        t0 = time.perf_counter()
        oappend.latents(x, L_keys, L_value, wl.dtype)
        t_app = time.perf_counter() - t0
    heads_done, t_dec = 0, 0.0
    for h in range(wl.num_q_heads):
        t0 = time.perf_counter()
        if rope_base is None:
            oattn.decode_head(q[b, h], Zk, Zv, R_blocks, R_value, bk, h, chunk=16384)
        else:
            orope.decode_head(q[b, h], Zk, Zv, R_blocks, R_value, bk, h, rope_base, chunk=16384)
        t_dec += time.perf_counter() - t0
        heads_done += 1
        if t_dec + t_app >= budget_s:
            break
    rows = wl.batch * Q * wl.num_q_heads
    # every (sequence, head) row of a full step costs about T_b / T_0 of a sampled row
    ctx_scale = sum(wl.seq_lens) / (wl.batch * T)
    step_s = t_app + t_dec / heads_done * rows * ctx_scale
    return {
        "value": wl.batch * Q / step_s,
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": ((f"oracle append of {wl.append_tokens} tokens ({t_app:.2f} s) + "
                    if wl.append_tokens and with_append else "")
                   + ("fp64 rotary decode of " if rope_base is not None else "fp64 decode of ")
                   + 
                   f"{heads_done} of {rows} (sequence, query, head) rows at {T} context tokens "
                   f"({t_dec:.2f} s), extrapolated to the full step ({step_s:.1f} s)"),
    }


def dense_cpu_baseline(wl, budget_s):
    """The oracle's uncompressed decode, as it stands, on a bounded sample: one
    sequence of the workload's head shape at a shorter context, extrapolated
    linearly in context length over the whole batch."""
    import numpy as np
    from oracle import dense as odense
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()
                       if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    g = np.random.default_rng(wl.seed)
    Hkv, d = wl.num_kv_heads, wl.head_dim
    T = min(max(wl.seq_lens), 4096)
    table = np.arange(-(-T // 64), dtype=np.int32)[None, :]
    pool = odense.new_pool(table.shape[1], Hkv, d)
    odense.pack(pool, table, 0, 0, g.standard_normal((T, Hkv, d)), g.standard_normal((T, Hkv, d)))
    q = g.standard_normal((1, wl.num_q_heads, d))
    t0 = time.perf_counter()
    odense.decode(q, pool, table, [T], Hkv)
    dt = time.perf_counter() - t0
    step_s = dt * sum(wl.seq_lens) / T
    return {"value": wl.batch / step_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"oracle uncompressed decode of one sequence of {T} tokens, all "
                       f"{wl.num_q_heads} heads ({dt:.2f} s), extrapolated to "
                       f"{sum(wl.seq_lens)} context tokens ({step_s:.1f} s)")}


def main_dense(args, torch, wl):
    """The uncompressed baseline: decode over a bf16 K/V cache of the workload's
    shape, same head map, pages and timing as the compressed path."""
    from paper_2607_24331_amd import dense_decode, dense_page_elems, dense_workspace_bytes
    Hq, Hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    pe = dense_page_elems(Hkv, d)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2000 + wl.seed)
    pool = torch.empty((wl.total_pages, pe), dtype=torch.bfloat16, device="cuda")
    for i in range(0, wl.total_pages, 256):       # fill in slices: no full-size fp32 temporary
        j = min(wl.total_pages, i + 256)
        pool[i:j] = torch.randn((j - i, pe), generator=gen, device="cuda").to(torch.bfloat16)
    pages = wl.pages_per_seq
    table = torch.zeros((wl.batch, wl.max_pages), dtype=torch.int32)
    pos = 0
    for b, n in enumerate(pages):
        table[b, :n] = torch.arange(pos, pos + n, dtype=torch.int32)
        pos += n
    table = table.cuda()
    seq_lens = torch.tensor(wl.seq_lens, dtype=torch.int32, device="cuda")
    q = torch.randn((wl.batch, Hq, d), generator=gen, device="cuda")
    max_ctx = max(wl.seq_lens)
    out = torch.empty((wl.batch, Hq, d), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(256, dense_workspace_bytes(Hq, Hkv, d, args.split_tokens, wl.batch, max_ctx)),
                     dtype=torch.uint8, device="cuda")

    def step(ev=None):
        dense_decode(q, pool, table, seq_lens, max_ctx, Hkv, split_tokens=args.split_tokens, out=out,
                     workspace=ws, events=ev)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    K = args.steps
    every = max(1, args.profile_every)
    ev = {k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for k in range(K) if k % every == 0}
    for a, b in ev.values():
        a.record()
        b.record()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record()
    for k in range(K):
        step(ev.get(k))
    t_end.record()
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / K
    kern_ms = sum(a.elapsed_time(b) for a, b in ev.values()) / len(ev)
    print(f"[bench] dense {wl.name}: {ms_step:.4f} ms/step, split kernel {kern_ms:.4f} ms",
          file=sys.stderr, flush=True)
    kv_bytes = sum(wl.seq_lens) * Hkv * d * 2 * 2
    achieved = kv_bytes / (kern_ms * 1e-3) / 1e9
    rec = {
        "metric": "uncompressed bf16 KV decode attention tokens/s (baseline; achieved HBM GB/s in roofline)",
        "value": wl.batch / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random keys, values and queries of the workload's shapes)",
        "config": {"workload": wl.name, "kv_cache": "uncompressed bf16", "batch": wl.batch,
                   "context_tokens": sum(wl.seq_lens), "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": d, "split_tokens": args.split_tokens or "auto"},
        "context_tokens_per_s": sum(wl.seq_lens) / (ms_step * 1e-3),
        "roofline": {"kernel": "uncompressed split-K attention (dense_split)", "bound": "hbm",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None, "kernel_ms": kern_ms,
                     "bytes_per_launch": kv_bytes, "kernel_launches_timed": len(ev)},
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = dense_cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU (got --gpus {args.gpus}); "
              "the multi-GPU sharding is a design note only", file=sys.stderr)
        sys.exit(2)
    import torch
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import paper_2607_24331_amd  # noqa: F401  (fails loudly when the library is not built)
    from workloads import make_workload

    if args.offline:
        return main_offline(args, torch)
    wl = make_workload(args.workload)
    if args.dense:
        return main_dense(args, torch, wl)
    copy = copy_peak(torch)
    rec = bench_compressed(args, torch, wl, copy)
    also = args.also
    if also == "auto":
        also = ("gqa8b_b4_t32k" if args.workload == "mha_long_t128k" and args.queries == 1
                and args.rope is None else "none")
    if also != "none":
        sub = bench_compressed(args, torch, make_workload(also), copy)
        for k in ("metric", "n_gpus", "higher_is_better", "scaling", "vs_baseline", "data", "warmup"):
            sub.pop(k, None)
        rec["also"] = {also: sub}
    print(json.dumps(rec), flush=True)


def copy_peak(torch, gib=2, reps=10):
    """Device-to-device copy of `gib` GiB timed with HIP events: the bytes read
    plus written over the time, a measured second denominator beside the
    published 8 TB/s."""
    n = gib << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    torch.cuda.empty_cache()
    gbs = 2.0 * n / (ms * 1e-3) / 1e9
    print(f"[bench] device copy of {gib} GiB: {ms:.3f} ms, {gbs:.0f} GB/s (read + write)",
          file=sys.stderr, flush=True)
    return {"gbs": gbs, "bytes_read_and_written": 2 * n, "ms": ms,
            "kind": f"device-to-device copy of {gib} GiB (torch copy_), read + written bytes / time"}


def bench_compressed(args, torch, wl, copy):
    """Time the compressed-KV step on one workload; returns its JSON record."""
    from paper_2607_24331_amd import Plan, decode, decode_rope, latent_append
    from workloads.inputs import random_pool_fill
    plan = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                wl.group_rank, wl.value_rank, wl.dtype, args.split_tokens, args.head_slices,
                args.decode_waves, args.queries, args.decode_passes)
    mfma = bool(plan.geometry["mfma_path"])
    Q = args.queries
    inp = device_inputs(wl, plan, torch, Q)
    max_ctx = max(wl.seq_lens)
    info = plan.launch_info(wl.batch, max_ctx)
    split_used = info["split_tokens"]
    out = torch.empty(tuple(inp["q"].shape), dtype=torch.float32, device="cuda")
    rope = args.rope is not None
    if rope:
        if Q != 1 or not mfma:
            sys.exit("bench.py: --rope runs one query a sequence on the bf16 MFMA path")
        split_used = min(plan.split_tokens or _auto_split(plan, wl, max_ctx), 1024)
        ws = torch.empty(max(256, plan.rope_workspace_bytes(wl.batch, max_ctx)), dtype=torch.uint8,
                         device="cuda")
    else:
        ws = plan.new_workspace(wl.batch, max_ctx)
    # Pool copies touched in turn, so that a step streams from HBM and not from
    # the 256 MB last-level cache (MALL): enough copies for > 512 MB a rotation.
    pool_bytes = wl.total_pages * plan.page_elems * wl.elem_bytes
    copies = args.pool_copies or max(1, math.ceil(600e6 / pool_bytes))
    pools = [inp["pool"]] + [random_pool_fill(wl.total_pages, plan.page_elems, wl.dtype,
                                              seed=wl.seed + 100 * c, device="cuda")
                             for c in range(1, copies)]
    append = bool(wl.append_tokens) and not args.decode_only

    def step(k, with_append=True):
        pool = pools[k % copies]
        if append and with_append:
            latent_append(plan, inp["x"], inp["L_keys"], inp["L_value"], inp["slot"], pool)
        if rope:
            decode_rope(plan, inp["q"], pool, inp["page_table"], inp["seq_lens"], max_ctx,
                        inp["R_keys"], inp["R_value"], rope_base=args.rope, out=out, workspace=ws)
        else:
            decode(plan, inp["q"], pool, inp["page_table"], inp["seq_lens"], max_ctx,
                   inp["R_keys"], inp["R_value"], out=out, workspace=ws)

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    print(f"[bench] {wl.name}: warmup done ({args.warmup} steps, {copies} pool cop"
          f"{'y' if copies == 1 else 'ies'})", file=sys.stderr, flush=True)

    K = args.steps
    every = max(1, args.profile_every)
    sampled = [k for k in range(K) if k % every == 0]
    ev = {k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for k in sampled}
    for a, b in ev.values():               # create the underlying HIP events
        a.record()
        b.record()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for k in range(K):
        if k in ev:
            plan.set_profile_events(*ev[k])
        elif k - 1 in ev:
            plan.set_profile_events(None, None)
        step(k)
    t_end.record()
    torch.cuda.synchronize()
    plan.set_profile_events(None, None)
    ms_step = t_start.elapsed_time(t_end) / K
    kern_ms = sum(a.elapsed_time(b) for a, b in ev.values()) / len(ev)
    # the decode call alone (no append), same rotation of pools
    if append:
        t_start.record()
        for k in range(K):
            step(k, with_append=False)
        t_end.record()
        torch.cuda.synchronize()
        ms_decode = t_start.elapsed_time(t_end) / K
    else:
        ms_decode = ms_step
    two_pass = info["kernels"] == 2
    print(f"[bench] {wl.name}: timed {K} steps: {ms_step:.4f} ms/step, decode call {ms_decode:.4f} ms, "
          f"{'key-rebuild' if rope else ('value-pass' if two_pass else 'split')} kernel {kern_ms:.4f} ms "
          f"(HIP events on {len(ev)} of the {K} steps)", file=sys.stderr, flush=True)

    nb = algorithmic_bytes(wl)
    launch = (f"split_tokens={split_used} head_slices={plan.geometry['head_slices']} "
              f"decode_waves={plan.geometry['decode_waves']}")
    if Q > 1:
        launch += f" queries_per_seq={Q}"
    # the two-pass value kernel: waves over pages for one row slice, all
    # waves over each page for several (the slices sharing one walk)
    vkern = "value_shared" if info["head_slices"] > 1 else "value_pages"
    if two_pass:
        launch = (f"two_pass chunk_tokens={split_used} head_slices={info['head_slices']} "
                  f"value_tiles={info['value_tiles']}")
        if Q > 1:
            launch += f" queries_per_seq={Q}"
    kernel_bytes = nb["value_latent"] if two_pass else nb["latent"]
    traffic = measured_traffic(wl, launch, Q, vkern if two_pass else "split_mfma") if mfma else None
    achieved = kernel_bytes / (kern_ms * 1e-3) / 1e9
    value = wl.batch * Q / (ms_step * 1e-3)
    decode_gbs = nb["decode_total"] / (ms_decode * 1e-3) / 1e9
    rec = {
        "metric": ("compressed-KV decode attention tokens/s (achieved HBM GB/s in roofline)" if Q == 1
                   else f"compressed-KV causal {Q}-query attention query tokens/s "
                        "(achieved HBM GB/s in roofline)"),
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if mfma else "f32",
        "data": "synthetic (seeded random latents, factors, queries and new tokens of the workload's shapes)",
        "config": {
            "workload": wl.name,
            "batch": wl.batch,
            "context_tokens": sum(wl.seq_lens),
            "appended_tokens": wl.append_tokens if append else 0,
            "q_heads": wl.num_q_heads, "kv_heads": wl.num_kv_heads, "head_dim": wl.head_dim,
            "hidden": wl.hidden, "group_sizes": list(wl.group_sizes),
            "group_ranks": list(wl.group_rank), "value_rank": wl.value_rank,
            "latent_dtype": wl.dtype, "split_tokens": split_used,
            "decode_kernels": ["portable", "single-pass", "two-pass"][info["kernels"]],
            "head_slices": info["head_slices"],
            "decode_waves": plan.geometry["decode_waves"],
            "queries_per_seq": Q,
            "pool_copies": copies, "pool_bytes": pool_bytes,
        },
        "context_tokens_per_s": sum(wl.seq_lens) / (ms_step * 1e-3),
        "step_hbm_gbs": (nb["decode_total"] + (nb["append"] if append else 0)) / (ms_step * 1e-3) / 1e9,
        "decode_call": {
            "ms": ms_decode, "bytes": nb["decode_total"], "hbm_gbs": decode_gbs,
            "frac": decode_gbs / HBM_PEAK_GBS, "frac_of_copy_peak": decode_gbs / copy["gbs"],
        },
        "copy_peak": copy,
        "roofline": {
            "kernel": (f"value pass of the two-pass decode ({vkern})" if two_pass else
                       "split-K latent attention (" + ("split_mfma" if mfma else "split_valu") + ")"),
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "frac_of_copy_peak": achieved / copy["gbs"],
            "traffic": traffic,
            "kernel_ms": kern_ms,
            "kernel_launches_timed": len(ev),
            "bytes_per_launch": kernel_bytes,
            "launch": launch,
        },
    }
    if rope:
        # the key rebuild is the dominant kernel: r_g * d_h MACs a token and KV head
        kv_ranks = sum(wl.group_rank[wl.group_of_kv[kv]] for kv in range(wl.num_kv_heads))
        flops = 2.0 * wl.head_dim * kv_ranks * sum(wl.seq_lens)
        tf = flops / (kern_ms * 1e-3) / 1e12
        rec["metric"] = ("compressed-KV rotary decode attention tokens/s "
                         "(key-rebuild MFMA TFLOP/s in roofline)")
        rec["config"]["rope_base"] = args.rope
        rec["config"]["split_tokens"] = split_used
        rec["roofline"] = {
            "kernel": "rotary key rebuild + scores + split softmax (rope_scores_res, bf16 MFMA)",
            "bound": "mfma", "achieved": tf, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": tf / MFMA_BF16_PEAK_TFLOPS,
            "traffic": measured_traffic(wl, f"split_tokens={split_used} rope", 1, "rope_scores"),
            "kernel_ms": kern_ms,
            "kernel_launches_timed": len(ev), "flops_per_launch": flops,
            "key_latent_bytes_per_launch": sum(wl.seq_lens) * wl.key_rank_total * wl.elem_bytes,
            "launch": f"split_tokens={split_used} rope",
        }
    if not args.no_cpu_baseline:
        print(f"[bench] {wl.name}: timing the CPU oracle sample", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, Q, append, args.rope)
    del pools, inp, ws
    torch.cuda.empty_cache()
    return rec


if __name__ == "__main__":
    main()
