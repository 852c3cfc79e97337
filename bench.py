#!/usr/bin/env python3
"""Throughput of LazyMAR's cached MAR transformer step on one MI355X.

One bench step = one whole 64-decoding-step LazyMAR schedule for a batch of
64 images x 2 guidance pathways at the MAR-L shape (16+16 blocks, width
1024, 16 heads, 320 tokens, bf16): the steps before the 5th and the first
step of every 9-step period are full steps (both pathways, every token);
the other steps are token-cached with N = 50 recomputed rows per sequence,
alternating conditional-only steps that reuse the stored guidance residual
with two-pathway steps that store a fresh one; every step ends with the
guidance combine.  Inputs of all 64 steps are resident in HBM before timing.

--schedule 32 runs the paper's other setting instead (32 decoding steps,
caching from the 4th step with tau = 5, about 250 of 320 tokens skipped per
cached step, so N = 70).

Other options: --workload (the MAR-B, MAR-H and 1088-token shapes), --rule
(the selection strategies of the paper's comparison), --score-source and
--fresh-kv (the method's variants), --profile-kind (which kernel class the
roofline reports, against the MFMA or the HBM peak).  --gemm-shapes,
--attention-shapes, --memory-shapes, --head-shapes and --calibrate-copy only
run single launches (or one head call) for trace and hardware-counter passes;
--library-gemms times the products against the vendor library's.

Prints one JSON line.  --gpus N with N > 1 exits: the measurement is one GPU's share of the work.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
# kernel class -> (what it is, the roof that bounds it)
KIND_ROOFLINE = {
    "fc1": ("fc1 product (bf16 MFMA, fp32 accumulate)", "mfma"),
    "qkv": ("QKV product with the key/value cache scatter (bf16 MFMA)", "mfma"),
    "proj": ("output projection + residual (bf16 MFMA)", "mfma"),
    "fc2": ("fc2 product + residual, output-cache scatter at the last block (bf16 MFMA)", "mfma"),
    "attention": ("attention of the computed queries against all keys (bf16 MFMA)", "mfma"),
    "layernorm": ("LayerNorm, with the row gather of the cached blocks", "hbm"),
    "scores": ("similarity of every token (fp64 sums)", "hbm"),
    "select": ("per-sequence ranking of the scores", "hbm"),
    "cfg": ("guidance combine with the condition cache", "hbm"),
}


# how the metric names each workload (the headline is MAR-L, 64 images x 2 pathways)
WORKLOAD_LABEL = {"mar-l": "MAR-L, 64x2 CFG", "mar-b": "MAR-B, 32x2 CFG", "mar-h": "MAR-H, 128x2 CFG",
                  "mar-l-hires": "MAR-L at 1088 tokens, 32x2 CFG"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3, help="timed schedules")
    ap.add_argument("--warmup", type=int, default=1, help="untimed schedules")
    ap.add_argument("--workload", default="mar-l", choices=["mar-l", "mar-b", "mar-h", "mar-l-hires"])
    ap.add_argument("--profile-kind", default="fc2", choices=list(KIND_ROOFLINE),
                    help="kernel class timed with HIP events for the roofline (default: fc2, the class with "
                         "the most GPU time in the MAR-L schedule)")
    ap.add_argument("--no-classes", action="store_true",
                    help="skip the per-class table (one extra schedule per kernel class, each class timed "
                         "with HIP events against its own roof)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--schedule", default="64", choices=list(SCHEDULES),
                    help="the paper's settings: 64 decoding steps (start 5, tau 9) or 32 (start 4, tau 5)")
    ap.add_argument("--score-source", default="values", choices=["values", "features"],
                    help="what the similarity compares (Sec. 4.4): block P-1's value rows or its output features")
    ap.add_argument("--fresh-kv", action="store_true",
                    help="recompute every row's keys/values at the first cached block")
    ap.add_argument("--rule", default="least", choices=list(RULES),
                    help="token selection of the cached steps (Table 3): least / most similar on the "
                         "device, or random / token-type rows chosen on the host")
    ap.add_argument("--gemm-shapes", default=None, choices=["qkv", "proj", "fc1", "fc2"],
                    help="only run one product class once per shape the 64-step MAR-L schedule "
                         "launches (for hardware-counter runs) and print each shape's launches per "
                         "schedule")
    ap.add_argument("--attention-shapes", action="store_true",
                    help="only run the attention once per shape the 64-step MAR-L schedule launches (for "
                         "hardware-counter runs) and print each shape's launches per schedule")
    ap.add_argument("--memory-shapes", action="store_true",
                    help="only run the memory-bound kernels (LayerNorm dense and gather, scores, select) once "
                         "each at the MAR-L schedule's shapes (for hardware-counter runs)")
    ap.add_argument("--head-shapes", action="store_true",
                    help="only run one call of the MAR-L diffusion head on 256 tokens (for trace and "
                         "hardware-counter runs)")
    ap.add_argument("--library-gemms", action="store_true",
                    help="only time the block products (bias epilogue) against the vendor library's "
                         "product of the same shape")
    ap.add_argument("--no-head", action="store_true",
                    help="skip the diffusion-head leg (the per-token head run for the tokens each decoding "
                         "step decodes, timed beside the transformer schedule)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy three times (the reference "
                         "dispatch that scales the HBM byte counters) and exit")
    return ap.parse_args()


COPY_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "{kind}_hbm_traffic_mar_l.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2503_12450_amd", "csrc", "gemm.hip")


def calibrate_copy():
    import torch
    a = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda:0")
    a.fill_(1)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "dispatches": 3}), flush=True)


def gemm_shapes(kind):
    """One product class of the 64-step MAR-L schedule, once per row count
    it launches: rows M -> launches per schedule.  Full steps run every
    block on every row of both pathways; cached steps the prefix blocks on
    every row and the rest on N rows per sequence.  Each launch goes through
    the class's own entry point and epilogue (QKV with the key/value cache
    scatter, fc1 with GELU, proj and fc2 with the fp32 residual)."""
    import torch

    from paper_2503_12450_amd import binding as B
    from paper_2503_12450_amd import schedule as sch
    from paper_2503_12450_amd.workload import WORKLOADS

    wl = WORKLOADS["mar-l"]
    d, n, img = wl.dims, wl.n_recompute, wl.images
    D, F, S, H = d.d_model, d.d_mlp, d.seq_len, d.n_heads
    N, K = {"qkv": (3 * D, D), "proj": (D, D), "fc1": (F, D), "fc2": (D, F)}[kind]
    counts = {}
    n_steps, start, tau, _ = SCHEDULES["64"]
    for p in sch.lazymar_schedule(n_steps, start, tau, "alternate"):
        seqs = 2 * img if (p.mode == sch.FULL or p.branches == sch.BOTH) else img
        if p.mode == sch.FULL:
            counts[seqs * S] = counts.get(seqs * S, 0) + d.n_layers
        else:
            counts[seqs * S] = counts.get(seqs * S, 0) + d.full_prefix
            counts[seqs * n] = counts.get(seqs * n, 0) + d.n_layers - d.full_prefix
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(0)
    w = (torch.randn(N, K, device=dev, generator=g) * 0.02).to(torch.bfloat16)
    bias = torch.zeros(N, device=dev)
    for m in sorted(counts, reverse=True):
        a = torch.randn(m, K, device=dev, generator=g).to(torch.bfloat16)
        per = S if m in (2 * img * S, img * S) else n   # dense rows: whole sequences
        seqs = m // per
        if kind == "qkv":
            q = torch.empty(m, D, device=dev, dtype=torch.bfloat16)
            kc = torch.empty(seqs, H, S, D // H, device=dev, dtype=torch.bfloat16)
            vc = torch.empty_like(kc)
            idx = None if per == S else torch.stack(
                [torch.randperm(S, device=dev, generator=g)[:per].sort().values for _ in range(seqs)]).to(torch.int32)
            B.k_qkv("bf16", a, w, bias, D, H, S, per, q_out=q, k_cache=kc, v_cache=vc, idx=idx)
        elif kind == "fc1":
            out = torch.empty(m, N, device=dev, dtype=torch.bfloat16)
            B.k_linear("bf16", a, w, bias, out, gelu=True)
        else:
            r = torch.randn(m, N, device=dev, generator=g)
            B.k_linear_residual("bf16", a, w, bias, r, r)
    torch.cuda.synchronize()
    print(json.dumps({f"{kind}_rows_to_launches_per_schedule": counts, "n": N, "k": K}), flush=True)


def attention_shapes():
    """The attention launches of one 64-step MAR-L schedule: (sequences, queries per
    sequence) -> launches.  Every key/value row of a block takes part; full steps and
    the prefix blocks of cached steps query all rows, the cached blocks N rows."""
    import torch

    from paper_2503_12450_amd import binding as B
    from paper_2503_12450_amd import schedule as sch
    from paper_2503_12450_amd.workload import WORKLOADS

    wl = WORKLOADS["mar-l"]
    d, n, img = wl.dims, wl.n_recompute, wl.images
    S, H, dh = d.seq_len, d.n_heads, d.d_model // d.n_heads
    counts = {}
    n_steps, start, tau, _ = SCHEDULES["64"]
    for p in sch.lazymar_schedule(n_steps, start, tau, "alternate"):
        seqs = 2 * img if (p.mode == sch.FULL or p.branches == sch.BOTH) else img
        if p.mode == sch.FULL:
            counts[(seqs, S)] = counts.get((seqs, S), 0) + d.n_layers
        else:
            counts[(seqs, S)] = counts.get((seqs, S), 0) + d.full_prefix
            counts[(seqs, n)] = counts.get((seqs, n), 0) + d.n_layers - d.full_prefix
    g = torch.Generator(device="cuda:0").manual_seed(0)
    for seqs, per in sorted(counts, key=lambda k: -k[0] * k[1]):
        q = torch.randn(seqs * per, d.d_model, device="cuda:0", generator=g).to(torch.bfloat16)
        kc = torch.randn(seqs, H, S, dh, device="cuda:0", generator=g).to(torch.bfloat16)
        vc = torch.randn(seqs, H, S, dh, device="cuda:0", generator=g).to(torch.bfloat16)
        out = torch.empty_like(q)
        B.k_attention("bf16", q, kc, vc, out, seqs, H, S, dh, per)
    torch.cuda.synchronize()
    shapes = {f"{seqs}x{per}": c for (seqs, per), c in sorted(counts.items(), key=lambda kv: -kv[0][0] * kv[0][1])}
    print(json.dumps({"attention_shapes_to_launches_per_schedule": shapes, "heads": H, "seq": S, "d_head": dh}),
          flush=True)


def head_shapes(tokens: int = 256):
    """One call of the MAR-L diffusion head on `tokens` tokens (the 64-step schedule decodes
    16384 tokens, 256 per step on average): 100 DDPM steps of both guidance branches, for
    trace and hardware-counter runs.  Inputs are random rows of a transformer output."""
    import torch

    from paper_2503_12450_amd import binding as B
    from paper_2503_12450_amd.device import upload_head
    from paper_2503_12450_amd.flops import head_flops_per_eval
    from paper_2503_12450_amd.workload import HEADS, head_weights

    dev = "cuda:0"
    hd = HEADS["mar-l"]
    from dataclasses import replace
    hd = replace(hd, max_rows=tokens)
    head = B.MarHead(hd, upload_head(head_weights(hd), hd.dtype, device=dev))
    g = torch.Generator(device=dev).manual_seed(0)
    y = torch.randn(tokens, hd.cond_dim, device=dev, generator=g)
    yu = torch.randn(tokens, hd.cond_dim, device=dev, generator=g)
    rows = torch.arange(tokens, device=dev, dtype=torch.int32)
    x0 = torch.randn(tokens, hd.token_dim, device=dev, generator=g)
    xi = torch.randn(hd.steps, tokens, hd.token_dim, device=dev, generator=g)
    xo = torch.empty(tokens, hd.token_dim, device=dev)
    head.sample(y, yu, rows, rows, x0, xi, 4.0, xo)
    torch.cuda.synchronize()
    flops = head_flops_per_eval(hd) * 2 * tokens * hd.steps
    print(json.dumps({"head": "mar-l", "width": hd.width, "depth": hd.depth, "tokens": tokens,
                      "ddpm_steps": hd.steps, "flops_per_call": flops}), flush=True)


def library_gemms():
    """The block products with the bias epilogue against the vendor library's product of the
    same shape (torch.nn.functional.linear, which dispatches to hipBLASLt), alternating, on the
    dense (40960 rows) and cached (3200 rows) MAR-L shapes.  A reference point only: the path's
    products carry fused epilogues the library call does not."""
    import torch

    from paper_2503_12450_amd import binding as B

    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(0)

    def timed(fn, reps=10):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    for name, M, N, K in (("qkv", 40960, 3072, 1024), ("proj", 40960, 1024, 1024), ("fc1", 40960, 4096, 1024),
                          ("fc2", 40960, 1024, 4096), ("qkv", 3200, 3072, 1024), ("proj", 3200, 1024, 1024),
                          ("fc1", 3200, 4096, 1024), ("fc2", 3200, 1024, 4096)):
        a = torch.randn(M, K, device=dev, generator=g).to(torch.bfloat16)
        w = (torch.randn(N, K, device=dev, generator=g) * 0.02).to(torch.bfloat16)
        b32 = torch.randn(N, device=dev, generator=g) * 0.1
        b16 = b32.to(torch.bfloat16)
        out = torch.empty(M, N, device=dev, dtype=torch.bfloat16)
        lib, ours = [], []
        for _ in range(2):
            lib.append(timed(lambda: torch.nn.functional.linear(a, w, b16)))
            ours.append(timed(lambda: B.k_linear("bf16", a, w, b32, out, gelu=False)))
        fl = 2.0 * M * N * K
        print(json.dumps({"product": name, "m": M, "n": N, "k": K, "library_us": round(min(lib), 1),
                          "path_us": round(min(ours), 1), "library_over_path_time": round(min(lib) / min(ours), 3),
                          "library_tflops": round(fl / min(lib) / 1e6), "path_tflops": round(fl / min(ours) / 1e6)}),
              flush=True)


def memory_shapes():
    """The memory-bound kernels once each at the shapes of the 64-step MAR-L schedule (for
    hardware-counter runs): the dense LayerNorm (both pathways, fp32 residual stream in, bf16
    out), the gather LayerNorm of the cached blocks (N rows per sequence, with the fp32 copy of
    the compact residual stream), the similarity scores with the reference update, and the
    selection.  Prints each launch's algorithmic bytes."""
    import torch

    from paper_2503_12450_amd import binding as B
    from paper_2503_12450_amd.workload import WORKLOADS

    wl = WORKLOADS["mar-l"]
    d, n, img = wl.dims, wl.n_recompute, wl.images
    S, D, H = d.seq_len, d.d_model, d.n_heads
    dh, seqs = D // H, 2 * img
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(0)
    w = torch.ones(D, device=dev)
    b = torch.zeros(D, device=dev)
    launches = []
    h = torch.randn(seqs * S, D, device=dev, generator=g)
    out = torch.empty(seqs * S, D, device=dev, dtype=torch.bfloat16)
    B.k_layernorm("bf16", h, w, b, 1e-6, out)
    launches.append(("layernorm (dense)", f"{seqs * S} rows", seqs * S * D * (4 + 2)))
    idx = torch.stack([torch.randperm(S, device=dev, generator=g)[:n].sort().values
                       for _ in range(seqs)]).to(torch.int32)
    og = torch.empty(seqs * n, D, device=dev, dtype=torch.bfloat16)
    cg = torch.empty(seqs * n, D, device=dev)
    B.k_layernorm("bf16", h, w, b, 1e-6, og, idx=idx, per_slot=n, seq=S, copy_f32=cg)
    launches.append(("layernorm (gather + fp32 copy)", f"{seqs} x {n} of {S} rows", seqs * n * D * (4 + 2 + 4)))
    vc = torch.randn(seqs, H, S, dh, device=dev, generator=g).to(torch.bfloat16)
    vr = torch.randn(seqs, H, S, dh, device=dev, generator=g).to(torch.bfloat16)
    sc = torch.empty(seqs, S, device=dev, dtype=torch.float64)
    B.k_scores("bf16", vc, vr, sc, update_ref=True)
    launches.append(("scores (+ reference update)", f"{seqs} x {S} tokens", 3 * seqs * S * D * 2 + seqs * S * 8))
    sel = torch.empty(seqs, n, device=dev, dtype=torch.int32)
    B.k_select(sc, n, sel)
    launches.append(("select", f"{seqs} x {S} -> {n}", seqs * S * 8 + seqs * n * 4))
    torch.cuda.synchronize()
    print(json.dumps({"memory_launches": launches}), flush=True)


def recorded_traffic(kind):
    """HBM bytes per launch of a product class from the committed counter
    runs, or None when there are none or the GEMM source changed since they
    were taken."""
    import hashlib
    try:
        text = open(TRAFFIC_FILE.format(kind=kind)).read()
        src = hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    vals = dict(kv.split("=", 1) for kv in text.split() if kv.startswith(("traffic_bytes_per_launch=",
                                                                           "gemm_source_sha256=")))
    if vals.get("gemm_source_sha256") != src or "traffic_bytes_per_launch" not in vals:
        return None
    return float(vals["traffic_bytes_per_launch"])


def cpu_baseline(dims, W, recipe, n, plans):
    """The oracle on the host cores: one full and one token-cached step of
    one sequence, composed into one image's schedule."""
    import numpy as np
    import threadpoolctl

    import oracle as O
    from paper_2503_12450_amd import schedule as sch
    from paper_2503_12450_amd.workload import step_input

    threads = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()), default=1)
    # a bounded sample: REPS full and REPS cached steps of one sequence
    # (decoding steps 20, 21, ...), the median of each
    reps = 5
    orc = O.MarOracle(dims, W)
    fulls, cacheds = [], []
    for r in range(reps):
        prev = step_input(recipe, 20 + 2 * r)[0]
        x = step_input(recipe, 21 + 2 * r)[0]
        t0 = time.perf_counter()
        orc.full_slot(0, prev)
        fulls.append(time.perf_counter() - t0)
        t0 = time.perf_counter()
        orc.cached_slot(0, x, n)
        cacheds.append(time.perf_counter() - t0)
    t_full, t_cached = float(np.median(fulls)), float(np.median(cacheds))
    full, cond, both = sch.counts(plans)
    seq_full = 2 * full
    seq_cached = 2 * both + cond
    t_sched = seq_full * t_full + seq_cached * t_cached
    tokens = len(plans) * dims.seq_len
    return {
        "value": tokens / t_sched, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
        "host_cpus": os.cpu_count(), "cpus_available": len(os.sched_getaffinity(0)),
        "threads_note": (f"the oracle's matrix products ran on {threads} BLAS threads; its other work "
                         "(the exactly rounded score sums, attention per head, LayerNorm) is single-threaded "
                         "numpy/Python"),
        "sample": (f"fp64 numpy oracle, one sequence: median of {reps} full steps ({t_full:.2f} s) and of {reps} "
                   f"token-cached steps N={n} ({t_cached:.2f} s) at the {dims.n_layers}-block width-{dims.d_model} "
                   f"shape; one image's schedule composed as {seq_full} full + {seq_cached} cached sequence-steps"),
    }


# the paper's two settings (Sec. 4.1): decoding steps, first cached step,
# refresh period tau, and tokens skipped per cached step at 320 tokens
# (None: the workload's own N)
SCHEDULES = {"64": (64, 5, 9, None), "32": (32, 4, 5, 250)}

# token-selection rules of the cached steps (Table 3's strategies)
RULES = {
    "least": "least similar computed (strategy V, LazyMAR)",
    "most": "most similar computed (strategy IV)",
    "random": "random rows (strategy III)",
    "decoded": "decoded tokens computed first (strategy I)",
    "undecoded": "not-yet-decoded tokens computed first (strategy II)",
}


def given_rows(rule, recipe, plans, slots, seq, n):
    """Host-chosen rows of every cached step for the random and token-type
    rules, in pinned host memory so that the step's upload stays
    asynchronous.  Buffer (condition) rows count as decoded."""
    import numpy as np
    import torch

    from paper_2503_12450_amd import schedule as sch
    from paper_2503_12450_amd import selection as SEL
    from paper_2503_12450_amd.workload import decoded_mask

    rng = np.random.Generator(np.random.Philox(4))
    out = {}
    for i, p in enumerate(plans):
        if p.mode == sch.FULL:
            continue
        if rule == "random":
            rows = SEL.random_rows(slots, seq, n, rng)
        else:
            img = decoded_mask(recipe, i)                       # [images, T]
            known = np.ones((img.shape[0], seq), dtype=bool)
            known[:, seq - img.shape[1]:] = img
            mask = np.concatenate([known, known])[:slots]     # both pathways share the state
            rows = SEL.observation_rows(mask, n, SEL.COMPUTE_DECODED if rule == "decoded"
                                        else SEL.COMPUTE_UNDECODED)
        t = torch.from_numpy(rows).pin_memory()
        out[i] = (t, t.numpy())
    return out


def head_leg(args, wl, dims, recipe, plans, cache, X, n, images, scale, dev):
    """One schedule with the diffusion head after every decoding step: the
    tokens decoded at that step (the cosine schedule) are sampled over 100
    DDPM steps, conditioned on their rows of the output cache (conditional
    slots) and on the unconditional rows of the same step (the output cache
    on two-pathway steps, the condition cache's reconstruction on reuse
    steps).  Timed with HIP events around the head calls; the transformer
    work between them runs as in the headline schedule."""
    import numpy as np
    import torch

    from paper_2503_12450_amd import binding as B
    from paper_2503_12450_amd import schedule as sch
    from paper_2503_12450_amd.device import upload_head
    from paper_2503_12450_amd.workload import BUFFER_ROWS, HEADS, decoded_at, head_weights
    from paper_2503_12450_amd.flops import head_flops_per_eval

    key = {"mar-l": "mar-l", "mar-b": "mar-b", "mar-h": "mar-h", "mar-l-hires": "mar-l"}[args.workload]
    S, D = dims.seq_len, dims.d_model
    per_step = [decoded_at(recipe, k) for k in range(len(plans))]
    R_max = max(r.size for r in per_step)
    from dataclasses import replace
    hd = replace(HEADS[key], cond_dim=D, max_rows=R_max)
    head = B.MarHead(hd, upload_head(head_weights(hd), hd.dtype, device=dev))
    rows = []
    for r in per_step:
        flat = (np.arange(images)[:, None] * S + BUFFER_ROWS + r).reshape(-1).astype(np.int32)
        rows.append(torch.from_numpy(flat).to(dev))
    g = torch.Generator(device=dev).manual_seed(5)
    x0 = [torch.randn(r.size, hd.token_dim, device=dev, generator=g) for r in per_step]
    xi = [torch.randn(hd.steps, r.size, hd.token_dim, device=dev, generator=g) for r in per_step]
    xo = [torch.empty(r.size, hd.token_dim, device=dev) for r in per_step]
    Y = cache.output()
    u_hat = torch.empty((images, S, D), dtype=torch.float32, device=dev)
    guided = torch.empty((images, S, D), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()

    def run(events=None):
        for i, p in enumerate(plans):
            slots = 2 * images if p.branches == sch.BOTH else images
            if p.mode == sch.FULL:
                cache.step(X[i], B.MAR_FULL)
            else:
                cache.step(X[i][:slots], B.MAR_TOKEN_CACHED, n, slot0=0)
            if p.cfg == sch.STORE:
                cache.cfg_combine(B.MAR_CFG_STORE, Y[:images], Y[images:2 * images], scale, guided)
                y_unc = Y[images:2 * images]
            else:
                cache.cfg_combine(B.MAR_CFG_REUSE, Y[:images], None, scale, guided, u_hat)
                y_unc = u_hat
            if events is not None:
                events[i][0].record()
            head.sample(Y[:images], y_unc, rows[i], rows[i], x0[i], xi[i], scale, xo[i])
            if events is not None:
                events[i][1].record()

    run()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in plans]
    t0 = time.perf_counter()
    run(ev)
    torch.cuda.synchronize()
    wall_ms = 1e3 * (time.perf_counter() - t0)
    head_ms = sum(a.elapsed_time(b) for a, b in ev)
    tokens = sum(r.size for r in per_step)
    fl = head_flops_per_eval(hd) * 2 * tokens * hd.steps
    return {
        "what": (f"per-token diffusion head (width {hd.width}, {hd.depth} blocks, {hd.steps} DDPM steps, both "
                 f"guidance branches) on the {tokens} tokens the {len(plans)}-step schedule decodes"),
        "schedule_with_head_ms": wall_ms, "head_ms": head_ms, "head_share": head_ms / wall_ms,
        "head_tflops": fl / (head_ms / 1e3) / 1e12, "head_frac_of_bf16_peak": fl / (head_ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
        "tokens": tokens, "max_tokens_per_step": R_max,
    }


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gemm_shapes:
        gemm_shapes(args.gemm_shapes)
        return
    if args.attention_shapes:
        attention_shapes()
        return
    if args.memory_shapes:
        memory_shapes()
        return
    if args.head_shapes:
        head_shapes()
        return
    if args.library_gemms:
        library_gemms()
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the cached step shards over images with no "
              "communication, so N GPUs each run this workload on 1/N of the images; the "
              "measurement is one GPU's share.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2503_12450_amd import binding as B
    from paper_2503_12450_amd import flops as FL
    from paper_2503_12450_amd import schedule as sch
    from paper_2503_12450_amd.device import upload_blocks
    from paper_2503_12450_amd.workload import WORKLOADS, all_block_weights, decode_recipe, step_inputs_device

    from dataclasses import replace
    wl = WORKLOADS[args.workload]
    dims = replace(wl.dims, score_source=args.score_source, fresh_kv=args.fresh_kv)
    n, images = wl.n_recompute, wl.images
    dev = "cuda:0"
    torch.cuda.set_device(0)
    W = all_block_weights(dims)
    blocks = upload_blocks(W, dims.dtype, device=dev)
    cache = B.MarCache(dims, blocks, device=dev)
    torch.cuda.synchronize()
    del blocks
    n_steps, start, tau, skipped = SCHEDULES[args.schedule]
    if skipped is not None:
        if dims.seq_len != 320:
            raise SystemExit("the 32-step setting is stated for 320-token sequences")
        n = dims.seq_len - skipped
    recipe = decode_recipe(dims, images, n_steps)
    X = step_inputs_device(recipe, range(n_steps), device=dev)
    cfg_rule = "paper" if args.workload == "mar-l-hires" else "alternate"
    plans = sch.lazymar_schedule(n_steps, start, tau, cfg_rule)
    Y = cache.output()
    guided = torch.empty((images, dims.seq_len, dims.d_model), dtype=torch.float32, device=dev)
    scale = 4.0

    given = given_rows(args.rule, recipe, plans, 2 * images, dims.seq_len, n) \
        if args.rule in ("random", "decoded", "undecoded") else {}
    ranked = B.MAR_TOKEN_CACHED_MOST_SIMILAR if args.rule == "most" else B.MAR_TOKEN_CACHED

    def one_step(i, p, x):
        slots = 2 * images if p.branches == sch.BOTH else images
        if p.mode == sch.FULL:
            cache.step(x, B.MAR_FULL)
        elif i in given:
            cache.step(x[:slots], B.MAR_TOKEN_GIVEN, n, slot0=0, sel_idx=given[i][1][:slots])
        else:
            cache.step(x[:slots], ranked, n, slot0=0)
        if p.cfg == sch.STORE:
            cache.cfg_combine(B.MAR_CFG_STORE, Y[:images], Y[images:2 * images], scale, guided)
        else:
            cache.cfg_combine(B.MAR_CFG_REUSE, Y[:images], None, scale, guided)

    def schedule_run(step_events=None):
        for i, p in enumerate(plans):
            if step_events is not None:
                step_events[i][0].record()
            one_step(i, p, X[i])
            if step_events is not None:
                step_events[i][1].record()

    for _ in range(args.warmup):
        schedule_run()
    torch.cuda.synchronize()

    # timed region: exactly `steps` schedules
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in plans] for _ in range(args.steps)]
    cache.profile_start(args.profile_kind)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        schedule_run(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    prof_ms, prof_n, prof_flops, prof_bytes = cache.profile_stop()

    per_mode = {"full": [], "cached_both": [], "cached_cond": []}
    for k in range(args.steps):
        for p, (a, b) in zip(plans, evs[k]):
            key = "full" if p.mode == sch.FULL else ("cached_both" if p.branches == sch.BOTH else "cached_cond")
            per_mode[key].append(a.elapsed_time(b))
    mean = {k: (float(np.mean(v)) if v else None) for k, v in per_mode.items()}

    ms_per_sched = 1e3 * wall / args.steps
    tokens_per_sched = len(plans) * images * dims.seq_len
    value = tokens_per_sched / (ms_per_sched / 1e3)
    sched_flops = 0
    for p in plans:
        if p.mode == sch.FULL:
            sched_flops += FL.step_flops(dims, 2 * images, "full")
        else:
            sched_flops += FL.step_flops(dims, (2 if p.branches == sch.BOTH else 1) * images, "cached", n)
    full_sched_ms = len(plans) * mean["full"]

    tflops = prof_flops / (prof_ms / 1e3) / 1e12 if prof_ms > 0 else None
    gbs = prof_bytes / (prof_ms / 1e3) / 1e9 if prof_ms > 0 else None
    what, bound = KIND_ROOFLINE[args.profile_kind]
    achieved, peak, unit = (tflops, PEAK_BF16_TFLOPS, "TFLOP/s") if bound == "mfma" else (gbs, PEAK_HBM_GBS, "GB/s")
    roofline = {
        "kernel": what,
        "bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
        "frac": (achieved / peak) if achieved else None,
        "traffic": recorded_traffic(args.profile_kind) if args.workload == "mar-l" else None,
        "launches": prof_n, "avg_launch_us": 1e3 * prof_ms / max(prof_n, 1),
        "flops_per_launch": prof_flops / max(prof_n, 1),
        "bytes_per_launch": prof_bytes / max(prof_n, 1),
        "tflops": tflops, "gbs": gbs,
    }
    line = {
        "metric": f"cached MAR step tokens/s ({WORKLOAD_LABEL[args.workload]}, {n_steps}-step LazyMAR schedule)",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_sched, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dims.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "images": images, "seq_len": dims.seq_len,
                   "n_recompute": n, "decode_steps": len(plans),
                   "schedule": f"start {start}, tau {tau}, " + cfg_rule + " guidance reuse",
                   "selection": RULES[args.rule],
                   "score_source": args.score_source, "fresh_kv": args.fresh_kv,
                   "step": f"one {n_steps}-decoding-step schedule"},
        "tflops": sched_flops / (ms_per_sched / 1e3) / 1e12,
        "step_ms": mean,
        "speedup_vs_full_recompute": full_sched_ms / ms_per_sched if mean["full"] else None,
        "speedup_cached_cond_vs_full": (mean["full"] / mean["cached_cond"]) if mean["cached_cond"] else None,
        "roofline": roofline,
    }
    if not args.no_classes:
        classes = {}
        for kind, (what_k, bound_k) in KIND_ROOFLINE.items():
            cache.profile_start(kind)
            schedule_run()
            torch.cuda.synchronize()
            ms_k, n_k, fl_k, by_k = cache.profile_stop()
            ach = (fl_k if bound_k == "mfma" else by_k) / (ms_k / 1e3) / (1e12 if bound_k == "mfma" else 1e9) \
                if ms_k > 0 else None
            pk = PEAK_BF16_TFLOPS if bound_k == "mfma" else PEAK_HBM_GBS
            classes[kind] = {"bound": bound_k, "ms_per_schedule": ms_k, "launches": n_k,
                             "avg_launch_us": 1e3 * ms_k / max(n_k, 1), "achieved": ach,
                             "unit": "TFLOP/s" if bound_k == "mfma" else "GB/s",
                             "frac": (ach / pk) if ach else None}
        total_k = sum(c["ms_per_schedule"] for c in classes.values())
        for c in classes.values():
            c["share_of_kernel_time"] = c["ms_per_schedule"] / total_k if total_k else None
        line["kernel_classes"] = classes
        line["dominant_class"] = max(classes, key=lambda k: classes[k]["ms_per_schedule"])
    if not args.no_head and args.rule == "least":
        line["diffusion_head"] = head_leg(args, wl, dims, recipe, plans, cache, X, n, images, scale, dev)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(dims, W, recipe, n, plans)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
