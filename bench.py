#!/usr/bin/env python3
"""Benchmark of budgeted in-place KV-cache repair on one MI355X.

Default workload: Llama-3-8B-shaped decoder (bf16, random-init N(0, 0.02)
weights), 5000-token context of uniform token ids, one 16-token in-place edit
at a seeded position in [1000, 4000], EditLocal K = 32 (48 recomputed rows),
batch 1.  One step = one kvr_repair call (all 32 layers) over a cache that is
already resident in HBM; repair is idempotent, so repeated steps need no cache
reset.  The same engine's full re-prefill of the edited 5000-token context is
timed for the speedup.

Prints one JSON line: ms per repair (value), algorithmic HBM GB/s, recomputed
tokens/s, prefill ms and speedup, the roofline of the dominant kernel (the
gate/up projection with SwiGLU, timed over the timed repairs with the HIP
events its dispatches record at the start and end of its execution), the
kernel time per step of the layer loop, and the fp64 CPU oracle's time on a
bounded sample of the same repair.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0

WORKLOADS = {
    "llama8b-k32": dict(shape="llama3-8b", n=5000, span=16, K=32, policy="edit_local", lo=1000, hi=4000),
    "qwen7b-k8": dict(shape="qwen2.5-7b", n=5000, span=16, K=8, policy="edit_local", lo=1000, hi=4000),
    "qwen7b-k32": dict(shape="qwen2.5-7b", n=5000, span=16, K=32, policy="edit_local", lo=1000, hi=4000),
    "qwen7b-k128": dict(shape="qwen2.5-7b", n=5000, span=16, K=128, policy="edit_local", lo=1000, hi=4000),
    "qwen7b-k512": dict(shape="qwen2.5-7b", n=5000, span=16, K=512, policy="edit_local", lo=1000, hi=4000),
    "qwen7b-random-k8": dict(shape="qwen2.5-7b", n=5000, span=16, K=8, policy="random", lo=1000, hi=4000),
    "qwen7b-random-k32": dict(shape="qwen2.5-7b", n=5000, span=16, K=32, policy="random", lo=1000, hi=4000),
    "qwen7b-random-k128": dict(shape="qwen2.5-7b", n=5000, span=16, K=128, policy="random", lo=1000, hi=4000),
    "qwen7b-random-k512": dict(shape="qwen2.5-7b", n=5000, span=16, K=512, policy="random", lo=1000, hi=4000),
    "mistral7b-end": dict(shape="mistral-7b", n=5000, span=16, K=32, policy="edit_local", lo=4900, hi=4900),
    "mistral7b-start": dict(shape="mistral-7b", n=5000, span=16, K=32, policy="edit_local", lo=200, hi=200),
    # 64 documents of 2000-8000 tokens, one 16-token edit each at 20-80 % of the
    # document, EditLocal K=32, repaired in one call (3072 rows)
    "llama8b-batch64": dict(shape="llama3-8b", docs=64, n_lo=2000, n_hi=8000, span=16, K=32, policy="edit_local"),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b-k32", choices=sorted(WORKLOADS))
    ap.add_argument("--seeds", type=int, default=5,
                    help="edit placements (seeds 0..S-1) timed for the per-seed report; value is seed 0's")
    ap.add_argument("--prefill-steps", type=int, default=5)
    ap.add_argument("--cpu-layers", type=int, default=32,
                    help="layers of the repair the CPU oracle runs for its bounded sample")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one 1 GiB device-to-device copy first (reference for HBM byte counters)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-adjacent", action="store_true",
                    help="skip the timings of the scoring forward, the selectors and transplant")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def plan_docs(wl, kvr, synth, label):
    """(n, edit start, A) of every document of the workload for edit seed `label`."""
    span, K = wl["span"], wl["K"]
    policy = kvr.KVR_EDIT_LOCAL if wl["policy"] == "edit_local" else kvr.KVR_RANDOM
    if "docs" not in wl:
        n = wl["n"]
        e = synth.edit_position(wl["lo"], wl["hi"], label=label)
        return [(n, e, kvr.kvr_select(policy, n, e, e + span, K, label))]
    out = []
    for i, n in enumerate(synth.doc_lengths(wl["docs"], wl["n_lo"], wl["n_hi"])):
        e = synth.edit_position(int(0.2 * n), int(0.8 * n) - span, label=1000 * label + i)
        out.append((n, e, kvr.kvr_select(policy, n, e, e + span, K, label + i)))
    return out


def repair_bytes(shape, plans, span):
    """Algorithmic HBM bytes of one repair call: every weight once, per document
    the KV rows [0, max P] of each kv head once and the fresh K/V writes, and
    the embedding rows."""
    es = 2
    b = shape.n_layers * shape.layer_params() * es + shape.d_model * es
    for n, e, A in plans:
        R = span + len(A)
        max_pos = max([e + span - 1] + list(A))
        b += (max_pos + 1) * shape.kv_bytes_per_pos(es) + R * shape.kv_bytes_per_pos(es) + R * shape.d_model * es
    return b


def repair_flops(shape, plans, span):
    """Algorithmic flops of one repair call: 2 per weight element per row, and
    per layer and row at position p: 4 * H_q * head_dim * (p + 1) of attention."""
    mat = shape.layer_params() - 2 * shape.d_model - (shape.q_dim + 2 * shape.kv_dim if shape.qkv_bias else 0)
    f = 0
    for n, e, A in plans:
        P = list(range(e, e + span)) + list(A)
        f += 2 * len(P) * shape.n_layers * mat
        f += shape.n_layers * 4 * shape.n_heads * shape.head_dim * sum(p + 1 for p in P)
    return f


def prefill_flops(shape, plans):
    """Algorithmic flops of the same engine's full prefill of every document:
    2 per weight element per position, and per layer 4 * H_q * head_dim * (p + 1)
    of causal attention for the position p."""
    mat = shape.layer_params() - 2 * shape.d_model - (shape.q_dim + 2 * shape.kv_dim if shape.qkv_bias else 0)
    f = 0
    for n, _, _ in plans:
        f += 2 * n * shape.n_layers * mat
        f += shape.n_layers * 4 * shape.n_heads * shape.head_dim * n * (n + 1) // 2
    return f


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); this build has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    import paper_2609_17983_amd as kvr
    import synth

    wl = WORKLOADS[args.workload]
    shape = synth.SHAPES[wl["shape"]]
    span, K = wl["span"], wl["K"]
    batched = "docs" in wl
    plans = plan_docs(wl, kvr, synth, 0)
    R = sum(span + len(A) for _, _, A in plans)
    n_max = max(n for n, _, _ in plans)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    L = shape.n_layers
    if batched:
        log(f"workload {args.workload}: {shape.name}, {len(plans)} docs of {min(n for n, _, _ in plans)}-{n_max} "
            f"tokens, {wl['policy']} K={K} -> {R} rows")
    else:
        n, e, A = plans[0]
        log(f"workload {args.workload}: {shape.name}, n={n}, edit [{e},{e + span}), {wl['policy']} K={K} -> {R} rows")

    if args.calibrate_copy:
        src = torch.empty(1 << 29, dtype=torch.int16, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration copy: 1 GiB read + 1 GiB written")
        del src, dst
    w = synth.make_weights(shape, dtype=torch.bfloat16, device="cuda")
    dims = kvr.dims_for(shape, kvr.KVR_BF16, max_ctx=n_max + ADJ_SLOTS, max_rows=max(R, 64))
    ctx = kvr.kvr_create(dims, kvr.weights_struct(w))

    # stale caches K(C) by the engine's own prefill, then the edited ids C'
    caches, olds, hiddens = [], [], []
    for i, (n, e, A) in enumerate(plans):
        toks = synth.make_tokens(n, shape.vocab, seed=synth.SEED_TOKENS + i).to(dev)
        cache = torch.empty((L, 2, shape.n_kv_heads, n, shape.head_dim), dtype=torch.bfloat16, device=dev)
        kvr.kvr_prefill(ctx, toks.data_ptr(), n, n, cache.data_ptr(), None, stream.cuda_stream)
        caches.append(cache)
        olds.append(toks)
        hiddens.append(torch.empty((span + len(A), shape.d_model), dtype=torch.float32, device=dev))
    torch.cuda.synchronize()

    def make_docs(plans_s, label):
        docs, news = [], []
        for i, (n, e, A) in enumerate(plans_s):
            new = synth.apply_edit(olds[i], e, span, shape.vocab, label=1000 * label + i)
            news.append(new)
            docs.append(kvr.make_doc(caches[i].data_ptr(), n, n, new.data_ptr(), e, e + span, A,
                                     hiddens[i].data_ptr() if len(A) + span == hiddens[i].shape[0] else None))
        return docs, news

    def timed(docs, steps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for i in range(steps):
            kvr.kvr_repair(ctx, docs, stream.cuda_stream)
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        return [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)], ev[0].elapsed_time(ev[-1]) / steps

    # ---- repair: W warmup, then K timed steps (HIP events on the stream the
    # kernels run on)
    docs, news = make_docs(plans, 0)
    for _ in range(args.warmup):
        kvr.kvr_repair(ctx, docs, stream.cuda_stream)
    torch.cuda.synchronize()  # the warm-up repairs finish outside the wall clock
    t_wall = time.perf_counter()
    step_ms, ms = timed(docs, args.steps)
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    log(f"repair: mean {ms:.3f} ms, median {statistics.median(step_ms):.3f}, min {min(step_ms):.3f} "
        f"(wall {wall_ms / args.steps:.3f} ms/step)")

    # ---- the same K repairs again with the library's step profiler on: every
    # kernel is launched with a pair of HIP events that its dispatch records at
    # the start and end of its execution on this stream.  That gives the kernel
    # time per step and the dominant kernel's launch time; recording the events
    # slows the launches down, so this loop is kept apart from the timed one.
    kvr.kvr_profile_enable(ctx, True)
    kvr.kvr_profile_read(ctx)
    _, profiled_ms = timed(docs, args.steps)
    prof = kvr.kvr_profile_read(ctx)
    kvr.kvr_profile_enable(ctx, False)
    log(f"repair with the step profiler on: {profiled_ms:.3f} ms")

    # ---- the other edit placements (single-document workloads): same protocol
    per_seed = [round(ms, 4)]
    seed_edits = [plans[0][1]] if not batched else []
    if not batched:
        for sd in range(1, args.seeds):
            ps = plan_docs(wl, kvr, synth, sd)
            d_s, _ = make_docs(ps, sd)
            for _ in range(args.warmup):
                kvr.kvr_repair(ctx, d_s, stream.cuda_stream)
            per_seed.append(round(timed(d_s, args.steps)[1], 4))
            seed_edits.append(ps[0][1])
        log(f"per edit seed ms: {per_seed} (edits at {seed_edits}); median {statistics.median(per_seed):.3f}")
        docs, news = make_docs(plans, 0)  # restore seed 0's edited ids for the prefill baseline

    # ---- same-engine full re-prefill of every C' (one scratch cache, reused)
    pcache = torch.empty((L, 2, shape.n_kv_heads, n_max, shape.head_dim), dtype=torch.bfloat16, device=dev)
    psteps = 1 if batched else args.prefill_steps

    def prefill_all():
        for i, (n, e, A) in enumerate(plans):
            kvr.kvr_prefill(ctx, news[i].data_ptr(), n, n_max, pcache.data_ptr(), None, stream.cuda_stream)

    prefill_all()
    torch.cuda.synchronize()
    pev = [torch.cuda.Event(enable_timing=True) for _ in range(psteps + 1)]
    pev[0].record(stream)
    for i in range(psteps):
        prefill_all()
        pev[i + 1].record(stream)
    torch.cuda.synchronize()
    prefill_ms = statistics.median([pev[i].elapsed_time(pev[i + 1]) for i in range(psteps)])
    pflops = prefill_flops(shape, plans)
    prefill_tflops = pflops / (prefill_ms * 1e-3) / 1e12
    log(f"prefill of every edited context: median {prefill_ms:.2f} ms, {prefill_tflops:.0f} TFLOP/s algorithmic")
    libref = None
    if not batched:
        # one more prefill with the step profiler on: kernel time per step,
        # set beside the vendor library's GEMM and attention at the same shapes
        kvr.kvr_profile_enable(ctx, True)
        kvr.kvr_profile_read(ctx)
        prefill_all()
        pprof = kvr.kvr_profile_read(ctx)
        kvr.kvr_profile_enable(ctx, False)
        try:
            libref = library_reference(torch, shape, plans[0][0], pprof)
        except Exception as ex:  # the reference leg never costs the bench line
            libref = {"error": f"{type(ex).__name__}: {ex}"}
            log(f"library reference skipped: {libref['error']}")
    del pcache

    steps_ms = {k: round(v[0] / args.steps, 4) for k, v in prof.items() if v[1]}
    gu_ms, gu_n = prof["gate_up_swiglu"]
    kern_ms = gu_ms / gu_n
    log(f"kernel execution ms per repair by step: {steps_ms} (sum {sum(steps_ms.values()):.3f})")
    d_, F_ = shape.d_model, shape.d_ffn
    if R <= 64:
        kern_bytes = 2 * F_ * d_ * 2 + R * d_ * 2 + R * F_ * 2
        achieved = kern_bytes / (kern_ms * 1e-3) / 1e9
        traffic = None
        # HBM bytes per launch from the FETCH_SIZE / WRITE_SIZE counter passes,
        # valid only while the kernel source is the one the counters were taken on
        tfile = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                             "gateup_swiglu_llama8b_r48_traffic.md")
        if wl["shape"] == "llama3-8b" and R == 48 and os.path.exists(tfile):
            with open(tfile) as f:
                kv = dict(l.split(": ", 1) for l in f.read().splitlines() if l.startswith(("hbm_bytes", "kernel_source")))
            if kv.get("kernel_source_sha") == _kernel_sha():
                traffic = int(kv["hbm_bytes_per_launch"])
        roof = {"kernel": "gate/up projection + SwiGLU (linear_skinny_kernel, SWIGLU epilogue)", "bound": "hbm",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "algorithmic_bytes_per_launch": kern_bytes, "avg_launch_us": round(kern_ms * 1e3, 2)}
    else:
        kern_flops = 2 * R * 2 * F_ * d_
        achieved = kern_flops / (kern_ms * 1e-3) / 1e12
        roof = {"kernel": "gate/up projection + SwiGLU (linear_tiled_kernel, SWIGLU epilogue)", "bound": "mfma",
                "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                "algorithmic_flops_per_launch": kern_flops, "avg_launch_us": round(kern_ms * 1e3, 2),
                "issued_mfma_frac": round(2 * achieved / MFMA_BF16_PEAK_TFLOPS, 4)}
    log(f"gate/up+SwiGLU kernel: {kern_ms * 1e3:.1f} us/launch, {roof['achieved']} {roof['unit']}")

    # ---- fp64 CPU oracle on a bounded sample of the same repair
    cpu = None
    if not args.no_cpu:
        n0, e0, A0 = plans[0]
        cpu = cpu_baseline(shape, w, n0, e0, span, A0, min(args.cpu_layers, L), len(plans), torch)

    adj = None
    if not batched and not args.no_adjacent:
        adj = adjacent_rows(kvr, synth, torch, ctx, shape, plans[0], olds[0], news[0], caches[0], span, stream,
                            max(3, args.steps // 4))

    rbytes = repair_bytes(shape, plans, span)
    rflops = repair_flops(shape, plans, span)
    if batched:
        cfg = {"workload": f"{shape.name}-shaped batched repair: {len(plans)} documents of "
                           f"{wl['n_lo']}-{wl['n_hi']} tokens, one {span}-token edit each, {wl['policy']} K={K}",
               "docs": len(plans), "rows": R, "K": K, "policy": wl["policy"],
               "n_ctx_total": sum(n for n, _, _ in plans)}
        metric = "ms per batched repair call (64 docs, 8B shape); MFMA TFLOP/s; speedup vs re-prefill of every doc"
    else:
        n, e, A = plans[0]
        cfg = {"workload": f"{shape.name}-shaped repair, n={n}, {span}-token edit at {e}, {wl['policy']} K={K}, "
                           f"batch 1", "n_ctx": n, "edit": [e, e + span], "K": K, "rows": R,
               "policy": wl["policy"], "batch": 1}
        metric = "ms per repair @5k ctx K=32 (8B shape), HBM GB/s; speedup vs full re-prefill"
    out = {
        "metric": metric,
        "value": round(ms, 4),
        "unit": "ms/repair",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: random-init N(0,0.02) bf16 weights, uniform token ids, seeded edit",
        "config": cfg,
        "median_ms": round(statistics.median(step_ms), 4),
        "min_ms": round(min(step_ms), 4),
        "hbm_gb_s": round(rbytes / (ms * 1e-3) / 1e9, 1),
        "hbm_frac": round(rbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "algorithmic_bytes_per_repair": rbytes,
        "mfma_tflops": round(rflops / (ms * 1e-3) / 1e12, 2),
        "mfma_frac": round(rflops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        "algorithmic_flops_per_repair": rflops,
        "recomputed_tokens_per_s": round(R / (ms * 1e-3), 1),
        "token_layers_per_s": round(R * L / (ms * 1e-3), 1),
        "prefill_ms": round(prefill_ms, 3),
        "speedup_vs_prefill": round(prefill_ms / ms, 2),
        # the prefill is MFMA-bound: its algorithmic rate against the bf16 peak,
        # and the issued rate (every product of a compensated operand pair is
        # two MFMAs, so issued = 2 x algorithmic)
        "prefill_algorithmic_flops": pflops,
        "prefill_tflops": round(prefill_tflops, 1),
        "prefill_mfma_frac": round(prefill_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "prefill_issued_mfma_frac": round(2 * prefill_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "token_layer_proxy_speedup": round(sum(n for n, _, _ in plans) / R, 2),
        "kernel_ms_per_repair_by_step": steps_ms,
        "profiled_loop_ms": round(profiled_ms, 4),
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    if not batched:
        out["per_seed_ms"] = per_seed
        out["per_seed_edits"] = seed_edits
        out["median_over_seeds_ms"] = round(statistics.median(per_seed), 4)
    if adj is not None:
        out["adjacent_rows"] = adj
    if libref is not None:
        out["prefill_vs_library"] = libref
    print(json.dumps(out), flush=True)
    kvr.kvr_destroy(ctx)


def library_reference(torch, shape, n, pprof):
    """The prefill's projections and attention beside the vendor library at the
    same shapes.  Every product of the engine's compensated operand pairs is two
    MFMAs, so the like-for-like library figure is torch.matmul (hipBLASLt) with
    2n bf16 rows (the hi and lo halves stacked: the same issued MFMA work); the
    n-row figure is a plain single-operand bf16 GEMM.  Attention is torch's
    causal scaled_dot_product_attention over single bf16 operands, with the key
    and value heads expanded to the query heads.  Times are µs per layer (the
    engine's from its step profiler over one prefill)."""
    dev = torch.device("cuda:0")
    L, d, F = shape.n_layers, shape.d_model, shape.d_ffn
    hd, hq, hkv = shape.head_dim, shape.n_heads, shape.n_kv_heads
    s = torch.cuda.current_stream()

    def t_us(fn, reps=10):
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            fn()
        e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    def eng_us(step):
        ms_, cnt = pprof.get(step, (0.0, 0))
        return round(ms_ * 1e3 / L, 1) if cnt else None

    out = {"rows": n, "library": f"torch {torch.__version__} matmul / scaled_dot_product_attention, bf16"}
    gemms = {"qkv_proj": (d, (hq + 2 * hkv) * hd), "o_proj": (hq * hd, d),
             "gate_up_swiglu": (d, 2 * F), "down_proj": (F, d)}
    for step, (K, N) in gemms.items():
        w = torch.randn(N, K, device=dev, dtype=torch.bfloat16)
        a = torch.randn(2 * n, K, device=dev, dtype=torch.bfloat16)
        lib2 = t_us(lambda: torch.matmul(a, w.t()))
        a1 = a[:n]
        lib1 = t_us(lambda: torch.matmul(a1, w.t()))
        del a, a1, w
        e = eng_us(step)
        out[step] = {"engine_us": e, "library_us_2n_rows": round(lib2, 1), "library_us_n_rows": round(lib1, 1),
                     "engine_tflops_algorithmic": round(2 * n * N * K / (e * 1e-6) / 1e12, 1) if e else None}
    q = torch.randn(1, hq, n, hd, device=dev, dtype=torch.bfloat16)
    k = torch.randn(1, hkv, n, hd, device=dev, dtype=torch.bfloat16).repeat_interleave(hq // hkv, dim=1)
    v = torch.randn(1, hkv, n, hd, device=dev, dtype=torch.bfloat16).repeat_interleave(hq // hkv, dim=1)
    lib = t_us(lambda: torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True))
    del q, k, v
    e = eng_us("attention")
    out["attention"] = {"engine_us": e, "library_us": round(lib, 1)}
    log(f"prefill vs library (us per layer): {out}")
    return out


ADJ_SLOTS = 64     # cache slots past the context for appended query/answer tokens
ADJ_QUERY = 16     # query tokens of the scoring forward and the Attention selector
ADJ_ANSWER = 8     # answer tokens scored after the query
ADJ_GEN = 16       # greedy tokens generated (the flip test's continuation length)


def adjacent_rows(kvr, synth, torch, ctx, shape, plan, old, new, cache, span, stream, reps):
    """Times the steps around the repair on the same workload: the fresh-query
    scoring forward (query + answer teacher-forced, and a greedy continuation),
    the CacheBlend and Attention selectors, transplant of the repaired set, and
    the host selectors.  Each is enqueued `reps` times after two warmup calls
    and timed with HIP events on the stream the kernels run on."""
    n, e, A = plan
    L, es = shape.n_layers, 2
    dev = cache.device
    ncap = n + ADJ_SLOTS
    kvpos = shape.kv_bytes_per_pos(es)
    wbytes = L * shape.layer_params() * es
    lm_bytes = shape.vocab * shape.d_model * es
    # a cache with room for appended tokens: the repaired cache's rows [0, n)
    work = torch.empty((L, 2, shape.n_kv_heads, ncap, shape.head_dim), dtype=torch.bfloat16, device=dev)
    work[:, :, :, :n].copy_(cache)
    q_ids = synth.make_tokens(ADJ_QUERY + ADJ_ANSWER, shape.vocab, seed=77).to(dev)
    toks = torch.cat([new.to(dev), q_ids, torch.zeros(ADJ_SLOTS, dtype=torch.int32, device=dev)])
    s = stream.cuda_stream

    def time_it(fn):
        for _ in range(2):
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(reps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / reps

    out = {}
    m = ADJ_QUERY + ADJ_ANSWER
    lp = torch.empty(m, dtype=torch.float32, device=dev)
    am = torch.empty(m, dtype=torch.int32, device=dev)
    t = time_it(lambda: kvr.kvr_score(ctx, work.data_ptr(), n, ncap, toks.data_ptr(), m, lp.data_ptr(), am.data_ptr(), s))
    b = wbytes + lm_bytes + (n + m) * kvpos
    out["score"] = {"what": f"kvr_score: {ADJ_QUERY}-token query + {ADJ_ANSWER}-token answer after the {n}-token "
                            f"cache, teacher-forced log-probs and argmax", "ms": round(t, 4),
                    "algorithmic_bytes": b, "hbm_gb_s": round(b / (t * 1e-3) / 1e9, 1)}
    gtoks = toks.clone()
    t = time_it(lambda: kvr.kvr_generate(ctx, work.data_ptr(), n, ncap, gtoks.data_ptr(), ADJ_QUERY, ADJ_GEN, s))
    b = ADJ_GEN * (wbytes + lm_bytes) + ADJ_GEN * (n + ADJ_QUERY + ADJ_GEN) * kvpos
    out["generate"] = {"what": f"kvr_generate: {ADJ_QUERY}-token query then {ADJ_GEN} greedy tokens",
                       "ms": round(t, 4), "ms_per_token": round(t / ADJ_GEN, 4), "algorithmic_bytes": b,
                       "hbm_gb_s": round(b / (t * 1e-3) / 1e9, 1)}

    K = len(A)
    sel = torch.empty(max(K, 1), dtype=torch.int32, device=dev)
    # CacheBlend: layer 0 and the key/value projection of layer 1 over the
    # suffix [e, n) of C' (an MFMA-bound partial prefill), deviation, top-K
    t = time_it(lambda: kvr.kvr_select_cacheblend(ctx, cache.data_ptr(), n, n, new.data_ptr(), e, e + span, K, 1,
                                                  sel.data_ptr(), None, s))
    rows = n - e
    d, f = shape.d_model, shape.d_ffn
    fl = 2 * rows * (shape.layer_params() + d * 2 * shape.kv_dim) + 4 * shape.n_heads * shape.head_dim * \
        sum(p + 1 for p in range(e, n))
    out["select_cacheblend"] = {"what": f"kvr_select_cacheblend layer 1 (the paper's layer 2): {rows} suffix rows",
                                "ms": round(t, 4), "algorithmic_flops": fl,
                                "mfma_tflops": round(fl / (t * 1e-3) / 1e12, 1)}
    mass = torch.empty(n, dtype=torch.float32, device=dev)
    def attn_sel():
        kvr.kvr_select_attention(ctx, work.data_ptr(), n, ncap, toks.data_ptr(), ADJ_QUERY, e, e + span, K,
                                 sel.data_ptr(), mass.data_ptr(), s)

    t = time_it(attn_sel)
    # kernel times from a separate loop with the step profiler on
    kvr.kvr_profile_enable(ctx, True)
    kvr.kvr_profile_read(ctx)
    time_it(attn_sel)
    prof = kvr.kvr_profile_read(ctx)
    kvr.kvr_profile_enable(ctx, False)
    b = wbytes + n * kvpos + n * kvpos // 2
    mass_ms, mass_n = prof.get("attention_mass", (0.0, 0))
    mass_bytes = n * kvpos // 2  # every stale key read once per layer
    out["select_attention"] = {
        "what": f"kvr_select_attention: {ADJ_QUERY}-token query over the {n}-token stale cache, attention mass, top-K",
        "ms": round(t, 4), "algorithmic_bytes": b, "hbm_gb_s": round(b / (t * 1e-3) / 1e9, 1),
        "attention_mass_kernel_us": round(mass_ms / max(mass_n, 1) * 1e3, 2),
        "attention_mass_kernel_gb_s": round(mass_bytes / L / (mass_ms / max(mass_n, 1) * 1e-3) / 1e9, 1)
        if mass_n else None}
    P = list(range(e, e + span)) + list(A)
    pos = sorted(P)
    t = time_it(lambda: kvr.kvr_transplant(ctx, work.data_ptr(), ncap, cache.data_ptr(), n, pos, s))
    b = 2 * len(pos) * kvpos
    out["transplant"] = {"what": f"kvr_transplant of the {len(pos)} repaired positions, every layer and kv head",
                         "ms": round(t, 4), "algorithmic_bytes": b, "hbm_gb_s": round(b / (t * 1e-3) / 1e9, 1)}
    import time as _t
    t0 = _t.perf_counter()
    for i in range(1000):
        kvr.kvr_select(kvr.KVR_RANDOM, n, e, e + span, 512, i)
    # per call through the Python binding (1000 calls: total ms = us per call)
    out["select_random_k512_host_us"] = round((_t.perf_counter() - t0) * 1e3, 3)
    t0 = _t.perf_counter()
    for i in range(1000):
        kvr.kvr_select_to_boundary(n, e, e + span, min(n - 1, e + span + 64))
    out["select_to_boundary_host_us"] = round((_t.perf_counter() - t0) * 1e3, 3)
    log("adjacent rows: " + ", ".join(f"{k} {v['ms']:.3f} ms" for k, v in out.items() if isinstance(v, dict)))
    del work
    return out


def _kernel_sha():
    import hashlib
    p = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2609_17983_amd", "csrc", "gemm_skinny.hip")
    with open(p, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def cpu_baseline(shape, w, n, e, span, A, layers, n_docs, torch):
    """The fp64 oracle repairing the first `layers` layers of the (first
    document's) repair (same weights, a synthetic stale cache of the same
    shape), scaled to all layers and documents."""
    import numpy as np
    import synth
    from oracle import decoder as od
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count()
    log(f"cpu baseline: oracle over {layers} of {shape.n_layers} layers, {threads} BLAS threads")
    host = {"embed": w["embed"].cpu(), "final_norm": w["final_norm"].cpu(),
            "layers": [{k: (None if v is None else v.cpu()) for k, v in w["layers"][l].items()} for l in range(layers)]}

    class HostWeights:
        final_norm = host["final_norm"].to(torch.float64).numpy()

        def embed_rows(self, ids):
            return host["embed"][torch.as_tensor(np.asarray(ids))].to(torch.float64).numpy()

        def layer(self, l):
            return {k: (None if v is None else v.to(torch.float64).numpy()) for k, v in host["layers"][l].items()}

    stale = synth.make_stale_cache(shape, n, device="cuda")[:layers].to(torch.float64).cpu().numpy()
    toks = synth.apply_edit(synth.make_tokens(n, shape.vocab), e, span, shape.vocab).numpy()
    runs = []
    for _ in range(3):
        work = stale.copy()
        t0 = time.perf_counter()
        od.repair(shape, HostWeights(), work, toks, e, e + span, A, n_layers=layers)
        runs.append(time.perf_counter() - t0)
    dt = statistics.median(runs)
    per_repair_ms = dt * 1e3 * shape.n_layers / layers * n_docs
    log(f"cpu baseline: {[round(r, 2) for r in runs]} s for {layers} layers -> median {per_repair_ms:.0f} ms per repair")
    return {"value": round(per_repair_ms, 1), "unit": "ms/repair", "cores": threads, "kind": "oracle",
            "blas_threads": threads, "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "runs_s": [round(r, 3) for r in runs],
            "sample": f"fp64 numpy oracle repair of layers 0-{layers - 1} of {shape.n_layers} ({span + len(A)} rows, "
                      f"n={n}, bf16->fp64 weight upcast included), median of 3 runs, scaled "
                      f"x{shape.n_layers / layers * n_docs:g}{' (layers x documents)' if n_docs > 1 else ''}; "
                      f"median run {dt:.1f} s"}

if __name__ == "__main__":
    main()
