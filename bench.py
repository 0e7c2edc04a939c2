"""Rollout benchmark: batched generation on one MI355X at the Qwen2.5-7B shape.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

A step is one decode step of the whole hot path (embedding, 28 layers of
RMSNorm / q|k|v projection + RoPE + KV append / split-KV attention /
o-projection / SwiGLU MLP, final norm, LM head, log-softmax + Gumbel-max
sampling + log-probability) over the sequences still generating.  The
workload is the GRPO rollout of 32 prompts x 16 samples (uniform prompt
lengths in [256, 1024], lognormal response lengths around 1500 capped at
4096) on a randomly initialised bf16 decoder.

After W warm-up steps of a separate rollout, the whole rollout runs twice.
The first pass is the measurement: nothing is instrumented, and K decode
steps spread evenly over the rollout (every step with K = 0) are each timed
between device synchronisations; the whole pass is timed as well.  `value`
is the generated tokens of the K steps over their wall time.  The second pass
times the kernel classes with HIP events on the library's stream during the
same K steps, for the roofline of the dominant kernel.  Inputs and weights
are resident in HBM before timing starts; the prefill that opens the rollout
is timed and reported separately.

Prints one JSON line: generated tokens/s over the timed steps, their
algorithmic HBM GB/s (nominal: every row's whole context; unique: each GRPO
group's shared prompt once) with the fraction of the 8 TB/s peak, the same
time-weighted over the whole rollout, the roofline of the dominant kernel,
and the CPU oracle timed on a bounded sample on this host.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA


# HBM traffic of the attention kernel per algorithmic byte, from two
# rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) of this benchmark's
# default command, over the 2 x 4095 x 28 attention launches of its two
# rollout passes, each counter scaled by what it reads for the library's
# plain copy kernel of known size (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0):
# 505.4 MB fetched + 24.1 MB written per launch against 483.5 MB algorithmic
# (unique K/V: each group's shared prompt once).  Valid for the attention
# kernel and work-item layout as of that measurement (shared-prompt items of
# 256 keys, shorter in steps with few rows); set to None when either changes
# until the counters are taken again.
ATTN_TRAFFIC_PER_ALG_BYTE = 1.0950


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="rollout: decode steps to time, spread evenly over the whole rollout (default 32, 0 = "
                         "every step); score: GRPO groups (default 4); switch: rounds (default 3)")
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default="qwen7b")
    ap.add_argument("--slots", type=int, default=256, help="--stage continuous: KV slots (sequences in flight)")
    ap.add_argument("--emit-every", type=int, default=64, help="--stage continuous: responses per emitted chunk")
    ap.add_argument("--rows", default="1,8,16,32,64,128,256,512",
                    help="--stage curve: batch sizes (comma-separated)")
    ap.add_argument("--ctx", type=int, default=2048, help="--stage curve: context of every row")
    ap.add_argument("--stage", choices=("rollout", "score", "switch", "continuous", "embodied", "curve"),
                    default="rollout",
                    help="rollout: the decode hot path (default); score: the inference stage "
                         "(log-probabilities of given responses, one GRPO group per call); switch: "
                         "context-switch cost (weights and live K/V to pinned host memory and back); "
                         "continuous: the rollout's 512 sequences through fewer slots, continuous batching "
                         "with chunked emission against static batches of the same size; embodied: the "
                         "Llama-2-7B-shaped policy over 256 environments, env steps of prefill + 6 decode steps; "
                         "curve: decode steps at fixed batch sizes (--rows) and context (--ctx), per-class times")
    ap.add_argument("--no-tune", action="store_true",
                    help="keep the cost-model GEMM plans (skip the measured plans taken before warm-up)")
    ap.add_argument("--kv-page-size", type=int, default=0,
                    help="rollout stage: paged K/V pool with pages of this many positions (0: one contiguous "
                         "block per slot); the pool holds exactly the pages the rollout's sequences reach, "
                         "each group's full prompt pages once")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run the library's plain copy kernel over this many MiB, 4 times "
                         "(calibrates the FETCH_SIZE / WRITE_SIZE counters against a known size)")
    return ap.parse_args()


# Batch sizes at which the decode GEMM plans are measured before warm-up; a
# step of n rows uses the plan of the smallest listed size >= n.
TUNE_SIZES = (1, 2, 4, 8, 12, 16, 20, 24, 32, 40, 48, 64, 80, 96, 112, 128, 160, 192, 224, 256, 288, 320, 384,
              448, 512)


def tune_gemms(eng, max_rows: int, skip: bool):
    """Measure the GEMM plans up to max_rows rows (untimed set-up, like the
    warm-up); returns what was done for the JSON line.  Mixture-of-experts
    models keep the cost-model plans (their experts have their own kernel)."""
    if skip or eng.shape.moe:
        return {"measured": False}
    sizes = [n for n in TUNE_SIZES if n < max_rows] + [max_rows]
    t0 = time.perf_counter()
    eng.tune_gemms(sizes)
    el = time.perf_counter() - t0
    # the measured table is part of the run's configuration (the plan decides the fp32 summation order)
    table = {c: [eng.gemm_plan("gemm_" + c, n)[0] for n in sizes] for c in ("qkv", "o", "gate_up", "down", "lm_head")}
    return {"measured": True, "sizes": sizes, "seconds": round(el, 2),
            "plan_codes": table}


def measured_peaks():
    """HBM and matrix-core peaks measured on this GPU with the library's probes
    (a read-only stream and a copy of 2 GiB; 1024 workgroups x 4 waves x 4000
    rounds of 8 MFMA 32x32x16 bf16), best of 5 launches each, HIP events."""
    import torch

    from paper_2509_15965_amd.rl_decode import probe_copy, probe_mfma, probe_read
    dev = torch.device("cuda:0")
    nbytes = 2 << 30
    src = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    words = torch.empty(8192, dtype=torch.int32, device=dev)
    acc = torch.empty(4 * 1024, dtype=torch.float32, device=dev)

    def best(fn):
        fn()
        ms = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            ms.append(a.elapsed_time(b))
        return min(ms)

    t_read = best(lambda: probe_read(src, nbytes, words))
    t_copy = best(lambda: probe_copy(dst, src, nbytes))
    iters = 4000
    # one and four waves per SIMD (256 and 1024 workgroups of four waves)
    mfma = {nb: nb * 4 * iters * 8 * 32768.0 / (best(lambda nb=nb: probe_mfma(nb, iters, acc)) * 1e9)
            for nb in (256, 1024)}
    out = {"hbm_read_GBps": round(nbytes / (t_read * 1e6), 1),
           "hbm_copy_GBps": round(2 * nbytes / (t_copy * 1e6), 1),
           "mfma_bf16_TFLOPs": round(max(mfma.values()), 1),
           "mfma_bf16_TFLOPs_by_waves_per_simd": {"1": round(mfma[256], 1), "4": round(mfma[1024], 1)},
           "probe": "read-only stream and copy of 2 GiB (copy counts read + write bytes); 256 or 1024 "
                    f"workgroups x 4 waves x {iters} x 8 MFMA 32x32x16 bf16; best of 5"}
    del src, dst, words, acc
    torch.cuda.empty_cache()
    return out


def copy_probe(mib: int):
    import torch

    from paper_2509_15965_amd.rl_decode import probe_copy
    n = mib << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(4):
        probe_copy(dst, src, n)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n, "launches": 4}), flush=True)


def cpu_baseline_score(shape, weights, seconds: float):
    """Oracle inference-stage tokens/s on this host's cores: score() of a
    short prompt + response, fed one token at a time, until `seconds`."""
    import numpy as np

    import oracle
    from paper_2509_15965_amd.inputs import weights_to_host
    cores = len(os.sched_getaffinity(0))
    oracle.set_threads(cores)
    host = weights_to_host(weights)
    om = oracle.OracleModel(shape.as_dict(), host, oracle.MODE_BF16)
    rng = np.random.default_rng(5)
    n = 0
    t0 = time.perf_counter()
    while True:
        prompt = rng.integers(0, shape.vocab, size=4)
        resp = rng.integers(0, shape.vocab, size=4)
        oracle.score(om, prompt, resp, 1.0)
        n += 7                                    # forwards: prompt + response - 1
        el = time.perf_counter() - t0
        if el >= seconds or n >= 512:
            break
    del om, host
    return {"value": n / el, "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{n} scored-sequence tokens of the 7B-shape decoder (4-token prompts + 4-token "
                      f"responses, KV-cached one token at a time, fp64 accumulation), {el:.1f} s"}


def roofline_of(stats, classes):
    """Roofline entry of the class with the largest measured time."""
    dom = max(classes, key=lambda c: stats[c]["total_ms"])
    d = stats[dom]
    avg_ms = d["total_ms"] / max(1, d["launches"])
    gbs = d["alg_bytes"] / (d["total_ms"] * 1e-3) / 1e9
    tflops = d["alg_flops"] / (d["total_ms"] * 1e-3) / 1e12
    intensity = d["alg_flops"] / max(1.0, d["alg_bytes"])
    if intensity > BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tflops / BF16_PEAK_TFLOPS, 4), "traffic": None}
    else:
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None}
    roof.update({"kernel": dom, "launches": d["launches"], "avg_launch_ms": round(avg_ms, 5),
                 "alg_bytes_per_launch": round(d["alg_bytes"] / max(1, d["launches"])),
                 "alg_flops_per_launch": round(d["alg_flops"] / max(1, d["launches"]))})
    return dom, roof


def score_main(args):
    """Inference stage on the 7B-shape rollout: every step scores one GRPO
    group (its prompt once + its 16 responses) with rl_score."""
    import numpy as np
    import torch

    from paper_2509_15965_amd.configs import WORKLOADS
    from paper_2509_15965_amd.inputs import make_weights, rollout_plan
    from paper_2509_15965_amd.rl_decode import KERNEL_CLASSES, RL_OPT_PROFILE, Engine

    wl = WORKLOADS[args.workload]
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    plan = rollout_plan(wl)
    G = wl.group
    steps = args.steps if args.steps else 4
    warm = max(0, min(args.warmup, 1))
    n_groups = min(wl.n_prompts, steps + warm)
    plens, resp = plan["prompt_lens"], plan["response_lens"]
    rng = np.random.default_rng(wl.seed + 7)
    groups = []
    for p in range(n_groups):
        rl = resp[p * G:(p + 1) * G]
        rt = rng.integers(0, shape.vocab, size=int(rl.sum())).astype(np.int32)
        groups.append({"prompt": torch.as_tensor(plan["prompts"][p], device=dev),
                       "poffs": np.array([0, plens[p]], dtype=np.int32),
                       "roffs": np.concatenate([[0], np.cumsum(rl)]).astype(np.int32),
                       "resp": torch.as_tensor(rt, device=dev),
                       "out": torch.empty(int(rl.sum()), dtype=torch.float32, device=dev),
                       "tokens": int(plens[p] + rl.sum()), "scored": int(rl.sum())})
    weights = make_weights(shape, wl.seed, device=dev, init=wl.init)
    max_ctx = max(int(plens[p] + resp[p * G:(p + 1) * G].max()) for p in range(n_groups))
    max_tok = max(g["tokens"] for g in groups)
    eng = Engine(shape, weights, max_seqs=G, max_ctx=max_ctx, max_prefill_tokens=max_tok, device=dev)
    stream = eng.stream
    slots = list(range(G))

    def run(g):
        eng.score(slots, g["poffs"], g["prompt"], g["roffs"], g["resp"], g["out"], group=G,
                  temperature=wl.temperature)

    for g in groups[:warm]:
        run(g)
    torch.cuda.synchronize()
    timed = groups[warm:warm + steps]
    prof_classes = ("attention", "gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down", "gemm_lm_head", "sample")
    mask = 0
    for c in prof_classes:
        mask |= 1 << KERNEL_CLASSES.index(c)
    eng.reset_stats()
    eng.set_option(RL_OPT_PROFILE, mask)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i, g in enumerate(timed):
        run(g)
        print(f"[bench] score step {i + 1}/{len(timed)} enqueued", file=sys.stderr, flush=True)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    stats = eng.kernel_stats()
    eng.set_option(RL_OPT_PROFILE, 0)
    finite = all(bool(torch.isfinite(g["out"]).all()) for g in timed)
    tokens = sum(g["tokens"] for g in timed)
    scored = sum(g["scored"] for g in timed)
    dom, roof = roofline_of(stats, prof_classes)
    gemm_flops = sum(stats[c]["alg_flops"] for c in prof_classes if c.startswith("gemm"))
    gemm_ms = sum(stats[c]["total_ms"] for c in prof_classes if c.startswith("gemm"))
    classes = {c: {"launches": stats[c]["launches"], "ms": round(stats[c]["total_ms"], 3),
                   "TFLOP/s": round(stats[c]["alg_flops"] / (stats[c]["total_ms"] * 1e9), 1)
                   if stats[c]["total_ms"] > 0 and stats[c]["alg_flops"] > 0 else None}
               for c in prof_classes}
    out = {
        "metric": "inference-stage tokens/sec (1 GPU) at 7B shape: prompt + response tokens through the "
                  "scoring forward",
        "value": round(tokens / wall, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": len(timed),
        "warmup": warm,
        "ms_per_step": round(wall * 1e3 / max(1, len(timed)), 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, uniform prompt and response tokens)",
        "config": {"workload": f"{wl.name} inference stage: one GRPO group ({G} responses of one prompt) per "
                               f"rl_score call; prompts U[{wl.prompt_len[0]},{wl.prompt_len[1]}], lognormal "
                               f"responses (median {wl.response_median}, cap {wl.response_cap})",
                   "tokens_timed": tokens, "scored_tokens_timed": scored},
        "scored_tokens_per_s": round(scored / wall, 1),
        "gpu_ms_timed": round(gpu_ms, 2),
        "gemm_TFLOPs": round(gemm_flops / (gemm_ms * 1e9), 1) if gemm_ms > 0 else None,
        "all_finite": finite,
        "roofline": roof,
        "timed_classes": classes,
    }
    eng.close()
    del eng
    torch.cuda.synchronize()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_score(shape, weights, args.cpu_seconds)
    print(json.dumps(out), flush=True)


PCIE_PEAK_GBS = 64.0           # PCIe 5.0 x16, one direction


def switch_main(args):
    """Temporal-mode context switch of the 7B-shape rollout engine: the
    weights (caller tensors) and the live K/V of the 512 sequences right
    after the rollout's prefill go to pinned host memory and come back."""
    import numpy as np
    import torch

    from paper_2509_15965_amd.configs import WORKLOADS
    from paper_2509_15965_amd.inputs import make_weights, rollout_plan
    from paper_2509_15965_amd.rl_decode import Engine

    wl = WORKLOADS[args.workload]
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    peaks = measured_peaks()
    print(f"[bench] measured peaks: {peaks}", file=sys.stderr, flush=True)
    plan = rollout_plan(wl)
    P, G = wl.n_prompts, wl.group
    n = P * G
    plens = plan["prompt_lens"]
    weights = make_weights(shape, wl.seed, device=dev, init=wl.init)
    eng = Engine(shape, weights, max_seqs=n, max_ctx=int(plens.max() + plan["response_lens"].max()),
                 max_prefill_tokens=int(plens.sum()), device=dev)
    slots = np.arange(n, dtype=np.int32)
    offs = np.concatenate([[0], np.cumsum(plens)]).astype(np.int32)
    tok = torch.as_tensor(np.concatenate(plan["prompts"]), dtype=torch.int32, device=dev)
    ot = torch.empty(n, dtype=torch.int32, device=dev)
    ol = torch.empty(n, dtype=torch.float32, device=dev)
    eng.prefill(slots, plan["uids"], offs, tok, ot, ol, group=G, seed=1)
    torch.cuda.synchronize()
    kv_bytes = eng.kv_offload_bytes(slots)
    host_kv = torch.empty(kv_bytes, dtype=torch.uint8, pin_memory=True)
    host_w = {k: torch.empty(v.shape, dtype=v.dtype, pin_memory=True) for k, v in weights.items()}
    w_bytes = sum(v.numel() * v.element_size() for v in weights.values())
    stream = eng.stream
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    res = []
    reps = max(1, args.steps if args.steps else 3)
    for r in range(reps + 1):
        torch.cuda.synchronize()
        ev[0].record(stream)
        with torch.cuda.stream(stream):
            for k, v in weights.items():
                host_w[k].copy_(v, non_blocking=True)
        ev[1].record(stream)
        eng.kv_offload(slots, host_kv)
        ev[2].record(stream)
        with torch.cuda.stream(stream):
            for k, v in weights.items():
                v.copy_(host_w[k], non_blocking=True)
        ev[3].record(stream)
        eng.kv_onload(slots, [eng.slot_length(int(s)) for s in slots], host_kv)
        ev[4].record(stream)
        torch.cuda.synchronize()
        if r > 0:                                 # the first round is warm-up
            res.append([ev[i].elapsed_time(ev[i + 1]) for i in range(4)])
        print(f"[bench] switch round {r + 1}/{reps + 1}", file=sys.stderr, flush=True)
    ms = np.median(np.array(res), axis=0)
    gbs = [w_bytes / (ms[0] * 1e6), kv_bytes / (ms[1] * 1e6), w_bytes / (ms[2] * 1e6), kv_bytes / (ms[3] * 1e6)]
    out = {
        "metric": "context-switch time (1 GPU) at 7B shape: weights + live K/V offloaded to pinned host memory "
                  "and reloaded",
        "value": round(float(ms.sum()) / 1e3, 4),
        "unit": "s",
        "n_gpus": 1,
        "steps": reps,
        "warmup": 1,
        "ms_per_step": round(float(ms.sum()), 2),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, the rollout's prefilled K/V)",
        "config": {"workload": f"{wl.name}: weights {w_bytes / 1e9:.2f} GB; live K/V of {n} sequences after the "
                               f"prefill ({int(plens.sum())} prompt tokens) {kv_bytes / 1e9:.3f} GB"},
        "ms": {"weights_offload": round(float(ms[0]), 2), "kv_offload": round(float(ms[1]), 2),
               "weights_onload": round(float(ms[2]), 2), "kv_onload": round(float(ms[3]), 2)},
        "GBps": {"weights_offload": round(gbs[0], 1), "kv_offload": round(gbs[1], 1),
                 "weights_onload": round(gbs[2], 1), "kv_onload": round(gbs[3], 1)},
        "roofline": {"bound": "pcie", "achieved": round((2 * w_bytes + 2 * kv_bytes) / (float(ms.sum()) * 1e6), 1),
                     "peak": PCIE_PEAK_GBS, "unit": "GB/s",
                     "frac": round((2 * w_bytes + 2 * kv_bytes) / (float(ms.sum()) * 1e6) / PCIE_PEAK_GBS, 4),
                     "traffic": None},
    }
    eng.close()
    print(json.dumps(out), flush=True)


def continuous_main(args):
    """The 7B rollout's 512 sequences (32 GRPO groups of 16) through
    args.slots slots: static batches one after another (each runs until its
    longest response ends) against continuous batching (groups admitted as
    slots free up), which also hands finished responses downstream in chunks
    of args.emit_every."""
    import numpy as np
    import torch

    from paper_2509_15965_amd.configs import WORKLOADS
    from paper_2509_15965_amd.inputs import make_weights, rollout_plan
    from paper_2509_15965_amd.rl_decode import Engine
    from paper_2509_15965_amd.rollout import ContinuousRollout, StaticRollout

    wl = WORKLOADS[args.workload]
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    peaks = measured_peaks()
    print(f"[bench] measured peaks: {peaks}", file=sys.stderr, flush=True)
    plan = rollout_plan(wl)
    P, G = wl.n_prompts, wl.group
    S = args.slots
    if S % G or S < G:
        raise SystemExit("--slots must be a multiple of the group size")
    plens, resp, uids = plan["prompt_lens"], plan["response_lens"], plan["uids"]
    weights = make_weights(shape, wl.seed, device=dev, init=wl.init)
    per = S // G                                          # prompts per static batch
    eng = Engine(shape, weights, max_seqs=S, max_ctx=int(plens.max() + resp.max()),
                 max_prefill_tokens=int(max(plens[i:i + per].sum() for i in range(0, P, per))), device=dev)
    seed, T = 20250919, wl.temperature
    tuning = tune_gemms(eng, S, args.no_tune)
    # warm-up: a short static run
    w = StaticRollout(eng, plan["prompts"][:per], G, np.minimum(resp[:S], 16), uids[:S], seed, T)
    w.run()
    torch.cuda.synchronize()
    # static batches of S sequences, one after another
    t0 = time.perf_counter()
    gen_static = 0
    for b in range(0, P, per):
        ro = StaticRollout(eng, plan["prompts"][b:b + per], G, resp[b * G:(b + per) * G], uids[b * G:(b + per) * G],
                           seed, T)
        gen_static += ro.run() + ro.n
        print(f"[bench] static batch {b // per + 1}/{-(-P // per)} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t_static = time.perf_counter() - t0
    # continuous batching over the same slots
    marks = []
    t0 = time.perf_counter()

    def on_emit(chunk):
        marks.append((time.perf_counter() - t0, len(chunk)))
        if len(marks) % 4 == 1:
            print(f"[bench] continuous: chunk {len(marks)} emitted", file=sys.stderr, flush=True)

    ro = ContinuousRollout(eng, plan["prompts"], G, resp, uids, seed, T, n_slots=S, emit_every=args.emit_every,
                           on_emit=on_emit)
    gen_cont = ro.run()
    torch.cuda.synchronize()
    t_cont = time.perf_counter() - t0
    eng.close()
    out = {
        "metric": f"continuous-batching rollout tokens/sec (1 GPU) at 7B shape, {P * G} sequences through {S} slots",
        "value": round(gen_cont / t_cont, 1),
        "unit": "generated tokens/s",
        "n_gpus": 1,
        "steps": ro.steps,
        "warmup": 16,
        "ms_per_step": round(t_cont * 1e3 / max(1, ro.steps), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init weights and uniform prompt tokens)",
        "config": {"workload": f"{wl.name}: {P} prompts x {G} samples, lognormal responses (median "
                               f"{wl.response_median}, cap {wl.response_cap}); {S} slots; chunks of "
                               f"{args.emit_every} responses",
                   "generated_tokens": int(gen_cont)},
        "static_batches": {"batches": -(-P // per), "seconds": round(t_static, 3),
                           "tokens_per_s": round(gen_static / t_static, 1)},
        "continuous": {"seconds": round(t_cont, 3), "decode_steps": ro.steps},
        "speedup_vs_static": round(t_static / t_cont, 3),
        "first_chunk_s": round(marks[0][0], 3) if marks else None,
        "chunk_times_s": [round(m[0], 2) for m in marks],
        "gemm_plans": tuning,
    }
    print(json.dumps(out), flush=True)


def rollout_step_bytes(shape, plens, resp, group, steps):
    """Algorithmic HBM bytes of every decode step of a static rollout (the
    sequences ordered longest first, decode step t appending position
    plen + t): the decode-read parameters, every active row's K/V context and
    new K/V row, its embedding row and 12 bytes of token / log-probability.
    Returns (nominal, unique): nominal counts every row's whole context;
    unique counts each GRPO group's shared prompt (whole 32-position steps,
    as the attention reads it) once per step while any member is active."""
    import numpy as np
    es = shape.elem_bytes
    kv_tok = shape.kv_bytes_per_token()
    fixed = shape.decode_params() * es
    plens = np.asarray(plens, dtype=np.int64)
    resp = np.asarray(resp, dtype=np.int64)
    n_seq = len(resp)
    seq_plen = np.repeat(plens, group)
    grp = np.arange(n_seq) // group
    shared = seq_plen // 32 * 32
    nominal = np.zeros(steps)
    unique = np.zeros(steps)
    for t in range(steps):
        act = resp > t + 1
        n = int(act.sum())
        ctx = seq_plen[act] + t + 1
        per_row = n * (kv_tok + shape.hidden * es + 12)
        if shape.moe:   # the experts that n rows reach (expected, uniform routing)
            fixed = shape.decode_params(active_experts=expected_experts(shape, n)) * es
        nominal[t] = fixed + per_row + float(ctx.sum()) * kv_tok
        own = ctx - (shared[act] if group > 1 else 0)
        groups_live = np.unique(grp[act]) if group > 1 else np.array([], dtype=np.int64)
        prompt_once = float(shared[groups_live * group].sum()) if group > 1 else 0.0
        unique[t] = fixed + per_row + (float(own.sum()) + prompt_once) * kv_tok
    return nominal, unique


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline_rollout(shape, weights, seconds: float):
    """Oracle decode tokens/s on this host: one new token per sequence at
    the 7B rollout's mean starting context (641), with a seeded N(0, 1) K/V
    cache of 640 positions, first on all host cores, then on one thread."""
    import numpy as np

    import oracle
    from paper_2509_15965_amd.inputs import weights_to_host
    cores = len(os.sched_getaffinity(0))
    host = weights_to_host(weights)
    om = oracle.OracleModel(shape.as_dict(), host, oracle.MODE_BF16)
    ctx = 640
    rng = np.random.default_rng(11)
    base = om.new_seq(ctx + 1)
    for l in range(shape.n_layers):
        for g in range(shape.n_kv_heads):
            K = rng.standard_normal((ctx, shape.head_dim))
            V = rng.standard_normal((ctx, shape.head_dim))
            base.set_kv_block(l, g, K, V)
    base.set_length(ctx)

    def timed(threads, budget, cap):
        oracle.set_threads(threads)
        n, el = 0, 0.0
        while el < budget and n < cap:
            s = base.clone()
            t0 = time.perf_counter()
            s.forward(1 + n)
            el += time.perf_counter() - t0
            n += 1
            del s
        return n, el, oracle.num_threads()

    n, el, used = timed(cores, seconds, 256)
    n1, el1, _ = timed(1, max(1.0, seconds * 0.6), 2)
    del om, host, base
    return {"value": round(n / el, 4), "unit": "tokens/s", "cores": used, "kind": "oracle",
            "sample": f"{n} decode tokens of the 7B-shape decoder at context {ctx + 1} (seeded N(0,1) K/V "
                      f"cache, one token per sequence, fp64 accumulation) in {el:.1f} s on {used} threads; "
                      f"single thread: {n1} tokens in {el1:.1f} s",
            "single_thread_value": round(n1 / el1, 4), "cpu_model": cpu_model()}


def describe_shape(m):
    mlp = (f"{m.n_experts} experts of width {m.expert_ffn}, top {m.top_k}" if m.moe else f"ffn {m.ffn}")
    return (f"{m.n_layers} layers, hidden {m.hidden}, {m.n_q_heads} q / {m.n_kv_heads} kv heads of {m.head_dim}, "
            f"{mlp}, vocab {m.vocab}, {m.dtype}")


def expected_experts(shape, n: int) -> float:
    """Distinct experts a layer reads for n rows when each row's top-k is a
    uniform draw without replacement (random-init routers are near uniform)."""
    E, k = shape.n_experts, shape.top_k
    return E * (1.0 - (1.0 - k / E) ** n)


def embodied_main(args):
    """The embodied workload (Llama-2-7B-shaped policy, 256 parallel
    environments), one env step at a time: every env's observation is a
    fresh prefill of 256 caller-provided patch rows (seeded N(0, 1) per env
    and step) plus 32 text tokens, then 6 decode steps for the remaining
    action tokens (7 per env step, the first sampled by the prefill); the K/V
    of the previous step is dropped.  K env steps are timed after W warm-up
    env steps."""
    import numpy as np
    import torch

    from paper_2509_15965_amd.configs import WORKLOADS
    from paper_2509_15965_amd.inputs import make_weights, patch_rows
    from paper_2509_15965_amd.rl_decode import Engine

    wl = WORKLOADS["llama7b-embodied"]
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    E, R, TXT, ACT = wl.n_prompts, wl.patch_rows, wl.prompt_len[0], wl.response_cap
    plen = R + TXT
    weights = make_weights(shape, wl.seed, device=dev, init=wl.init)
    eng = Engine(shape, weights, max_seqs=E, max_ctx=plen + ACT, max_prefill_tokens=E * plen, device=dev)
    stream = eng.stream
    tuning = tune_gemms(eng, E, args.no_tune)
    slots = np.arange(E, dtype=np.int32)
    offs = (np.arange(E + 1) * plen).astype(np.int32)
    rng = np.random.default_rng(wl.seed)
    text = torch.as_tensor(rng.integers(0, shape.vocab, size=(E, TXT)).astype(np.int32), device=dev)
    # prompt ids: -(e*R + r) - 1 selects patch row r of env e, then the text tokens
    rows_id = -(torch.arange(E * R, device=dev, dtype=torch.int32).view(E, R) + 1)
    tokens = torch.cat([rows_id, text], dim=1).reshape(-1).contiguous()
    toks = torch.empty((ACT, E), dtype=torch.int32, device=dev)
    logps = torch.empty((ACT, E), dtype=torch.float32, device=dev)
    n_env_steps = args.steps if args.steps else 4
    warm = min(args.warmup, 1)
    seed, T = 20250919, wl.temperature
    kv_tok = shape.kv_bytes_per_token()

    def observe(k):
        return patch_rows(E * R, shape.hidden, wl.seed * 1000 + k, device=dev)

    def env_step(k, emb, timing=None):
        uids = (np.arange(E, dtype=np.uint64) * np.uint64(wl.env_steps) + np.uint64(k))
        eng.release(slots)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(stream)
        eng.prefill(slots, uids, offs, tokens, toks[0], logps[0], group=1, embeds=emb, seed=seed, temperature=T)
        ev[1].record(stream)
        for j in range(1, ACT):
            eng.step(slots, uids, toks[j - 1], toks[j], logps[j], seed=seed, temperature=T)
        ev[2].record(stream)
        if timing is not None:
            timing.append(ev)

    for k in range(warm):
        env_step(10_000 + k, observe(10_000 + k))
    # the observations (the environments' output) exist before the timed region
    obs = [observe(k) for k in range(n_env_steps)]
    torch.cuda.synchronize()
    timing = []
    t0 = time.perf_counter()
    for k in range(n_env_steps):
        env_step(k, obs[k], timing)
        print(f"[bench] env step {k + 1}/{n_env_steps} enqueued", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    pre_ms = sum(e[0].elapsed_time(e[1]) for e in timing)
    dec_ms = sum(e[1].elapsed_time(e[2]) for e in timing)
    # decode-step algorithmic bytes: parameters + every env's K/V context and new row + embedding row
    dec_bytes = sum(shape.decode_params() * shape.elem_bytes + E * ((plen + j + 1) * kv_tok + kv_tok +
                                                                    shape.hidden * shape.elem_bytes + 12)
                    for j in range(ACT - 1)) * n_env_steps
    L, H, F, V = shape.n_layers, shape.hidden, shape.ffn, shape.vocab
    qkv = (shape.n_q_heads + 2 * shape.n_kv_heads) * shape.head_dim
    pre_flops = (2.0 * E * plen * (L * (H * qkv + shape.n_q_heads * shape.head_dim * H + 3 * H * F)) +
                 2.0 * E * H * V + 4.0 * L * shape.n_q_heads * shape.head_dim * E * plen * (plen + 1) / 2) * n_env_steps
    finite = bool(torch.isfinite(logps).all())
    out = {
        "metric": "embodied rollout env-steps/sec (1 GPU), Llama-2-7B-shaped policy, 256 envs",
        "value": round(E * n_env_steps / wall, 2),
        "unit": "env steps/s",
        "n_gpus": 1,
        "steps": n_env_steps,
        "warmup": warm,
        "ms_per_step": round(wall * 1e3 / n_env_steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": f"synthetic (seeded random-init weights, {wl.init} init; N(0,1) patch rows, uniform text tokens)",
        "config": {"workload": f"{wl.name}: {describe_shape(shape)}; {E} envs, each env step a fresh prefill of "
                               f"{R} patch rows + {TXT} text tokens then {ACT - 1} decode steps ({ACT} action "
                               f"tokens), K/V dropped between env steps"},
        "action_tokens_per_s": round(E * ACT * n_env_steps / wall, 1),
        "prefill_ms_per_env_step": round(pre_ms / n_env_steps, 3),
        "decode_ms_per_env_step": round(dec_ms / n_env_steps, 3),
        "prefill_TFLOPs": round(pre_flops / (pre_ms * 1e9), 1),
        "prefill_mfma_frac": round(pre_flops / (pre_ms * 1e9) / BF16_PEAK_TFLOPS, 4),
        "decode_step_alg_GBps": round(dec_bytes / (dec_ms * 1e6), 1),
        "decode_step_hbm_frac": round(dec_bytes / (dec_ms * 1e6) / HBM_PEAK_GBS, 4),
        "all_finite": finite,
        "gemm_plans": tuning,
    }
    eng.close()
    print(json.dumps(out), flush=True)


def curve_main(args):
    """Decode-step time against batch size: for every n in --rows, n rows of
    --ctx positions each (own K/V, no shared prompt; seeded N(0, 1) cache),
    W warm-up steps, then K timed steps (one event pair around all K), then
    the same K steps again with every kernel class timed by HIP events.
    Algorithmic bytes per step: the decode-read parameters plus every row's
    K/V context, new K/V row, embedding row and 12 bytes of token /
    log-probability; algorithmic flops: 2 per parameter and row plus the
    attention's 4 * q-heads * head_dim per row and key."""
    import torch

    from paper_2509_15965_amd.configs import WORKLOADS
    from paper_2509_15965_amd.inputs import make_weights
    from paper_2509_15965_amd.rl_decode import KERNEL_CLASSES, RL_OPT_PROFILE, Engine

    wl = WORKLOADS[args.workload]
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rows = [int(x) for x in args.rows.split(",")]
    K = args.steps if args.steps else 10
    W = min(args.warmup, 3)
    ctx = args.ctx
    weights = make_weights(shape, wl.seed, device=dev, init=wl.init)
    eng = Engine(shape, weights, max_seqs=max(rows), max_ctx=ctx + W + 2 * K + 2, max_prefill_tokens=8,
                 device=dev)
    stream = eng.stream
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seed)
    kc, vc = eng.kv_views()
    kc.normal_(generator=gen)
    vc.normal_(generator=gen)
    tuning = tune_gemms(eng, max(rows), args.no_tune)
    es, kv_tok = shape.elem_bytes, shape.kv_bytes_per_token()
    all_mask = (1 << len(KERNEL_CLASSES)) - 1
    curve = []
    for n in rows:
        slots = list(range(n))
        tok = torch.randint(0, shape.vocab, (n,), dtype=torch.int32, device=dev, generator=gen)
        ot = torch.empty(n, dtype=torch.int32, device=dev)
        ol = torch.empty(n, dtype=torch.float32, device=dev)
        eng.set_lengths(slots, [ctx] * n)
        for _ in range(W):
            eng.step(slots, slots, tok, ot, ol)
        eng.set_lengths(slots, [ctx] * n)
        torch.cuda.synchronize()
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ea.record(stream)
        for _ in range(K):
            eng.step(slots, slots, tok, ot, ol)
        eb.record(stream)
        torch.cuda.synchronize()
        ms = ea.elapsed_time(eb) / K
        eng.set_lengths(slots, [ctx] * n)
        eng.reset_stats()
        eng.set_option(RL_OPT_PROFILE, all_mask)
        for _ in range(K):
            eng.step(slots, slots, tok, ot, ol)
        eng.set_option(RL_OPT_PROFILE, 0)
        torch.cuda.synchronize()
        st = eng.kernel_stats()
        # mean context over the K timed steps: ctx + (K - 1) / 2 keys before the new one
        mean_ctx = ctx + (K - 1) / 2.0
        step_bytes = shape.decode_params() * es + n * ((mean_ctx + 1) * kv_tok + kv_tok + shape.hidden * es + 12)
        classes = {}
        for c in KERNEL_CLASSES:
            d = st[c]
            if d["launches"] == 0:
                continue
            e = {"ms_per_step": round(d["total_ms"] / K, 4)}
            if c.startswith("gemm") and d["total_ms"] > 0:
                tf = d["alg_flops"] / (d["total_ms"] * 1e9)
                e.update({"TFLOPs": round(tf, 1), "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4),
                          "GBps": round(d["alg_bytes"] / (d["total_ms"] * 1e6), 1)})
            elif d["total_ms"] > 0:
                e["GBps"] = round(d["alg_bytes"] / (d["total_ms"] * 1e6), 1)
            classes[c] = e
        gbs = step_bytes / (ms * 1e6)
        curve.append({"rows": n, "ctx": ctx, "ms_per_step": round(ms, 4),
                      "tokens_per_s": round(n / (ms * 1e-3), 1), "alg_GBps": round(gbs, 1),
                      "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                      "profiled_ms_per_step": round(sum(st[c]["total_ms"] for c in KERNEL_CLASSES) / K, 4),
                      "classes": classes})
        print(f"[bench] rows {n}: {ms:.3f} ms per step", file=sys.stderr, flush=True)
    eng.close()
    out = {"metric": "decode-step time by batch size (1 GPU)", "unit": "ms/step", "n_gpus": 1, "steps": K,
           "warmup": W, "higher_is_better": False, "dtype": "bf16",
           "data": f"synthetic (seeded random-init weights, {wl.init} init; N(0,1) K/V cache)",
           "config": {"workload": f"{wl.name}: {describe_shape(shape)}; every row {ctx} positions of its own "
                                  f"K/V (no shared prompt)"},
           "gemm_plans": tuning, "curve": curve}
    print(json.dumps(out), flush=True)


def sample_steps(max_steps: int, k: int):
    """k decode steps spread evenly over the rollout (all steps when k <= 0
    or k >= max_steps)."""
    if k <= 0 or k >= max_steps:
        return list(range(max_steps))
    if k == 1:
        return [0]
    return sorted({round(j * (max_steps - 1) / (k - 1)) for j in range(k)})


def main():
    args = parse()
    if args.copy_probe_mib > 0:
        copy_probe(args.copy_probe_mib)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    if args.stage == "score":
        score_main(args)
        return
    if args.stage == "switch":
        switch_main(args)
        return
    if args.stage == "continuous":
        continuous_main(args)
        return
    if args.stage == "embodied":
        embodied_main(args)
        return
    if args.stage == "curve":
        curve_main(args)
        return
    import numpy as np
    import torch

    from paper_2509_15965_amd.configs import WORKLOADS
    from paper_2509_15965_amd.inputs import make_weights, rollout_plan
    from paper_2509_15965_amd.rl_decode import KERNEL_CLASSES, RL_OPT_PROFILE, Engine
    from paper_2509_15965_amd.rollout import StaticRollout

    wl = WORKLOADS[args.workload]
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    peaks = measured_peaks()
    print(f"[bench] measured peaks: {peaks}", file=sys.stderr, flush=True)
    plan = rollout_plan(wl)
    P, G = wl.n_prompts, wl.group
    n_seq = P * G
    plens = plan["prompt_lens"]
    resp = plan["response_lens"]
    weights = make_weights(shape, wl.seed, device=dev, init=wl.init)
    max_ctx = int(plens.max() + resp.max())
    page = args.kv_page_size
    if shape.moe and page == 0:
        # the mixture-of-experts workload's contiguous pool (512 slots x 5120
        # positions x 98 KB) would not fit beside its 61 GB of weights
        page = 256
    # a finished sequence keeps its pages until the next prefill, so the pool
    # needs the pages of every sequence's final length; a group holds the
    # pages its prompt fills once
    final_len = np.repeat(plens, G) + resp
    shared = np.repeat(plens // page, G) if page else 0
    kv_pages = int((plens // page).sum() + ((final_len + page - 1) // page - shared).sum()) if page else 0
    eng = Engine(shape, weights, max_seqs=n_seq, max_ctx=max_ctx, max_prefill_tokens=int(plens.sum()),
                 device=dev, kv_page_size=page, kv_pages=kv_pages)
    kv_pool = {"page": page or None, "pages": kv_pages or n_seq, "bytes": eng.kv_nbytes}
    stream = eng.stream

    # the rollout driver orders slots by response length (longest first), so
    # the active set of decode step t is always a prefix of that order
    seed, T = 20250919, wl.temperature
    ro = StaticRollout(eng, plan["prompts"], G, resp, plan["uids"], seed=seed, temperature=T)
    max_steps = ro.max_steps
    sampled = sample_steps(max_steps, 32 if args.steps is None else args.steps)
    is_sampled = np.zeros(max_steps, dtype=bool)
    is_sampled[sampled] = True
    nominal, unique = rollout_step_bytes(shape, plens, resp, G, max_steps)

    # ---- measured GEMM plans and warm-up (untimed) ----
    tuning = tune_gemms(eng, n_seq, args.no_tune)
    print(f"[bench] GEMM plans: {tuning}", file=sys.stderr, flush=True)
    ro.prefill()
    for t in range(min(args.warmup, max_steps)):
        ro.step(t)
    torch.cuda.synchronize()
    print(f"[bench] warm-up done; timing {len(sampled)} of {max_steps} decode steps", file=sys.stderr, flush=True)

    # ---- pass 1: the whole rollout, profiling off; the sampled steps are
    # each bracketed by device synchronisation and timed ----
    t_pf0 = time.perf_counter()
    ro.prefill()
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - t_pf0
    ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e_all0, e_all1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall_t, gpu_t, gen_t = [], [], []
    gen_all = 0
    torch.cuda.synchronize()
    t_all0 = time.perf_counter()
    e_all0.record(stream)
    last_print = t_all0
    for t in range(max_steps):
        if is_sampled[t]:
            torch.cuda.synchronize()
            w0 = time.perf_counter()
            ea.record(stream)
            n = ro.step(t)
            eb.record(stream)
            torch.cuda.synchronize()
            wall_t.append(time.perf_counter() - w0)
            gpu_t.append(ea.elapsed_time(eb) * 1e-3)
            gen_t.append(n)
        else:
            n = ro.step(t)
        gen_all += n
        now = time.perf_counter()
        if now - last_print > 20.0:
            print(f"[bench] measured pass: step {t + 1}/{max_steps}", file=sys.stderr, flush=True)
            last_print = now
    e_all1.record(stream)
    torch.cuda.synchronize()
    rollout_wall = time.perf_counter() - t_all0
    rollout_gpu = e_all0.elapsed_time(e_all1) * 1e-3

    # ---- pass 2: the same rollout again, kernel classes timed with HIP
    # events on the library's stream during the sampled steps only ----
    prof_classes = ("attention", "gemm_gate_up", "gemm_down", "gemm_lm_head", "gemm_qkv", "gemm_o")
    if shape.moe:
        prof_classes = ("attention", "moe_experts", "moe_route", "gemm_lm_head", "gemm_qkv", "gemm_o")
    mask = 0
    for c in prof_classes:
        mask |= 1 << KERNEL_CLASSES.index(c)
    ro.prefill()
    torch.cuda.synchronize()
    eng.reset_stats()
    last_print = time.perf_counter()
    for t in range(max_steps):
        if is_sampled[t]:
            eng.set_option(RL_OPT_PROFILE, mask)
            ro.step(t)
            eng.set_option(RL_OPT_PROFILE, 0)
        else:
            ro.step(t)
        now = time.perf_counter()
        if now - last_print > 20.0:
            print(f"[bench] profiled pass: step {t + 1}/{max_steps}", file=sys.stderr, flush=True)
            last_print = now
    torch.cuda.synchronize()
    stats = eng.kernel_stats()

    dom, roof = roofline_of(stats, prof_classes)
    roof.pop("alg_flops_per_launch")
    roof["frac_of_measured_peak"] = round(roof["achieved"] / (peaks["hbm_read_GBps"] if roof["bound"] == "hbm"
                                                              else peaks["mfma_bf16_TFLOPs"]), 4)
    d = stats[dom]
    if dom == "attention" and ATTN_TRAFFIC_PER_ALG_BYTE is not None:
        roof["traffic"] = round(ATTN_TRAFFIC_PER_ALG_BYTE * d["alg_bytes"] / max(1, d["launches"]))
    classes = {c: {"launches": stats[c]["launches"],
                   "avg_launch_ms": round(stats[c]["total_ms"] / max(1, stats[c]["launches"]), 5),
                   "alg_bytes_per_launch": round(stats[c]["alg_bytes"] / max(1, stats[c]["launches"])),
                   "frac_of_peak": round(stats[c]["alg_flops"] / (stats[c]["total_ms"] * 1e9) / BF16_PEAK_TFLOPS, 4)
                   if c.startswith("gemm") and stats[c]["total_ms"] > 0 else
                   round(stats[c]["alg_bytes"] / (stats[c]["total_ms"] * 1e6) / HBM_PEAK_GBS, 4)
                   if stats[c]["total_ms"] > 0 else None}
               for c in prof_classes}

    wall_s, gpu_s, gen = sum(wall_t), sum(gpu_t), sum(gen_t)
    nom_b = float(nominal[is_sampled].sum())
    uni_b = float(unique[is_sampled].sum())
    step_gbs = nom_b / gpu_s / 1e9
    step_gbs_u = uni_b / gpu_s / 1e9
    roll_gbs = float(nominal.sum()) / rollout_gpu / 1e9
    roll_gbs_u = float(unique.sum()) / rollout_gpu / 1e9
    prompt_tokens = int(plens.sum())
    out = {
        "metric": "rollout tokens/sec (1 GPU) at 7B shape; decode-step HBM GB/s vs peak" if wl.name == "qwen7b"
                  else f"rollout tokens/sec (1 GPU), {wl.name} workload; decode-step HBM GB/s vs peak",
        "value": round(gen / wall_s, 1),
        "unit": "generated tokens/s",
        "n_gpus": 1,
        "steps": len(sampled),
        "warmup": args.warmup,
        "ms_per_step": round(wall_s * 1e3 / len(sampled), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": f"synthetic (seeded random-init weights, {wl.init} init, and uniform prompt tokens)",
        "config": {"workload": f"{wl.name}: {describe_shape(shape)}; {P} prompts x {G} samples, prompts "
                               f"U[{wl.prompt_len[0]},{wl.prompt_len[1]}], lognormal responses (median "
                               f"{wl.response_median}, sigma {wl.response_sigma}, cap {wl.response_cap}); the timed "
                               f"steps are spread evenly over the whole rollout",
                   "n_seqs": n_seq, "prompt_tokens": prompt_tokens, "decode_steps_in_rollout": max_steps,
                   "timed_steps": sampled if len(sampled) <= 64 else f"all {len(sampled)}",
                   "generated_tokens_timed": gen},
        "gpu_ms_timed": round(gpu_s * 1e3, 3),
        "decode_step_alg_GBps": round(step_gbs, 1),
        "decode_step_hbm_frac": round(step_gbs / HBM_PEAK_GBS, 4),
        "decode_step_unique_GBps": round(step_gbs_u, 1),
        "decode_step_unique_hbm_frac": round(step_gbs_u / HBM_PEAK_GBS, 4),
        "rollout": {"decode_s": round(rollout_wall, 3), "gpu_s": round(rollout_gpu, 3),
                    "generated_tokens": gen_all, "tokens_per_s": round(gen_all / rollout_wall, 1),
                    "alg_GBps": round(roll_gbs, 1), "hbm_frac": round(roll_gbs / HBM_PEAK_GBS, 4),
                    "unique_alg_GBps": round(roll_gbs_u, 1),
                    "unique_hbm_frac": round(roll_gbs_u / HBM_PEAK_GBS, 4),
                    "alg_TB": round(float(nominal.sum()) / 1e12, 2),
                    "unique_alg_TB": round(float(unique.sum()) / 1e12, 2),
                    "prefill_s": round(prefill_s, 4),
                    "paper_style_tokens_per_s": round((prompt_tokens + gen_all + n_seq) /
                                                      (rollout_wall + prefill_s), 1)},
        "roofline": roof,
        "measured_peaks": peaks,
        "timed_classes": classes,
        "gemm_plans": tuning,
        "kv_pool": kv_pool,
    }
    eng.close()
    del eng, ro
    torch.cuda.synchronize()
    if shape.moe:
        out["data"] += "; expert bytes counted for the experts n rows reach under uniform routing"
    if not args.no_cpu_baseline and not shape.moe:   # (the oracle would need a 61 GB host copy of the experts)
        out["cpu_baseline"] = cpu_baseline_rollout(shape, weights, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
