"""Profiler (RLinf Sec. 3.4 "Profiler"): measure each component's execution
time at several data-parallel sizes, extrapolate with a polynomial, and hand
the estimates to the worker scheduling policy.

On one GPU a data-parallel size N is measured as one device's share of the
batch: the first M/N sequences (whole GRPO groups) of the 7B rollout
workload.  Components:
  rollout     StaticRollout of the share (prefill + every decode step);
  inference   rl_score of the share, one call per GRPO group;
  training    not built here: a stand-in at 3x the inference time (forward +
              backward of the same tokens), so that the scheduler has a
              three-stage GRPO graph to place.
Fit (a reading: the paper names polynomial extrapolation, not the
variable or degree): T(N) = a + b/N, least squares over the measured N -- a
fixed part (for the rollout, mostly its longest response) plus work divided
over the devices.  (--degree 2 adds c/N^2; with three measured sizes that
interpolates them exactly and extrapolates worse.)

    python -m paper_2509_15965_amd.profiler [--dp 1,2,4] [--check 8,16]
    python -m paper_2509_15965_amd.profiler --measurements out.json   # refit on the CPU

prints one JSON object: the profiled component times, the fits, the
estimate of a temporal iteration (the sum of the components' estimates)
against an independently timed end-to-end iteration -- at the measured
sizes and at held-out sizes the fit extrapolates to -- and the schedules the
policy picks for 1..1024 devices with these estimates.
"""
import argparse
import json
import sys
import time
from typing import Dict, List, Sequence

import numpy as np


def fit_inverse_poly(ns: Sequence[float], ts: Sequence[float], deg: int = 1):
    """Least-squares T(N) = sum_k c_k N^-k, k = 0..deg (deg capped by the
    number of points - 1) with every c_k >= 0 (a time has no negative fixed
    or per-item part); returns (coefficients, callable)."""
    from scipy.optimize import nnls
    ns = np.asarray(ns, dtype=np.float64)
    ts = np.asarray(ts, dtype=np.float64)
    deg = min(deg, len(ns) - 1)
    X = np.stack([ns ** (-k) for k in range(deg + 1)], axis=1)
    coef, _ = nnls(X, ts)

    def f(n):
        n = np.asarray(n, dtype=np.float64)
        return sum(coef[k] * n ** (-k) for k in range(len(coef)))

    return coef, f


def _shard(plan, group: int, n_prompts: int):
    return (plan["prompts"][:n_prompts], plan["response_lens"][:n_prompts * group], plan["uids"][:n_prompts * group])


def run_share(shape, weights, plan, group, n_prompts, seed, T, dev, score_seed=7):
    """One device's share of a temporal GRPO iteration: the rollout of the
    first n_prompts groups, then the inference stage over the same
    responses (one rl_score call per group).  Engines are created and warmed
    up first.  Profiling pass: each component timed on its own; then an
    independent end-to-end pass running the two back to back.  Returns
    (rollout s, inference s, end-to-end s)."""
    import torch

    from .rl_decode import Engine
    from .rollout import StaticRollout
    prompts, resp, uids = _shard(plan, group, n_prompts)
    plens = np.array([len(p) for p in prompts])
    ro_eng = Engine(shape, weights, max_seqs=len(uids), max_ctx=int(plens.max() + resp.max()),
                    max_prefill_tokens=int(plens.sum()), device=dev)
    StaticRollout(ro_eng, prompts, group, np.minimum(resp, 8), uids, seed, T).run()
    ro = StaticRollout(ro_eng, prompts, group, resp, uids, seed, T)
    rng = np.random.default_rng(score_seed)
    calls = []
    for p in range(n_prompts):
        rl = resp[p * group:(p + 1) * group]
        calls.append((torch.as_tensor(prompts[p], device=dev), np.array([0, len(prompts[p])], dtype=np.int32),
                      np.concatenate([[0], np.cumsum(rl)]).astype(np.int32),
                      torch.as_tensor(rng.integers(0, shape.vocab, size=int(rl.sum())).astype(np.int32), device=dev),
                      torch.empty(int(rl.sum()), dtype=torch.float32, device=dev), len(prompts[p]) + int(rl.sum())))
    sc_eng = Engine(shape, weights, max_seqs=group,
                    max_ctx=max(len(prompts[p]) + int(resp[p * group:(p + 1) * group].max()) for p in range(n_prompts)),
                    max_prefill_tokens=max(c[5] for c in calls), device=dev)
    slots = list(range(group))
    c = calls[0]
    sc_eng.score(slots, c[1], c[0], c[2], c[3], c[4], group=group, temperature=T)     # warm-up
    torch.cuda.synchronize()

    def rollout():
        ro.run()

    def inference():
        for c in calls:
            sc_eng.score(slots, c[1], c[0], c[2], c[3], c[4], group=group, temperature=T)

    t0 = time.perf_counter()
    rollout()
    torch.cuda.synchronize()
    t_r = time.perf_counter() - t0
    t0 = time.perf_counter()
    inference()
    torch.cuda.synchronize()
    t_i = time.perf_counter() - t0
    t0 = time.perf_counter()
    rollout()
    inference()
    torch.cuda.synchronize()
    t_e = time.perf_counter() - t0
    ro_eng.close()
    sc_eng.close()
    del ro_eng, sc_eng, ro
    torch.cuda.empty_cache()
    return t_r, t_i, t_e


def schedules(E: Dict[str, callable], M: int, state_bytes: Dict[str, float], switch_bw: float,
              devices: Sequence[int], min_micro: int = 1) -> List[dict]:
    """Run the scheduling policy on the GRPO chain rollout -> inference ->
    training.  E_c(N) estimates a component on N devices for the whole batch
    M, i.e. a per-device share of M/N items; b items on n devices are the
    same share as M items on n*M/b devices, so time(n, b) = E_c(n*M/b): a
    small micro-batch keeps the fixed part of the estimate (for the rollout,
    its longest response) and loses only the divisible part.  Micro-batches
    hold at least min_micro items (whole GRPO groups: a group's responses
    are normalised together downstream)."""
    from .scheduler import Component, Scheduler, Workflow
    comps = {name: Component(name, (lambda n, b, f=f: float(f(n * M / b))), state_bytes[name])
             for name, f in E.items()}
    wf = Workflow(comps, [("rollout", "inference"), ("inference", "training")])
    out = []
    for N in devices:
        t0 = time.perf_counter()
        t, s = Scheduler(wf, switch_bw=switch_bw, min_micro=min_micro).schedule(N, M)
        out.append({"devices": N, "estimate_s": round(t, 3), "schedule": s.describe(),
                    "search_s": round(time.perf_counter() - t0, 4)})
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="qwen7b")
    ap.add_argument("--dp", default="1,2,4", help="data-parallel sizes measured (device shares)")
    ap.add_argument("--check", default="8", help="held-out data-parallel sizes: predicted, then measured")
    ap.add_argument("--switch-gbps", type=float, default=56.5, help="host link GB/s per device (measured)")
    ap.add_argument("--degree", type=int, default=1, help="degree of the fit in 1/N")
    ap.add_argument("--measurements", default="", help="JSON written by an earlier run: refit it, no GPU")
    args = ap.parse_args()
    from .configs import WORKLOADS
    wl = WORKLOADS[args.workload]
    shape = wl.model
    G, P = wl.group, wl.n_prompts
    M = P * G
    dps = [int(x) for x in args.dp.split(",")]
    checks = [int(x) for x in args.check.split(",") if x]
    if args.measurements:
        old = json.load(open(args.measurements))
        meas = {c: {int(k): v for k, v in old["measured_s"][c].items()} for c in old["measured_s"]}
        n_params = old["n_params"]
        wbytes = old["weight_bytes"]
    else:
        import torch

        from .inputs import make_weights, rollout_plan
        dev = torch.device("cuda:0")
        torch.cuda.set_device(dev)
        plan = rollout_plan(wl)
        weights = make_weights(shape, wl.seed, device=dev, init=wl.init)
        n_params = sum(v.numel() for v in weights.values())
        wbytes = sum(v.numel() * v.element_size() for v in weights.values())
        seed, T = 20250919, wl.temperature
        meas = {"rollout": {}, "inference": {}, "iteration": {}}
        for N in dps + checks:
            r, i, e = run_share(shape, weights, plan, G, P // N, seed, T, dev)
            meas["rollout"][N], meas["inference"][N], meas["iteration"][N] = r, i, e
            print(f"[profiler] N={N}: rollout {r:.2f} s, inference {i:.2f} s, iteration {e:.2f} s",
                  file=sys.stderr, flush=True)
    fits, E = {}, {}
    for c in ("rollout", "inference"):
        coef, f = fit_inverse_poly(dps, [meas[c][n] for n in dps], args.degree)
        fits[c] = [float(x) for x in coef]
        E[c] = f
    E["training"] = lambda n, f=E["inference"]: 3.0 * f(n)
    est = []
    for N in dps + checks:
        pr, pi = float(E["rollout"](N)), float(E["inference"](N))
        est.append({"devices": N, "held_out": N in checks,
                    "rollout_pred_s": round(pr, 3), "rollout_meas_s": round(meas["rollout"][N], 3),
                    "inference_pred_s": round(pi, 3), "inference_meas_s": round(meas["inference"][N], 3),
                    "iteration_pred_s": round(pr + pi, 3), "iteration_meas_s": round(meas["iteration"][N], 3),
                    "iteration_err": round((pr + pi) / meas["iteration"][N] - 1, 4)})
    state = {"rollout": float(wbytes), "inference": float(wbytes), "training": float(16 * n_params)}
    sched = schedules(E, M, state, args.switch_gbps * 1e9, [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024],
                      min_micro=G)
    out = {"workload": wl.name, "batch": M, "n_params": int(n_params), "weight_bytes": int(wbytes),
           "measured_s": meas, "fit_coefficients_of_N^-k": fits, "fit_degree": args.degree,
           "estimates": est, "state_bytes_per_device": state,
           "switch_GBps": args.switch_gbps, "schedules": sched}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
