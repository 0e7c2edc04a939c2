"""The worker scheduling policy (Alg. 1) on the CPU: graph preprocessing,
s-t cuts, the two cost models, and the memoised search against exhaustive
enumeration of the same schedule space."""
import math
import time

import pytest

from paper_2509_15965_amd.scheduler import (INF, Component, Scheduler, Workflow, brute_force, collapse_cycles,
                                            micro_batches, pipelining_time, st_cuts, strongly_connected)


def lin(c, fixed=0.0):
    """time(n, b) = fixed + c * b / n (perfectly data parallel)."""
    return lambda n, b: fixed + c * b / n


def test_strongly_connected_and_collapse():
    comps = strongly_connected(["env", "policy", "train", "ref"],
                               [("env", "policy"), ("policy", "env"), ("policy", "train"), ("ref", "train")])
    assert sorted(map(tuple, comps)) == [("env", "policy"), ("ref",), ("train",)]
    wf = Workflow({"env": Component("env", lin(1.0), 10), "policy": Component("policy", lin(2.0), 5),
                   "train": Component("train", lin(4.0), 7)},
                  [("env", "policy"), ("policy", "env"), ("policy", "train")])
    g = collapse_cycles(wf)
    assert set(g.components) == {"env+policy", "train"}
    assert g.edges == [("env+policy", "train")]
    c = g.components["env+policy"]
    assert c.time(2, 8) == pytest.approx(1.0 * 4 + 2.0 * 4)      # members run one after another
    assert c.state_bytes == 15


def test_st_cuts_of_a_diamond():
    nodes = frozenset("abcd")
    edges = [("a", "b"), ("a", "c"), ("b", "d"), ("c", "d")]
    cuts = {(tuple(sorted(S)), tuple(sorted(T))) for S, T in st_cuts(nodes, edges)}
    assert cuts == {(("a",), ("b", "c", "d")), (("a", "b"), ("c", "d")), (("a", "c"), ("b", "d")),
                    (("a", "b", "c"), ("d",))}


def test_pipelining_time_formula():
    # 4 micro-batches through stages of 2 s and 3 s: 2 + 3 + 3 * 3
    assert pipelining_time(2.0, 3.0, 8, 2) == pytest.approx(14.0)
    assert micro_batches(12) == [1, 2, 4, 12]
    assert micro_batches(8) == [1, 2, 4, 8]
    assert micro_batches(512, 16) == [16, 32, 64, 128, 256, 512]


def test_single_node_is_its_estimate():
    wf = Workflow({"gen": Component("gen", lin(3.0, 1.0))})
    t, s = Scheduler(wf).schedule(4, 16)
    assert t == pytest.approx(1.0 + 3.0 * 16 / 4)
    assert s.describe() == "gen@4"


def test_temporal_wins_without_switch_cost_and_spatial_with_it():
    """Two perfectly parallel stages: sharing all devices costs the sum of
    their times; a pipeline adds a warm-up, so temporal wins -- until the
    temporal mode pays for offloading and reloading device state."""
    wf = Workflow({"gen": Component("gen", lin(1.0), state_bytes=4e9),
                   "train": Component("train", lin(1.0), state_bytes=4e9)}, [("gen", "train")])
    t, s = Scheduler(wf).schedule(8, 64)
    assert s.kind == "temporal"
    assert t == pytest.approx(2 * 64 / 8)
    t2, s2 = Scheduler(wf, switch_bw=1e9).schedule(8, 64)     # 8 s of offload + reload
    assert s2.kind == "pipeline"
    assert s2.parts[0].devices == 4 and s2.micro_batch == 1
    # balanced halves, micro-batch 1: (1/4 + 1/4) + 63 * 1/4
    assert t2 == pytest.approx(0.5 + 63 * 0.25)


def test_memory_fit_forces_spreading():
    """A stage that only fits on >= 4 devices is never given fewer."""
    wf = Workflow({"gen": Component("gen", lin(1.0), fits=lambda n, b: n >= 4),
                   "train": Component("train", lin(1.0))}, [("gen", "train")])
    t, s = Scheduler(wf, switch_bw=1e30).schedule(4, 16)
    assert s.kind == "temporal" and t < INF
    t, s = Scheduler(wf).schedule(3, 16)
    assert t == INF and s is None


@pytest.mark.parametrize("N,M", [(1, 8), (2, 8), (3, 4), (5, 8), (6, 4)])
@pytest.mark.parametrize("bw", [INF, 2e9])
def test_search_equals_exhaustive_enumeration(N, M, bw):
    """A 3-stage GRPO-shaped chain with a fixed cost per call (so
    micro-batching is not free) and uneven parallel efficiency."""
    wf = Workflow({
        "rollout": Component("rollout", lambda n, b: 0.3 + 2.0 * b / n ** 0.9, state_bytes=3e9),
        "inference": Component("inference", lambda n, b: 0.1 + 0.5 * b / n, state_bytes=1e9),
        "training": Component("training", lambda n, b: 0.2 + 1.5 * b / n ** 0.95, state_bytes=5e9),
    }, [("rollout", "inference"), ("inference", "training")])
    t, s = Scheduler(wf, switch_bw=bw).schedule(N, M)
    assert t == pytest.approx(brute_force(wf, N, M, switch_bw=bw), rel=1e-12)
    assert s is not None


def test_search_on_a_branching_graph_equals_enumeration():
    wf = Workflow({
        "actor_gen": Component("actor_gen", lambda n, b: 0.5 + 1.0 * b / n, 2e9),
        "reward": Component("reward", lambda n, b: 0.05 + 0.2 * b / n, 1e9),
        "critic": Component("critic", lambda n, b: 0.1 + 0.4 * b / n, 1e9),
        "train": Component("train", lambda n, b: 0.2 + 0.8 * b / n, 3e9),
    }, [("actor_gen", "reward"), ("actor_gen", "critic"), ("reward", "train"), ("critic", "train")])
    for N in (2, 4):
        t, _ = Scheduler(wf, switch_bw=4e9).schedule(N, 8)
        assert t == pytest.approx(brute_force(wf, N, 8, switch_bw=4e9), rel=1e-12)


def test_search_time_stays_small_at_many_devices():
    wf = Workflow({
        "rollout": Component("rollout", lambda n, b: 0.3 + 2.0 * b / n ** 0.9, state_bytes=3e9),
        "inference": Component("inference", lambda n, b: 0.1 + 0.5 * b / n, state_bytes=1e9),
        "training": Component("training", lambda n, b: 0.2 + 1.5 * b / n ** 0.95, state_bytes=5e9),
    }, [("rollout", "inference"), ("inference", "training")])
    t0 = time.perf_counter()
    t, s = Scheduler(wf, switch_bw=50e9).schedule(256, 512)
    assert time.perf_counter() - t0 < 60.0
    assert math.isfinite(t) and s is not None


def test_profiler_fit_recovers_the_model_form():
    import numpy as np

    from paper_2509_15965_amd.profiler import fit_inverse_poly
    ns = [1, 2, 4]
    ts = [3.0 + 8.0 / n + 0.5 / n ** 2 for n in ns]
    coef, f = fit_inverse_poly(ns, ts, deg=2)
    assert np.allclose(coef, [3.0, 8.0, 0.5])
    assert f(8) == pytest.approx(3.0 + 1.0 + 0.5 / 64)
    coef2, f2 = fit_inverse_poly([1, 2, 4, 8], [1.0 + 2.0 / n for n in (1, 2, 4, 8)])
    assert np.allclose(coef2, [1.0, 2.0], atol=1e-12)
    assert f2(16) == pytest.approx(1.125)
    # no negative parts: data below the proportional line clamps the fixed part at 0
    coef3, _ = fit_inverse_poly([1, 2, 4], [10.0, 4.9, 2.4])
    assert coef3[0] == 0.0 and coef3[1] > 0


def test_profiler_schedules_use_the_policy():
    from paper_2509_15965_amd.profiler import schedules
    E = {"rollout": lambda n: 40.0 / n + 2.0, "inference": lambda n: 10.0 / n + 0.5,
         "training": lambda n: 30.0 / n + 1.5}
    out = schedules(E, 512, {"rollout": 15e9, "inference": 15e9, "training": 120e9}, 56.5e9, [1, 4, 16])
    assert [o["devices"] for o in out] == [1, 4, 16]
    assert out[0]["schedule"] == "((rollout@1 ; inference@1) ; training@1)"
    for o in out:
        assert o["estimate_s"] > 0 and o["search_s"] >= 0


def test_search_with_a_minimum_micro_batch_equals_enumeration():
    wf = Workflow({
        "rollout": Component("rollout", lambda n, b: 0.3 + 2.0 * b / n ** 0.9, state_bytes=3e9),
        "inference": Component("inference", lambda n, b: 0.01 + 0.5 * b / n, state_bytes=1e9),
        "training": Component("training", lambda n, b: 0.02 + 1.5 * b / n, state_bytes=5e9),
    }, [("rollout", "inference"), ("inference", "training")])
    for N in (3, 5):
        t, s = Scheduler(wf, switch_bw=2e9, min_micro=4).schedule(N, 16)
        assert t == pytest.approx(brute_force(wf, N, 16, switch_bw=2e9, min_micro=4), rel=1e-12)
        assert all(p.micro_batch == 0 or p.micro_batch >= 4 for p in (s,) + s.parts)
