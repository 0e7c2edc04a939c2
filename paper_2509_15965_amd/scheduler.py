"""Worker scheduling policy (RLinf Sec. 3.4, Alg. 1).

Given a workflow graph, an execution-time estimate for every component and
a device count, find the placement that minimises the time of one
iteration:
  - cycles of the graph are collapsed into single nodes first (their members
    run one after another on the devices given to the node);
  - a (sub)graph is split along every s-t cut into an upstream part G_s and
    a downstream part G_t (no edge from G_t back to G_s), and for each cut
    - temporal: G_s and G_t share all N devices, G_t starts after G_s, and
      the switch between them costs moving G_s's device state out and G_t's
      in (Sec. 3.4);
    - spatial: G_s gets N_s devices and G_t the other N_t, and they run as a
      pipeline over micro-batches of m items, one micro-batch's time through
      both stages plus (M/m - 1) times the slower stage (Sec. 3.4);
  - a single node's time is its estimate E;
  - the best time of every (subgraph, devices, batch) is cached, so each is
    solved once however many cuts reach it.

Readings (the paper leaves these open):
  - a pipeline's micro-batch times are the subgraphs' own estimates at batch
    m on their devices, t_s and t_t; T_critical = t_s + t_t (one micro-batch
    through both stages) and T_bottleneck = max(t_s, t_t);
  - m ranges over the powers of two dividing the batch M that are at least
    a given minimum (1 by default), and M itself;
  - N_s ranges over 1 .. N-1 for N <= 64 and over the multiples of N/64
    above (keeps the search under seconds at 1024 devices);
  - a collapsed cycle's estimate is the sum of its members' estimates;
  - a schedule that does not fit device memory (Component.fits) is
    infeasible (time +inf).
"""
from dataclasses import dataclass, field
from typing import Callable, Dict, FrozenSet, Iterable, List, Optional, Sequence, Tuple

INF = float("inf")


@dataclass
class Component:
    """A workflow node.  time(n_devices, batch) -> seconds for `batch` items
    data-parallel over n_devices; state_bytes: per-device bytes offloaded
    when it is switched out (and reloaded when switched in); fits(n, batch)
    -> whether it fits device memory."""
    name: str
    time: Callable[[int, int], float]
    state_bytes: float = 0.0
    fits: Optional[Callable[[int, int], bool]] = None


@dataclass
class Workflow:
    components: Dict[str, Component]
    edges: List[Tuple[str, str]] = field(default_factory=list)   # data flows u -> v


# ---------------------------------------------------------------------------
# graph preprocessing
# ---------------------------------------------------------------------------

def strongly_connected(nodes: Sequence[str], edges: Iterable[Tuple[str, str]]) -> List[List[str]]:
    """Strongly connected components (Tarjan), each sorted, in a stable order."""
    adj = {u: [] for u in nodes}
    for u, v in edges:
        adj[u].append(v)
    index, low, on, stack, out = {}, {}, set(), [], []
    counter = [0]

    def visit(u):
        index[u] = low[u] = counter[0]
        counter[0] += 1
        stack.append(u)
        on.add(u)
        for v in adj[u]:
            if v not in index:
                visit(v)
                low[u] = min(low[u], low[v])
            elif v in on:
                low[u] = min(low[u], index[v])
        if low[u] == index[u]:
            comp = []
            while True:
                w = stack.pop()
                on.discard(w)
                comp.append(w)
                if w == u:
                    break
            out.append(sorted(comp))

    for u in nodes:
        if u not in index:
            visit(u)
    return out


def collapse_cycles(wf: Workflow) -> Workflow:
    """One node per strongly connected component; a multi-member node runs
    its members one after another (times and device state add up)."""
    comps = strongly_connected(list(wf.components), wf.edges)
    of = {}
    nodes = {}
    for comp in comps:
        name = "+".join(comp)
        for u in comp:
            of[u] = name
        if len(comp) == 1:
            nodes[name] = wf.components[comp[0]]
            continue
        members = [wf.components[u] for u in comp]

        def t(n, b, members=members):
            return sum(c.time(n, b) for c in members)

        def f(n, b, members=members):
            return all(c.fits is None or c.fits(n, b) for c in members)

        nodes[name] = Component(name, t, sum(c.state_bytes for c in members), f)
    edges = sorted({(of[u], of[v]) for u, v in wf.edges if of[u] != of[v]})
    return Workflow(nodes, edges)


def st_cuts(nodes: FrozenSet[str], edges: Sequence[Tuple[str, str]]) -> List[Tuple[FrozenSet[str], FrozenSet[str]]]:
    """Every split of a DAG's nodes into a non-empty upstream set S and a
    non-empty downstream set T with no edge from T to S."""
    ns = sorted(nodes)
    inner = [(u, v) for u, v in edges if u in nodes and v in nodes]
    out = []
    for mask in range(1, (1 << len(ns)) - 1):
        S = frozenset(ns[i] for i in range(len(ns)) if mask >> i & 1)
        if any(v in S and u not in S for u, v in inner):   # an edge T -> S
            continue
        out.append((S, nodes - S))
    return out


# ---------------------------------------------------------------------------
# schedules
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Schedule:
    kind: str                      # "node", "temporal" or "pipeline"
    devices: int
    batch: int
    node: str = ""
    parts: Tuple["Schedule", ...] = ()
    micro_batch: int = 0

    def describe(self) -> str:
        if self.kind == "node":
            return f"{self.node}@{self.devices}"
        a, b = (p.describe() for p in self.parts)
        if self.kind == "temporal":
            return f"({a} ; {b})"
        return f"({a} | {b} m={self.micro_batch})"


def micro_batches(M: int, min_micro: int = 1) -> List[int]:
    out = []
    m = 1
    while m < M:
        if M % m == 0 and m >= min_micro:
            out.append(m)
        m *= 2
    out.append(M)
    return out


def device_splits(N: int) -> List[int]:
    if N <= 64:
        return list(range(1, N))
    step = N // 64
    return [k for k in range(step, N, step)]


def pipelining_time(t_s: float, t_t: float, M: int, m: int) -> float:
    """Two stages over M/m micro-batches: T_critical + (M/m - 1) T_bottleneck."""
    return (t_s + t_t) + (M // m - 1) * max(t_s, t_t)


class Scheduler:
    """Schedule search over a workflow; switch_bw = host link bytes/s per
    device for the temporal mode's offload + reload.

    best(nodes, N, M) is the minimum over the candidates of every s-t cut of
    `nodes`: the temporal candidate, and the pipeline candidates of every
    (device split, micro-batch), whose stage times come from a table of the
    two sides' best times at each device count.  Results are cached per
    (nodes, N, M)."""

    def __init__(self, wf: Workflow, switch_bw: float = INF, min_micro: int = 1):
        self.wf = collapse_cycles(wf)
        self.switch_bw = switch_bw
        self.min_micro = min_micro
        self.memo: Dict[Tuple[FrozenSet[str], int, int], Tuple[float, Optional[Schedule]]] = {}
        self._cuts: Dict[FrozenSet[str], List[Tuple[FrozenSet[str], FrozenSet[str]]]] = {}

    def switch_cost(self, S: FrozenSet[str], T: FrozenSet[str]) -> float:
        if self.switch_bw == INF:
            return 0.0
        b = sum(self.wf.components[u].state_bytes for u in S) + sum(self.wf.components[u].state_bytes for u in T)
        return b / self.switch_bw

    def node_time(self, name: str, N: int, M: int) -> float:
        c = self.wf.components[name]
        if c.fits is not None and not c.fits(N, M):
            return INF
        return c.time(N, M)

    def cuts(self, nodes: FrozenSet[str]):
        if nodes not in self._cuts:
            self._cuts[nodes] = st_cuts(nodes, self.wf.edges)
        return self._cuts[nodes]

    # -- candidates ------------------------------------------------------------
    def _temporal(self, S, T, N, M):
        ts, ss = self.best(S, N, M)
        tt, st = self.best(T, N, M)
        return ts + tt + self.switch_cost(S, T), Schedule("temporal", N, M, parts=(ss, st))

    def _pipelines(self, S, T, N, M):
        splits = device_splits(N)
        for m in micro_batches(M, self.min_micro):
            up = {n: self.best(S, n, m) for n in splits}
            down = {n: self.best(T, n, m) for n in {N - k for k in splits}}
            for Ns in splits:
                (a, sa), (b, sb) = up[Ns], down[N - Ns]
                if a < INF and b < INF:
                    yield pipelining_time(a, b, M, m), Schedule("pipeline", N, M, parts=(sa, sb), micro_batch=m)

    def _candidates(self, nodes, N, M):
        for S, T in self.cuts(nodes):
            yield self._temporal(S, T, N, M)
            yield from self._pipelines(S, T, N, M)

    def best(self, nodes: FrozenSet[str], N: int, M: int) -> Tuple[float, Optional[Schedule]]:
        key = (nodes, N, M)
        hit = self.memo.get(key)
        if hit is not None:
            return hit
        if len(nodes) == 1:
            (u,) = tuple(nodes)
            res = (self.node_time(u, N, M), Schedule("node", N, M, node=u))
        else:
            res = (INF, None)
            for cand in self._candidates(nodes, N, M):
                if cand[0] < res[0]:
                    res = cand
        self.memo[key] = res
        return res

    find = best

    def schedule(self, N: int, M: int) -> Tuple[float, Optional[Schedule]]:
        return self.best(frozenset(self.wf.components), N, M)


def brute_force(wf: Workflow, N: int, M: int, switch_bw: float = INF, min_micro: int = 1) -> float:
    """Best time by exhaustive enumeration of the same schedule space, with no
    memo and no pruning (small graphs and device counts only)."""
    sch = Scheduler(wf, switch_bw, min_micro)
    g = sch.wf

    def all_times(nodes, n, b):
        if len(nodes) == 1:
            (u,) = tuple(nodes)
            yield sch.node_time(u, n, b)
            return
        for S, T in st_cuts(nodes, g.edges):
            for ts in all_times(S, n, b):
                for tt in all_times(T, n, b):
                    yield ts + tt + sch.switch_cost(S, T)
            for Ns in device_splits(n):
                for m in micro_batches(b, min_micro):
                    for a in all_times(S, Ns, m):
                        for c in all_times(T, n - Ns, m):
                            if a < INF and c < INF:
                                yield pipelining_time(a, c, b, m)

    return min(all_times(frozenset(g.components), N, M), default=INF)
