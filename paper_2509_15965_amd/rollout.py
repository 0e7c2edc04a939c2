"""Rollout drivers over the C ABI (host-side scheduling only; every token is
produced by the library's prefill and decode steps).

Generation in GRPO samples `group` responses per prompt (Sec. 2.1).  The
response lengths are given up front (random-init models have no meaningful
end token), counting the token sampled by the prefill.

  StaticRollout      one batch: every sequence gets a slot, the prefill opens
                     them all, and each decode step runs over the sequences
                     still generating (slots ordered longest first, so the
                     active set is always a prefix) until the longest ends.
  ContinuousRollout  more sequences than slots: whole prompt groups are
                     admitted into free slots as earlier sequences finish, so
                     the batch stays full instead of draining into a long
                     tail, and finished responses are handed downstream in
                     chunks of m as soon as m are ready -- the one-GPU core of
                     elastic pipelining (Sec. 3.3: a stage forwards output
                     once a batch of the configured size is ready).

Sampling noise is keyed by (seed, sequence uid, position), so a sequence's
tokens do not depend on which slot or batch it ran in (bit-identical in the
fp32 model).
"""
from dataclasses import dataclass
from typing import Callable, List, Optional, Sequence

import numpy as np
import torch


@dataclass
class Response:
    uid: int
    prompt: int                    # prompt index
    tokens: np.ndarray             # int32 [length]
    logps: np.ndarray              # float32 [length]


class StaticRollout:
    """prompts: list of int32 arrays (one per prompt); resp_lens: [P*group]
    lengths (sample k of prompt p at p*group + k); uids: [P*group]."""

    def __init__(self, engine, prompts: Sequence[np.ndarray], group: int, resp_lens: Sequence[int],
                 uids: Sequence[int], seed: int, temperature: float):
        self.eng = engine
        dev = engine.device
        self.P, self.G = len(prompts), group
        n = self.P * group
        self.n = n
        resp = np.asarray(resp_lens, dtype=np.int64)
        self.resp = resp
        self.seed, self.T = seed, temperature
        order = np.argsort(-resp, kind="stable")          # slot k holds the k-th longest sequence
        slot_of = np.empty(n, dtype=np.int64)
        slot_of[order] = np.arange(n)
        self.order = order
        self.slot_of = slot_of
        self.uids_sorted = np.asarray(uids, dtype=np.uint64)[order]
        self.pre_slots = slot_of.astype(np.int32)
        self.pre_uids = np.asarray(uids, dtype=np.uint64)
        plens = [len(p) for p in prompts]
        self.offs = np.concatenate([[0], np.cumsum(plens)]).astype(np.int32)
        self.prompt_tok = torch.as_tensor(np.concatenate(prompts).astype(np.int32), device=dev)
        self.max_steps = int(resp.max()) - 1
        resp_sorted = resp[order]
        self.active = np.array([(resp_sorted > t + 1).sum() for t in range(self.max_steps)], dtype=np.int64)
        self.slots_sorted = np.arange(n, dtype=np.int32)
        self.toks = torch.zeros((self.max_steps + 1, n), dtype=torch.int32, device=dev)
        self.logps = torch.zeros((self.max_steps + 1, n), dtype=torch.float32, device=dev)
        self._ft = torch.empty(n, dtype=torch.int32, device=dev)
        self._fl = torch.empty(n, dtype=torch.float32, device=dev)
        self._perm = torch.as_tensor(self.pre_slots.astype(np.int64), device=dev)

    def prefill(self):
        self.eng.release(self.slots_sorted)
        self.eng.prefill(self.pre_slots, self.pre_uids, self.offs, self.prompt_tok, self._ft, self._fl,
                         group=self.G, seed=self.seed, temperature=self.T)
        self.toks[0].index_copy_(0, self._perm, self._ft)
        self.logps[0].index_copy_(0, self._perm, self._fl)

    def step(self, t: int) -> int:
        """Decode step t (0-based); returns the number of sequences stepped."""
        n = int(self.active[t])
        self.eng.step(self.slots_sorted[:n], self.uids_sorted[:n], self.toks[t, :n], self.toks[t + 1, :n],
                      self.logps[t + 1, :n], seed=self.seed, temperature=self.T)
        return n

    def run(self, steps: Optional[int] = None) -> int:
        self.prefill()
        steps = self.max_steps if steps is None else min(steps, self.max_steps)
        return sum(self.step(t) for t in range(steps))

    def responses(self) -> List[Response]:
        toks = self.toks.cpu().numpy()
        lps = self.logps.cpu().numpy()
        out = []
        for s in range(self.n):
            k = int(self.slot_of[s])
            m = int(self.resp[s])
            out.append(Response(int(self.pre_uids[s]), s // self.G, toks[:m, k].copy(), lps[:m, k].copy()))
        return out


class ContinuousRollout:
    """Continuous batching over `n_slots` slots (<= the engine's max_seqs):
    prompt groups wait in order and are prefilled together whenever enough
    slots are free; each decode step runs over every generating sequence;
    a sequence that reaches its length frees its slot.  Finished responses
    are passed to on_emit(list[Response]) in chunks of `emit_every` (the
    last chunk may be smaller).

    Device-side bookkeeping needs no per-step host-to-device copy: the
    generating sequences occupy rows 0..n-1 of a row order (a finished row
    is replaced by the last one), `cur[r]` holds row r's last token, and
    step t's outputs land in row t of a step table; the host remembers which
    sequence each row held at each step and gathers a response's tokens when
    it is emitted."""

    def __init__(self, engine, prompts: Sequence[np.ndarray], group: int, resp_lens: Sequence[int],
                 uids: Sequence[int], seed: int, temperature: float, n_slots: int, emit_every: int,
                 on_emit: Optional[Callable[[List[Response]], None]] = None):
        if n_slots < group or n_slots > engine.cfg.max_seqs:
            raise ValueError("n_slots must hold a prompt group and fit the engine's slots")
        self.eng = engine
        self.dev = engine.device
        self.prompts = [np.asarray(p, dtype=np.int32) for p in prompts]
        self.G = group
        self.resp = np.asarray(resp_lens, dtype=np.int64)
        self.uids = np.asarray(uids, dtype=np.uint64)
        self.seed, self.T = seed, temperature
        self.n_slots = n_slots
        self.emit_every = max(1, emit_every)
        self.on_emit = on_emit
        self.cur = torch.zeros(n_slots, dtype=torch.int32, device=self.dev)
        self.block = 256                   # steps per table block
        self.tab_tok: List[torch.Tensor] = []
        self.tab_lp: List[torch.Tensor] = []
        self.first: dict = {}              # sequence -> (token tensor, logp tensor, index)
        self.where: dict = {}              # sequence -> flat step-table indices of its tokens 1..
        self.emitted: List[List[Response]] = []
        self.steps = 0
        self.generated = 0

    def _table(self, t: int):
        while len(self.tab_tok) * self.block <= t:
            self.tab_tok.append(torch.zeros((self.block, self.n_slots), dtype=torch.int32, device=self.dev))
            self.tab_lp.append(torch.zeros((self.block, self.n_slots), dtype=torch.float32, device=self.dev))
        return self.tab_tok[t // self.block][t % self.block], self.tab_lp[t // self.block][t % self.block]

    def _emit(self, seqs: List[int]):
        if not seqs:
            return
        tok = torch.cat([b.reshape(-1) for b in self.tab_tok]) if self.tab_tok else None
        lp = torch.cat([b.reshape(-1) for b in self.tab_lp]) if self.tab_lp else None
        chunk = []
        for q in seqs:
            ft, fl, i = self.first.pop(q)
            idx = self.where.pop(q)
            t0 = ft[i:i + 1]
            l0 = fl[i:i + 1]
            if idx:
                ix = torch.as_tensor(np.asarray(idx, dtype=np.int64), device=self.dev)
                t0 = torch.cat([t0, tok.index_select(0, ix)])
                l0 = torch.cat([l0, lp.index_select(0, ix)])
            chunk.append(Response(int(self.uids[q]), q // self.G, t0.cpu().numpy(), l0.cpu().numpy()))
        self.emitted.append(chunk)
        if self.on_emit is not None:
            self.on_emit(chunk)

    def run(self) -> int:
        eng, G = self.eng, self.G
        free = list(range(self.n_slots))[::-1]
        waiting = list(range(len(self.prompts)))
        rows: List[int] = []               # row -> sequence
        slot_of: dict = {}                 # sequence -> slot
        made: dict = {}                    # sequence -> tokens produced so far
        done: List[int] = []
        def retire():
            # complete responses leave: the last row moves into the gap
            nonlocal done
            r = 0
            fin_slots = []
            while r < len(rows):
                q = rows[r]
                if made[q] < self.resp[q]:
                    r += 1
                    continue
                last = len(rows) - 1
                if r != last:
                    self.cur[r:r + 1].copy_(self.cur[last:last + 1])
                    rows[r] = rows[last]
                rows.pop()
                fin_slots.append(slot_of.pop(q))
                done.append(q)
            if fin_slots:
                eng.release(fin_slots)
                free.extend(fin_slots)
            while len(done) >= self.emit_every:
                self._emit(done[:self.emit_every])
                done = done[self.emit_every:]

        while waiting or rows:
            retire()
            # admit whole groups while they fit; their first tokens become new rows
            adm = []
            while waiting and len(free) >= G * (len(adm) + 1):
                adm.append(waiting.pop(0))
            if adm:
                seqs = [p * G + k for p in adm for k in range(G)]
                slots = [free.pop() for _ in seqs]
                offs = np.concatenate([[0], np.cumsum([len(self.prompts[p]) for p in adm])]).astype(np.int32)
                ptok = torch.as_tensor(np.concatenate([self.prompts[p] for p in adm]), device=self.dev)
                n0 = len(rows)
                ft = self.cur[n0:n0 + len(seqs)]
                fl = torch.empty(len(seqs), dtype=torch.float32, device=self.dev)
                eng.prefill(slots, self.uids[seqs], offs, ptok, ft, fl, group=G, seed=self.seed, temperature=self.T)
                ft_keep = ft.clone()
                for i, (q, s) in enumerate(zip(seqs, slots)):
                    rows.append(q)
                    slot_of[q] = s
                    made[q] = 1
                    self.first[q] = (ft_keep, fl, i)
                    self.where[q] = []
                self.generated += len(seqs)
                retire()                   # one-token responses are complete after the prefill
            if not rows:
                continue
            # one decode step over rows 0..n-1
            n = len(rows)
            tt, tl = self._table(self.steps)
            eng.step(np.asarray([slot_of[q] for q in rows], dtype=np.int32), self.uids[rows], self.cur[:n],
                     tt[:n], tl[:n], seed=self.seed, temperature=self.T)
            self.cur[:n].copy_(tt[:n])
            base = self.steps * self.n_slots
            for i, q in enumerate(rows):
                self.where[q].append(base + i)
                made[q] += 1
            self.steps += 1
            self.generated += n
        self._emit(done)
        return self.generated
