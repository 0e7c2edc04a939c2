"""Rollout drivers' host logic on the CPU, against a stand-in engine whose
"model" is a fixed function of (uid, position, previous token): the static
and the continuous-batching drivers must produce the same responses, every
response exactly once, in chunks of the configured size, never more
sequences in flight than slots, and never a slot used twice at once."""
import numpy as np
import pytest
import torch

from paper_2509_15965_amd.rollout import ContinuousRollout, StaticRollout

V = 997


def first_token(uid, plen):
    return (uid * 131 + plen * 17) % V


def next_token(uid, pos, prev):
    return (prev * 31 + uid * 7 + pos * 3) % V


class FakeEngine:
    class _Cfg:
        pass

    def __init__(self, max_seqs):
        self.device = torch.device("cpu")
        self.cfg = self._Cfg()
        self.cfg.max_seqs = max_seqs
        self.len = [0] * max_seqs
        self.busy = set()
        self.max_busy = 0
        self.steps = 0

    def release(self, slots):
        for s in np.asarray(slots).tolist():
            self.len[s] = 0
            self.busy.discard(s)

    def prefill(self, slots, uids, offs, ptok, ft, fl, group, seed, temperature):
        slots = np.asarray(slots).tolist()
        uids = np.asarray(uids, dtype=np.uint64).tolist()
        for s in slots:
            assert s not in self.busy, "prefill into a slot in use"
            self.busy.add(s)
        self.max_busy = max(self.max_busy, len(self.busy))
        for i, (s, u) in enumerate(zip(slots, uids)):
            p = i // group
            plen = int(offs[p + 1] - offs[p])
            self.len[s] = plen
            ft[i] = first_token(u, plen)
            fl[i] = -float(u % 5) - 0.25

    def step(self, slots, uids, in_tok, out_tok, out_lp, seed, temperature):
        slots = np.asarray(slots).tolist()
        uids = np.asarray(uids, dtype=np.uint64).tolist()
        assert len(set(slots)) == len(slots)
        vals = in_tok.clone()
        for i, (s, u) in enumerate(zip(slots, uids)):
            assert s in self.busy
            pos = self.len[s] + 1
            out_tok[i] = next_token(u, pos, int(vals[i]))
            out_lp[i] = -float((u + pos) % 7) - 0.5
            self.len[s] += 1
        self.steps += 1


def reference(prompts, group, resp, uids):
    out = {}
    for q, u in enumerate(uids):
        plen = len(prompts[q // group])
        t = [first_token(u, plen)]
        lp = [-float(u % 5) - 0.25]
        for j in range(1, resp[q]):
            pos = plen + j
            t.append(next_token(u, pos, t[-1]))
            lp.append(-float((u + pos) % 7) - 0.5)
        out[u] = (np.array(t), np.array(lp, dtype=np.float32))
    return out


def workload(P=7, G=4, seed=0):
    rng = np.random.default_rng(seed)
    prompts = [rng.integers(0, V, size=int(n)).astype(np.int32) for n in rng.integers(3, 12, size=P)]
    resp = rng.integers(1, 20, size=P * G)
    resp[3] = 1                                   # a response that ends with the prefill
    uids = (1000 + np.arange(P * G) * 3).astype(np.uint64)
    return prompts, G, resp, uids


def check(responses, ref, resp, uids):
    got = {r.uid: r for r in responses}
    assert sorted(got) == sorted(int(u) for u in uids)
    for q, u in enumerate(uids):
        r = got[int(u)]
        assert len(r.tokens) == resp[q]
        assert np.array_equal(r.tokens, ref[int(u)][0])
        assert np.array_equal(r.logps, ref[int(u)][1])


def test_static_driver_matches_the_reference():
    prompts, G, resp, uids = workload()
    eng = FakeEngine(len(uids))
    ro = StaticRollout(eng, prompts, G, resp, uids, seed=1, temperature=1.0)
    gen = ro.run()
    assert gen == int(resp.sum()) - len(uids)     # decode steps produce all but the first token
    check(ro.responses(), reference(prompts, G, resp, uids), resp, uids)


@pytest.mark.parametrize("n_slots,emit", [(4, 1), (8, 3), (12, 5), (28, 28)])
def test_continuous_driver_matches_the_reference(n_slots, emit):
    prompts, G, resp, uids = workload()
    eng = FakeEngine(32)
    chunks = []
    ro = ContinuousRollout(eng, prompts, G, resp, uids, seed=1, temperature=1.0, n_slots=n_slots,
                           emit_every=emit, on_emit=chunks.append)
    gen = ro.run()
    assert gen == int(resp.sum())
    assert eng.max_busy <= n_slots
    assert all(len(c) == emit for c in chunks[:-1]) and 1 <= len(chunks[-1]) <= emit
    check([r for c in chunks for r in c], reference(prompts, G, resp, uids), resp, uids)
    assert not eng.busy                           # every slot released at the end


def test_continuous_keeps_the_batch_fuller_than_static():
    """With twice as many sequences as slots, continuous batching needs
    fewer decode steps than two static batches one after the other."""
    prompts, G, resp, uids = workload(P=8, G=4, seed=3)
    half = len(uids) // 2
    st_steps = 0
    for part in (slice(0, half), slice(half, None)):
        eng = FakeEngine(half)
        ro = StaticRollout(eng, prompts[part.start // G if part.start else 0:(part.stop // G if part.stop else None)],
                           G, resp[part], uids[part], seed=1, temperature=1.0)
        ro.run()
        st_steps += eng.steps
    eng = FakeEngine(half)
    ro = ContinuousRollout(eng, prompts, G, resp, uids, seed=1, temperature=1.0, n_slots=half, emit_every=4)
    ro.run()
    assert eng.steps < st_steps
