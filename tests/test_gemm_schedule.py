"""CPU model of the direct-to-LDS GEMM's DMA issue order and wait counts.

gemm_dma128_kernel (paper_2509_15965_amd/csrc/k_gemm_lds.hip) streams the
activation tile through a ring of SA LDS stages and the weight tile through a
ring of SW stages.  Each wave issues AQ (activation) and BQ (weight) DMA
instructions per stage; the hardware load counter retires them in issue
order, and the kernel waits with `s_waitcnt vmcnt(n)` where n comes from its
after_stage() formula, rounded down by wait_vm_atmost().

This model replays the kernel's program order for one wave (all waves run the
same sequence) and checks, for every ring pair the library instantiates and
every stage count up to 100 plus the K of the real projections:
  - every DMA targets a stage in [0, nk) and each stage is issued once;
  - a stage is read only after a wait that retired all of its DMAs and a
    barrier behind that wait;
  - a ring slot is refilled only after a barrier that follows the last read
    of its previous stage;
  - every vmcnt immediate is in range and nothing is in flight at the end.
Two schedules known to be wrong (a prologue that starts at -SW, a steady
state bounded by SW when SA > SW) must fail it.
"""
import pytest

# (AQ, BQ, SA, SW) of the instantiated kernels: 256x256 / 8 waves, 128x128 /
# 4 waves, 128x256 / 8 waves, 128x128 deep / 4 waves
INSTANTIATED = [(4, 4, 2, 3), (4, 4, 2, 3), (2, 4, 3, 3), (4, 4, 4, 4)]
NK_CASES = list(range(1, 101)) + [112, 148, 296]


def wait_rounded(n):
    """wait_vm_atmost: the largest available immediate <= n."""
    for v in (48, 32, 24, 16, 12, 8, 6, 4, 2):
        if n >= v:
            return v
    return 0


class Schedule:
    def __init__(self, AQ, BQ, SA, SW, nk, prologue_from=None, steady_bound=None):
        self.AQ, self.BQ, self.SA, self.SW, self.nk = AQ, BQ, SA, SW, nk
        self.SMAX = max(SA, SW)
        self.prologue_from = -self.SMAX if prologue_from is None else prologue_from
        self.steady_bound = self.SMAX if steady_bound is None else steady_bound
        self.queue = []               # (kind, stage) per DMA instruction, issue order
        self.done = 0                 # retired prefix of the queue
        self.done_at_barrier = 0
        self.t = 0
        self.last_barrier = -1
        self.last_read = {}
        self.reads = {}
        self.issued = set()

    # -- the kernel's wait-count formula -----------------------------------
    def after_stage(self, s, last):
        SA, SW, AQ, BQ, nk = self.SA, self.SW, self.AQ, self.BQ, self.nk
        ia, iw = s - SA, s - SW
        n = 0
        if ia > iw:
            i0 = ia
            n += BQ if 0 <= i0 + SW < nk else 0
        else:
            i0 = iw
        for i in range(i0 + 1, last + 1):
            n += (AQ if 0 <= i + SA < nk else 0) + (BQ if 0 <= i + SW < nk else 0)
        return n

    # -- events ----------------------------------------------------------------
    def _tick(self):
        self.t += 1

    def issue(self, kind, s):
        self._tick()
        assert 0 <= s < self.nk, ("DMA outside [0, nk)", kind, s)
        assert (kind, s) not in self.issued, ("stage issued twice", kind, s)
        prev = s - (self.SA if kind == "A" else self.SW)
        if prev >= 0:
            assert self.reads.get(prev, 0) >= 4, ("slot refilled before its stage was read", kind, s)
            assert self.last_read[prev] < self.last_barrier, ("slot refilled without a barrier", kind, s)
        self.issued.add((kind, s))
        self.queue.extend([(kind, s)] * (self.AQ if kind == "A" else self.BQ))

    def issue_iter(self, i):
        if 0 <= i + self.SA < self.nk:
            self.issue("A", i + self.SA)
        if 0 <= i + self.SW < self.nk:
            self.issue("W", i + self.SW)

    def wait(self, n):
        self._tick()
        assert 0 <= n, n
        r = wait_rounded(n)
        assert r < 64
        self.done = max(self.done, len(self.queue) - r)

    def barrier(self):
        self._tick()
        self.last_barrier = self.t
        self.done_at_barrier = self.done

    def read(self, s, sub):
        self._tick()
        for kind in ("A", "W"):
            pos = [i for i, e in enumerate(self.queue) if e == (kind, s)]
            assert pos, ("read of a stage never issued", kind, s)
            assert max(pos) < self.done_at_barrier, ("read before the DMA retired", kind, s, sub)
        self.reads[s] = self.reads.get(s, 0) + 1
        self.last_read[s] = self.t

    # -- the kernel's program order --------------------------------------------
    def run(self):
        nk = self.nk
        for i in range(self.prologue_from, 0):
            self.issue_iter(i)
        if nk > 0:
            self.wait(self.after_stage(0, -1))
        self.barrier()
        self.read(0, 0)
        kt = 0
        while kt + self.steady_bound < nk:          # steady state: both issues unconditional
            for sub in (1, 2, 3):
                self.read(kt, sub)
            self.wait(self.after_stage(kt + 1, kt - 1))
            self.barrier()
            self.read(kt + 1, 0)
            self.issue("A", kt + self.SA)
            self.issue("W", kt + self.SW)
            kt += 1
        while kt < nk:
            for sub in (1, 2, 3):
                self.read(kt, sub)
            self.wait(self.after_stage(kt + 1, kt - 1) if kt + 1 < nk else 0)
            self.barrier()
            self.issue_iter(kt)
            self.read(kt + 1 if kt + 1 < nk else kt, 0)
            kt += 1
        assert self.done == len(self.queue), "DMAs still in flight at the end"
        assert self.issued == {(k, s) for k in ("A", "W") for s in range(nk)}
        return self


@pytest.mark.parametrize("AQ,BQ,SA,SW", sorted(set(INSTANTIATED)))
def test_instantiated_ring_schedules_are_safe(AQ, BQ, SA, SW):
    for nk in NK_CASES:
        Schedule(AQ, BQ, SA, SW, nk).run()


@pytest.mark.parametrize("AQ,BQ,SA,SW", [(4, 4, 3, 2), (4, 4, 2, 4), (2, 4, 5, 3)])
def test_other_ring_pairs_are_safe(AQ, BQ, SA, SW):
    """The formula is written for any ring pair, SA > SW included."""
    for nk in NK_CASES:
        Schedule(AQ, BQ, SA, SW, nk).run()


def test_model_rejects_known_bad_schedules():
    # prologue from -SW with SA > SW: stage 0's activations are never loaded
    with pytest.raises(AssertionError):
        for nk in range(1, 20):
            Schedule(4, 4, 3, 2, nk, prologue_from=-2).run()
    # steady state bounded by SW < SA: it issues activation stages past nk
    with pytest.raises(AssertionError):
        for nk in range(1, 20):
            Schedule(4, 4, 3, 2, nk, steady_bound=2).run()
    # a wait count one stage too generous lets a read overtake its DMA
    class Loose(Schedule):
        def after_stage(self, s, last):
            return super().after_stage(s, last) + self.AQ + self.BQ
    with pytest.raises(AssertionError):
        for nk in range(4, 30):
            Loose(4, 4, 2, 3, nk).run()
