"""The allocation-free sampler entry point against rl_sample_logits (needs an
MI355X).

rl_sample_logits_noalloc keeps the sampler's chunk partials in a fixed device
array of the library instead of a context's workspace.  Its tokens and
log-probabilities must equal those of rl_sample_logits on the same logits and
noise keys, bit for bit, on consecutive calls that reuse the array (the
second with fewer rows, so stale partials of the first are left behind), with
and without forced tokens, at T = 1, 0.6 and 0, and for batches whose rows
take one vocabulary chunk (no partials).
"""
import numpy as np
import pytest
import torch

from paper_2509_15965_amd.configs import ModelShape
from paper_2509_15965_amd.inputs import make_weights
from paper_2509_15965_amd.rl_decode import RL_ERR_INVALID_ARG, Engine, RLError, sample_logits_noalloc

pytestmark = pytest.mark.gpu

DEV = "cuda"
V = 152064
SHAPE = ModelShape(1, 64, 1, 1, 64, 64, V, 1e-6, 1e4, "bf16")


def _case(n, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    logits = torch.randn((n, V), generator=g, device=DEV, dtype=torch.float32) * 2.0
    uids = torch.randint(0, 1 << 40, (n,), generator=g, device=DEV, dtype=torch.int64)
    pos = torch.randint(0, 5000, (n,), generator=g, device=DEV, dtype=torch.int32)
    forced = torch.randint(0, V, (n,), generator=g, device=DEV, dtype=torch.int32)
    return logits, uids, pos, forced


@pytest.mark.parametrize("T", [1.0, 0.6, 0.0])
def test_noalloc_sampler_equals_workspace_sampler(T):
    eng = Engine(SHAPE, make_weights(SHAPE, 1, device=DEV), max_seqs=2600, max_ctx=8, max_prefill_tokens=8)
    try:
        for n, seed, use_forced in ((37, 1, False), (5, 2, True), (2600, 3, False), (1, 4, True)):
            logits, uids, pos, forced = _case(n, seed + int(10 * T))
            f = forced if use_forced else None
            t_ref = torch.empty(n, dtype=torch.int32, device=DEV)
            l_ref = torch.empty(n, dtype=torch.float32, device=DEV)
            eng.sample_logits(logits, uids.cpu().numpy().astype(np.uint64), pos.cpu().numpy(), t_ref, l_ref,
                              forced=f, seed=99, temperature=T)
            t_na = torch.full((n,), -1, dtype=torch.int32, device=DEV)
            l_na = torch.full((n,), float("nan"), dtype=torch.float32, device=DEV)
            sample_logits_noalloc(logits, uids, pos, t_na, l_na, forced=f, seed=99, temperature=T,
                                  stream=eng.stream)
            torch.cuda.synchronize()
            assert torch.equal(t_na, t_ref), (n, T)
            assert torch.equal(l_na, l_ref), (n, T)
    finally:
        eng.close()


def test_noalloc_sampler_rejects_bad_sizes():
    logits = torch.zeros((2, 16), dtype=torch.float32, device=DEV)
    u = torch.zeros(2, dtype=torch.int64, device=DEV)
    p = torch.zeros(2, dtype=torch.int32, device=DEV)
    t = torch.empty(2, dtype=torch.int32, device=DEV)
    l = torch.empty(2, dtype=torch.float32, device=DEV)
    with pytest.raises(RLError) as e:
        sample_logits_noalloc(logits[:, :14], u, p, t, l)          # vocab not a multiple of 4
    assert e.value.status == RL_ERR_INVALID_ARG
