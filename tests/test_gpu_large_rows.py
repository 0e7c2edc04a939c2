"""Row blocks of the bf16 GEMMs (needs an MI355X).

The tile kernels address their operands with 32-bit per-lane byte offsets,
so an activation matrix spanning 4 GiB or more is run in row blocks.  A
one-layer decoder of the 7B shape scores 60 sequences of 2000 tokens
(120,000 rows: the down projection's 120,000 x 18944 bf16 activations take
two row blocks).  With one GEMM kernel forced for every projection, every
row is computed the same way wherever it lies, so the log-probabilities of
sequences whose rows lie in the second block equal those of the same
sequences scored alone, bit for bit.
"""
import dataclasses
import gc

import numpy as np
import pytest
import torch

from paper_2509_15965_amd.configs import WORKLOADS
from paper_2509_15965_amd.inputs import make_weights
from paper_2509_15965_amd.rl_decode import RL_GEMM_T256, RL_OPT_GEMM_PLAN, Engine, gemm_plan_code

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _i32(a):
    return torch.as_tensor(np.asarray(a, dtype=np.int32), device=DEV)


def test_rows_beyond_4gib_of_activations_match_the_same_sequences_alone():
    shape = dataclasses.replace(WORKLOADS["qwen7b"].model, n_layers=1)
    n, plen, rlen = 60, 1900, 100
    assert n * (plen + rlen) * shape.ffn * 2 >= 1 << 32
    rng = np.random.default_rng(17)
    prompts = [rng.integers(0, shape.vocab, size=plen).astype(np.int32) for _ in range(n)]
    resps = [rng.integers(0, shape.vocab, size=rlen).astype(np.int32) for _ in range(n)]
    w = make_weights(shape, 23, device=DEV)
    eng = Engine(shape, w, max_seqs=n, max_ctx=plen + rlen, max_prefill_tokens=n * (plen + rlen))
    eng.set_option(RL_OPT_GEMM_PLAN, gemm_plan_code(RL_GEMM_T256))
    big = torch.empty(n * rlen, dtype=torch.float32, device=DEV)
    eng.score(list(range(n)), np.arange(n + 1) * plen, _i32(np.concatenate(prompts)), np.arange(n + 1) * rlen,
              _i32(np.concatenate(resps)), big)
    torch.cuda.synchronize()
    big = big.cpu().numpy()
    assert np.isfinite(big).all()
    for k in (n - 3, n - 1):
        one = torch.empty(rlen, dtype=torch.float32, device=DEV)
        eng.score([0], [0, plen], _i32(prompts[k]), [0, rlen], _i32(resps[k]), one)
        torch.cuda.synchronize()
        assert np.array_equal(one.cpu().numpy(), big[k * rlen:(k + 1) * rlen]), k
    eng.close()
    del w, eng
    gc.collect()
    torch.cuda.empty_cache()
