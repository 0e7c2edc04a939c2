"""CPU oracle of the RL-rollout decode step (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this package.  It shares no code with the GPU library.
"""
from .oracle import (  # noqa: F401
    OracleModel, OracleSeq, load, philox4x32_10, noise_word, gumbel_of_word,
    gumbel_argmax_u, sample, sample_margin, logprob, score, round_bf16, rmsnorm, rope, rope_cos_sin,
    attend, matvec, route, set_threads, num_threads, MODE_FP64, MODE_FP32, MODE_BF16,
)
