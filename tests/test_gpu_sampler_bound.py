"""The sampler's noise filter (needs an MI355X).

The Gumbel-max sampler skips the exact fp64 noise of a vocabulary entry when
an upper bound of that noise cannot lift the entry's score to the best seen
so far.  The sample equals the exhaustive arg-max only if the bounds hold for
every 32-bit noise word; this evaluates them with the sampler's own device
code over all 2^32 words.
"""
import pytest

from paper_2509_15965_amd.rl_decode import probe_gumbel_bound

pytestmark = pytest.mark.gpu


def test_gumbel_noise_bounds_hold_for_every_word():
    violations, margin = probe_gumbel_bound(0, 1 << 32, n_blocks=8192)
    print(f"violations {violations}, smallest margin of the fp32 bound {margin:.6f}", flush=True)
    assert violations == 0
    # the bound adds 0.01 to an fp32 estimate within 1e-4 of the noise
    assert margin > 0.005
