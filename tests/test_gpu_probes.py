"""The measurement probes (read-only stream, matrix-core rate) through the C ABI:
their outputs prove the work was done and was the work claimed.  Needs an MI355X."""
import numpy as np
import pytest
import torch

from paper_2509_15965_amd.rl_decode import RLError, lib, probe_mfma, probe_read

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("nbytes,blocks", [(64 << 20, 512), ((1 << 20) + 48, 3), (16, 1)])
def test_read_probe_xor_covers_every_word(nbytes, blocks):
    rng = np.random.default_rng(nbytes)
    words = rng.integers(0, 2 ** 32, size=nbytes // 4, dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(words.view(np.int32)).to(DEV)
    out = torch.empty(blocks, dtype=torch.int32, device=DEV)
    probe_read(src, nbytes, out)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(words)


def test_mfma_probe_counts_every_product():
    n_blocks, iters = 16, 100
    out = torch.full((4 * n_blocks,), -1.0, dtype=torch.float32, device=DEV)
    probe_mfma(n_blocks, iters, out)
    torch.cuda.synchronize()
    assert torch.all(out == 128.0 * iters)


def test_probes_refuse_bad_arguments():
    out = torch.empty(4, dtype=torch.int32, device=DEV)
    src = torch.zeros(8, dtype=torch.int32, device=DEV)
    s = torch.cuda.current_stream().cuda_stream
    assert lib().rl_probe_read(src.data_ptr(), 24, 1, out.data_ptr(), s) == 1      # not a multiple of 16
    assert lib().rl_probe_read(src.data_ptr(), 16, 0, out.data_ptr(), s) == 1      # no workgroup
    assert lib().rl_probe_mfma(0, 10, out.data_ptr(), s) == 1
    assert lib().rl_probe_mfma(1, 0, out.data_ptr(), s) == 1
    with pytest.raises(ValueError):
        probe_mfma(2, 10, torch.empty(4, dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()
