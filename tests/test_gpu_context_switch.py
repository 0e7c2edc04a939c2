"""Context switching: live K/V offloaded to pinned host memory and reloaded
(rl_kv_offload / rl_kv_onload), and the context pointed at new device
buffers (rl_decode_rebind), through the C ABI (needs an MI355X).

A rollout that is switched out and back in (pool wiped, or weights, pool
and workspace replaced by new allocations; slots renumbered) must continue
bit-identically to one that never left the GPU (dense and
mixture-of-experts models).
"""
import numpy as np
import pytest
import torch

from harness import build_models
from paper_2509_15965_amd.configs import WORKLOADS, ModelShape
from paper_2509_15965_amd.inputs import uniform_tokens
from paper_2509_15965_amd.rl_decode import RL_OPT_SHARED_PREFIX, Engine, RLError

pytestmark = pytest.mark.gpu

DEV = "cuda"
GQA = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e4, "bf16")
MOE = ModelShape(2, 256, 4, 2, 64, 0, 512, 1e-6, 1e6, "bf16", n_experts=8, top_k=2, expert_ffn=128)


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _i32(a):
    return torch.as_tensor(np.asarray(a, dtype=np.int32), device=DEV)


def _engine(shape, w_dev, max_seqs=12):
    eng = Engine(shape, w_dev, max_seqs=max_seqs, max_ctx=128, max_prefill_tokens=128)
    eng.set_option(RL_OPT_SHARED_PREFIX, 0)
    return eng


def _prefill(eng, slots, prompts, group):
    n = len(slots)
    offs = np.concatenate([[0], np.cumsum([len(p) for p in prompts])]).astype(np.int32)
    ot = torch.empty(n, dtype=torch.int32, device=DEV)
    ol = torch.empty(n, dtype=torch.float32, device=DEV)
    eng.prefill(slots, list(range(n)), offs, _i32(np.concatenate(prompts)), ot, ol, group=group, seed=3)


def _step(eng, slots, k, vocab):
    n = len(slots)
    lg = torch.empty((n, vocab), dtype=torch.float32, device=DEV)
    ot = torch.empty(n, dtype=torch.int32, device=DEV)
    ol = torch.empty(n, dtype=torch.float32, device=DEV)
    eng.step(slots, list(range(n)), _i32(uniform_tokens(n, vocab, 70 + k)), ot, ol, seed=3, out_logits=lg)
    torch.cuda.synchronize()
    return lg.cpu().numpy(), ot.cpu().numpy(), ol.cpu().numpy()


def _case(shape):
    rng = np.random.default_rng(61)
    return [rng.integers(0, shape.vocab, size=n).astype(np.int32) for n in (37, 58)]


@pytest.mark.parametrize("shape", [GQA, WORKLOADS["tiny"].model, MOE], ids=["bf16", "fp32", "moe"])
@pytest.mark.parametrize("rebind", [False, True], ids=["wipe-pool", "new-buffers"])
def test_switch_out_and_back_continues_bit_identically(shape, rebind):
    w_dev, _, _ = build_models(shape, 62)
    prompts = _case(shape)
    old = list(range(6))
    new = [11, 7, 9, 6, 10, 8]                         # renumbered slots after the switch
    ref = _engine(shape, w_dev)
    _prefill(ref, old, prompts, 3)
    expect = [_step(ref, old, k, shape.vocab) for k in range(5)]
    ref.close()

    eng = _engine(shape, w_dev)
    _prefill(eng, old, prompts, 3)
    got = [_step(eng, old, k, shape.vocab) for k in range(3)]
    lengths = [eng.slot_length(s) for s in old]
    nbytes = eng.kv_offload_bytes(old)
    L, Hkv, d = shape.n_layers, shape.n_kv_heads, shape.head_dim
    es = 2 if shape.dtype == "bf16" else 4
    assert nbytes == sum(L * Hkv * (n + (n + 7) // 8 * 8) * d * es for n in lengths)
    host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    eng.kv_offload(old, host)
    torch.cuda.synchronize()
    eng.release(old)
    if rebind:
        # the caller frees everything and comes back with new allocations
        w2 = {k: v.clone() for k, v in w_dev.items()}
        kv2 = torch.full_like(eng.kv, 0x7F)
        ws2 = torch.full_like(eng.ws, 0x3C)
        eng.kv.zero_()
        eng.rebind(w2, kv2, ws2)
    else:
        eng.kv.zero_()
    eng.kv_onload(new, lengths, host)
    for s, n in zip(new, lengths):
        assert eng.slot_length(s) == n
    got += [_step(eng, new, k, shape.vocab) for k in range(3, 5)]
    eng.close()
    for k in range(5):
        for a, b in zip(got[k], expect[k]):
            assert np.array_equal(a, b), (k, rebind)


def test_packed_layout_is_the_documented_one():
    """Slot by slot, layer by layer, head by head: K rows then V blocks."""
    shape = GQA
    w_dev, _, _ = build_models(shape, 63)
    eng = _engine(shape, w_dev)
    _prefill(eng, [4, 2], [_case(shape)[0]], 2)
    _step(eng, [2], 0, shape.vocab)                      # slot 2 one longer than slot 4
    slots = [2, 4]
    lens = [eng.slot_length(s) for s in slots]
    host = torch.empty(eng.kv_offload_bytes(slots), dtype=torch.uint8, pin_memory=True)
    eng.kv_offload(slots, host)
    torch.cuda.synchronize()
    K, V = eng.kv_views()
    parts = []
    for s, n in zip(slots, lens):
        n8 = (n + 7) // 8 * 8
        for l in range(shape.n_layers):
            for h in range(shape.n_kv_heads):
                parts.append(K[l, s, h, :n].contiguous().view(torch.uint8).reshape(-1))
                parts.append(V[l, s, h, :n8 // 8].contiguous().view(torch.uint8).reshape(-1))
    expect = torch.cat(parts).cpu()
    assert torch.equal(host, expect)
    eng.close()


def test_switch_argument_errors():
    shape = GQA
    w_dev, _, _ = build_models(shape, 64)
    eng = _engine(shape, w_dev)
    _prefill(eng, [0, 1], [_case(shape)[1]], 2)
    n = eng.kv_offload_bytes([0, 1])
    small = torch.empty(n - 16, dtype=torch.uint8, pin_memory=True)
    with pytest.raises(RLError):
        eng.kv_offload([0, 1], small)
    with pytest.raises(RLError):
        eng.kv_offload([0, 0], torch.empty(2 * n, dtype=torch.uint8, pin_memory=True))
    with pytest.raises(RLError):
        eng.kv_onload([3], [129], torch.empty(n, dtype=torch.uint8, pin_memory=True))   # > max_ctx
    with pytest.raises(RLError):
        eng.kv_onload([3], [58], small[:100])                                            # too small
    assert eng.kv_offload_bytes([99]) == 0
    eng.close()


@pytest.mark.parametrize("shape", [GQA, WORKLOADS["tiny"].model], ids=["bf16", "fp32"])
def test_switched_continuation_matches_oracle(shape):
    """After offload, new device buffers (rebind) and onload into renumbered
    slots, the continuation's logits and log-probabilities against the
    oracle run of the same sequences, at the stated bars (bf16) or 1e-4
    (fp32)."""
    import oracle
    from harness import (F32_LOGIT_REL_TOL, F32_LOGP_ABS_TOL, LOGIT_REL_TOL, LOGP_ABS_TOL, OracleRollout,
                         row_rel_err)
    w_dev, _, om = build_models(shape, 65)
    prompts = _case(shape)
    old, new = list(range(6)), [11, 7, 9, 6, 10, 8]
    group = 3
    eng = _engine(shape, w_dev)
    _prefill(eng, old, prompts, group)
    orc = OracleRollout(om, 128)
    for p, pr in enumerate(prompts):
        orc.prefill(old[p * group], pr)
        for k in range(1, group):
            orc.seqs[old[p * group + k]] = orc.seqs[old[p * group]].clone()
    for k in range(3):
        _step(eng, old, k, shape.vocab)
        tin = uniform_tokens(len(old), shape.vocab, 70 + k)
        for i, s in enumerate(old):
            orc.step(s, tin[i])
    lengths = [eng.slot_length(s) for s in old]
    host = torch.empty(eng.kv_offload_bytes(old), dtype=torch.uint8, pin_memory=True)
    eng.kv_offload(old, host)
    torch.cuda.synchronize()
    eng.release(old)
    w2 = {k: v.clone() for k, v in w_dev.items()}
    kv2 = torch.full_like(eng.kv, 0x7F)
    ws2 = torch.full_like(eng.ws, 0x3C)
    eng.kv.zero_()
    eng.rebind(w2, kv2, ws2)
    eng.kv_onload(new, lengths, host)
    tol = (LOGIT_REL_TOL, LOGP_ABS_TOL) if shape.dtype == "bf16" else (F32_LOGIT_REL_TOL, F32_LOGP_ABS_TOL)
    for k in range(3, 6):
        lg, ot, ol = _step(eng, new, k, shape.vocab)
        tin = uniform_tokens(len(new), shape.vocab, 70 + k)
        for i, s in enumerate(old):
            z = orc.step(s, tin[i])
            assert row_rel_err(lg[i], z) < tol[0], (k, i)
            assert abs(ol[i] - oracle.logprob(z.astype(np.float32), 1.0, int(ot[i]))) < tol[1], (k, i)
    eng.close()
