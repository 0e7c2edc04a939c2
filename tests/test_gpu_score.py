"""Inference-stage scoring (rl_score) vs the CPU oracle, through the C ABI
(needs an MI355X).

rl_score computes, for every response token, its log-probability given the
prompt and the response tokens before it, in one causal forward over all
tokens with each prompt computed once per group.  The oracle feeds every
sequence one token at a time through its own KV-cached forward and takes a
plain fp64 log-softmax at each response token.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from harness import F32_LOGP_ABS_TOL, LOGP_ABS_TOL, build_models
from paper_2509_15965_amd.configs import WORKLOADS, ModelShape
from paper_2509_15965_amd.inputs import patch_rows, uniform_tokens
from paper_2509_15965_amd.rl_decode import RL_OPT_ATTN_CHUNK, RL_OPT_GEMM_PLAN, RL_OPT_PREFILL_ATTENTION, \
    RL_GEMM_T128, Engine, gemm_plan_code

pytestmark = pytest.mark.gpu

DEV = "cuda"

GQA = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e4, "bf16")      # group 4, d 128
G7 = ModelShape(2, 448, 14, 2, 64, 640, 776, 1e-6, 1e6, "bf16")         # group 7 (7B ratio), d 64
MHA = ModelShape(2, 256, 4, 4, 64, 512, 520, 1e-5, 1e4, "bf16")         # group 1


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _i32(a):
    return torch.as_tensor(np.asarray(a, dtype=np.int32), device=DEV)


def make_case(shape, n_prompts, group, plens, rlens, seed):
    rng = np.random.default_rng(seed)
    prompts = [rng.integers(0, shape.vocab, size=int(n)).astype(np.int32) for n in plens]
    resp = [rng.integers(0, shape.vocab, size=int(m)).astype(np.int32) for m in rlens]
    assert len(prompts) == n_prompts and len(resp) == n_prompts * group
    return prompts, resp


def run_score(shape, w_dev, prompts, group, resp, T, *, embeds=None, chunk=0, gemm_plan=0, max_seqs=None,
              slots=None, prefill_items=False):
    n_seq = len(prompts) * group
    plens = [len(p) for p in prompts]
    rlens = [len(r) for r in resp]
    max_ctx = max(plens[s // group] + rlens[s] for s in range(n_seq))
    eng = Engine(shape, w_dev, max_seqs=max_seqs or n_seq, max_ctx=max_ctx,
                 max_prefill_tokens=sum(plens) + sum(rlens))
    if chunk:
        eng.set_option(RL_OPT_ATTN_CHUNK, chunk)
    if gemm_plan:
        eng.set_option(RL_OPT_GEMM_PLAN, gemm_plan)
    if prefill_items:
        eng.set_option(RL_OPT_PREFILL_ATTENTION, 1)
    slots = slots if slots is not None else list(reversed(range(n_seq)))
    poffs = np.concatenate([[0], np.cumsum(plens)]).astype(np.int32)
    roffs = np.concatenate([[0], np.cumsum(rlens)]).astype(np.int32)
    out = torch.full((int(roffs[-1]),), 123.0, dtype=torch.float32, device=DEV)
    eng.score(slots, poffs, _i32(np.concatenate(prompts)), roffs, _i32(np.concatenate(resp)), out,
              group=group, embeds=None if embeds is None else embeds.to(DEV), temperature=T)
    torch.cuda.synchronize()
    for s in slots:
        assert eng.slot_length(s) == 0          # scratch slots are released
    got = out.cpu().numpy().astype(np.float64)
    eng.close()
    return got


def oracle_scores(om, prompts, group, resp, T, embeds=None):
    emb = None
    if embeds is not None:
        from paper_2509_15965_amd.inputs import to_host_numpy
        emb = to_host_numpy(embeds)
    return np.concatenate([oracle.score(om, prompts[s // group], resp[s], T, embeds=emb)
                           for s in range(len(resp))])


def _check(got, ref, tol, what):
    assert got.shape == ref.shape
    assert np.isfinite(got).all(), what
    assert np.all(got <= 1e-6), what
    err = np.abs(got - ref).max()
    assert err < tol, (what, err)
    return err


def test_score_tiny_fp32_matches_oracle():
    """The tiny fp32 decoder: 2 prompts x 4 responses, ragged prompts and
    responses (1 to 32 tokens), slots in reverse order."""
    shape = WORKLOADS["tiny"].model
    w_dev, _, om = build_models(shape, 31)
    prompts, resp = make_case(shape, 2, 4, [32, 17], [1, 5, 32, 20, 9, 31, 2, 16], 32)
    got = run_score(shape, w_dev, prompts, 4, resp, 1.0)
    ref = oracle_scores(om, prompts, 4, resp, 1.0)
    _check(got, ref, F32_LOGP_ABS_TOL, "tiny fp32")


@pytest.mark.parametrize("T", [1.0, 0.6, 0.0])
def test_score_bf16_gqa_matches_oracle(T):
    """Group-4 bf16 decoder: 3 prompts x 3 responses over several attention
    blocks and GEMM tiles with ragged tails; T = 0 reports T = 1 values."""
    w_dev, _, om = build_models(GQA, 33)
    prompts, resp = make_case(GQA, 3, 3, [40, 70, 9], [1, 60, 33, 17, 2, 45, 58, 7, 26], 34)
    got = run_score(GQA, w_dev, prompts, 3, resp, T)
    ref = oracle_scores(om, prompts, 3, resp, T)
    _check(got, ref, LOGP_ABS_TOL, f"gqa T={T}")


@pytest.mark.parametrize("shape", [G7, MHA], ids=["group7", "mha"])
def test_score_head_groupings_match_oracle(shape):
    w_dev, _, om = build_models(shape, 35)
    prompts, resp = make_case(shape, 2, 2, [23, 51], [38, 1, 64, 19], 36)
    got = run_score(shape, w_dev, prompts, 2, resp, 1.0)
    ref = oracle_scores(om, prompts, 2, resp, 1.0)
    _check(got, ref, LOGP_ABS_TOL, shape)


@pytest.mark.parametrize("shape", [GQA, G7, MHA], ids=["group4", "group7", "mha"])
def test_score_both_prefill_attention_kernels(shape):
    """The LDS-shared tile kernel (default) and the split-KV item kernel
    both match the oracle, over tiles cut short at sequence ends."""
    w_dev, _, om = build_models(shape, 47)
    prompts, resp = make_case(shape, 2, 2, [33, 70], [45, 2, 64, 29], 48)
    ref = oracle_scores(om, prompts, 2, resp, 1.0)
    for items in (False, True):
        got = run_score(shape, w_dev, prompts, 2, resp, 1.0, prefill_items=items)
        _check(got, ref, LOGP_ABS_TOL, (shape, items))


def test_score_split_kv_chunks_and_forced_tile_kernel():
    """32-position split-KV chunks (every long row combines several partial
    sums) and a forced 128x128 tile GEMM give the same scores."""
    w_dev, _, om = build_models(GQA, 37)
    prompts, resp = make_case(GQA, 2, 2, [90, 41], [120, 3, 77, 150], 38)
    ref = oracle_scores(om, prompts, 2, resp, 1.0)
    got = run_score(GQA, w_dev, prompts, 2, resp, 1.0, chunk=32, prefill_items=True)
    _check(got, ref, LOGP_ABS_TOL, "chunk 32")
    got2 = run_score(GQA, w_dev, prompts, 2, resp, 1.0, gemm_plan=gemm_plan_code(RL_GEMM_T128))
    _check(got2, ref, LOGP_ABS_TOL, "tile 128")


def test_score_embedding_prompt_rows():
    """Prompts that start with caller-provided embedding rows (ids < 0)."""
    w_dev, _, om = build_models(GQA, 39)
    rows = patch_rows(12, GQA.hidden, 40)
    rng = np.random.default_rng(41)
    prompts = [np.concatenate([-(np.arange(12) + 1), rng.integers(0, GQA.vocab, size=5)]).astype(np.int32),
               np.concatenate([-(np.arange(4) + 1), rng.integers(0, GQA.vocab, size=9)]).astype(np.int32)]
    resp = [rng.integers(0, GQA.vocab, size=m).astype(np.int32) for m in (14, 6)]
    got = run_score(GQA, w_dev, prompts, 1, resp, 1.0, embeds=rows)
    ref = oracle_scores(om, prompts, 1, resp, 1.0, embeds=rows)
    _check(got, ref, LOGP_ABS_TOL, "embeds")


def test_score_out_of_range_target_is_nan_and_chunked_lm_head():
    """An id outside the vocabulary scores NaN (its row still embeds as
    zeros, as in decoding); with this small workspace (max_seqs = 3, 28
    rows) the LM head runs in several 4-row chunks; the other entries match
    the oracle run on the same ids."""
    shape = WORKLOADS["tiny"].model
    w_dev, _, om = build_models(shape, 42)
    prompts, resp = make_case(shape, 1, 2, [12], [9, 7], 43)
    resp[1][4] = shape.vocab + 5
    got = run_score(shape, w_dev, prompts, 2, resp, 1.0, max_seqs=3, slots=[2, 0])
    bad = 9 + 4
    assert math.isnan(got[bad])
    # the oracle embeds an out-of-range id as zeros too: build its reference
    # with an explicit zero row
    zero = np.zeros((1, shape.hidden), dtype=np.float32)
    r1 = oracle.score(om, prompts[0], resp[0], 1.0)
    seq = om.new_seq(64)
    for t in prompts[0]:
        z = seq.forward(int(t))
    r2 = []
    for j, y in enumerate(resp[1]):
        r2.append(oracle.logprob(z.astype(np.float32), 1.0, int(y)))
        if j + 1 < len(resp[1]):
            z = seq.forward(int(y)) if 0 <= y < shape.vocab else seq.forward(-1, embed_row=zero[0])
    ref = np.concatenate([r1, np.array(r2)])
    keep = np.arange(len(ref)) != bad
    assert math.isnan(ref[bad])
    _check(got[keep], ref[keep], F32_LOGP_ABS_TOL, "nan target")


def test_score_equals_teacher_forced_decode_fp32():
    """Scoring a sequence equals prefill + teacher-forced decoding of it in
    the fp32 model (the same log-probabilities, different launch shapes)."""
    shape = WORKLOADS["tiny"].model
    w_dev, _, _ = build_models(shape, 44)
    prompts, resp = make_case(shape, 2, 2, [20, 31], [24, 24, 24, 24], 45)
    got = run_score(shape, w_dev, prompts, 2, resp, 0.8)
    n = 4
    eng = Engine(shape, w_dev, max_seqs=n, max_ctx=31 + 24, max_prefill_tokens=51)
    R = np.stack(resp)                                    # [n][24]
    ot = torch.empty(n, dtype=torch.int32, device=DEV)
    ol = torch.empty(n, dtype=torch.float32, device=DEV)
    dec = np.zeros((n, 24))
    eng.prefill(list(range(n)), list(range(n)), [0, 20, 51], _i32(np.concatenate(prompts)), ot, ol, group=2,
                forced=_i32(R[:, 0]), temperature=0.8)
    dec[:, 0] = ol.cpu().numpy()
    for j in range(1, 24):
        eng.step(list(range(n)), list(range(n)), _i32(R[:, j - 1]), ot, ol, forced=_i32(R[:, j]), temperature=0.8)
        dec[:, j] = ol.cpu().numpy()
    eng.close()
    err = np.abs(got - dec.reshape(-1)).max()
    assert err < F32_LOGP_ABS_TOL, err


def test_score_rejects_bad_arguments():
    shape = WORKLOADS["tiny"].model
    w_dev, _, _ = build_models(shape, 46)
    eng = Engine(shape, w_dev, max_seqs=4, max_ctx=16, max_prefill_tokens=20)
    p = _i32(uniform_tokens(8, shape.vocab, 1))
    r = _i32(uniform_tokens(16, shape.vocab, 2))
    out = torch.empty(16, dtype=torch.float32, device=DEV)
    from paper_2509_15965_amd.rl_decode import RLError
    with pytest.raises(RLError):                          # prompt + response > max_ctx
        eng.score([0, 1], [0, 8], p, [0, 9, 16], r, out, group=2)
    with pytest.raises(RLError):                          # empty response
        eng.score([0, 1], [0, 4], p, [0, 0, 4], r, out, group=2)
    with pytest.raises(RLError):                          # duplicate slot
        eng.score([1, 1], [0, 4], p, [0, 4, 8], r, out, group=2)
    with pytest.raises(RLError):                          # more tokens than max_prefill_tokens
        eng.score([0, 1, 2, 3], [0, 4, 8], p, [0, 4, 8, 12, 16], r, out, group=2)
    with pytest.raises(RLError):                          # negative temperature
        eng.score([0, 1], [0, 4], p, [0, 4, 8], r, out, group=2, temperature=-1.0)
    eng.score([0, 1], [0, 4], p, [0, 4, 8], r, out, group=2)   # the valid call still works
    torch.cuda.synchronize()
    assert np.isfinite(out[:8].cpu().numpy()).all()
    eng.close()
