"""GPU path vs the CPU oracle, through the C ABI (needs an MI355X).

Sizes here are small enough for the oracle to finish in seconds while
spanning several GEMM and attention tiles with ragged tails.
"""
import numpy as np
import pytest
import torch

import oracle
from harness import (F32_LOGIT_REL_TOL, F32_LOGP_ABS_TOL, LOGIT_REL_TOL, LOGP_ABS_TOL, OracleRollout,
                     build_models, check_token, inject_random_kv, row_rel_err)
from paper_2509_15965_amd.configs import WORKLOADS, ModelShape
from paper_2509_15965_amd.inputs import rollout_plan, uniform_tokens
from paper_2509_15965_amd.rl_decode import (RL_GEMM_DIRECT, RL_GEMM_GEMV, RL_GEMM_GEMV_WIDE, RL_GEMM_T128,
                                           RL_GEMM_T128_DEEP,
                                           RL_GEMM_T128X256, RL_GEMM_T256, RL_OPT_ATTN_CHUNK, RL_OPT_GEMM_PLAN,
                                           Engine, RLError, gemm_plan_code)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _i32(a):
    return torch.as_tensor(np.asarray(a, dtype=np.int32), device=DEV)


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def teacher_forced_run(shape, seed, prompts, group, n_steps, T=1.0, sample_seed=5, max_ctx=None,
                       embed_rows=None, gemm_plan=0, tune_sizes=None):
    """Prefill `prompts` (group slots each), then n_steps decode steps that feed
    seeded forced tokens.  Returns per-step (gpu logits, oracle logits, gpu
    logp, oracle logp, gpu tokens, oracle sampled tokens)."""
    w_dev, w_host, om = build_models(shape, seed)
    n_seq = len(prompts) * group
    plens = [len(p) for p in prompts]
    max_ctx = max_ctx or (max(plens) + n_steps + 2)
    eng = Engine(shape, w_dev, max_seqs=n_seq, max_ctx=max_ctx, max_prefill_tokens=sum(plens))
    if gemm_plan:
        eng.set_option(RL_OPT_GEMM_PLAN, gemm_plan)
    if tune_sizes:
        eng.tune_gemms(tune_sizes)
    slots = list(range(n_seq))
    uids = [1000 + i for i in range(n_seq)]
    offs = np.concatenate([[0], np.cumsum(plens)]).astype(np.int32)
    toks = _i32(np.concatenate(prompts))
    forced = [uniform_tokens(n_seq, shape.vocab, seed + 100 + s) for s in range(n_steps + 1)]
    out_tok = torch.empty(n_seq, dtype=torch.int32, device=DEV)
    out_lp = torch.empty(n_seq, dtype=torch.float32, device=DEV)
    logits_p = torch.empty((len(prompts), shape.vocab), dtype=torch.float32, device=DEV)
    emb = None if embed_rows is None else embed_rows.to(DEV)
    eng.prefill(slots, uids, offs, toks, out_tok, out_lp, group=group, forced=_i32(forced[0]),
                seed=sample_seed, temperature=T, out_logits=logits_p, embeds=emb)
    torch.cuda.synchronize()
    emb_host = None
    if embed_rows is not None:
        from paper_2509_15965_amd.inputs import to_host_numpy
        emb_host = to_host_numpy(embed_rows)
    orc = OracleRollout(om, max_ctx)
    zo_p = []
    for p in range(len(prompts)):
        zo_p.append(orc.prefill(p * group, prompts[p], emb_host))
        for k in range(1, group):
            orc.seqs[p * group + k] = orc.seqs[p * group].clone()
    zg = logits_p.cpu().numpy()
    zo = np.stack(zo_p)
    lo = np.array([oracle.sample(zo[i // group].astype(np.float32), T, sample_seed, uids[i], plens[i // group],
                                 forced=int(forced[0][i]))[1] for i in range(n_seq)])
    so = [oracle.sample(zo[i // group].astype(np.float32), T, sample_seed, uids[i], plens[i // group])[0]
          for i in range(n_seq)]
    res = [(zg, zo, out_lp.cpu().numpy(), lo, out_tok.cpu().numpy(), np.array(so))]
    logits = torch.empty((n_seq, shape.vocab), dtype=torch.float32, device=DEV)
    for s in range(1, n_steps + 1):
        in_tok = _i32(forced[s - 1])
        eng.step(slots, uids, in_tok, out_tok, out_lp, forced=_i32(forced[s]), seed=sample_seed,
                 temperature=T, out_logits=logits)
        torch.cuda.synchronize()
        zg = logits.cpu().numpy()
        zo = np.stack([orc.step(i, forced[s - 1][i]) for i in range(n_seq)])
        pos_new = [orc.length(i) for i in range(n_seq)]
        lo = np.array([oracle.sample(zo[i].astype(np.float32), T, sample_seed, uids[i], pos_new[i],
                                     forced=int(forced[s][i]))[1] for i in range(n_seq)])
        so = [oracle.sample(zo[i].astype(np.float32), T, sample_seed, uids[i], pos_new[i])[0] for i in range(n_seq)]
        res.append((zg, zo, out_lp.cpu().numpy(), lo, out_tok.cpu().numpy(), np.array(so)))
    for i in range(n_seq):
        assert eng.slot_length(i) == plens[i // group] + n_steps
    eng.close()
    return res


def test_sampler_matches_oracle_on_given_logits():
    shape = WORKLOADS["tiny"].model
    w_dev, _, _ = build_models(shape, 3)
    n, V = 37, shape.vocab
    eng = Engine(shape, w_dev, max_seqs=64, max_ctx=16, max_prefill_tokens=16)
    rng = np.random.default_rng(0)
    z = rng.normal(0, 2.5, size=(n, V)).astype(np.float32)
    z[5, 100] = z[5, 7] = 30.0                                # exact tie for greedy
    zt = torch.from_numpy(z).to(DEV)
    uids = [int(u) for u in rng.integers(0, 2 ** 63, size=n, dtype=np.int64)]
    pos = [int(p) for p in rng.integers(0, 5000, size=n)]
    forced = rng.integers(0, V, size=n).astype(np.int32)
    out_tok = torch.empty(n, dtype=torch.int32, device=DEV)
    out_lp = torch.empty(n, dtype=torch.float32, device=DEV)
    for T in (1.0, 0.6, 0.0):
        for use_forced in (False, True):
            eng.sample_logits(zt, uids, pos, out_tok, out_lp, seed=0xABCDEF0123, temperature=T,
                              forced=_i32(forced) if use_forced else None)
            torch.cuda.synchronize()
            gt, gl = out_tok.cpu().numpy(), out_lp.cpu().numpy()
            for i in range(n):
                ot, ol = oracle.sample(z[i], T, 0xABCDEF0123, uids[i], pos[i],
                                       forced=int(forced[i]) if use_forced else -1)
                assert gt[i] == ot, (T, i)
                assert abs(gl[i] - ol) < 1e-5, (T, i, gl[i], ol)
    assert out_tok.cpu().numpy()[5] in (7, 100)
    eng.close()


@pytest.mark.parametrize("n", [6, 2048], ids=["merged-chunks", "single-chunk"])
def test_sampler_nan_rows_never_index_outside_the_row(n):
    """A NaN score never wins a comparison.  A row of NaN logits ranks no
    entry: token -1 and a NaN log-probability (no logit outside the row is
    read).  A row with some NaN entries samples among its other entries (the
    oracle's sample with the NaN entries at -inf) and has a NaN
    log-probability (its log-sum-exp is NaN).  The other rows are unchanged.
    Both the merge kernel (few rows, several vocabulary chunks per row) and
    the single-chunk path (2048 rows) are covered."""
    shape = WORKLOADS["tiny"].model
    w_dev, _, _ = build_models(shape, 5)
    V = shape.vocab
    eng = Engine(shape, w_dev, max_seqs=n, max_ctx=16, max_prefill_tokens=16)
    rng = np.random.default_rng(2)
    z = rng.normal(0, 2.0, size=(n, V)).astype(np.float32)
    z[0, :] = np.nan
    z[1, ::3] = np.nan
    zt = torch.from_numpy(z).to(DEV)
    z_inf = np.where(np.isnan(z[1]), -np.inf, z[1]).astype(np.float32)
    uids = [int(u) for u in rng.integers(0, 2 ** 63, size=n, dtype=np.int64)]
    pos = [int(p) for p in rng.integers(0, 5000, size=n)]
    forced = rng.integers(0, V, size=n).astype(np.int32)
    out_tok = torch.empty(n, dtype=torch.int32, device=DEV)
    out_lp = torch.empty(n, dtype=torch.float32, device=DEV)
    for T in (1.0, 0.0):
        for use_forced in (False, True):
            eng.sample_logits(zt, uids, pos, out_tok, out_lp, seed=91, temperature=T,
                              forced=_i32(forced) if use_forced else None)
            torch.cuda.synchronize()
            gt, gl = out_tok.cpu().numpy(), out_lp.cpu().numpy()
            assert gt[0] == -1 and np.isnan(gl[0]), (T, use_forced)
            assert gt[1] == oracle.sample(z_inf, T, 91, uids[1], pos[1])[0] and np.isnan(gl[1]), (T, use_forced)
            for i in range(2, min(n, 40)):
                ot, ol = oracle.sample(z[i], T, 91, uids[i], pos[i], forced=int(forced[i]) if use_forced else -1)
                assert gt[i] == ot and abs(gl[i] - ol) < 1e-5, (T, use_forced, i)
    eng.close()


def test_sampler_single_chunk_rows_match_oracle():
    """From 2048 rows each row's vocabulary is one chunk: the sampling
    workgroup finishes the row itself (no merge kernel)."""
    shape = WORKLOADS["tiny"].model
    w_dev, _, _ = build_models(shape, 4)
    n, V = 2048, shape.vocab
    eng = Engine(shape, w_dev, max_seqs=n, max_ctx=16, max_prefill_tokens=16)
    rng = np.random.default_rng(1)
    z = rng.normal(0, 2.0, size=(n, V)).astype(np.float32)
    uids = [int(u) for u in rng.integers(0, 2 ** 63, size=n, dtype=np.int64)]
    pos = [int(p) for p in rng.integers(0, 5000, size=n)]
    out_tok = torch.empty(n, dtype=torch.int32, device=DEV)
    out_lp = torch.empty(n, dtype=torch.float32, device=DEV)
    eng.sample_logits(torch.from_numpy(z).to(DEV), uids, pos, out_tok, out_lp, seed=77, temperature=0.8)
    torch.cuda.synchronize()
    gt, gl = out_tok.cpu().numpy(), out_lp.cpu().numpy()
    for i in range(0, n, 7):
        ot, ol = oracle.sample(z[i], 0.8, 77, uids[i], pos[i])
        assert gt[i] == ot, i
        assert abs(gl[i] - ol) < 1e-5, (i, gl[i], ol)
    eng.close()


def test_tiny_fp32_rollout_bit_exact_tokens():
    """The tiny fp32 workload end to end: 2 prompts x 4 samples, 32 prompt
    tokens, 32 generated tokens, seeded Gumbel noise at T = 1.  Every GPU token
    equals the oracle's (near ties excused and counted); the oracle follows
    the GPU's tokens so one excused tie does not end the comparison."""
    wl = WORKLOADS["tiny"]
    shape = wl.model
    plan = rollout_plan(wl)
    w_dev, _, om = build_models(shape, wl.seed)
    G, P = wl.group, wl.n_prompts
    n = P * G
    max_ctx = 64
    eng = Engine(shape, w_dev, max_seqs=n, max_ctx=max_ctx, max_prefill_tokens=64)
    prompts = plan["prompts"]
    offs = np.concatenate([[0], np.cumsum([len(p) for p in prompts])]).astype(np.int32)
    uids = [int(u) for u in plan["uids"]]
    slots = list(range(n))
    seed, T = 777, wl.temperature
    out_tok = torch.empty(n, dtype=torch.int32, device=DEV)
    out_lp = torch.empty(n, dtype=torch.float32, device=DEV)
    lg_p = torch.empty((P, shape.vocab), dtype=torch.float32, device=DEV)
    lg = torch.empty((n, shape.vocab), dtype=torch.float32, device=DEV)
    eng.prefill(slots, uids, offs, _i32(np.concatenate(prompts)), out_tok, out_lp, group=G, seed=seed,
                temperature=T, out_logits=lg_p)
    torch.cuda.synchronize()
    orc = {}
    excused = []
    toks = out_tok.cpu().numpy().copy()
    lps = out_lp.cpu().numpy().copy()
    zg = lg_p.cpu().numpy()
    for i in range(n):
        s = om.new_seq(max_ctx)
        for t in prompts[i // G]:
            z = s.forward(int(t))
        orc[i] = s
        assert row_rel_err(zg[i // G], z) < F32_LOGIT_REL_TOL
        assert check_token(int(toks[i]), z, T, seed, uids[i], len(prompts[i // G]), excused), (i, 0)
        _, ol = oracle.sample(z.astype(np.float32), T, seed, uids[i], len(prompts[i // G]), forced=int(toks[i]))
        assert abs(lps[i] - ol) < F32_LOGP_ABS_TOL
    all_tokens = [toks.copy()]
    for step in range(1, wl.response_cap):
        eng.step(slots, uids, out_tok.clone(), out_tok, out_lp, seed=seed, temperature=T, out_logits=lg)
        torch.cuda.synchronize()
        new = out_tok.cpu().numpy().copy()
        lps = out_lp.cpu().numpy()
        zg = lg.cpu().numpy()
        for i in range(n):
            z = orc[i].forward(int(toks[i]))
            assert row_rel_err(zg[i], z) < F32_LOGIT_REL_TOL, (i, step)
            assert check_token(int(new[i]), z, T, seed, uids[i], orc[i].length, excused), (i, step)
            _, ol = oracle.sample(z.astype(np.float32), T, seed, uids[i], orc[i].length, forced=int(new[i]))
            assert abs(lps[i] - ol) < F32_LOGP_ABS_TOL
        toks = new
        all_tokens.append(new)
    assert len(excused) <= 2, excused
    # samples of one prompt differ (uid-keyed noise) though their prefill logits are equal
    first = all_tokens[0]
    assert len(set(first[:G].tolist())) > 1 or len(set(first[G:].tolist())) > 1
    eng.close()


@pytest.mark.parametrize("shape", [
    # GQA group 4, head_dim 128, ragged hidden/ffn/vocab tiles
    ModelShape(2, 320, 8, 2, 128, 712, 1000, 1e-6, 1e6, "bf16"),
    # MHA, head_dim 64
    ModelShape(2, 256, 4, 4, 64, 520, 776, 1e-5, 1e4, "bf16"),
    # group 7 (the 7B shape's ratio), head_dim 128
    ModelShape(1, 448, 7, 1, 128, 384, 512, 1e-6, 1e6, "bf16"),
])
def test_bf16_prefill_and_decode_teacher_forced(shape):
    rng = np.random.default_rng(11)
    lens = [1, 7, 33, 70]
    prompts = [rng.integers(0, shape.vocab, size=n).astype(np.int32) for n in lens]
    res = teacher_forced_run(shape, 21, prompts, group=2, n_steps=6, T=1.0)
    agree = total = 0
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, k
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, k
        agree += int((tg == to).sum())
        total += len(tg)
    assert agree >= 0.8 * total          # sampled tokens mostly agree despite bf16 round-off


def test_bf16_prefill_with_embedding_rows_and_temperature():
    shape = ModelShape(2, 256, 4, 2, 64, 512, 640, 1e-5, 1e4, "bf16")
    from paper_2509_15965_amd.inputs import patch_rows
    rows = patch_rows(12, shape.hidden, 3)
    rng = np.random.default_rng(4)
    p0 = np.concatenate([-(np.arange(12) + 1), rng.integers(0, shape.vocab, size=5)]).astype(np.int32)
    p1 = rng.integers(0, shape.vocab, size=9).astype(np.int32)
    res = teacher_forced_run(shape, 8, [p0, p1], group=3, n_steps=3, T=0.6, embed_rows=rows)
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, k
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, k


def test_split_kv_long_context_matches_oracle_and_any_chunk():
    """Injected caches up to 3000 positions: the split-KV decode step matches
    the oracle, and every chunk size gives the same result up to bf16
    probability rounding."""
    shape = ModelShape(2, 256, 8, 2, 128, 512, 1024, 1e-6, 1e6, "bf16")
    w_dev, _, om = build_models(shape, 31)
    lengths = [3000, 1, 31, 32, 33, 777]
    n = len(lengths)
    eng = Engine(shape, w_dev, max_seqs=n, max_ctx=3008, max_prefill_tokens=8)
    slots = list(range(n))
    uids = list(range(n))
    tok = uniform_tokens(n, shape.vocab, 2)
    results = {}
    for chunk in (0, 32, 64, 256, 4096):
        seqs = inject_random_kv(eng, om, slots, lengths, seed=99)
        eng.set_option(RL_OPT_ATTN_CHUNK, chunk)
        logits = torch.empty((n, shape.vocab), dtype=torch.float32, device=DEV)
        ot = torch.empty(n, dtype=torch.int32, device=DEV)
        ol = torch.empty(n, dtype=torch.float32, device=DEV)
        eng.step(slots, uids, _i32(tok), ot, ol, seed=1, out_logits=logits)
        torch.cuda.synchronize()
        results[chunk] = logits.cpu().numpy()
        if chunk == 0:
            zo = np.stack([seqs[s].forward(int(tok[s])) for s in slots])
            assert row_rel_err(results[0], zo) < LOGIT_REL_TOL
    for chunk, z in results.items():
        assert row_rel_err(z, results[4096]) < 1e-2, chunk
    eng.close()


def test_decode_is_deterministic():
    """Two identical runs give the same bits; a third run that asks for no
    logits (the benchmark's calls) samples the same tokens with the same
    log-probabilities."""
    shape = ModelShape(2, 256, 4, 2, 64, 512, 512, 1e-6, 1e6, "bf16")
    w_dev, _, _ = build_models(shape, 5)
    outs = []
    for r in range(3):
        eng = Engine(shape, w_dev, max_seqs=4, max_ctx=64, max_prefill_tokens=64)
        toks = _i32(uniform_tokens(40, shape.vocab, 1))
        ot = torch.empty(4, dtype=torch.int32, device=DEV)
        ol = torch.empty(4, dtype=torch.float32, device=DEV)
        lg = torch.empty((4, shape.vocab), dtype=torch.float32, device=DEV)
        eng.prefill([0, 1, 2, 3], [9, 8, 7, 6], [0, 10, 40], toks, ot, ol, group=2, seed=3)
        run = []
        for _ in range(5):
            eng.step([0, 1, 2, 3], [9, 8, 7, 6], ot.clone(), ot, ol, seed=3, out_logits=lg if r < 2 else None)
            run.append((ot.cpu().numpy().copy(), ol.cpu().numpy().copy(), lg.cpu().numpy().copy()))
        outs.append(run)
        eng.close()
    for a, b, c in zip(*outs):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
        assert np.array_equal(a[0], c[0]) and np.array_equal(a[1], c[1])


def test_step_rejects_bad_arguments_without_side_effects():
    shape = ModelShape(1, 64, 2, 1, 64, 64, 64, 1e-6, 1e4, "bf16")
    w_dev, _, _ = build_models(shape, 1)
    eng = Engine(shape, w_dev, max_seqs=4, max_ctx=8, max_prefill_tokens=8)
    ot = torch.empty(4, dtype=torch.int32, device=DEV)
    ol = torch.empty(4, dtype=torch.float32, device=DEV)
    t = _i32([1, 2, 3, 4])
    from paper_2509_15965_amd.rl_decode import RLError
    with pytest.raises(RLError) as e:
        eng.step([0, 0], [1, 2], t, ot, ol)                    # duplicate slot
    assert e.value.status == 1
    with pytest.raises(RLError) as e:
        eng.step([0, 9], [1, 2], t, ot, ol)                    # slot out of range
    assert e.value.status == 1
    with pytest.raises(RLError) as e:
        eng.step([0], [1], t, ot, ol, temperature=-1.0)
    assert e.value.status == 1
    eng.set_lengths([1], [8])
    with pytest.raises(RLError) as e:
        eng.step([1], [1], t, ot, ol)                          # full slot
    assert e.value.status == 3
    assert eng.slot_length(0) == 0 and eng.slot_length(1) == 8
    with pytest.raises(RLError) as e:
        eng.prefill([0], [1], [0, 8], t, ot, ol)               # prompt of max_ctx tokens
    assert e.value.status == 3
    # options: out-of-range values are refused and leave the setting as it was
    from paper_2509_15965_amd.rl_decode import (RL_OPT_ATTN_CHUNK, RL_OPT_PREFILL_ATTENTION,
                                               RL_OPT_SHARED_PREFIX)
    for opt, bad in [(RL_OPT_ATTN_CHUNK, 16), (RL_OPT_ATTN_CHUNK, 33), (RL_OPT_ATTN_CHUNK, 65568),
                     (RL_OPT_ATTN_CHUNK, -32), (RL_OPT_SHARED_PREFIX, 2), (RL_OPT_PREFILL_ATTENTION, -1),
                     (RL_OPT_GEMM_PLAN, 8), (RL_OPT_GEMM_PLAN, 5 | (33 << 8)), (RL_OPT_GEMM_PLAN, 5 | (2 << 16)),
                     (99, 0)]:
        with pytest.raises(RLError) as e:
            eng.set_option(opt, bad)
        assert e.value.status == 1, (opt, bad)
    eng.set_option(RL_OPT_ATTN_CHUNK, 65536)
    eng.set_option(RL_OPT_ATTN_CHUNK, 0)
    eng.set_lengths([1], [0])
    eng.step([0, 1], [1, 2], t, ot, ol)                        # still usable after the refusals
    assert eng.slot_length(0) == 1 and eng.slot_length(1) == 1
    eng.close()


def test_empty_calls_are_no_ops_and_empty_prompts_are_refused():
    """Zero rows is a no-op for every per-row entry point (nothing enqueued,
    no length changed); an empty prompt or response, or a prefill of no
    prompts, is refused; the engine decodes normally afterwards."""
    shape = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e6, "bf16")
    w_dev, _, _ = build_models(shape, 7)
    eng = Engine(shape, w_dev, max_seqs=4, max_ctx=16, max_prefill_tokens=16)
    i0 = torch.empty(0, dtype=torch.int32, device=DEV)
    f0 = torch.empty(0, dtype=torch.float32, device=DEV)
    eng.step([], [], i0, i0, f0)
    eng.sample_logits(torch.empty((0, shape.vocab), dtype=torch.float32, device=DEV), [], [], i0, f0)
    eng.release([])
    eng.set_lengths([], [])
    assert eng.kv_offload_bytes([]) == 0
    assert all(eng.slot_length(i) == 0 for i in range(4))
    t = _i32([3, 4, 5])
    ot = torch.empty(4, dtype=torch.int32, device=DEV)
    ol = torch.empty(4, dtype=torch.float32, device=DEV)
    for args in (([], [], [0]), ([0], [1], [0, 0]), ([0, 1], [1, 2], [0, 2, 2])):
        with pytest.raises(RLError) as e:
            eng.prefill(*args, t, ot, ol)
        assert e.value.status == 1, args
    lp = torch.empty(4, dtype=torch.float32, device=DEV)
    with pytest.raises(RLError) as e:
        eng.score([0, 1], [0, 2], t, [0, 2, 2], t, lp, group=2)   # second response empty
    assert e.value.status == 1
    assert all(eng.slot_length(i) == 0 for i in range(4))
    eng.prefill([0], [1], [0, 3], t, ot, ol)
    eng.step([0], [1], ot[:1], ot[1:2], ol[:1])
    assert eng.slot_length(0) == 4
    eng.close()


def test_one_token_prompts_match_oracle():
    """Prompts of a single token (each query attends to one key at prefill),
    shared by a group of 2, then decoding."""
    shape = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e6, "bf16")
    prompts = [np.array([5], dtype=np.int32), np.array([1031], dtype=np.int32), np.array([0, 9], dtype=np.int32)]
    res = teacher_forced_run(shape, 313, prompts, group=2, n_steps=3, T=1.0)
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, k
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, k


@pytest.mark.parametrize("n_prompts,plen", [(100, 3), (140, 4), (9, 70)])
def test_large_batch_gemm_tiles_match_oracle(n_prompts, plen):
    """Batches above 64 rows take the LDS-tiled GEMM (128- and 256-row tiles,
    split K for the narrow matrices) in both prefill and decode."""
    shape = ModelShape(2, 512, 8, 2, 128, 1096, 1032, 1e-6, 1e6, "bf16")
    rng = np.random.default_rng(n_prompts)
    prompts = [rng.integers(0, shape.vocab, size=plen).astype(np.int32) for _ in range(n_prompts)]
    res = teacher_forced_run(shape, 40 + n_prompts, prompts, group=1, n_steps=2, T=1.0)
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, k
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, k


_FORCED_PLANS = [
    ("gemv", gemm_plan_code(RL_GEMM_GEMV)),
    ("direct_s4", gemm_plan_code(RL_GEMM_DIRECT, 4)),
    ("gemv_wide", gemm_plan_code(RL_GEMM_GEMV_WIDE)),
    ("gemv_wide_s3", gemm_plan_code(RL_GEMM_GEMV_WIDE, 3)),
    ("gemv_wide_s8", gemm_plan_code(RL_GEMM_GEMV_WIDE, 8)),
    ("t256", gemm_plan_code(RL_GEMM_T256)),
    ("t256_s4", gemm_plan_code(RL_GEMM_T256, 4)),
    ("t256_s3", gemm_plan_code(RL_GEMM_T256, 3)),
    ("t256_s8", gemm_plan_code(RL_GEMM_T256, 8)),          # split-K 8 and 16: one split per XCD
    ("t128_s16", gemm_plan_code(RL_GEMM_T128, 16)),
    ("t128x256_s8", gemm_plan_code(RL_GEMM_T128X256, 8)),
    ("t128x256_s6", gemm_plan_code(RL_GEMM_T128X256, 6)),
    ("t128x256_s2", gemm_plan_code(RL_GEMM_T128X256, 2)),
    ("t128", gemm_plan_code(RL_GEMM_T128)),
    ("t128deep_s8", gemm_plan_code(RL_GEMM_T128_DEEP, 8)),
    ("t256+t128", gemm_plan_code(RL_GEMM_T256, 0, RL_GEMM_T128)),
    ("t256+t128x256", gemm_plan_code(RL_GEMM_T256, 0, RL_GEMM_T128X256)),
    ("t128x256+t128deep", gemm_plan_code(RL_GEMM_T128X256, 0, RL_GEMM_T128_DEEP)),
]


@pytest.mark.parametrize("name,code", _FORCED_PLANS, ids=[n for n, _ in _FORCED_PLANS])
def test_every_gemm_kernel_matches_oracle(name, code):
    """Each bf16 GEMM tile kernel, split-K count and two-segment launch, forced
    for every projection of a model whose dimensions are multiples of 64
    (vocab ragged): prefill of 144 rows (tile kernels; the GEMV and direct-load
    overrides fall back to the planner there) and decode at 24 rows."""
    shape = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e6, "bf16")
    rng = np.random.default_rng(77)
    prompts = [rng.integers(0, shape.vocab, size=6).astype(np.int32) for _ in range(24)]
    res = teacher_forced_run(shape, 91, prompts, group=1, n_steps=2, T=1.0, gemm_plan=code)
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, (name, k)
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, (name, k)


@pytest.mark.parametrize("rows,splits", [(1, 0), (5, 4), (16, 0), (40, 2), (64, 0), (64, 8)])
def test_wide_gemv_every_row_tile_count_matches_oracle(rows, splits):
    """The wide GEMV (64 weight rows per workgroup) at one, two and four
    16-row activation tiles, ragged and full, with and without split-K (at
    split 8 the 64- and 128-wide K slices leave some of a workgroup's four
    waves without k blocks), forced for every projection in decode and in
    prefills of at most 64 rows; the 1032-entry vocabulary leaves a partial
    last weight group."""
    shape = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e6, "bf16")
    rng = np.random.default_rng(300 + rows)
    prompts = [rng.integers(0, shape.vocab, size=3).astype(np.int32) for _ in range(rows)]
    res = teacher_forced_run(shape, 301 + rows, prompts, group=1, n_steps=2, T=1.0,
                             gemm_plan=gemm_plan_code(RL_GEMM_GEMV_WIDE, splits))
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, k
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, k


def test_measured_gemm_plans_match_oracle():
    """Plans chosen by measurement (rl_decode_tune_gemms) at 1, 8 and 24 rows:
    decode at 24 rows uses the plans measured there and matches the oracle;
    the plan query reports them with their time, and the cost model (time
    -1) beyond the largest measured size."""
    shape = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e6, "bf16")
    rng = np.random.default_rng(78)
    prompts = [rng.integers(0, shape.vocab, size=6).astype(np.int32) for _ in range(24)]
    res = teacher_forced_run(shape, 92, prompts, group=1, n_steps=2, T=1.0, tune_sizes=[1, 8, 24])
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, k
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, k
    w_dev, _, _ = build_models(shape, 93)
    eng = Engine(shape, w_dev, max_seqs=24, max_ctx=16, max_prefill_tokens=144)
    eng.tune_gemms([1, 8, 24])
    for kc in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down", "gemm_lm_head"):
        for rows in (1, 5, 8, 20, 24):
            code, us = eng.gemm_plan(kc, rows)
            assert code != 0 and us > 0, (kc, rows)
        code, us = eng.gemm_plan(kc, 100)
        assert code != 0 and us == -1.0, kc
    assert all(eng.slot_length(i) == 0 for i in range(24))
    eng.tune_gemms([])
    assert eng.gemm_plan("gemm_o", 8)[1] == -1.0
    for bad in ([0], [8, 8], [25], [4, 2]):
        with pytest.raises(RLError):
            eng.tune_gemms(bad)
    eng.set_lengths([3], [5])                # a live sequence: refused, table untouched
    with pytest.raises(RLError):
        eng.tune_gemms([8])
    assert eng.slot_length(3) == 5 and eng.gemm_plan("gemm_o", 8)[1] == -1.0
    eng.close()


@pytest.mark.parametrize("n_prompts", [64, 20])
def test_wide_hidden_residual_norm_paths(n_prompts):
    """hidden 4608 > 4096 (more than one float4 per thread of a 1024-wide
    workgroup): the split-K o / down slices are summed with the residual and
    normed in one grouped pass per row from 64 rows, by the wide reduction and
    a separate norm below (split-K 4 forced for every projection)."""
    shape = ModelShape(1, 4608, 36, 6, 128, 640, 512, 1e-6, 1e6, "bf16")
    rng = np.random.default_rng(n_prompts)
    prompts = [rng.integers(0, shape.vocab, size=2).astype(np.int32) for _ in range(n_prompts)]
    res = teacher_forced_run(shape, 90 + n_prompts, prompts, group=1, n_steps=1, T=1.0,
                             gemm_plan=gemm_plan_code(RL_GEMM_T256, 4))
    for k, (zg, zo, lg, lo, tg, to) in enumerate(res):
        assert row_rel_err(zg, zo) < LOGIT_REL_TOL, k
        assert np.max(np.abs(lg - lo)) < LOGP_ABS_TOL, k
