"""Paged K/V pool (kv_page_size > 0) through the C ABI.  The paged pool changes
only where a position's K/V lives, so every output must equal, bit for bit,
the same calls on a contiguous pool; one case is also checked against the
oracle.  Pages are handed out in a scrambled order (other slots take and
return pages first) and sequences cross page boundaries while decoding.
Needs an MI355X."""
import numpy as np
import pytest
import torch

from harness import LOGIT_REL_TOL, LOGP_ABS_TOL, build_models, row_rel_err
from paper_2509_15965_amd.configs import WORKLOADS, ModelShape
from paper_2509_15965_amd.rl_decode import RL_ERR_CAPACITY, Engine, RLError

pytestmark = pytest.mark.gpu
DEV = "cuda"
GQA = ModelShape(2, 512, 8, 2, 128, 1024, 1032, 1e-6, 1e4, "bf16")
G7 = ModelShape(2, 512, 14, 2, 128, 1024, 1032, 1e-6, 1e4, "bf16")


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _i32(a):
    return torch.as_tensor(np.asarray(a, dtype=np.int32), device=DEV)


def _scramble(eng, page, max_ctx):
    """Slots 0-3 take pages and slots 0 and 2 give theirs back, so the pages
    that follow come from the middle of the pool, out of order."""
    eng.set_lengths([0, 1, 2, 3], [min(max_ctx, n) for n in (2 * page + 5, page + 1, 2 * page, 5)])
    eng.release([0, 2])


def _run(shape, w_dev, prompts, group, n_steps, T, page=0, pages=0, slot0=4, max_ctx=None, seed=11, tune=None):
    """Prefill + n_steps teacher-forced decode steps on slots slot0.. (after
    measuring GEMM plans at the `tune` batch sizes, if given); returns every
    logits row, log-prob and token, in call order."""
    n_seq = len(prompts) * group
    plens = [len(p) for p in prompts]
    max_ctx = max_ctx or max(plens) + n_steps + 2
    eng = Engine(shape, w_dev, max_seqs=slot0 + n_seq, max_ctx=max_ctx, max_prefill_tokens=sum(plens),
                 kv_page_size=page, kv_pages=pages)
    if tune:
        total = eng.kv_free_pages()
        eng.tune_gemms(tune)                     # its measuring steps take pages and give them all back
        assert eng.kv_free_pages() == total
    if page:
        _scramble(eng, page, max_ctx)
    slots = list(range(slot0, slot0 + n_seq))
    uids = [1000 + i for i in range(n_seq)]
    offs = np.concatenate([[0], np.cumsum(plens)]).astype(np.int32)
    rng = np.random.default_rng(seed)
    forced = [rng.integers(0, shape.vocab, size=n_seq).astype(np.int32) for _ in range(n_steps + 1)]
    ot = torch.empty(n_seq, dtype=torch.int32, device=DEV)
    ol = torch.empty(n_seq, dtype=torch.float32, device=DEV)
    zp = torch.empty((len(prompts), shape.vocab), dtype=torch.float32, device=DEV)
    eng.prefill(slots, uids, offs, _i32(np.concatenate(prompts)), ot, ol, group=group, forced=_i32(forced[0]),
                seed=5, temperature=T, out_logits=zp)
    out = [(zp.cpu().numpy(), ol.cpu().numpy(), ot.cpu().numpy())]
    z = torch.empty((n_seq, shape.vocab), dtype=torch.float32, device=DEV)
    for s in range(1, n_steps + 1):
        eng.step(slots, uids, _i32(forced[s - 1]), ot, ol, forced=_i32(forced[s]), seed=5, temperature=T,
                 out_logits=z)
        out.append((z.cpu().numpy(), ol.cpu().numpy(), ot.cpu().numpy()))
    for i, sl in enumerate(slots):
        assert eng.slot_length(sl) == plens[i // group] + n_steps
    eng.close()
    return out


def _assert_same(a, b):
    assert len(a) == len(b)
    for k, (x, y) in enumerate(zip(a, b)):
        for u, v in zip(x, y):
            assert np.array_equal(u, v), k


@pytest.mark.parametrize("page,group", [(32, 1), (32, 4), (64, 4), (96, 4), (128, 1)])
def test_paged_decode_equals_contiguous(page, group):
    """Prompts of 37-90 tokens, 40 decode steps (every sequence crosses at
    least one page boundary while decoding), shared prompts with group 4."""
    w_dev, _, _ = build_models(GQA, 61)
    rng = np.random.default_rng(62)
    prompts = [rng.integers(0, GQA.vocab, size=n).astype(np.int32) for n in (37, 64, 90)]
    ref = _run(GQA, w_dev, prompts, group, 40, 1.0)
    got = _run(GQA, w_dev, prompts, group, 40, 1.0, page=page)
    _assert_same(got, ref)


def test_paged_lds_shared_chunks_group16_equals_contiguous():
    """The 7B rollout's attention path (7 q-heads per kv-head, groups of 16:
    LDS-staged workgroups over shared prompt chunks) on a paged pool."""
    w_dev, _, _ = build_models(G7, 63)
    rng = np.random.default_rng(64)
    prompts = [rng.integers(0, G7.vocab, size=650).astype(np.int32)]
    ref = _run(G7, w_dev, prompts, 16, 4, 1.0)
    got = _run(G7, w_dev, prompts, 16, 4, 1.0, page=256)
    _assert_same(got, ref)


def test_paged_fp32_equals_contiguous():
    shape = WORKLOADS["tiny"].model
    w_dev, _, _ = build_models(shape, 65)
    rng = np.random.default_rng(66)
    prompts = [rng.integers(0, shape.vocab, size=n).astype(np.int32) for n in (20, 45)]
    ref = _run(shape, w_dev, prompts, 2, 30, 1.0)
    got = _run(shape, w_dev, prompts, 2, 30, 1.0, page=32)
    _assert_same(got, ref)


@pytest.mark.parametrize("tune", [None, [1, 4, 8]], ids=["cost-model", "measured-plans"])
def test_paged_decode_matches_oracle(tune):
    """A paged pool against the oracle at the stated bars (group 2, pages of
    32), with the cost model's GEMM plans or plans measured on the paged
    engine first."""
    from harness import OracleRollout
    import oracle
    w_dev, _, om = build_models(GQA, 67)
    rng = np.random.default_rng(68)
    prompts = [rng.integers(0, GQA.vocab, size=n).astype(np.int32) for n in (30, 41)]
    group, n_steps = 2, 6
    got = _run(GQA, w_dev, prompts, group, n_steps, 1.0, page=32, seed=69, tune=tune)
    max_ctx = max(len(p) for p in prompts) + n_steps + 2
    orc = OracleRollout(om, max_ctx)
    zo = [orc.prefill(p * group, prompts[p]) for p in range(len(prompts))]
    for p in range(len(prompts)):
        for k in range(1, group):
            orc.seqs[p * group + k] = orc.seqs[p * group].clone()
    assert row_rel_err(got[0][0], np.stack(zo)) < LOGIT_REL_TOL
    frng = np.random.default_rng(69)
    n_seq = len(prompts) * group
    forced = [frng.integers(0, GQA.vocab, size=n_seq).astype(np.int32) for _ in range(n_steps + 1)]
    for s in range(1, n_steps + 1):
        z = np.stack([orc.step(i, forced[s - 1][i]) for i in range(n_seq)])
        assert row_rel_err(got[s][0], z) < LOGIT_REL_TOL, s
        lo = np.array([oracle.sample(z[i].astype(np.float32), 1.0, 5, 1000 + i, orc.length(i),
                                     forced=int(forced[s][i]))[1] for i in range(n_seq)])
        assert np.max(np.abs(got[s][1] - lo)) < LOGP_ABS_TOL, s


def test_paged_score_equals_contiguous():
    w_dev, _, _ = build_models(GQA, 70)
    rng = np.random.default_rng(71)
    prompts = [rng.integers(0, GQA.vocab, size=n).astype(np.int32) for n in (33, 70)]
    group = 3
    resp = rng.integers(20, 60, size=len(prompts) * group)
    out = []
    for page in (0, 32):
        eng = Engine(GQA, w_dev, max_seqs=4 + len(resp), max_ctx=140, max_prefill_tokens=int(sum(map(len, prompts)) + resp.sum()),
                     kv_page_size=page)
        if page:
            _scramble(eng, page, 140)
        slots = list(range(4, 4 + len(resp)))
        poffs = np.concatenate([[0], np.cumsum([len(p) for p in prompts])]).astype(np.int32)
        roffs = np.concatenate([[0], np.cumsum(resp)]).astype(np.int32)
        rtok = _i32(np.random.default_rng(72).integers(0, GQA.vocab, size=int(resp.sum())))
        lp = torch.empty(int(resp.sum()), dtype=torch.float32, device=DEV)
        eng.score(slots, poffs, _i32(np.concatenate(prompts)), roffs, rtok, lp, group=group, temperature=1.0)
        out.append(lp.cpu().numpy())
        assert all(eng.slot_length(s) == 0 for s in slots)
        eng.close()
    assert np.array_equal(out[0], out[1])


def test_paged_offload_onload_continues_bit_identically():
    """Offload the K/V of sequences on a paged pool, release them, onload into
    other slots (new pages), and continue: equal to the run that never left."""
    w_dev, _, _ = build_models(GQA, 73)
    rng = np.random.default_rng(74)
    prompts = [rng.integers(0, GQA.vocab, size=n).astype(np.int32) for n in (50, 77)]
    n_seq, steps = 2, 12
    forced = [rng.integers(0, GQA.vocab, size=n_seq).astype(np.int32) for _ in range(2 * steps + 1)]
    res = []
    for switch in (False, True):
        eng = Engine(GQA, w_dev, max_seqs=8, max_ctx=128, max_prefill_tokens=200, kv_page_size=32)
        _scramble(eng, 32, 128)
        slots, uids = [4, 5], [1, 2]
        offs = np.array([0, 50, 127], dtype=np.int32)
        ot = torch.empty(n_seq, dtype=torch.int32, device=DEV)
        ol = torch.empty(n_seq, dtype=torch.float32, device=DEV)
        z = torch.empty((n_seq, GQA.vocab), dtype=torch.float32, device=DEV)
        eng.prefill(slots, uids, offs, _i32(np.concatenate(prompts)), ot, ol, forced=_i32(forced[0]))
        for s in range(1, steps + 1):
            eng.step(slots, uids, _i32(forced[s - 1]), ot, ol, forced=_i32(forced[s]))
        if switch:
            lens = [eng.slot_length(s) for s in slots]
            host = torch.empty(eng.kv_offload_bytes(slots), dtype=torch.uint8, pin_memory=True)
            eng.kv_offload(slots, host)
            torch.cuda.synchronize()
            eng.release(slots)
            eng.set_lengths([1, 3], [70, 9])       # other sequences take pages meanwhile
            slots = [6, 7]
            eng.kv_onload(slots, lens, host)
        outs = []
        for s in range(steps + 1, 2 * steps + 1):
            eng.step(slots, uids, _i32(forced[s - 1]), ot, ol, forced=_i32(forced[s]), out_logits=z)
            outs.append(z.cpu().numpy())
        res.append(outs)
        eng.close()
    for a, b in zip(*res):
        assert np.array_equal(a, b)


def test_paged_pool_exhaustion_is_refused_without_side_effects():
    w_dev, _, _ = build_models(GQA, 75)
    # 6 pages of 32 positions for 4 slots of up to 100 positions
    eng = Engine(GQA, w_dev, max_seqs=4, max_ctx=100, max_prefill_tokens=200, kv_page_size=32, kv_pages=6)
    rng = np.random.default_rng(76)
    p = rng.integers(0, GQA.vocab, size=90).astype(np.int32)
    ot = torch.zeros(2, dtype=torch.int32, device=DEV)
    ol = torch.empty(2, dtype=torch.float32, device=DEV)
    eng.prefill([0], [1], [0, 90], _i32(p), ot, ol)            # 3 pages
    with pytest.raises(RLError) as e:                            # 3 + 3 pages wanted, 3 left
        eng.prefill([1, 2], [2, 3], [0, 90, 180], _i32(np.concatenate([p, p])), ot, ol)
    assert e.value.status == RL_ERR_CAPACITY
    assert [eng.slot_length(s) for s in range(4)] == [90, 0, 0, 0]
    eng.prefill([1], [2], [0, 90], _i32(p), ot, ol)            # the other 3 pages
    with pytest.raises(RLError) as e:                            # position 96 needs a fourth page
        eng.set_lengths([0], [97])
    assert e.value.status == RL_ERR_CAPACITY
    for _ in range(6):                                           # positions 90..95 stay in page 3
        eng.step([0, 1], [1, 2], ot, ot, ol)
    with pytest.raises(RLError) as e:
        eng.step([0, 1], [1, 2], ot, ot, ol)
    assert e.value.status == RL_ERR_CAPACITY
    assert eng.slot_length(0) == 96 and eng.slot_length(1) == 96
    eng.release([1])
    eng.step([0], [1], ot, ot, ol)                               # a page is free again
    assert eng.slot_length(0) == 97
    torch.cuda.synchronize()
    eng.close()


def test_group_prompt_pages_are_shared_and_counted():
    """A group's full prompt pages are held once for all its slots; each slot's
    partial last prompt page is its own.  Releasing slots gives back exactly the
    pages no other slot holds."""
    w_dev, _, _ = build_models(GQA, 77)
    rng = np.random.default_rng(78)
    prompts = [rng.integers(0, GQA.vocab, size=n).astype(np.int32) for n in (70, 100)]
    eng = Engine(GQA, w_dev, max_seqs=8, max_ctx=128, max_prefill_tokens=170, kv_page_size=32, kv_pages=40)
    assert eng.kv_free_pages() == 40
    ot = torch.zeros(8, dtype=torch.int32, device=DEV)
    ol = torch.empty(8, dtype=torch.float32, device=DEV)
    eng.prefill(list(range(8)), list(range(8)), [0, 70, 170], _i32(np.concatenate(prompts)), ot, ol, group=4)
    # prompt 0: 2 shared + 4 own (positions 64..69); prompt 1: 3 shared + 4 own (96..99)
    assert eng.kv_free_pages() == 40 - 6 - 7
    eng.release([0, 1, 2])
    assert eng.kv_free_pages() == 40 - 13 + 3
    eng.release([3])
    assert eng.kv_free_pages() == 40 - 7
    eng.release([4, 5, 6, 7])
    assert eng.kv_free_pages() == 40
    assert Engine(GQA, w_dev, max_seqs=2, max_ctx=64, max_prefill_tokens=8).kv_free_pages() == -1
    eng.close()


def _truncated_group_run(page, cut_slot, cut_len, steps=6):
    w_dev, _, _ = build_models(GQA, 79)
    rng = np.random.default_rng(80)
    prompt = rng.integers(0, GQA.vocab, size=100).astype(np.int32)
    eng = Engine(GQA, w_dev, max_seqs=4, max_ctx=128, max_prefill_tokens=100, kv_page_size=page)
    slots = [0, 1, 2, 3]
    ot = torch.zeros(4, dtype=torch.int32, device=DEV)
    ol = torch.empty(4, dtype=torch.float32, device=DEV)
    z = torch.empty((4, GQA.vocab), dtype=torch.float32, device=DEV)
    eng.prefill(slots, slots, [0, 100], _i32(prompt), ot, ol, group=4)
    free0 = eng.kv_free_pages()
    eng.set_lengths([cut_slot], [cut_len])
    free1 = eng.kv_free_pages()
    frng = np.random.default_rng(81)
    outs = []
    for _ in range(steps):
        tin = _i32(frng.integers(0, GQA.vocab, size=4))
        eng.step(slots, slots, tin, ot, ol, out_logits=z)
        outs.append(z.cpu().numpy())
    eng.close()
    return outs, free0, free1


def test_cutting_into_a_shared_page_copies_it():
    """A slot cut back into its group's shared prompt page writes its next rows
    into a copy of that page: every slot of the group decodes as on the
    contiguous pool (the others' prompt rows are untouched)."""
    ref, _, _ = _truncated_group_run(0, 1, 50)
    got, free0, free1 = _truncated_group_run(32, 1, 50)
    _assert_same(got, ref)
    # slot 1 let go of shared page 2 (still held by three) and of its own page 3,
    # and took one page for the copy of page 1
    assert free1 == free0
