"""The CPU oracle against what the paper and the mathematics fix.

Each test pins one part of the oracle to something other than itself:
published known-answer values, hand-worked cases, closed forms,
invariants, a library routine in a special case, or a brute-force
second formulation.  No GPU is needed.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from bruteforce import forward_all
from paper_2509_15965_amd.configs import ModelShape
from paper_2509_15965_amd.inputs import make_weights, weights_to_host

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

SMALL = ModelShape(n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16, ffn=96,
                   vocab=128, rms_eps=1e-6, rope_theta=1e4, dtype="fp32")


def small_cfg(shape=SMALL):
    return shape.as_dict()


def small_model(mode, dtype="fp32", seed=7, shape=SMALL):
    s = ModelShape(**{**shape.as_dict(), "dtype": dtype})
    w = weights_to_host(make_weights(s, seed))
    return oracle.OracleModel(s.as_dict(), w, mode), w, s


# --------------------------------------------------------------------------
# Philox4x32-10 and the noise stream
# --------------------------------------------------------------------------

def test_philox_known_answers():
    n = 0
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(x, 16) for x in line.split()]
            assert oracle.philox4x32_10(v[0:4], v[4:6]) == v[6:10]
            n += 1
    assert n == 3


def test_noise_word_counter_layout():
    # word v % 4 of the block at counter (v/4, pos, uid lo, uid hi), key (seed lo, seed hi)
    seed, uid, pos = 0x1234_5678_9ABC_DEF0, 0x0000_0007_0000_0003, 41
    for v in (0, 1, 2, 3, 4, 7, 1001):
        blk = oracle.philox4x32_10([v // 4, pos, uid & 0xFFFFFFFF, uid >> 32],
                                   [seed & 0xFFFFFFFF, seed >> 32])
        assert oracle.noise_word(seed, uid, pos, v) == blk[v % 4]


def test_noise_words_uniform():
    # chi-square of the top 4 bits over 65536 words: 15 dof, p = 1e-4 bound ~ 45.3
    words = np.array([oracle.noise_word(99, 5, p, v) for p in range(16) for v in range(4096)],
                     dtype=np.uint64)
    counts = np.bincount((words >> 28).astype(np.int64), minlength=16)
    e = len(words) / 16
    chi2 = float(((counts - e) ** 2 / e).sum())
    assert chi2 < 45.3


def test_gumbel_of_word_matches_definition_endpoints():
    # u = (x + 1/2) 2^-32 never reaches 0 or 1; both extremes stay finite
    lo = oracle.gumbel_of_word(0)
    hi = oracle.gumbel_of_word(0xFFFFFFFF)
    u0 = 0.5 * 2.0 ** -32
    assert lo == pytest.approx(-math.log(-math.log(u0)), rel=1e-6)
    assert np.isfinite(lo) and np.isfinite(hi) and lo < -3.0 and hi > 22.0


# --------------------------------------------------------------------------
# Gumbel-max sampling and log-probabilities
# --------------------------------------------------------------------------

def _hand_cases():
    with open(os.path.join(GOLDEN, "gumbel_hand_cases.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            T, z, u, exp, _ = [p.strip() for p in line.split(";")]
            yield (float(T), [float(x) for x in z.split(",")], [float(x) for x in u.split(",")], int(exp))


def test_gumbel_hand_cases():
    cases = list(_hand_cases())
    assert len(cases) == 7
    for T, z, u, exp in cases:
        assert oracle.gumbel_argmax_u(z, u, T) == exp, (T, z, u)


def test_logprob_hand_values():
    # z = [0, 0, ln 2]: LSE = ln 4, so logp(2) = -ln 2 and logp(0) = -ln 4
    z = np.array([0.0, 0.0, math.log(2.0)], dtype=np.float32)
    _, lp2 = oracle.sample(z, 1.0, 1, 2, 3, forced=2)
    _, lp0 = oracle.sample(z, 1.0, 1, 2, 3, forced=0)
    zf = z.astype(np.float64)
    assert lp2 == pytest.approx(zf[2] - math.log(2.0 + math.exp(zf[2])), abs=1e-12)
    assert lp2 == pytest.approx(-math.log(2.0), abs=1e-7)
    assert lp0 == pytest.approx(-math.log(4.0), abs=1e-7)


def test_logprobs_normalise_and_are_nonpositive():
    rng = np.random.default_rng(0)
    for T in (1.0, 0.6):
        z = rng.normal(0, 3, size=257).astype(np.float32)
        lps = np.array([oracle.sample(z, T, 5, 6, 7, forced=v)[1] for v in range(len(z))])
        assert np.all(lps <= 0.0)
        assert abs(np.exp(lps).sum() - 1.0) < 1e-12


def test_shift_invariance():
    rng = np.random.default_rng(1)
    z = (np.round(rng.normal(0, 2, size=300) * 1024) / 1024).astype(np.float32)  # shift is exact
    for uid in range(20):
        t0, l0 = oracle.sample(z, 1.0, 11, uid, 9)
        t1, l1 = oracle.sample(z + np.float32(8.0), 1.0, 11, uid, 9)
        assert t0 == t1
        assert l0 == pytest.approx(l1, abs=1e-12)


def test_temperature_divides_logits():
    rng = np.random.default_rng(2)
    z = (np.round(rng.normal(0, 2, size=200) * 256) / 256).astype(np.float32)
    for uid in range(20):
        assert oracle.sample(z, 0.5, 3, uid, 4) == oracle.sample(2 * z, 1.0, 3, uid, 4)


def test_greedy_at_zero_temperature():
    z = np.array([0.5, 3.0, -1.0, 3.0], dtype=np.float32)
    tok, lp = oracle.sample(z, 0.0, 1, 1, 1)
    assert tok == 1                                   # first of the tied maxima
    zf = z.astype(np.float64)
    assert lp == pytest.approx(zf[1] - math.log(np.exp(zf).sum()), abs=1e-12)


def test_dominant_logit_always_chosen():
    z = np.zeros(64, dtype=np.float32)
    z[17] = 50.0
    assert all(oracle.sample(z, 1.0, 8, uid, 3)[0] == 17 for uid in range(200))


def test_gumbel_max_frequencies_match_softmax():
    # Gumbel-max draws follow softmax(z / T): chi-square over 40000 draws
    p = np.array([0.05, 0.1, 0.15, 0.2, 0.5])
    z = np.log(p).astype(np.float32)
    draws = np.array([oracle.sample(z, 1.0, 2024, uid, 0)[0] for uid in range(40000)])
    counts = np.bincount(draws, minlength=5)
    e = p * len(draws)
    chi2 = float(((counts - e) ** 2 / e).sum())
    assert chi2 < 23.5            # 4 dof, p = 1e-4


def test_uniform_logits_uniform_frequencies():
    z = np.zeros(8, dtype=np.float32)
    draws = np.array([oracle.sample(z, 1.0, 77, uid, 5)[0] for uid in range(40000)])
    counts = np.bincount(draws, minlength=8)
    e = len(draws) / 8
    assert float(((counts - e) ** 2 / e).sum()) < 31.3   # 7 dof, p = 1e-4


def test_sample_margin_hand_cases():
    """Top-two perturbed scores of a draw (what excuses a near-tie token flip
    in fp32 parity): at T = 0 the scores are the logits themselves, so the
    best, runner-up and margin are read off by hand."""
    cases = [
        ([0.5, 3.0, -1.0, 2.0], (1, 3, 1.0)),
        ([0.5, 3.0, -1.0, 3.0], (1, 3, 0.0)),      # exact tie: lowest index first, the other second
        ([4.0, 1.0, 2.0], (0, 2, 2.0)),             # runner-up found after the best
        ([1.0, 2.0, 3.0], (2, 1, 1.0)),             # each new best pushes the old one to second
        ([-2.0, -2.0], (0, 1, 0.0)),
    ]
    for z, exp in cases:
        assert oracle.sample_margin(np.array(z, dtype=np.float32), 0.0, 1, 2, 3) == exp, z


@pytest.mark.parametrize("T", [1.0, 0.6])
def test_sample_margin_matches_sorted_scores(T):
    """With noise: the perturbed scores fl32(fl32(z/T) + g_v) formed here in
    NumPy from the noise words, sorted by (score desc, index asc); the top two
    and their fp64 difference equal sample_margin, and its best is the
    sampler's token."""
    rng = np.random.default_rng(33)
    for trial in range(40):
        V = int(rng.integers(2, 400))
        z = rng.normal(0, 2, size=V).astype(np.float32)
        if trial % 4 == 0:
            z[:] = np.float32(0.25)                   # equal logits: the noise decides alone
        seed, uid, pos = 1000 + trial, 7 * trial, trial % 5
        g = np.array([oracle.gumbel_of_word(oracle.noise_word(seed, uid, pos, v)) for v in range(V)],
                     dtype=np.float32)
        sc = (z / np.float32(T)).astype(np.float32) + g
        order = np.lexsort((np.arange(V), -sc.astype(np.float64)))
        a, b, m = oracle.sample_margin(z, T, seed, uid, pos)
        assert (a, b) == (int(order[0]), int(order[1]))
        assert m == float(sc[order[0]]) - float(sc[order[1]])
        assert a == oracle.sample(z, T, seed, uid, pos)[0]


def test_noise_depends_on_uid_and_position():
    z = np.zeros(512, dtype=np.float32)
    a = [oracle.sample(z, 1.0, 1, uid, 0)[0] for uid in range(8)]
    b = [oracle.sample(z, 1.0, 1, 0, pos)[0] for pos in range(8)]
    assert len(set(a)) > 4 and len(set(b)) > 4


# --------------------------------------------------------------------------
# bf16 rounding
# --------------------------------------------------------------------------

def test_round_bf16_ties_to_even():
    one = 1.0
    assert oracle.round_bf16(one + 2.0 ** -8) == 1.0                 # tie -> even (1.0)
    assert oracle.round_bf16(one + 3 * 2.0 ** -8) == one + 2.0 ** -6  # tie -> even
    assert oracle.round_bf16(one + 2.0 ** -8 + 2.0 ** -30) == one + 2.0 ** -7
    assert oracle.round_bf16(-(one + 2.0 ** -8 + 2.0 ** -30)) == -(one + 2.0 ** -7)


def test_round_bf16_matches_torch_on_fp32_values():
    # for values exact in fp32, double->bf16 equals torch's fp32->bf16 (RNE)
    rng = np.random.default_rng(3)
    x = rng.normal(0, 10, size=5000).astype(np.float32)
    x[:8] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 3.0e38, -7.5e-39, 1e-40, 0.0, -0.0, 65504.0]
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.round_bf16(float(v)) for v in x])
    assert np.array_equal(got, ref)


# --------------------------------------------------------------------------
# building blocks
# --------------------------------------------------------------------------

def test_rmsnorm_constant_vector_closed_form():
    c, eps, H = 0.37, 1e-6, 32
    g = np.linspace(0.5, 1.5, H).astype(np.float32)
    out = oracle.rmsnorm(np.full(H, c), g, eps, oracle.MODE_FP64)
    assert np.allclose(out, c / math.sqrt(c * c + eps) * g.astype(np.float64), rtol=1e-15, atol=0)


def test_rmsnorm_scale_invariance():
    rng = np.random.default_rng(4)
    x = rng.normal(size=96)
    g = np.ones(96, dtype=np.float32)
    a = oracle.rmsnorm(x, g, 0.0, oracle.MODE_FP64)
    b = oracle.rmsnorm(7.25 * x, g, 0.0, oracle.MODE_FP64)
    assert np.allclose(a, b, rtol=1e-14, atol=1e-15)
    assert np.mean(a * a) == pytest.approx(1.0, rel=1e-14)


def test_matvec_matches_numpy_on_bf16_inputs():
    rng = np.random.default_rng(5)
    Wf = torch.from_numpy(rng.normal(0, 0.02, size=(37, 200)).astype(np.float32)).to(torch.bfloat16)
    Wb = Wf.view(torch.int16).numpy().view(np.uint16)
    x = rng.normal(size=200)
    ref = Wf.to(torch.float64).numpy() @ x
    assert np.allclose(oracle.matvec(Wb, x), ref, rtol=1e-13, atol=1e-15)


def test_rope_position_zero_is_identity():
    v = np.random.default_rng(6).normal(size=64)
    assert np.array_equal(oracle.rope(v, 0, 1e4), v)


def test_rope_two_dims_is_rotation_by_position():
    # D = 2: one pair with frequency theta^0 = 1, so the angle is the position
    for p in (1, 5, 1000):
        out = oracle.rope([1.0, 0.0], p, 1e6)
        assert out[0] == float(np.float32(math.cos(p)))
        assert out[1] == float(np.float32(math.sin(p)))
        out = oracle.rope([0.0, 1.0], p, 1e6)
        assert out[0] == -float(np.float32(math.sin(p)))


def test_rope_frequency_of_second_pair():
    # D = 4, pair i = 1 rotates by p * theta^(-1/2)
    theta, p = 1e4, 3
    c, s = oracle.rope_cos_sin(p, 1, 4, theta)
    assert c == float(np.float32(math.cos(p / 100.0)))
    assert s == float(np.float32(math.sin(p / 100.0)))


def test_rope_norm_and_relative_position():
    rng = np.random.default_rng(7)
    q, k = rng.normal(size=128), rng.normal(size=128)
    for p in (0, 17, 4095, 8703):
        assert np.linalg.norm(oracle.rope(q, p, 1e6)) == pytest.approx(np.linalg.norm(q), rel=2e-7)
    # <R_p q, R_p' k> depends only on p - p' (fp32-rounded cos/sin: ~1e-7)
    ref = np.dot(oracle.rope(q, 100, 1e6), oracle.rope(k, 37, 1e6))
    for shift in (1, 500, 8000):
        got = np.dot(oracle.rope(q, 100 + shift, 1e6), oracle.rope(k, 37 + shift, 1e6))
        assert got == pytest.approx(ref, abs=2e-5 * np.linalg.norm(q) * np.linalg.norm(k))


def test_attention_single_key_returns_its_value():
    rng = np.random.default_rng(8)
    q, K, V = rng.normal(size=16), rng.normal(size=(1, 16)), rng.normal(size=(1, 16))
    assert np.array_equal(oracle.attend(q, K, V), V[0])


def test_attention_zero_query_averages_values():
    rng = np.random.default_rng(9)
    K, V = rng.normal(size=(13, 16)), rng.normal(size=(13, 16))
    assert np.allclose(oracle.attend(np.zeros(16), K, V), V.mean(axis=0), rtol=1e-13, atol=1e-14)


def test_attention_peaked_key_selects_its_value():
    rng = np.random.default_rng(10)
    K, V = rng.normal(size=(40, 64)), rng.normal(size=(40, 64))
    q = 50.0 * K[23] / np.linalg.norm(K[23])
    K[23] = q                                          # score 50^2/8 = 312.5 above the rest
    assert np.allclose(oracle.attend(q, K, V), V[23], atol=1e-12)


def test_attention_matches_scipy_softmax():
    from scipy.special import softmax
    rng = np.random.default_rng(11)
    q, K, V = rng.normal(size=32), rng.normal(size=(50, 32)), rng.normal(size=(50, 32))
    ref = softmax(K @ q / math.sqrt(32)) @ V
    assert np.allclose(oracle.attend(q, K, V), ref, rtol=1e-13, atol=1e-14)


# --------------------------------------------------------------------------
# whole decoder
# --------------------------------------------------------------------------

@pytest.mark.parametrize("shape", [
    SMALL,
    ModelShape(1, 48, 3, 3, 16, 80, 96, 1e-5, 1e4, "fp32"),      # MHA (group 1)
    ModelShape(2, 64, 8, 1, 8, 64, 64, 1e-6, 1e6, "fp32"),       # MQA (group 8)
])
def test_incremental_decode_equals_bruteforce_full_sequence(shape):
    """KV-cached one-token-at-a-time decode (fp64 storage) = full causal
    forward with a mask matrix, at every position."""
    m, w, s = small_model(oracle.MODE_FP64, "fp32", seed=12, shape=shape)
    toks = [int(t) for t in np.random.default_rng(13).integers(0, s.vocab, size=24)]
    seq = m.new_seq(32)
    inc = np.stack([seq.forward(t) for t in toks])
    ref = forward_all(s.as_dict(), w, toks)
    err = np.abs(inc - ref).max() / np.abs(ref).max()
    assert err < 1e-10, err


@pytest.mark.parametrize("mode,dtype", [(oracle.MODE_FP32, "fp32"), (oracle.MODE_BF16, "bf16")])
def test_kv_cached_decode_equals_recompute(mode, dtype):
    """Storage modes: the last logits of every prefix are bit-identical
    whether reached incrementally or by re-feeding the prefix."""
    m, _, s = small_model(mode, dtype, seed=14)
    toks = [int(t) for t in np.random.default_rng(15).integers(0, s.vocab, size=10)]
    seq = m.new_seq(16)
    inc = [seq.forward(t) for t in toks]
    for k in (1, 4, 10):
        fresh = m.new_seq(16)
        for t in toks[:k]:
            last = fresh.forward(t)
        assert np.array_equal(last, inc[k - 1])


MHA = ModelShape(1, 48, 3, 3, 16, 80, 96, 1e-5, 1e4, "fp32")
MQA = ModelShape(2, 64, 8, 1, 8, 64, 64, 1e-6, 1e6, "fp32")


def test_bruteforce_round_bf16_matches_torch():
    """The brute force's own bf16 rounding (frexp/rint) against torch's
    fp32 -> bf16 conversion on fp32-exact values, ties and subnormals included."""
    from bruteforce import round_bf16
    rng = np.random.default_rng(30)
    x = rng.normal(0, 10, size=20000).astype(np.float32)
    x[:10] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 3.0e38, -7.5e-39, 1e-40, 0.0, 2.0 ** -130,
              65504.0, 255.5]
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(round_bf16(x.astype(np.float64)), ref)


@pytest.mark.parametrize("shape", [SMALL, MHA, MQA], ids=["gqa", "mha", "mqa"])
@pytest.mark.parametrize("mode,dtype,bmode", [(oracle.MODE_FP32, "fp32", "fp32"), (oracle.MODE_BF16, "bf16", "bf16")],
                         ids=["fp32", "bf16"])
def test_storage_modes_equal_bruteforce_with_same_rounding(shape, mode, dtype, bmode):
    """The oracle's storage modes against the brute-force full-sequence
    forward that rounds at the same declared sites (normed projection inputs,
    q and k after RoPE, v, attention output, SwiGLU product; fp32 residual
    and logits), written independently in NumPy.  Both accumulate in fp64, so
    they agree to fp64 round-off; a storage rounding missing on either side
    moves the logits by about one storage ulp (~1e-3 in bf16, ~1e-7 in fp32)."""
    m, w, s = small_model(mode, dtype, seed=31, shape=shape)
    toks = [int(t) for t in np.random.default_rng(32).integers(0, s.vocab, size=24)]
    seq = m.new_seq(32)
    inc = np.stack([seq.forward(t) for t in toks])
    ref = forward_all(s.as_dict(), w, toks, mode=bmode)
    scale = np.abs(ref).max()
    assert np.abs(inc - ref).max() / scale < 1e-10
    # the rounding is visible at this size: the fp64 forward differs
    ref64 = forward_all(s.as_dict(), w, toks, mode="fp64")
    assert np.abs(ref - ref64).max() / scale > (1e-4 if dtype == "bf16" else 1e-8)


def test_storage_rounding_is_small_against_fp64():
    """bf16 storage moves the logits by a small relative amount vs fp64."""
    s = ModelShape(**{**SMALL.as_dict(), "dtype": "bf16"})
    w = weights_to_host(make_weights(s, 16))
    toks = [int(t) for t in np.random.default_rng(17).integers(0, s.vocab, size=8)]
    a = oracle.OracleModel(s.as_dict(), w, oracle.MODE_FP64).new_seq(8)
    b = oracle.OracleModel(s.as_dict(), w, oracle.MODE_BF16).new_seq(8)
    za = np.stack([a.forward(t) for t in toks])
    zb = np.stack([b.forward(t) for t in toks])
    rel = np.abs(za - zb).max() / np.abs(za).max()
    assert 0 < rel < 3e-2


def test_embedding_override_row_equals_token_row():
    m, w, s = small_model(oracle.MODE_FP32, "fp32", seed=18)
    a, b = m.new_seq(4), m.new_seq(4)
    za = a.forward(9)
    zb = b.forward(-1, embed_row=w["embed"][9])
    assert np.array_equal(za, zb)


def test_resume_from_prefix_reproduces_sampling():
    """Counter-keyed noise: re-prefilling prompt + generated prefix and
    continuing gives the same tokens as the uninterrupted rollout."""
    m, _, s = small_model(oracle.MODE_FP32, "fp32", seed=19)
    prompt = [3, 14, 15, 92, 65]
    seed, uid, T = 4242, 77, 1.0

    def run(prefix, n_new):
        seq = m.new_seq(32)
        for t in prefix[:-1]:
            seq.forward(t)
        z = seq.forward(prefix[-1])
        out = []
        for _ in range(n_new):
            tok, _ = oracle.sample(z.astype(np.float32), T, seed, uid, seq.length)
            out.append(tok)
            z = seq.forward(tok)
        return out

    full = run(prompt, 8)
    tail = run(prompt + full[:3], 5)
    assert tail == full[3:]


def test_kv_injection_then_decode_matches_natural_cache():
    """Writing a cache the oracle itself produced back through set_kv gives
    the same next logits (the step is a function of KV, token, position)."""
    m, _, s = small_model(oracle.MODE_BF16, "bf16", seed=20)
    toks = [5, 6, 7, 8, 9]
    a = m.new_seq(8)
    for t in toks[:-1]:
        a.forward(t)
    b = m.new_seq(8)
    for l in range(s.n_layers):
        for g in range(s.n_kv_heads):
            K = np.stack([a.get_kv(l, p, g)[0] for p in range(4)])
            V = np.stack([a.get_kv(l, p, g)[1] for p in range(4)])
            b.set_kv_block(l, g, K, V)
    b.set_length(4)
    assert np.array_equal(a.forward(toks[-1]), b.forward(toks[-1]))


# --------------------------------------------------------------------------
# Inference stage: log-probabilities of given responses
# --------------------------------------------------------------------------

def test_logprob_closed_forms():
    V = 1000
    assert oracle.logprob(np.zeros(V, np.float32), 1.0, 17) == pytest.approx(-math.log(V), abs=1e-12)
    z = np.array([0.0, 0.0, math.log(2.0)], dtype=np.float32)
    zf = z.astype(np.float64)
    assert oracle.logprob(z, 1.0, 2) == pytest.approx(zf[2] - math.log(2.0 + math.exp(zf[2])), abs=1e-12)
    # two entries: log-sigmoid of the difference / T
    a, b, T = 1.25, -0.5, 0.5
    z2 = np.array([a, b], dtype=np.float32)
    assert oracle.logprob(z2, T, 0) == pytest.approx(-math.log1p(math.exp(-(a - b) / T)), abs=1e-12)
    # T == 0 reports the T = 1 value; ids outside the vocabulary give NaN
    rng = np.random.default_rng(21)
    z3 = rng.normal(0, 2, size=50).astype(np.float32)
    assert oracle.logprob(z3, 0.0, 7) == oracle.logprob(z3, 1.0, 7)
    assert math.isnan(oracle.logprob(z3, 1.0, 50)) and math.isnan(oracle.logprob(z3, 1.0, -1))


def test_logprob_normalises_and_matches_sampler_report():
    rng = np.random.default_rng(22)
    for T in (1.0, 0.6):
        z = rng.normal(0, 3, size=301).astype(np.float32)
        lps = np.array([oracle.logprob(z, T, v) for v in range(len(z))])
        assert np.all(lps <= 0.0)
        assert abs(np.exp(lps).sum() - 1.0) < 1e-12
        # exactly the quantity the sampler reports for a forced token
        for v in (0, 150, 300):
            assert oracle.logprob(z, T, v) == oracle.sample(z, T, 3, 4, 5, forced=v)[1]


@pytest.mark.parametrize("T", [1.0, 0.6])
@pytest.mark.parametrize("shape", [
    SMALL,
    ModelShape(2, 64, 8, 1, 8, 64, 64, 1e-6, 1e6, "fp32"),       # MQA (group 8)
])
def test_score_equals_bruteforce_log_softmax(shape, T):
    """score() = log-softmax of the full causal forward over prompt +
    response, read at each response token (fp64 storage, no cache)."""
    from scipy.special import logsumexp
    m, w, s = small_model(oracle.MODE_FP64, "fp32", seed=23, shape=shape)
    rng = np.random.default_rng(24)
    prompt = [int(t) for t in rng.integers(0, s.vocab, size=9)]
    resp = [int(t) for t in rng.integers(0, s.vocab, size=14)]
    got = oracle.score(m, prompt, resp, T)
    ref = forward_all(s.as_dict(), w, prompt + resp)
    P = len(prompt)
    for j, y in enumerate(resp):
        zt = ref[P - 1 + j] / T
        exp = zt[y] - logsumexp(zt)
        assert got[j] == pytest.approx(exp, abs=2e-5), (j, got[j], exp)


def test_score_embedding_prompt_rows():
    """Prompt ids < 0 read rows of the caller's embedding table: with rows
    equal to token rows the scores are identical."""
    m, w, s = small_model(oracle.MODE_BF16, "bf16", seed=25)
    rng = np.random.default_rng(26)
    prompt = [int(t) for t in rng.integers(0, s.vocab, size=6)]
    resp = [int(t) for t in rng.integers(0, s.vocab, size=5)]
    embeds = w["embed"][np.array(prompt[:3])]
    mixed = [-1, -2, -3] + prompt[3:]
    assert np.array_equal(oracle.score(m, prompt, resp, 1.0), oracle.score(m, mixed, resp, 1.0, embeds=embeds))
