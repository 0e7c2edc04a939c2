"""The oracle's mixture-of-experts MLP (the Qwen3-30B-A3B policy of
Sec. 5.1.1) pinned to things other than itself: hand-worked routing cases,
a sort-based routing, the dense MLP it reduces to, and the brute-force
full-sequence forward written independently in NumPy.  No GPU is needed."""
import numpy as np
import pytest

import oracle
from bruteforce import forward_all
from paper_2509_15965_amd.configs import ModelShape
from paper_2509_15965_amd.inputs import make_weights, weights_to_host

MOE = ModelShape(2, 64, 4, 2, 16, 0, 128, 1e-6, 1e4, "fp32", n_experts=8, top_k=2, expert_ffn=32)
DENSE = ModelShape(2, 64, 4, 2, 16, 32, 128, 1e-6, 1e4, "fp32")


def test_route_hand_cases():
    sel, w = oracle.route([1.0, 3.0, 3.0, 0.0], 2)          # equal logits: the lower expert first
    assert list(sel) == [1, 2] and np.allclose(w, [0.5, 0.5], rtol=0, atol=1e-15)
    sel, w = oracle.route([0.0, np.log(3.0), -5.0], 2)       # weights are the softmax of the chosen two
    assert list(sel) == [1, 0] and np.allclose(w, [0.75, 0.25], rtol=0, atol=1e-15)
    sel, w = oracle.route([2.0, -1.0, 7.0], 1)
    assert list(sel) == [2] and w[0] == 1.0


def test_route_matches_stable_sort():
    rng = np.random.default_rng(3)
    for trial in range(200):
        E = int(rng.integers(2, 40))
        k = int(rng.integers(1, E + 1))
        r = rng.integers(-3, 4, size=E).astype(np.float64) if trial % 2 else rng.normal(size=E)
        sel, w = oracle.route(r, k)
        ref = np.argsort(-r, kind="stable")[:k]
        assert np.array_equal(sel, ref)
        e = np.exp(r[ref] - r[ref].max())
        assert np.allclose(w, e / e.sum(), rtol=1e-14, atol=0)


def _dense_as_single_expert(dtype):
    s = ModelShape(**{**DENSE.as_dict(), "dtype": dtype})
    w = weights_to_host(make_weights(s, 41))
    m = ModelShape(**{**s.as_dict(), "n_experts": 1, "top_k": 1, "expert_ffn": s.ffn})
    wm = {k: v for k, v in w.items() if k not in ("w_gate_up", "w_down")}
    L, H = s.n_layers, s.hidden
    wm["w_router"] = np.zeros((L, 1, H), dtype=w["w_o"].dtype)
    wm["w_exp_gate_up"] = w["w_gate_up"][:, None]
    wm["w_exp_down"] = w["w_down"][:, None]
    return s, w, m, wm


@pytest.mark.parametrize("mode,dtype", [(oracle.MODE_FP64, "fp32"), (oracle.MODE_BF16, "bf16")])
def test_single_expert_equals_dense_mlp(mode, dtype):
    """One expert chosen with weight 1 is the dense SwiGLU MLP: same logits, bit for bit."""
    s, w, m, wm = _dense_as_single_expert(dtype)
    dense = oracle.OracleModel(s.as_dict(), w, mode).new_seq(16)
    moe = oracle.OracleModel(m.as_dict(), wm, mode).new_seq(16)
    for t in np.random.default_rng(42).integers(0, s.vocab, size=8):
        assert np.array_equal(dense.forward(int(t)), moe.forward(int(t)))


def test_identical_experts_equal_the_dense_mlp():
    """Any routing over experts that all equal the dense MLP gives the dense
    MLP (the selected weights sum to one)."""
    s, w, m, wm = _dense_as_single_expert("fp32")
    E = 5
    m = ModelShape(**{**m.as_dict(), "n_experts": E, "top_k": 3})
    rng = np.random.default_rng(43)
    wm["w_router"] = rng.normal(size=(s.n_layers, E, s.hidden)).astype(np.float32)
    wm["w_exp_gate_up"] = np.repeat(w["w_gate_up"][:, None], E, axis=1)
    wm["w_exp_down"] = np.repeat(w["w_down"][:, None], E, axis=1)
    dense = oracle.OracleModel(s.as_dict(), w, oracle.MODE_FP64).new_seq(16)
    moe = oracle.OracleModel(m.as_dict(), wm, oracle.MODE_FP64).new_seq(16)
    for t in rng.integers(0, s.vocab, size=8):
        a, b = dense.forward(int(t)), moe.forward(int(t))
        assert np.abs(a - b).max() / np.abs(a).max() < 1e-12


@pytest.mark.parametrize("mode,dtype,bmode", [(oracle.MODE_FP64, "fp32", "fp64"), (oracle.MODE_FP32, "fp32", "fp32"),
                                              (oracle.MODE_BF16, "bf16", "bf16")], ids=["fp64", "fp32", "bf16"])
def test_moe_decode_equals_bruteforce(mode, dtype, bmode):
    """KV-cached decode through the oracle's expert MLP against the brute-force
    full-sequence forward (sort-based routing, experts applied per expert over
    all the rows that chose it), with the same storage roundings."""
    s = ModelShape(**{**MOE.as_dict(), "dtype": dtype})
    w = weights_to_host(make_weights(s, 44, init="fanin"))
    m = oracle.OracleModel(s.as_dict(), w, mode)
    toks = [int(t) for t in np.random.default_rng(45).integers(0, s.vocab, size=20)]
    seq = m.new_seq(24)
    inc = np.stack([seq.forward(t) for t in toks])
    ref = forward_all(s.as_dict(), w, toks, mode=bmode)
    assert np.abs(inc - ref).max() / np.abs(ref).max() < 1e-10


def test_routing_changes_the_output():
    """The router matters: swapping two experts' weights changes the logits
    unless neither is ever chosen (guards against an expert index that is
    ignored)."""
    s = MOE
    w = weights_to_host(make_weights(s, 46, init="fanin"))
    toks = [int(t) for t in np.random.default_rng(47).integers(0, s.vocab, size=6)]
    base = forward_all(s.as_dict(), w, toks)
    w2 = dict(w)
    for name in ("w_exp_gate_up", "w_exp_down"):
        a = w[name].copy()
        a[:, [0, 1]] = a[:, [1, 0]]
        w2[name] = a
    seq = oracle.OracleModel(s.as_dict(), w2, oracle.MODE_FP64).new_seq(8)
    swapped = np.stack([seq.forward(t) for t in toks])
    seq = oracle.OracleModel(s.as_dict(), w, oracle.MODE_FP64).new_seq(8)
    same = np.stack([seq.forward(t) for t in toks])
    assert np.abs(same - base).max() / np.abs(base).max() < 1e-10
    assert np.abs(swapped - base).max() / np.abs(base).max() > 1e-6
