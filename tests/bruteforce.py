"""Brute-force full-sequence causal forward in NumPy (test helper).

An independent second formulation of the decoder used to pin the oracle:
it processes the whole sequence at once with a causal mask matrix instead of
a KV cache, and shares no code with the oracle.  Used only on tiny shapes.

Storage modes (the precision model of the decoder, written out here from its
definition rather than taken from the oracle):
  "fp64"  no rounding anywhere;
  "fp32"  every stored activation rounded to fp32;
  "bf16"  every stored activation rounded to bf16 (round to nearest, ties to
          even), the residual stream and the logits to fp32.
The stored activations are: the normed rows that enter a projection (both
RMSNorms of every layer and the final one), q and k after RoPE, v, the
attention output and the SwiGLU product.  Accumulation is fp64 throughout.
"""
import numpy as np

from paper_2509_15965_amd.inputs import host_values_f64


def round_bf16(x):
    """Nearest bf16 value of float64 x, ties to even (8 significant bits).

    Written with frexp/rint: x = m * 2**e with 0.5 <= |m| < 1, so m * 2**8 has
    its 8 significant bits left of the binary point and rint (half to even)
    rounds the rest away.  Below the smallest normal (2**-126) bf16 values are
    multiples of 2**-133."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    r = np.ldexp(np.rint(m * 256.0), e - 8)
    small = np.abs(x) < 2.0 ** -126
    r = np.where(small, np.rint(x * 2.0 ** 133) * 2.0 ** -133, r)
    big = np.abs(r) > 3.3895313892515355e38
    return np.where(big, np.copysign(np.inf, x), r)


def round_fp32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def _storage(mode):
    if mode == "fp64":
        return (lambda a: a), (lambda a: a)
    if mode == "fp32":
        return round_fp32, round_fp32
    if mode == "bf16":
        return round_bf16, round_fp32
    raise ValueError(mode)


def _rms(X, g, eps):
    return X / np.sqrt(np.mean(X * X, axis=-1, keepdims=True) + eps) * g


def _rope_tables(n, D, theta):
    half = D // 2
    i = np.arange(half, dtype=np.float64)
    w = np.array([theta ** (-2.0 * k / D) for k in i])
    ang = np.arange(n, dtype=np.float64)[:, None] * w[None, :]
    # angles in fp64, cos/sin rounded to fp32 (part of the definition)
    return np.cos(ang).astype(np.float32).astype(np.float64), np.sin(ang).astype(np.float32).astype(np.float64)


def _rotate(X, c, s):
    """X [n, heads, D]; rotate-half pairs (i, i + D/2)."""
    half = X.shape[-1] // 2
    a, b = X[..., :half], X[..., half:]
    c = c[:, None, :]
    s = s[:, None, :]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def _moe(cfg, W, l, Hn, st, res):
    """Mixture-of-experts MLP output [n, H]: router logits stored like the
    residual, the k largest per row (a stable sort, so equal logits keep the
    lower expert first), softmax over those k, then the weighted sum of the
    selected SwiGLU experts."""
    k, Fe = cfg["top_k"], cfg["expert_ffn"]
    R = res(Hn @ W["w_router"][l].T)                              # [n, E]
    idx = np.argsort(-R, axis=1, kind="stable")[:, :k]
    sel = np.take_along_axis(R, idx, axis=1)
    wts = np.exp(sel - sel[:, :1])
    wts = wts / wts.sum(axis=1, keepdims=True)
    out = np.zeros((Hn.shape[0], Hn.shape[1]))
    for e in np.unique(idx):
        rows, slot = np.nonzero(idx == e)
        GU = Hn[rows] @ W["w_exp_gate_up"][l, e].T
        a, b = GU[:, :Fe], GU[:, Fe:]
        M = st(a / (1.0 + np.exp(-a)) * b)
        out[rows] += wts[rows, slot][:, None] * (M @ W["w_exp_down"][l, e].T)
    return out


def forward_all(cfg, weights, tokens, mode="fp64"):
    """Logits [n, V] at every position of `tokens` (list of ids >= 0)."""
    st, res = _storage(mode)
    W = {k: host_values_f64(v) for k, v in weights.items()}
    L, H, Hq, Hkv, D, F = (cfg["n_layers"], cfg["hidden"], cfg["n_q_heads"], cfg["n_kv_heads"],
                           cfg["head_dim"], cfg["ffn"])
    eps, theta = cfg["rms_eps"], cfg["rope_theta"]
    n = len(tokens)
    G = Hq // Hkv
    X = res(W["embed"][np.asarray(tokens)])
    c, s = _rope_tables(n, D, theta)
    mask = np.triu(np.full((n, n), -np.inf), k=1)       # key t > query p is hidden
    for l in range(L):
        Hn = st(_rms(X, W["attn_norm"][l], eps))
        QKV = Hn @ W["w_qkv"][l].T
        Q = QKV[:, :Hq * D].reshape(n, Hq, D)
        K = QKV[:, Hq * D:(Hq + Hkv) * D].reshape(n, Hkv, D)
        Vv = st(QKV[:, (Hq + Hkv) * D:].reshape(n, Hkv, D))
        Q = st(_rotate(Q, c, s))
        K = st(_rotate(K, c, s))
        K = np.repeat(K, G, axis=1)                      # contiguous q-head groups
        Vv = np.repeat(Vv, G, axis=1)
        S = np.einsum("phd,thd->hpt", Q, K) / np.sqrt(D) + mask[None]
        S = S - S.max(axis=-1, keepdims=True)
        P = np.exp(S)
        P = P / P.sum(axis=-1, keepdims=True)
        O = st(np.einsum("hpt,thd->phd", P, Vv).reshape(n, Hq * D))
        X = res(X + O @ W["w_o"][l].T)
        Hn = st(_rms(X, W["mlp_norm"][l], eps))
        if cfg.get("n_experts", 0) > 0:
            X = res(X + _moe(cfg, W, l, Hn, st, res))
            continue
        GU = Hn @ W["w_gate_up"][l].T
        a, b = GU[:, :F], GU[:, F:]
        M = st(a / (1.0 + np.exp(-a)) * b)
        X = res(X + M @ W["w_down"][l].T)
    Hf = st(_rms(X, W["final_norm"], eps))
    return res(Hf @ W["lm_head"].T)
