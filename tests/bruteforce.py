"""Brute-force full-sequence causal forward in NumPy fp64 (test helper).

An independent second formulation of the decoder used to pin the oracle:
it processes the whole sequence at once with a causal mask matrix instead of
a KV cache, applies no storage rounding, and shares no code with the oracle.
Used only on tiny shapes.
"""
import numpy as np

from paper_2509_15965_amd.inputs import host_values_f64


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


def forward_all(cfg, weights, tokens):
    """Logits [n, V] at every position of `tokens` (list of ids >= 0)."""
    W = {k: host_values_f64(v) for k, v in weights.items()}
    L, H, Hq, Hkv, D, F = (cfg["n_layers"], cfg["hidden"], cfg["n_q_heads"], cfg["n_kv_heads"],
                           cfg["head_dim"], cfg["ffn"])
    eps, theta = cfg["rms_eps"], cfg["rope_theta"]
    n = len(tokens)
    G = Hq // Hkv
    X = W["embed"][np.asarray(tokens)]
    c, s = _rope_tables(n, D, theta)
    mask = np.triu(np.full((n, n), -np.inf), k=1)       # key t > query p is hidden
    for l in range(L):
        Hn = _rms(X, W["attn_norm"][l], eps)
        QKV = Hn @ W["w_qkv"][l].T
        Q = QKV[:, :Hq * D].reshape(n, Hq, D)
        K = QKV[:, Hq * D:(Hq + Hkv) * D].reshape(n, Hkv, D)
        Vv = QKV[:, (Hq + Hkv) * D:].reshape(n, Hkv, D)
        Q = _rotate(Q, c, s)
        K = _rotate(K, c, s)
        K = np.repeat(K, G, axis=1)                      # contiguous q-head groups
        Vv = np.repeat(Vv, G, axis=1)
        S = np.einsum("phd,thd->hpt", Q, K) / np.sqrt(D) + mask[None]
        S = S - S.max(axis=-1, keepdims=True)
        P = np.exp(S)
        P = P / P.sum(axis=-1, keepdims=True)
        O = np.einsum("hpt,thd->phd", P, Vv).reshape(n, Hq * D)
        X = X + O @ W["w_o"][l].T
        Hn = _rms(X, W["mlp_norm"][l], eps)
        GU = Hn @ W["w_gate_up"][l].T
        a, b = GU[:, :F], GU[:, F:]
        M = a / (1.0 + np.exp(-a)) * b
        X = X + M @ W["w_down"][l].T
    Hf = _rms(X, W["final_norm"], eps)
    return Hf @ W["lm_head"].T
