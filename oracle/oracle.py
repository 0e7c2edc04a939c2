"""ctypes wrapper of the C oracle (oracle/rl_oracle.c).

Test infrastructure only: the GPU library never imports this module.
Every function here forwards to the C oracle; the arithmetic lives there.
"""
import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

MODE_FP64, MODE_FP32, MODE_BF16 = 0, 1, 2
W_F32, W_BF16 = 0, 1

_lib = None


class _Model(C.Structure):
    _fields_ = [
        ("L", C.c_int32), ("H", C.c_int32), ("Hq", C.c_int32), ("Hkv", C.c_int32),
        ("D", C.c_int32), ("F", C.c_int32), ("V", C.c_int32),
        ("eps", C.c_double), ("theta", C.c_double),
        ("mode", C.c_int32), ("wdt", C.c_int32),
        ("embed", C.c_void_p), ("attn_norm", C.c_void_p), ("w_qkv", C.c_void_p),
        ("w_o", C.c_void_p), ("mlp_norm", C.c_void_p), ("w_gate_up", C.c_void_p),
        ("w_down", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p),
        ("E", C.c_int32), ("topk", C.c_int32), ("Fe", C.c_int32),
        ("w_router", C.c_void_p), ("w_exp_gate_up", C.c_void_p), ("w_exp_down", C.c_void_p),
    ]


_dp = C.POINTER(C.c_double)
_fp = C.POINTER(C.c_float)


def load():
    """Load liboracle.so, building it with gcc if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _b
        _b.build()
    lib = C.CDLL(LIB_PATH)
    lib.orc_round_bf16.restype = C.c_double
    lib.orc_round_bf16.argtypes = [C.c_double]
    lib.orc_philox4x32_10.argtypes = [C.POINTER(C.c_uint32), C.POINTER(C.c_uint32), C.POINTER(C.c_uint32)]
    lib.orc_noise_word.restype = C.c_uint32
    lib.orc_noise_word.argtypes = [C.c_uint64, C.c_uint64, C.c_int32, C.c_int64]
    lib.orc_gumbel_of_word.restype = C.c_float
    lib.orc_gumbel_of_word.argtypes = [C.c_uint32]
    lib.orc_gumbel_argmax_u.restype = C.c_int32
    lib.orc_gumbel_argmax_u.argtypes = [_fp, _dp, C.c_int32, C.c_float]
    lib.orc_sample.argtypes = [_fp, C.c_int32, C.c_float, C.c_uint64, C.c_uint64, C.c_int32,
                               C.c_int32, C.POINTER(C.c_int32), _dp]
    lib.orc_logprob.restype = C.c_double
    lib.orc_logprob.argtypes = [_fp, C.c_int32, C.c_float, C.c_int32]
    lib.orc_sample_margin.argtypes = [_fp, C.c_int32, C.c_float, C.c_uint64, C.c_uint64, C.c_int32,
                                      C.POINTER(C.c_int32), C.POINTER(C.c_int32), _dp]
    lib.orc_rmsnorm.argtypes = [_dp, C.c_int, C.c_void_p, C.c_size_t, C.c_int32, C.c_double, C.c_int, _dp]
    lib.orc_matvec.argtypes = [C.c_int, C.c_void_p, C.c_size_t, C.c_int32, C.c_int32, _dp, _dp]
    lib.orc_rope_cos_sin.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_double, _dp, _dp]
    lib.orc_rope.argtypes = [_dp, C.c_int32, C.c_int32, C.c_double]
    lib.orc_attend.argtypes = [_dp, _dp, _dp, C.c_int64, C.c_int32, C.c_int32, _dp]
    lib.orc_route.argtypes = [_dp, C.c_int32, C.c_int32, C.POINTER(C.c_int32), _dp]
    lib.orc_seq_create.restype = C.c_void_p
    lib.orc_seq_create.argtypes = [C.POINTER(_Model), C.c_int32]
    lib.orc_seq_destroy.argtypes = [C.c_void_p]
    lib.orc_seq_clone.restype = C.c_void_p
    lib.orc_seq_clone.argtypes = [C.POINTER(_Model), C.c_void_p]
    lib.orc_seq_route_margin.restype = C.c_double
    lib.orc_seq_route_margin.argtypes = [C.c_void_p]
    lib.orc_seq_len.restype = C.c_int32
    lib.orc_seq_len.argtypes = [C.c_void_p]
    lib.orc_seq_set_len.argtypes = [C.c_void_p, C.c_int32]
    lib.orc_seq_set_kv.argtypes = [C.POINTER(_Model), C.c_void_p, C.c_int32, C.c_int32, C.c_int32, _dp, _dp]
    lib.orc_seq_set_kv_block.argtypes = [C.POINTER(_Model), C.c_void_p, C.c_int32, C.c_int32, C.c_int32,
                                         _dp, _dp]
    lib.orc_seq_get_kv.argtypes = [C.POINTER(_Model), C.c_void_p, C.c_int32, C.c_int32, C.c_int32, _dp, _dp]
    lib.orc_forward_token.restype = C.c_int
    lib.orc_forward_token.argtypes = [C.POINTER(_Model), C.c_void_p, C.c_int32, C.c_void_p, _dp]
    lib.orc_num_threads.restype = C.c_int
    lib.orc_set_num_threads.argtypes = [C.c_int]
    lib.orc_model_size.restype = C.c_size_t
    if lib.orc_model_size() != C.sizeof(_Model):
        raise RuntimeError("oracle model struct layout mismatch")
    _lib = lib
    return lib


def _d(a):
    return a.ctypes.data_as(_dp)


def _f(a):
    return a.ctypes.data_as(_fp)


def set_threads(n: int) -> None:
    load().orc_set_num_threads(int(n))


def num_threads() -> int:
    return int(load().orc_num_threads())


def round_bf16(x: float) -> float:
    return float(load().orc_round_bf16(float(x)))


def philox4x32_10(ctr, key):
    c = (C.c_uint32 * 4)(*[int(v) & 0xFFFFFFFF for v in ctr])
    k = (C.c_uint32 * 2)(*[int(v) & 0xFFFFFFFF for v in key])
    o = (C.c_uint32 * 4)()
    load().orc_philox4x32_10(c, k, o)
    return [int(v) for v in o]


def noise_word(seed: int, uid: int, pos_new: int, v: int) -> int:
    return int(load().orc_noise_word(seed, uid, pos_new, v))


def gumbel_of_word(x: int) -> float:
    return float(load().orc_gumbel_of_word(x))


def gumbel_argmax_u(z, u, T: float = 1.0) -> int:
    z = np.ascontiguousarray(z, dtype=np.float32)
    u = np.ascontiguousarray(u, dtype=np.float64)
    return int(load().orc_gumbel_argmax_u(_f(z), _d(u), len(z), T))


def sample(z, T: float, seed: int, uid: int, pos_new: int, forced: int = -1):
    """Returns (token, logp) for fp32 logits z."""
    z = np.ascontiguousarray(z, dtype=np.float32)
    tok = C.c_int32()
    lp = C.c_double()
    load().orc_sample(_f(z), len(z), T, seed, uid, pos_new, forced, C.byref(tok), C.byref(lp))
    return int(tok.value), float(lp.value)


def logprob(z, T: float, y: int) -> float:
    """log softmax(fl32(z / T))[y] for fp32 logits z (T == 0: the T = 1 value)."""
    z = np.ascontiguousarray(z, dtype=np.float32)
    return float(load().orc_logprob(_f(z), len(z), T, int(y)))


def sample_margin(z, T: float, seed: int, uid: int, pos_new: int):
    """Returns (best, runner_up, margin) of the perturbed scores."""
    z = np.ascontiguousarray(z, dtype=np.float32)
    a, b, m = C.c_int32(), C.c_int32(), C.c_double()
    load().orc_sample_margin(_f(z), len(z), T, seed, uid, pos_new, C.byref(a), C.byref(b), C.byref(m))
    return int(a.value), int(b.value), float(m.value)


def _w(arr):
    """numpy weight array -> (encoding, array kept alive)."""
    if arr.dtype == np.uint16:
        return W_BF16, np.ascontiguousarray(arr)
    return W_F32, np.ascontiguousarray(arr, dtype=np.float32)


def rmsnorm(x, g, eps: float, mode: int):
    x = np.ascontiguousarray(x, dtype=np.float64)
    wdt, g = _w(g)
    out = np.empty_like(x)
    load().orc_rmsnorm(_d(x), wdt, g.ctypes.data, 0, len(x), eps, mode, _d(out))
    return out


def matvec(W, x):
    wdt, W = _w(W)
    x = np.ascontiguousarray(x, dtype=np.float64)
    R, K = W.shape
    y = np.empty(R, dtype=np.float64)
    load().orc_matvec(wdt, W.ctypes.data, 0, R, K, _d(x), _d(y))
    return y


def rope_cos_sin(pos: int, i: int, D: int, theta: float):
    c, s = C.c_double(), C.c_double()
    load().orc_rope_cos_sin(pos, i, D, theta, C.byref(c), C.byref(s))
    return c.value, s.value


def rope(v, pos: int, theta: float):
    v = np.array(v, dtype=np.float64, copy=True)
    load().orc_rope(_d(v), len(v), pos, theta)
    return v


def route(r, k: int):
    """Top-k routing of one row of router logits: (experts, weights)."""
    r = np.ascontiguousarray(r, dtype=np.float64)
    sel = np.empty(k, dtype=np.int32)
    w = np.empty(k, dtype=np.float64)
    load().orc_route(_d(r), len(r), int(k), sel.ctypes.data_as(C.POINTER(C.c_int32)), _d(w))
    return sel, w


def attend(q, K, V):
    q = np.ascontiguousarray(q, dtype=np.float64)
    K = np.ascontiguousarray(K, dtype=np.float64)
    V = np.ascontiguousarray(V, dtype=np.float64)
    n, D = K.shape
    out = np.empty(D, dtype=np.float64)
    load().orc_attend(_d(q), _d(K), _d(V), D, n, D, _d(out))
    return out


class OracleModel:
    """Decoder weights (host numpy arrays) plus the precision mode.

    weights: dict with embed [V,H], attn_norm [L,H], w_qkv [L,(Hq+2Hkv)D,H],
    w_o [L,H,Hq*D], mlp_norm [L,H], w_gate_up [L,2F,H], w_down [L,H,F],
    final_norm [H], lm_head [V,H]; all float32 or all uint16 (bf16 bits).
    A mixture-of-experts model (cfg n_experts E > 0, top_k, expert_ffn Fe)
    has w_router [L,E,H], w_exp_gate_up [L,E,2Fe,H] and w_exp_down
    [L,E,H,Fe] instead of w_gate_up and w_down.
    """

    NAMES = ("embed", "attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up",
             "w_down", "final_norm", "lm_head", "w_router", "w_exp_gate_up", "w_exp_down")

    def __init__(self, cfg, weights, mode: int):
        self.lib = load()
        self.cfg = cfg
        self._keep = {}
        wdts = set()
        for n in self.NAMES:
            if n not in weights:
                continue
            wdt, arr = _w(weights[n])
            wdts.add(wdt)
            self._keep[n] = arr
        if len(wdts) != 1:
            raise ValueError("all weights must share one encoding")
        m = _Model()
        m.L, m.H, m.Hq, m.Hkv = cfg["n_layers"], cfg["hidden"], cfg["n_q_heads"], cfg["n_kv_heads"]
        m.D, m.F, m.V = cfg["head_dim"], cfg["ffn"], cfg["vocab"]
        m.eps, m.theta = float(cfg["rms_eps"]), float(cfg["rope_theta"])
        m.mode, m.wdt = int(mode), wdts.pop()
        m.E, m.topk, m.Fe = int(cfg.get("n_experts", 0)), int(cfg.get("top_k", 0)), int(cfg.get("expert_ffn", 0))
        need = self.NAMES[:5] + self.NAMES[7:9] + (self.NAMES[9:] if m.E > 0 else self.NAMES[5:7])
        for n in need:
            if n not in self._keep:
                raise ValueError(f"missing weight {n}")
        for n in self.NAMES:
            setattr(m, n, self._keep[n].ctypes.data if n in self._keep else None)
        self.m = m
        self.wdt = m.wdt
        self.mode = mode

    def new_seq(self, max_ctx: int) -> "OracleSeq":
        return OracleSeq(self, max_ctx)


class OracleSeq:
    """One sequence's KV cache ([L][max_ctx][Hkv][D] doubles) and length."""

    def __init__(self, model: OracleModel, max_ctx: int, _handle=None):
        self.model = model
        self.lib = model.lib
        self.h = _handle if _handle else self.lib.orc_seq_create(C.byref(model.m), int(max_ctx))
        if not self.h:
            raise MemoryError("oracle sequence allocation failed")
        self.max_ctx = max_ctx

    def clone(self) -> "OracleSeq":
        h = self.lib.orc_seq_clone(C.byref(self.model.m), self.h)
        if not h:
            raise MemoryError("oracle sequence allocation failed")
        return OracleSeq(self.model, self.max_ctx, _handle=h)

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            self.lib.orc_seq_destroy(h)
            self.h = None

    @property
    def length(self) -> int:
        return int(self.lib.orc_seq_len(self.h))

    @property
    def route_margin(self) -> float:
        """Smallest gap between a chosen router logit and the largest one left
        out, over every token routed so far (inf for a dense model)."""
        return float(self.lib.orc_seq_route_margin(self.h))

    def set_length(self, n: int) -> None:
        self.lib.orc_seq_set_len(self.h, int(n))

    def forward(self, tok: int, embed_row=None):
        """Feed one token (or an embedding row when tok < 0); returns logits (float64 [V])."""
        cfg = self.model.cfg
        logits = np.empty(cfg["vocab"], dtype=np.float64)
        row_ptr = None
        keep = None
        if tok < 0:
            if embed_row is None:
                raise ValueError("tok < 0 needs embed_row")
            wdt, keep = _w(np.asarray(embed_row))
            if wdt != self.model.wdt:
                raise ValueError("embedding row encoding must match the weights")
            row_ptr = keep.ctypes.data
        rc = self.lib.orc_forward_token(C.byref(self.model.m), self.h, int(tok), row_ptr, _d(logits))
        if rc != 0:
            raise RuntimeError(f"oracle forward failed ({rc})")
        del keep
        return logits

    def set_kv(self, layer: int, pos: int, kvh: int, k, v) -> None:
        k = np.ascontiguousarray(k, dtype=np.float64)
        v = np.ascontiguousarray(v, dtype=np.float64)
        self.lib.orc_seq_set_kv(C.byref(self.model.m), self.h, layer, pos, kvh, _d(k), _d(v))

    def set_kv_block(self, layer: int, kvh: int, K, V) -> None:
        """K, V: [n, D] rows for positions 0..n-1 of (layer, kv-head)."""
        K = np.ascontiguousarray(K, dtype=np.float64)
        V = np.ascontiguousarray(V, dtype=np.float64)
        if K.shape != V.shape or K.shape[0] > self.max_ctx:
            raise ValueError("bad KV block shape")
        self.lib.orc_seq_set_kv_block(C.byref(self.model.m), self.h, layer, kvh, K.shape[0], _d(K), _d(V))

    def get_kv(self, layer: int, pos: int, kvh: int):
        D = self.model.cfg["head_dim"]
        k = np.empty(D, dtype=np.float64)
        v = np.empty(D, dtype=np.float64)
        self.lib.orc_seq_get_kv(C.byref(self.model.m), self.h, layer, pos, kvh, _d(k), _d(v))
        return k, v


def score(model: OracleModel, prompt, response, T: float, embeds=None, return_margin: bool = False):
    """Inference-stage log-probabilities of one response (Sec. 2.1, GRPO:
    after generation the log-probabilities of the responses are computed by a
    forward pass over them).

    Entry j is log softmax(z_j / T)[response[j]], where z_j are the logits
    after prompt + response[:j].  The sequence is fed one token at a time
    through the oracle's KV-cached forward; prompt ids < 0 select rows of
    `embeds` (row -id-1).  Returns a float64 array of len(response), and
    with return_margin also the sequence's smallest routing margin (inf for
    a dense model)."""
    response = [int(t) for t in response]
    seq = model.new_seq(len(prompt) + len(response))
    z = None
    for t in prompt:
        t = int(t)
        z = seq.forward(t, None if t >= 0 else embeds[-t - 1])
    out = np.empty(len(response), dtype=np.float64)
    for j, y in enumerate(response):
        out[j] = logprob(z.astype(np.float32), T, y)
        if j + 1 < len(response):
            z = seq.forward(y)
    return (out, seq.route_margin) if return_margin else out
