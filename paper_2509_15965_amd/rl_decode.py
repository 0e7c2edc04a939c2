"""Python binding of the C ABI in include/rl_decode.h (argument marshalling only).

PyTorch supplies device memory (weights, KV pool, workspace, token and output
buffers) and the stream; every step of the decoder runs in the library's HIP
kernels.  There is no fallback: if librl_decode.so is missing or a call
fails, an exception is raised.
"""
import ctypes as C
import os
from typing import Dict, Optional, Sequence

import numpy as np
import torch

from .configs import ModelShape

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "librl_decode.so")

RL_OK, RL_ERR_INVALID_ARG, RL_ERR_UNSUPPORTED, RL_ERR_CAPACITY, RL_ERR_HIP, RL_ERR_STATE = range(6)
RL_DTYPE_FP32, RL_DTYPE_BF16 = 0, 1
RL_OPT_ATTN_CHUNK, RL_OPT_PROFILE, RL_OPT_GEMM_PLAN, RL_OPT_SHARED_PREFIX, RL_OPT_PREFILL_ATTENTION = 1, 2, 3, 4, 5
(RL_GEMM_DIRECT, RL_GEMM_GEMV, RL_GEMM_T256, RL_GEMM_T128X256, RL_GEMM_T128, RL_GEMM_T128_DEEP,
 RL_GEMM_GEMV_WIDE) = 1, 2, 3, 4, 5, 6, 7


def gemm_plan_code(kernel: int, splits: int = 0, second: int = 0) -> int:
    """Value of RL_OPT_GEMM_PLAN: tile kernel, split-K count, second-half kernel."""
    return int(kernel) | (int(splits) << 8) | (int(second) << 16)
KERNEL_CLASSES = ("embed", "rmsnorm", "gemm_qkv", "rope_append", "attention", "attn_combine",
                  "gemm_o", "gemm_gate_up", "gemm_down", "gemm_lm_head", "splitk_reduce", "sample",
                  "moe_route", "moe_experts")

EXPORTS = ("rl_decode_kv_bytes", "rl_decode_workspace_bytes", "rl_decode_create", "rl_decode_destroy",
           "rl_prefill", "rl_score", "rl_decode_step", "rl_sample_logits", "rl_release_slots",
           "rl_set_slot_lengths", "rl_slot_length", "rl_kv_free_pages", "rl_kv_offload_bytes", "rl_kv_offload", "rl_kv_onload",
           "rl_decode_rebind", "rl_decode_set_option", "rl_decode_kernel_stats",
           "rl_decode_reset_stats", "rl_decode_attn_plan_stats", "rl_probe_copy", "rl_probe_read", "rl_probe_mfma",
           "rl_probe_gumbel_bound",
           "rl_sample_logits_noalloc", "rl_decode_tune_gemms", "rl_decode_gemm_plan", "rl_status_string",
           "rl_decode_last_error")


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("dtype", C.c_int32), ("rms_eps", C.c_double),
                ("rope_theta", C.c_double), ("max_seqs", C.c_int32), ("max_ctx", C.c_int32),
                ("max_prefill_tokens", C.c_int32), ("kv_page_size", C.c_int32), ("kv_pages", C.c_int32),
                ("n_experts", C.c_int32), ("top_k", C.c_int32), ("expert_ffn", C.c_int32),
                ("reserved", C.c_int32)]


class Weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("embed", "attn_norm", "w_qkv", "w_o", "mlp_norm",
                                          "w_gate_up", "w_down", "final_norm", "lm_head",
                                          "w_router", "w_exp_gate_up", "w_exp_down")]


def _weights_struct(weights: Dict[str, torch.Tensor]) -> "Weights":
    """Device pointers of the weight tensors (absent ones NULL: the dense MLP
    of a mixture of experts, the experts of a dense model)."""
    w = Weights()
    for name, _ in Weights._fields_:
        setattr(w, name, weights[name].data_ptr() if name in weights else None)
    return w


class SampleParams(C.Structure):
    _fields_ = [("seed", C.c_uint64), ("temperature", C.c_float), ("reserved", C.c_int32)]


class KernelStats(C.Structure):
    _fields_ = [("launches", C.c_int64), ("total_ms", C.c_double), ("alg_bytes", C.c_double),
                ("alg_flops", C.c_double), ("name", C.c_char * 48)]


class AttnPlanStats(C.Structure):
    _fields_ = [("steps", C.c_int64), ("items", C.c_int64), ("shared_items", C.c_int64),
                ("pair_items", C.c_int64), ("lds_workgroups", C.c_int64)]


_lib = None


def lib():
    """Load librl_decode.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2509_15965_amd.build`")
    L = C.CDLL(LIB_PATH)
    vp, i32, u64, sz = C.c_void_p, C.c_int32, C.c_uint64, C.c_size_t
    cfgp = C.POINTER(ModelConfig)
    L.rl_decode_kv_bytes.restype = sz
    L.rl_decode_kv_bytes.argtypes = [cfgp]
    L.rl_decode_workspace_bytes.restype = sz
    L.rl_decode_workspace_bytes.argtypes = [cfgp]
    L.rl_decode_create.restype = C.c_int
    L.rl_decode_create.argtypes = [cfgp, C.POINTER(Weights), vp, sz, vp, sz, vp, C.POINTER(vp)]
    L.rl_decode_destroy.restype = C.c_int
    L.rl_decode_destroy.argtypes = [vp]
    L.rl_prefill.restype = C.c_int
    L.rl_prefill.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp, i32, vp, C.POINTER(SampleParams), vp, vp, vp]
    L.rl_score.restype = C.c_int
    L.rl_score.argtypes = [vp, i32, i32, vp, vp, vp, vp, i32, vp, vp, C.c_float, vp]
    L.rl_decode_step.restype = C.c_int
    L.rl_decode_step.argtypes = [vp, i32, vp, vp, vp, vp, C.POINTER(SampleParams), vp, vp, vp]
    L.rl_sample_logits.restype = C.c_int
    L.rl_sample_logits.argtypes = [vp, i32, vp, vp, vp, vp, C.POINTER(SampleParams), vp, vp]
    L.rl_release_slots.restype = C.c_int
    L.rl_release_slots.argtypes = [vp, i32, vp]
    L.rl_set_slot_lengths.restype = C.c_int
    L.rl_set_slot_lengths.argtypes = [vp, i32, vp, vp]
    L.rl_slot_length.restype = i32
    L.rl_slot_length.argtypes = [vp, i32]
    L.rl_kv_free_pages.restype = C.c_int64
    L.rl_kv_free_pages.argtypes = [vp]
    L.rl_kv_offload_bytes.restype = sz
    L.rl_kv_offload_bytes.argtypes = [vp, i32, vp]
    L.rl_kv_offload.restype = C.c_int
    L.rl_kv_offload.argtypes = [vp, i32, vp, vp, sz]
    L.rl_kv_onload.restype = C.c_int
    L.rl_kv_onload.argtypes = [vp, i32, vp, vp, vp, sz]
    L.rl_decode_rebind.restype = C.c_int
    L.rl_decode_rebind.argtypes = [vp, C.POINTER(Weights), vp, sz, vp, sz]
    L.rl_decode_set_option.restype = C.c_int
    L.rl_decode_set_option.argtypes = [vp, i32, C.c_int64]
    L.rl_decode_tune_gemms.restype = C.c_int
    L.rl_decode_tune_gemms.argtypes = [vp, i32, vp]
    L.rl_decode_gemm_plan.restype = C.c_int
    L.rl_decode_gemm_plan.argtypes = [vp, i32, i32, C.POINTER(C.c_int64), C.POINTER(C.c_float)]
    L.rl_decode_kernel_stats.restype = C.c_int
    L.rl_decode_kernel_stats.argtypes = [vp, i32, C.POINTER(KernelStats)]
    L.rl_decode_reset_stats.restype = C.c_int
    L.rl_decode_reset_stats.argtypes = [vp]
    L.rl_decode_attn_plan_stats.restype = C.c_int
    L.rl_decode_attn_plan_stats.argtypes = [vp, C.POINTER(AttnPlanStats)]
    L.rl_probe_copy.restype = C.c_int
    L.rl_probe_copy.argtypes = [vp, vp, sz, vp]
    L.rl_probe_read.restype = C.c_int
    L.rl_probe_read.argtypes = [vp, sz, i32, vp, vp]
    L.rl_probe_mfma.restype = C.c_int
    L.rl_probe_mfma.argtypes = [i32, i32, vp, vp]
    L.rl_sample_logits_noalloc.restype = C.c_int
    L.rl_sample_logits_noalloc.argtypes = [i32, i32, vp, i32, vp, vp, vp, C.POINTER(SampleParams), vp, vp, vp]
    L.rl_probe_gumbel_bound.restype = C.c_int
    L.rl_probe_gumbel_bound.argtypes = [C.c_uint32, C.c_uint64, i32, vp, vp, vp]
    L.rl_status_string.restype = C.c_char_p
    L.rl_status_string.argtypes = [C.c_int]
    L.rl_decode_last_error.restype = C.c_char_p
    L.rl_decode_last_error.argtypes = [vp]
    _lib = L
    return L


class RLError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{lib().rl_status_string(status).decode()} ({status}): {msg}")
        self.status = status


def make_config(shape: ModelShape, max_seqs: int, max_ctx: int, max_prefill_tokens: int,
                kv_page_size: int = 0, kv_pages: int = 0) -> ModelConfig:
    c = ModelConfig()
    c.n_layers, c.hidden, c.n_q_heads = shape.n_layers, shape.hidden, shape.n_q_heads
    c.n_kv_heads, c.head_dim, c.ffn, c.vocab = shape.n_kv_heads, shape.head_dim, shape.ffn, shape.vocab
    c.dtype = RL_DTYPE_BF16 if shape.dtype == "bf16" else RL_DTYPE_FP32
    c.rms_eps, c.rope_theta = float(shape.rms_eps), float(shape.rope_theta)
    c.max_seqs, c.max_ctx, c.max_prefill_tokens = max_seqs, max_ctx, max_prefill_tokens
    c.kv_page_size, c.kv_pages, c.reserved = kv_page_size, kv_pages, 0
    c.n_experts, c.top_k, c.expert_ffn = shape.n_experts, shape.top_k, shape.expert_ffn
    return c


def kv_bytes(cfg: ModelConfig) -> int:
    return int(lib().rl_decode_kv_bytes(C.byref(cfg)))


def workspace_bytes(cfg: ModelConfig) -> int:
    return int(lib().rl_decode_workspace_bytes(C.byref(cfg)))


def _p(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _host_u64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.uint64))


class Engine:
    """One decode context: borrowed weights, a KV pool and a workspace
    allocated here with torch, and the current torch stream."""

    def __init__(self, shape: ModelShape, weights: Dict[str, torch.Tensor], max_seqs: int,
                 max_ctx: int, max_prefill_tokens: int, device="cuda", stream=None,
                 kv_page_size: int = 0, kv_pages: int = 0):
        L = lib()
        self.shape = shape
        self.cfg = make_config(shape, max_seqs, max_ctx, max_prefill_tokens, kv_page_size, kv_pages)
        self.kv_nbytes = kv_bytes(self.cfg)
        self.ws_nbytes = workspace_bytes(self.cfg)
        if self.kv_nbytes == 0 or self.ws_nbytes == 0:
            raise RLError(RL_ERR_INVALID_ARG, "configuration rejected")
        self.device = torch.device(device)
        self.kv = torch.empty(self.kv_nbytes, dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(self.ws_nbytes, dtype=torch.uint8, device=self.device)
        self.weights = weights
        w = _weights_struct(weights)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        h = C.c_void_p()
        st = L.rl_decode_create(C.byref(self.cfg), C.byref(w), self.kv.data_ptr(), self.kv_nbytes,
                                self.ws.data_ptr(), self.ws_nbytes, self.stream.cuda_stream, C.byref(h))
        if st != RL_OK:
            raise RLError(st, "rl_decode_create failed")
        self.h = h

    # -- helpers ----------------------------------------------------------
    def _check(self, st: int, what: str):
        if st != RL_OK:
            raise RLError(st, f"{what}: {lib().rl_decode_last_error(self.h).decode()}")

    def close(self):
        if getattr(self, "h", None):
            lib().rl_decode_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- entry points -----------------------------------------------------
    def prefill(self, slots: Sequence[int], uids: Sequence[int], prompt_offsets: Sequence[int],
                tokens: torch.Tensor, out_tok: torch.Tensor, out_logp: torch.Tensor, *, group: int = 1,
                embeds: Optional[torch.Tensor] = None, forced: Optional[torch.Tensor] = None,
                seed: int = 0, temperature: float = 1.0, out_logits: Optional[torch.Tensor] = None):
        slots, uids, offs = _host_i32(slots), _host_u64(uids), _host_i32(prompt_offsets)
        n_prompts = len(offs) - 1
        sp = SampleParams(seed, temperature, 0)
        n_rows = 0 if embeds is None else int(embeds.shape[0])
        st = lib().rl_prefill(self.h, n_prompts, group, slots.ctypes.data, uids.ctypes.data,
                              offs.ctypes.data, _p(tokens), _p(embeds), n_rows, _p(forced), C.byref(sp),
                              _p(out_tok), _p(out_logp), _p(out_logits))
        self._check(st, "rl_prefill")

    def score(self, slots: Sequence[int], prompt_offsets: Sequence[int], prompt_tokens: torch.Tensor,
              resp_offsets: Sequence[int], resp_tokens: torch.Tensor, out_logp: torch.Tensor, *,
              group: int = 1, embeds: Optional[torch.Tensor] = None, temperature: float = 1.0):
        slots, poffs, roffs = _host_i32(slots), _host_i32(prompt_offsets), _host_i32(resp_offsets)
        n_rows = 0 if embeds is None else int(embeds.shape[0])
        st = lib().rl_score(self.h, len(poffs) - 1, group, slots.ctypes.data, poffs.ctypes.data,
                            _p(prompt_tokens), _p(embeds), n_rows, roffs.ctypes.data, _p(resp_tokens),
                            float(temperature), _p(out_logp))
        self._check(st, "rl_score")

    def step(self, slots: Sequence[int], uids: Sequence[int], in_tok: torch.Tensor, out_tok: torch.Tensor,
             out_logp: torch.Tensor, *, forced: Optional[torch.Tensor] = None, seed: int = 0,
             temperature: float = 1.0, out_logits: Optional[torch.Tensor] = None):
        slots, uids = _host_i32(slots), _host_u64(uids)
        sp = SampleParams(seed, temperature, 0)
        st = lib().rl_decode_step(self.h, len(slots), slots.ctypes.data, uids.ctypes.data, _p(in_tok),
                                  _p(forced), C.byref(sp), _p(out_tok), _p(out_logp), _p(out_logits))
        self._check(st, "rl_decode_step")

    def sample_logits(self, logits: torch.Tensor, uids: Sequence[int], pos_new: Sequence[int],
                      out_tok: torch.Tensor, out_logp: torch.Tensor, *, forced=None, seed: int = 0,
                      temperature: float = 1.0):
        uids, pos = _host_u64(uids), _host_i32(pos_new)
        sp = SampleParams(seed, temperature, 0)
        st = lib().rl_sample_logits(self.h, len(uids), _p(logits), uids.ctypes.data, pos.ctypes.data,
                                    _p(forced), C.byref(sp), _p(out_tok), _p(out_logp))
        self._check(st, "rl_sample_logits")

    def release(self, slots: Sequence[int]):
        s = _host_i32(slots)
        self._check(lib().rl_release_slots(self.h, len(s), s.ctypes.data), "rl_release_slots")

    def set_lengths(self, slots: Sequence[int], lengths: Sequence[int]):
        s, l = _host_i32(slots), _host_i32(lengths)
        self._check(lib().rl_set_slot_lengths(self.h, len(s), s.ctypes.data, l.ctypes.data),
                    "rl_set_slot_lengths")

    def slot_length(self, slot: int) -> int:
        return int(lib().rl_slot_length(self.h, slot))

    def kv_free_pages(self) -> int:
        """Free pages of a paged K/V pool (-1 for a contiguous pool)."""
        return int(lib().rl_kv_free_pages(self.h))

    def kv_offload_bytes(self, slots: Sequence[int]) -> int:
        s = _host_i32(slots)
        return int(lib().rl_kv_offload_bytes(self.h, len(s), s.ctypes.data))

    def kv_offload(self, slots: Sequence[int], host: torch.Tensor):
        """Live K/V of `slots` into `host` (a pinned uint8 CPU tensor)."""
        s = _host_i32(slots)
        self._check(lib().rl_kv_offload(self.h, len(s), s.ctypes.data, host.data_ptr(), host.numel()),
                    "rl_kv_offload")

    def kv_onload(self, slots: Sequence[int], lengths: Sequence[int], host: torch.Tensor):
        s, l = _host_i32(slots), _host_i32(lengths)
        self._check(lib().rl_kv_onload(self.h, len(s), s.ctypes.data, l.ctypes.data, host.data_ptr(),
                                       host.numel()), "rl_kv_onload")

    def rebind(self, weights: Dict[str, torch.Tensor], kv: torch.Tensor, ws: torch.Tensor):
        """Point the context at new device buffers (weights, KV pool, workspace)."""
        w = _weights_struct(weights)
        self._check(lib().rl_decode_rebind(self.h, C.byref(w), kv.data_ptr(), kv.numel(), ws.data_ptr(),
                                           ws.numel()), "rl_decode_rebind")
        self.weights, self.kv, self.ws = weights, kv, ws

    def set_option(self, option: int, value: int):
        self._check(lib().rl_decode_set_option(self.h, option, value), "rl_decode_set_option")

    def tune_gemms(self, sizes: Sequence[int]):
        """Measure the GEMM plans at these batch sizes (increasing); [] clears."""
        s = _host_i32(sizes)
        self._check(lib().rl_decode_tune_gemms(self.h, len(s), s.ctypes.data if len(s) else None),
                    "rl_decode_tune_gemms")

    def gemm_plan(self, kclass: str, rows: int):
        """(RL_OPT_GEMM_PLAN code, measured us per layer or -1) of a GEMM class at `rows` rows."""
        code, us = C.c_int64(0), C.c_float(0.0)
        self._check(lib().rl_decode_gemm_plan(self.h, KERNEL_CLASSES.index(kclass), rows, C.byref(code),
                                              C.byref(us)), "rl_decode_gemm_plan")
        return int(code.value), float(us.value)

    def kernel_stats(self) -> Dict[str, dict]:
        out = {}
        for k, name in enumerate(KERNEL_CLASSES):
            s = KernelStats()
            self._check(lib().rl_decode_kernel_stats(self.h, k, C.byref(s)), "rl_decode_kernel_stats")
            out[name] = {"launches": s.launches, "total_ms": s.total_ms, "alg_bytes": s.alg_bytes,
                         "alg_flops": s.alg_flops}
        return out

    def attn_plan_stats(self) -> Dict[str, int]:
        s = AttnPlanStats()
        self._check(lib().rl_decode_attn_plan_stats(self.h, C.byref(s)), "rl_decode_attn_plan_stats")
        return {name: int(getattr(s, name)) for name, _ in AttnPlanStats._fields_}

    def reset_stats(self):
        self._check(lib().rl_decode_reset_stats(self.h), "rl_decode_reset_stats")

    # -- KV pool views (layout of include/rl_decode.h) --------------------
    def kv_views(self):
        """(K, V) torch views of a contiguous pool: K [L][S][Hkv][cap][d],
        V [L][S][Hkv][cap/8][d][8] (8-position blocks), model dtype."""
        if self.cfg.kv_page_size:
            raise ValueError("a paged pool has no per-slot views")
        s = self.shape
        cap = (self.cfg.max_ctx + 31) // 32 * 32
        dt = torch.float32 if s.dtype == "fp32" else torch.bfloat16
        half = self.kv_nbytes // 2
        K = self.kv[:half].view(dt).view(s.n_layers, self.cfg.max_seqs, s.n_kv_heads, cap, s.head_dim)
        V = self.kv[half:].view(dt).view(s.n_layers, self.cfg.max_seqs, s.n_kv_heads, cap // 8, s.head_dim, 8)
        return K, V


def probe_copy(dst: torch.Tensor, src: torch.Tensor, nbytes: int, stream=None):
    stream = stream if stream is not None else torch.cuda.current_stream(dst.device)
    st = lib().rl_probe_copy(dst.data_ptr(), src.data_ptr(), nbytes, stream.cuda_stream)
    if st != RL_OK:
        raise RLError(st, "rl_probe_copy")


def probe_read(src: torch.Tensor, nbytes: int, out: torch.Tensor, stream=None):
    """Read-only stream of nbytes of src by out.numel() workgroups (out: int32, one word each)."""
    stream = stream if stream is not None else torch.cuda.current_stream(src.device)
    st = lib().rl_probe_read(src.data_ptr(), nbytes, out.numel(), out.data_ptr(), stream.cuda_stream)
    if st != RL_OK:
        raise RLError(st, "rl_probe_read")


def probe_mfma(n_blocks: int, iters: int, out: torch.Tensor, stream=None):
    """n_blocks x 4 waves x iters x 8 MFMA 32x32x16 bf16 (out: float32 [4 * n_blocks])."""
    if out.numel() < 4 * n_blocks or out.dtype != torch.float32:
        raise ValueError("out must hold 4 * n_blocks float32")
    stream = stream if stream is not None else torch.cuda.current_stream(out.device)
    st = lib().rl_probe_mfma(n_blocks, iters, out.data_ptr(), stream.cuda_stream)
    if st != RL_OK:
        raise RLError(st, "rl_probe_mfma")


def probe_gumbel_bound(lo: int, count: int, n_blocks: int = 4096, device="cuda"):
    """Run the sampler's noise-bound check over words [lo, lo + count);
    returns (violations, smallest margin of the fp32 bound)."""
    viol = torch.empty(n_blocks, dtype=torch.int32, device=device)
    mm = torch.empty(n_blocks, dtype=torch.float32, device=device)
    stream = torch.cuda.current_stream(torch.device(device))
    st = lib().rl_probe_gumbel_bound(int(lo), int(count), n_blocks, viol.data_ptr(), mm.data_ptr(),
                                     stream.cuda_stream)
    if st != RL_OK:
        raise RLError(st, "rl_probe_gumbel_bound")
    torch.cuda.synchronize(device)
    return int(viol.to(torch.int64).sum().item()), float(mm.min().item())


def sample_logits_noalloc(logits: torch.Tensor, uids: torch.Tensor, pos_new: torch.Tensor, out_tok: torch.Tensor,
                          out_logp: torch.Tensor, *, forced: Optional[torch.Tensor] = None, seed: int = 0,
                          temperature: float = 1.0, stream=None):
    """rl_sample_logits_noalloc: logits [n][ld] fp32, uids uint64 (int64
    tensor) and pos_new int32 on the device."""
    n, ld = int(logits.shape[0]), int(logits.stride(0))
    stream = stream if stream is not None else torch.cuda.current_stream(logits.device)
    sp = SampleParams(seed, temperature, 0)
    st = lib().rl_sample_logits_noalloc(n, int(logits.shape[1]), logits.data_ptr(), ld, uids.data_ptr(),
                                        pos_new.data_ptr(), _p(forced), C.byref(sp), out_tok.data_ptr(),
                                        out_logp.data_ptr(), stream.cuda_stream)
    if st != RL_OK:
        raise RLError(st, "rl_sample_logits_noalloc")
