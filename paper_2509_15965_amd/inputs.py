"""Seeded synthetic inputs shared by the GPU path's tests, the oracle's tests
and the benchmark.

This module draws random numbers and lays them out; it holds none of the
decoder's arithmetic.  Weights are drawn in fp32 and rounded once to the
model dtype (torch's round-to-nearest-even for bf16); RMSNorm gains are 1.0.
Two initialisations:
  "normal"  every linear and embedding matrix i.i.d. N(0, 0.02);
  "fanin"   unit-variance (fan-in) init: every matrix N(0, 1/fan_in), with
            the residual-branch output projections (w_o, w_down, and the
            experts' w_exp_down) further
            divided by sqrt(2 L) and embedding rows N(0, 1) (the scale of
            caller-provided N(0, 1) embedding rows).  The residual stream then
            starts at the scale of its inputs and each layer adds a bounded
            fraction to it, so one storage ulp changed anywhere is not
            amplified across the depth.
Prompts are uniform
token ids; prompt lengths are uniform integers in the workload's range;
response lengths are lognormal around the workload's median, clamped to
[1, cap] (the long tail of Sec. 2.2, Fig. 2).
"""
import math
from typing import Dict, Optional

import numpy as np
import torch

from .configs import ModelShape, Workload

INIT_STD = 0.02


def torch_dtype(shape: ModelShape):
    return torch.float32 if shape.dtype == "fp32" else torch.bfloat16


def weight_shapes(m: ModelShape) -> Dict[str, tuple]:
    """Shapes of the model's weight tensors; a mixture of experts has a router
    and stacked experts (gate rows first in each expert's gate|up) in place of
    w_gate_up and w_down."""
    L, H, F, V = m.n_layers, m.hidden, m.ffn, m.vocab
    out = {
        "embed": (V, H),
        "attn_norm": (L, H),
        "w_qkv": (L, m.qkv_rows, H),
        "w_o": (L, H, m.n_q_heads * m.head_dim),
        "mlp_norm": (L, H),
    }
    if m.moe:
        E, Fe = m.n_experts, m.expert_ffn
        out.update({"w_router": (L, E, H), "w_exp_gate_up": (L, E, 2 * Fe, H), "w_exp_down": (L, E, H, Fe)})
    else:
        out.update({"w_gate_up": (L, 2 * F, H), "w_down": (L, H, F)})
    out.update({"final_norm": (H,), "lm_head": (V, H)})
    return out


INITS = ("normal", "fanin")


def init_std(m: ModelShape, name: str, init: str) -> float:
    """Standard deviation of weight matrix `name` under initialisation `init`."""
    if init not in INITS:
        raise ValueError(f"unknown init {init!r}")
    if init == "normal":
        return INIT_STD
    if name == "embed":
        return 1.0
    fan_in = {"w_o": m.n_q_heads * m.head_dim, "w_down": m.ffn, "w_exp_down": m.expert_ffn}.get(name, m.hidden)
    if name in ("w_o", "w_down", "w_exp_down"):
        return 1.0 / math.sqrt(fan_in * 2.0 * m.n_layers)
    return 1.0 / math.sqrt(fan_in)


def make_weights(m: ModelShape, seed: int, device="cpu", init: str = "normal") -> Dict[str, torch.Tensor]:
    """Random-init decoder weights on `device`, drawn one layer slice at a time
    (bounded temporary memory) from a single seeded generator."""
    dt = torch_dtype(m)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    out = {}
    for name, shp in weight_shapes(m).items():
        t = torch.empty(shp, dtype=dt, device=device)
        if name.endswith("norm"):
            t.fill_(1.0)
        elif len(shp) == 4:   # stacked experts: one (layer, expert) slice at a time
            std = init_std(m, name, init)
            for l in range(shp[0]):
                for e in range(shp[1]):
                    r = torch.randn(shp[2:], generator=gen, device=device, dtype=torch.float32)
                    t[l, e].copy_(r.mul_(std))
                    del r
        elif len(shp) == 3:
            std = init_std(m, name, init)
            for l in range(shp[0]):
                r = torch.randn(shp[1:], generator=gen, device=device, dtype=torch.float32)
                t[l].copy_(r.mul_(std))
                del r
        else:
            rows = shp[0]
            step = max(1, (1 << 26) // shp[1])
            for r0 in range(0, rows, step):
                r1 = min(rows, r0 + step)
                r = torch.randn((r1 - r0, shp[1]), generator=gen, device=device, dtype=torch.float32)
                t[r0:r1].copy_(r.mul_(init_std(m, name, init)))
                del r
        out[name] = t
    return out


def to_host_numpy(t: torch.Tensor) -> np.ndarray:
    """Host copy: float32 stays float32, bfloat16 becomes its uint16 bit pattern."""
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def weights_to_host(w: Dict[str, torch.Tensor]) -> Dict[str, np.ndarray]:
    return {k: to_host_numpy(v) for k, v in w.items()}


def bf16_bits_to_f64(a: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) to float64 values (exact)."""
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def host_values_f64(a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f64(a) if a.dtype == np.uint16 else a.astype(np.float64)


def rollout_plan(w: Workload, seed: Optional[int] = None, n_prompts: Optional[int] = None):
    """Prompt lengths, prompt tokens (uniform ids), response lengths and uids.

    Response length R counts every generated token, including the first one
    sampled by the prefill; R = clamp(round(exp(ln(median) + sigma*z)), 1, cap).
    Sample k of prompt p has uid p*group + k.
    """
    rng = np.random.default_rng(w.seed if seed is None else seed)
    P = w.n_prompts if n_prompts is None else n_prompts
    lo, hi = w.prompt_len
    plen = rng.integers(lo, hi + 1, size=P)
    prompts = [rng.integers(0, w.model.vocab, size=int(n)).astype(np.int32) for n in plen]
    n = P * w.group
    if w.response_sigma > 0:
        z = rng.standard_normal(n)
        r = np.rint(np.exp(math.log(w.response_median) + w.response_sigma * z))
        resp = np.clip(r, 1, w.response_cap).astype(np.int64)
    else:
        resp = np.full(n, w.response_median, dtype=np.int64)
    uids = np.arange(n, dtype=np.uint64)
    return {"prompt_lens": plen.astype(np.int64), "prompts": prompts,
            "response_lens": resp, "uids": uids}


def uniform_tokens(n: int, vocab: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, vocab, size=n).astype(np.int32)


def patch_rows(n_rows: int, hidden: int, seed: int, dtype=torch.bfloat16, device="cpu") -> torch.Tensor:
    """Caller-provided embedding rows (N(0, 1)), e.g. image patch embeddings."""
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    return torch.randn((n_rows, hidden), generator=gen, device=device, dtype=torch.float32).to(dtype)


def random_kv_rows(L: int, n_seqs: int, Hkv: int, ctx: int, d: int, seed: int,
                   dtype=torch.bfloat16, device="cpu"):
    """Seeded N(0,1) key and value rows [L][n_seqs][Hkv][ctx][d] in the model dtype."""
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    K = torch.randn((L, n_seqs, Hkv, ctx, d), generator=gen, device=device, dtype=torch.float32).to(dtype)
    V = torch.randn((L, n_seqs, Hkv, ctx, d), generator=gen, device=device, dtype=torch.float32).to(dtype)
    return K, V
