"""The five synthetic rollout workloads (shapes only; no arithmetic).

Each workload is a randomly initialised decoder shaped like a policy model the
paper trains (Sec. 5.1.1: Qwen2.5 1.5B / 7B / 32B with GRPO, rollout batch
512; Sec. 5.1.2: OpenVLA on a Llama-2-7B backbone, 256 parallel ManiSkill
environments), plus the batch structure of its rollout.
"""
from dataclasses import dataclass, field, asdict
from typing import Optional, Tuple


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rms_eps: float
    rope_theta: float
    dtype: str  # "fp32" or "bf16"
    # mixture of experts (n_experts > 0): each layer's MLP is n_experts SwiGLU
    # experts of width expert_ffn, of which each token uses its top_k
    n_experts: int = 0
    top_k: int = 0
    expert_ffn: int = 0

    def as_dict(self):
        return asdict(self)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "fp32" else 2

    @property
    def moe(self) -> bool:
        return self.n_experts > 0

    def expert_params(self) -> int:
        """Parameters of one expert (gate, up and down rows)."""
        return 3 * self.hidden * self.expert_ffn

    def decode_params(self, active_experts: Optional[float] = None) -> int:
        """Parameters a decode step reads: every layer matrix, the norms, the LM head
        (a mixture of experts: the router and `active_experts` experts per layer,
        all of them when None)."""
        L, H, Hq, Hkv, d, F, V = (self.n_layers, self.hidden, self.n_q_heads, self.n_kv_heads,
                                  self.head_dim, self.ffn, self.vocab)
        attn = H * (Hq + 2 * Hkv) * d + Hq * d * H + 2 * H
        if self.moe:
            a = self.n_experts if active_experts is None else active_experts
            return int(L * (attn + self.n_experts * H + a * self.expert_params()) + H * V + H)
        return L * (attn + 3 * H * F) + H * V + H

    def kv_bytes_per_token(self) -> int:
        return self.n_layers * 2 * self.n_kv_heads * self.head_dim * self.elem_bytes


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    n_prompts: int
    group: int
    prompt_len: Tuple[int, int]         # inclusive uniform range
    response_median: int                # lognormal median (or fixed length when sigma == 0)
    response_sigma: float
    response_cap: int
    temperature: float = 1.0
    patch_rows: int = 0                 # embodied workload: caller-provided embedding rows
    env_steps: int = 0                  # embodied workload: env steps per rollout
    seed: int = 20250919
    init: str = "fanin"                 # weight initialisation (inputs.make_weights)

    @property
    def n_seqs(self) -> int:
        return self.n_prompts * self.group

    @property
    def max_prompt(self) -> int:
        return self.prompt_len[1] + self.patch_rows

    @property
    def max_ctx(self) -> int:
        return self.max_prompt + self.response_cap


TINY = ModelShape(2, 256, 4, 2, 64, 688, 4096, 1e-6, 1e4, "fp32")
QWEN_1_5B = ModelShape(28, 1536, 12, 2, 128, 8960, 151936, 1e-6, 1e6, "bf16")
LLAMA2_7B = ModelShape(32, 4096, 32, 32, 128, 11008, 32000, 1e-5, 1e4, "bf16")
QWEN_7B = ModelShape(28, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1e6, "bf16")
QWEN_32B = ModelShape(64, 5120, 40, 8, 128, 27648, 152064, 1e-6, 1e6, "bf16")
# Qwen3-30B-A3B shape (Sec. 5.1.1's MoE policy): 128 experts of width 768, top 8
QWEN3_MOE = ModelShape(48, 2048, 32, 4, 128, 768, 151936, 1e-6, 1e6, "bf16",
                       n_experts=128, top_k=8, expert_ffn=768)

WORKLOADS = {
    # tiny fp32 decoder: 2 prompts x 4 samples, 32-token prompts, 32 generated tokens
    "tiny": Workload("tiny", TINY, 2, 4, (32, 32), 32, 0.0, 32, seed=20250919 + 0, init="normal"),
    # Qwen2.5-1.5B shape: 64 prompts x 8, prompts U[128,512], lognormal(600) capped at 1024
    "qwen1.5b": Workload("qwen1.5b", QWEN_1_5B, 64, 8, (128, 512), 600, 0.5, 1024, seed=20250919 + 1),
    # Llama-2-7B embodied shape: 256 envs, 256 patch rows + 32 text tokens, 7 action tokens per env step
    "llama7b-embodied": Workload("llama7b-embodied", LLAMA2_7B, 256, 1, (32, 32), 7, 0.0, 7,
                                 patch_rows=256, env_steps=50, seed=20250919 + 2),
    # Qwen2.5-7B shape: 32 prompts x 16, prompts U[256,1024], lognormal(1500) capped at 4096
    "qwen7b": Workload("qwen7b", QWEN_7B, 32, 16, (256, 1024), 1500, 0.5, 4096, seed=20250919 + 3),
    # Qwen2.5-32B shape: 8 prompts x 8, 512-token prompts, lognormal(4000) capped at 8192
    "qwen32b": Workload("qwen32b", QWEN_32B, 8, 8, (512, 512), 4000, 0.5, 8192, seed=20250919 + 4),
    # Qwen3-30B-A3B shape (mixture of experts): 32 prompts x 16, prompts U[256,1024],
    # lognormal(1500) capped at 4096 (the 7B rollout's batch and lengths)
    "qwen3moe": Workload("qwen3moe", QWEN3_MOE, 32, 16, (256, 1024), 1500, 0.5, 4096, seed=20250919 + 5),
}
