"""The five workload configurations, as plain data (no arithmetic of the method)."""
from dataclasses import dataclass, field, replace
from typing import Optional


@dataclass(frozen=True)
class ModelCfg:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int          # dense SwiGLU hidden size (0 for MoE)
    vocab: int
    dtype: str            # "f32" or "bf16"
    weight_seed: int
    rope_theta: float = 10000.0
    rms_eps: float = 1e-6
    n_experts: int = 0
    top_k: int = 0
    expert_ffn: int = 0

    @property
    def eos_id(self) -> int:
        return self.vocab - 1

    @property
    def is_moe(self) -> bool:
        return self.n_experts > 0


@dataclass(frozen=True)
class RunCfg:
    n_prompts: int
    prompt_len: int
    m: int                # redundant rollout size per prompt (M'_i)
    k: int                # kept group size (M)
    cap: int              # max new tokens (system length limit)
    len_median: float
    len_sigma: float
    len_tail: bool        # 5% of draws replaced by U(5,10) x median
    workload_seed: int
    sample_seed: int
    temperature: float = 1.0
    L: int = 1            # dual-end long side size (paper sets L=1)
    m_up: Optional[int] = None   # default 2k
    kv_pool_gb: float = 0.0      # 0: size the pool to the worst case

    @property
    def m_up_eff(self) -> int:
        return self.m_up if self.m_up is not None else 2 * self.k


TINY = (ModelCfg("tiny", 2, 128, 4, 4, 32, 512, 512, "f32", 0),
        RunCfg(4, 16, 8, 4, 64, 24.0, 0.8, False, 0, 0))
DENSE_SMALL = (ModelCfg("dense-small", 8, 1024, 16, 4, 64, 4096, 32000, "bf16", 2),
               RunCfg(32, 256, 16, 8, 4096, 800.0, 0.8, False, 2, 2))
QWEN3_8B = (ModelCfg("qwen3-8b-shaped", 36, 4096, 32, 8, 128, 12288, 151936, "bf16", 3,
                     rope_theta=1e6),
            RunCfg(32, 512, 16, 8, 8192, 1200.0, 1.0, True, 3, 3, kv_pool_gb=150.0))
QWEN3_30B_A3B = (ModelCfg("qwen3-30b-a3b-shaped", 48, 2048, 32, 4, 128, 0, 151936, "bf16", 4,
                          rope_theta=1e6, n_experts=128, top_k=8, expert_ffn=768),
                 RunCfg(64, 512, 16, 8, 16384, 1000.0, 1.1, True, 4, 4, kv_pool_gb=160.0))

CONFIGS = {
    "tiny": TINY,
    "dense-small": DENSE_SMALL,
    "qwen3-8b": QWEN3_8B,
    "qwen3-30b-a3b": QWEN3_30B_A3B,
}

# Kernel sweep (bf16, data seed 1, no model).
SWEEP = dict(
    seed=1,
    attn_rows=1024, attn_hq=32, attn_hkv=8, attn_hd=128,
    attn_ctx_median=1500.0, attn_ctx_sigma=1.0, attn_ctx_min=16, attn_ctx_max=32768,
    page=16,
    samp_rows=1024, samp_vocab=151936, samp_std=3.0,
    sel_traj=65536, sel_m=16, sel_k=8, sel_cap=8192, sel_len_median=1000.0,
)


# Reduced shapes used only by parity tests: the Qwen3-30B-A3B-shaped MoE layer
# at full width (d 2048, 32/4 heads x 128, 128 experts top-8, expert FFN 768)
# with 2 layers and a 4096-token vocabulary, 2 prompts x 32 tokens, m 16,
# k 8, cap 20 (early stop fires inside a 20-token window).
PARITY = {
    "moe-full-width": (replace(QWEN3_30B_A3B[0], name="moe-full-width", n_layers=2, vocab=4096),
                       replace(QWEN3_30B_A3B[1], n_prompts=2, prompt_len=32, cap=20, len_median=10.0,
                               len_tail=False, kv_pool_gb=0.0)),
}


def get_config(name: str, **run_overrides):
    model, run = CONFIGS[name] if name in CONFIGS else PARITY[name]
    if run_overrides:
        run = replace(run, **run_overrides)
    return model, run
