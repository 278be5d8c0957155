"""Workload shapes for the MoE-decode hot path.

Each workload is a stack of MoE layers shaped like a published MoE model, decoded
token by token with synthetic hidden states.  Notation follows the paper's notation
table (Sec. IV-C): ``E`` experts (the paper's N), ``k`` routed experts, ``d`` hidden
size, ``I`` expert intermediate size, ``C`` HBM cache slots per layer, ``tau`` the
coverage target, ``k_max`` the cap on the prefetch-set size k + delta_hat.

Values the workload descriptions leave open are fixed here and listed with the other
readings in the design notes: the Granite-3B cache and cap (C = 16, k_max = 16) and
the OLMoE cap and target (k_max = 16, tau = 0.9, 256 steps).
"""
from dataclasses import dataclass
from typing import Tuple


@dataclass(frozen=True)
class MoEConfig:
    name: str
    cfg_id: int            # seed component, one per workload
    L: int                 # MoE layers
    d: int                 # hidden size
    E: int                 # experts per layer (the paper's N)
    k: int                 # routed experts per token
    I: int                 # SwiGLU intermediate size
    C: int                 # HBM cache slots per layer
    k_max: int             # cap on the prefetch-set size
    tau: float             # coverage target
    steps: int             # decode steps
    batches: Tuple[int, ...] = (1,)
    taus: Tuple[float, ...] = ()       # tau sweep, if any
    bias_skew: bool = False            # per-expert logit bias ~N(0,1) (Zipf-like load)
    heads: int = 0                     # attention query heads (0: d / 64)
    kv_heads: int = 0                  # attention key/value heads (0: as many as heads)
    shared: int = 0                    # always-active shared experts per layer
    I_shared: int = 0                  # their SwiGLU intermediate size (0: I)

    @property
    def n_heads(self) -> int:
        return self.heads or self.d // 64

    @property
    def n_kv_heads(self) -> int:
        return self.kv_heads or self.n_heads

    @property
    def head_dim(self) -> int:
        return self.d // self.n_heads

    @property
    def shared_I(self) -> int:
        return self.I_shared or self.I

    @property
    def expert_bytes(self) -> int:
        """Bytes of one bf16 SwiGLU expert: W1, W3 (I x d) and W2 (d x I)."""
        return 3 * self.d * self.I * 2

    def ffn_bytes(self, n_experts: int) -> int:
        return n_experts * self.expert_bytes


# Attention shapes (heads / key-value heads) follow the published model configurations;
# they only shape the decode-attention window that the prefetch overlaps.
TINY = MoEConfig("tiny", 0, L=1, d=256, E=8, k=2, I=512, C=4, k_max=4, tau=0.9,
                 steps=64, heads=4, kv_heads=2)
GRANITE_1B = MoEConfig("granite-1b-a400m", 1, L=24, d=1024, E=32, k=8, I=512, C=16,
                       k_max=16, tau=0.9, steps=256, heads=16, kv_heads=8)
GRANITE_3B = MoEConfig("granite-3b-a800m", 2, L=32, d=1536, E=40, k=8, I=512, C=16,
                       k_max=16, tau=0.9, steps=256, batches=(1, 8),
                       taus=(0.8, 0.9, 0.95, 0.99), heads=24, kv_heads=8)
OLMOE = MoEConfig("olmoe-1b-7b", 3, L=16, d=2048, E=64, k=8, I=1024, C=24, k_max=16,
                  tau=0.9, steps=256, batches=(1, 16, 64), bias_skew=True, heads=16,
                  kv_heads=16)
MIXTRAL = MoEConfig("mixtral-8x7b", 4, L=8, d=4096, E=8, k=2, I=14336, C=4, k_max=4,
                    tau=0.9, steps=128, batches=(1, 8, 32), heads=32, kv_heads=8)

# The paper's other two evaluated models (Sec. V-A).  d from the per-layer router sizes of
# its overhead table (d N + 2N parameters per layer); I from the total and active
# parameter counts in the model names, I = (P_total - P_active) / (L (N - k) 3 d), rounded
# to a multiple of 64 (Phi: 7B and 2.4B over 32 layers; DeepSeek: 16B and 2.4B over its 26
# MoE layers, the dense first layer left out).  DeepSeek's two shared experts run for
# every token outside the adaptive decision.  Cache sizes and k_max follow the other
# workloads (half of E at small E, C = 24 of 64 as OLMoE).
PHI_7B = MoEConfig("phi-7b", 5, L=32, d=4096, E=16, k=2, I=832, C=8, k_max=6, tau=0.9,
                   steps=256, batches=(1, 8), heads=32, kv_heads=8)
DEEPSEEK_16B = MoEConfig("deepseek-16b", 6, L=26, d=2048, E=64, k=6, I=1472, C=24, k_max=16,
                         tau=0.9, steps=256, batches=(1, 16), heads=16, kv_heads=16, shared=2)

CONFIGS = {c.name: c for c in (TINY, GRANITE_1B, GRANITE_3B, OLMOE, MIXTRAL, PHI_7B,
                               DEEPSEEK_16B)}
BY_ID = {c.cfg_id: c for c in CONFIGS.values()}


def get(name_or_id) -> MoEConfig:
    if isinstance(name_or_id, int):
        return BY_ID[name_or_id]
    return CONFIGS[name_or_id]
