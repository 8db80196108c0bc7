"""Frozen synthetic workload configurations for the TopoEP planner.

Each configuration fixes the EP topology (R ranks as M nodes x G GPUs), the
expert count E (main instances contiguous, E/R per rank), top-k, local tokens
T, the per-rank replica budget N, the two-level cost matrix (0 on the
diagonal, ``c_intra`` inside a node, ``c_inter`` across nodes), the routed
activation size S_tok and the expert parameter size ||W_e|| (Section 4.1 of
the paper: system model), and how the synthetic routing is skewed.

S_tok = hidden x 2 bytes (BF16 activations).  ||W_e|| = 3 x hidden x
intermediate x 2 bytes (a SwiGLU expert in BF16).  The Qwen3 dimensions are
the ones of the paper's model table (Section 6.1, 2048 hidden / 768
intermediate, 9 MiB per expert as in the placement-cost example of Section
2.3); Mixtral-8x7B and DeepSeek-V3 dimensions are their public model
configurations; Tiny uses a small synthetic expert.

This module holds parameters only, none of the planner's arithmetic.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Config:
    name: str
    cfg_id: int          # seed component
    R: int               # EP ranks
    G: int               # ranks per node (NVLink / xGMI domain)
    E: int               # logical experts
    k: int               # top-k
    T: int               # local tokens per rank
    N: int               # replica slots per rank
    c_intra: int         # per-byte cost between two ranks of one node
    c_inter: int         # per-byte cost between ranks of different nodes
    S: int               # bytes per routed activation (S_tok)
    W: int               # bytes per expert (||W_e||)
    layers: int          # MoE layers planned per microbatch
    microbatches: int    # microbatches (only the drifting config uses > 1)
    zipf_s: float        # Zipf exponent of expert popularity
    drift_positions: int = 0     # expert-order positions re-permuted per microbatch
    node_limit: int = 0          # tokens draw experts from at most this many nodes (0: off)
    adversarial: tuple = ()      # experts each included per token with prob adv_p
    adv_p: float = 0.0
    extra: dict = field(default_factory=dict, compare=False, hash=False)

    @property
    def M(self) -> int:
        return self.R // self.G

    @property
    def P(self) -> int:
        return self.E // self.R

    @property
    def assignments(self) -> int:
        return self.T * self.k


def _swiglu_bytes(hidden: int, inter: int) -> int:
    return 3 * hidden * inter * 2


TINY = Config("tiny", 1, R=8, G=4, E=16, k=2, T=512, N=1, c_intra=1, c_inter=4,
              S=2048 * 2, W=_swiglu_bytes(512, 512), layers=1, microbatches=1,
              zipf_s=1.2)

MIXTRAL = Config("mixtral", 2, R=8, G=8, E=8, k=2, T=4096, N=1, c_intra=1, c_inter=8,
                 S=4096 * 2, W=_swiglu_bytes(4096, 14336), layers=32, microbatches=1,
                 zipf_s=1.0)

QWEN3 = Config("qwen3", 3, R=32, G=8, E=128, k=8, T=4096, N=2, c_intra=1, c_inter=8,
               S=2048 * 2, W=_swiglu_bytes(2048, 768), layers=48, microbatches=4,
               zipf_s=1.1, drift_positions=13)

DSV3 = Config("dsv3", 4, R=32, G=8, E=256, k=8, T=8192, N=2, c_intra=1, c_inter=8,
              S=7168 * 2, W=_swiglu_bytes(7168, 2048), layers=58, microbatches=1,
              zipf_s=1.0, node_limit=4)

STRESS = Config("stress", 5, R=256, G=8, E=512, k=8, T=16384, N=4, c_intra=1, c_inter=16,
                S=2048 * 2, W=_swiglu_bytes(2048, 768), layers=16, microbatches=1,
                zipf_s=1.4, adversarial=(0, 1, 2, 3), adv_p=0.6)

CONFIGS = {c.name: c for c in (TINY, MIXTRAL, QWEN3, DSV3, STRESS)}


def get(name: str) -> Config:
    return CONFIGS[name]
