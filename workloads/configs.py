"""The workloads the path is specified on: five, and an fp32 twin of the second.

Shapes follow the models the paper evaluates (Section 4, "Base Models"):
Llama-3.1-8B (d=4096, d_ff=14336, 32 MLP layers) and Qwen3-8B (d=4096,
d_ff=12288, 36 MLP layers), plus one small fp32 layer.  Weights, inputs,
token ids and route tables are synthetic and seeded (see ``synth``).

Sparsity targets are CATS percentile levels k (Section 2, Eq. 3): the per-layer
threshold is the k-quantile of |SiLU(x W_gate)| pooled over ``n_cal``
calibration tokens propagated through the dense stack.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Tuple


@dataclass(frozen=True)
class Config:
    index: int                 # 0-based position in the list below; seeds derive from it
    name: str
    n_layers: int
    d: int
    d_ff: int
    dtype: str                 # "f32" or "bf16": storage type of x, weights and out
    n_cal: int                 # calibration tokens for the CATS percentile (Eq. 3)
    k_fixed: Optional[float]   # one CATS level for every layer ...
    k_range: Optional[Tuple[float, float]]  # ... or k_l ~ U[lo, hi] per layer
    vocab: Optional[int]       # None: no route table, every token takes the sparse path
    n_dense_ids: int           # vocabulary ids whose table entry selects the base path
    id_dist: Optional[str]     # "uniform" or "zipf"
    zipf_s: float
    batches: Tuple[int, ...]   # decode batch sizes the workload is run at

    @property
    def seed(self) -> int:
        return 1000 * (self.index + 1)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


CONFIGS = (
    Config(0, "c1_small_f32", 1, 512, 1536, "f32", 256, 0.50, None,
           1000, 300, "uniform", 0.0, (1,)),
    Config(1, "c2_llama8b_layer_bf16", 1, 4096, 14336, "bf16", 1024, 0.50, None,
           None, 0, None, 0.0, (1,)),
    Config(2, "c3_llama8b_stack32_bf16", 32, 4096, 14336, "bf16", 1024, None, (0.40, 0.70),
           128256, 32064, "zipf", 1.1, (1,)),
    Config(3, "c4_qwen3_8b_stack36_bf16", 36, 4096, 12288, "bf16", 1024, 0.70, None,
           128256, 32064, "zipf", 1.1, (1, 4, 16)),
    Config(4, "c5_llama8b_stack32_b64_bf16", 32, 4096, 14336, "bf16", 1024, 0.60, None,
           128256, 51302, "zipf", 1.1, (64,)),
    # the second workload with fp32 weights and activations: the precision the
    # paper's own throughput figures are measured in (Section 4)
    Config(5, "c2_llama8b_layer_f32", 1, 4096, 14336, "f32", 1024, 0.50, None,
           None, 0, None, 0.0, (1,)),
)


def get_config(key) -> Config:
    if isinstance(key, int):
        return CONFIGS[key]
    for c in CONFIGS:
        if c.name == key or c.name.startswith(key):
            return c
    raise KeyError(key)
