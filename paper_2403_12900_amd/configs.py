"""Model shapes and workload recipes of the five decode configurations.

Section IV (Methodology) serves Llama 2 with three generation-directive levels:
L0 (no directive), L1 ("brief"), L2 ("very brief").  No trained weights or
datasets are used here: every model is random-init from a seed and every
prompt is seeded synthetic token ids whose lengths follow the recipe below.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-5
    bf16: bool = True
    kv_bf16: Optional[bool] = None   # KV-cache format; None: the weight format

    @property
    def kv_is_bf16(self) -> bool:
        return self.bf16 if self.kv_bf16 is None else self.kv_bf16

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def weight_elements_per_step(self) -> int:
        """Elements of every matrix a decode step streams (projections of all layers + LM head)."""
        d, hd, f = self.d_model, self.head_dim, self.d_ff
        per_layer = self.qkv_rows * d + d * self.n_heads * hd + 2 * f * d + d * f
        return self.n_layers * per_layer + self.vocab * d

    @property
    def weight_bytes(self) -> int:
        return 2 if self.bf16 else 4

    def kv_bytes_per_token(self) -> int:
        """K and V of one position over all layers."""
        return 2 * self.n_layers * self.n_kv_heads * self.head_dim * (2 if self.kv_is_bf16 else 4)


@dataclasses.dataclass(frozen=True)
class WorkloadRecipe:
    batch: int
    # Fixed user-prompt lengths (tiny / latency configs) or a lognormal recipe.
    prompt_lens: Optional[Tuple[int, ...]] = None
    prompt_median: float = 0.0
    prompt_clip: Tuple[int, int] = (1, 1)
    # Directive prefix length per level L0/L1/L2; a single-level recipe uses one entry.
    prefix_lens: Tuple[int, ...] = (0,)
    stop_lens: Optional[Tuple[int, ...]] = None
    stop_medians: Tuple[float, ...] = ()
    stop_clip: Tuple[int, int] = (1, 1)
    sigma: float = 0.6


@dataclasses.dataclass(frozen=True)
class DecodeConfig:
    name: str
    model: ModelConfig
    workload: WorkloadRecipe
    weight_seed: int
    workload_seed: int


TINY = ModelConfig(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ff=688, vocab=1024, bf16=False)
LLAMA2_7B = ModelConfig(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128, d_ff=11008, vocab=32000)
LLAMA2_13B = ModelConfig(n_layers=40, d_model=5120, n_heads=40, n_kv_heads=40, head_dim=128, d_ff=13824, vocab=32000)
# The 70B shape keeps its (grouped, 8x smaller per token) KV cache in fp32.
# With a bf16 cache, two implementations that compute each key/value before
# rounding in different but valid arithmetic (fp64 and fp32) already differ by
# 0.061 in max-abs logit on a 16-token request at this shape (the oracle alone,
# tests/test_kv_rounding_floor.py), above the 5e-2 parity tolerance; with an
# fp32 cache they differ by 1.1e-4.  fp32 costs ~3% of the step's bytes.
LLAMA2_70B = ModelConfig(n_layers=80, d_model=8192, n_heads=64, n_kv_heads=8, head_dim=128, d_ff=28672, vocab=32000,
                         kv_bf16=False)

_DIRECTIVE_STOPS = (400.0, 120.0, 40.0)   # generation-length medians for L0 / L1 / L2

CONFIGS = {
    "c1": DecodeConfig("c1_tiny_fp32_b4", TINY,
                       WorkloadRecipe(batch=4, prompt_lens=(16, 24, 32, 8), prefix_lens=(6,),
                                      stop_lens=(32, 8, 16, 4)), 1001, 2001),
    "c2": DecodeConfig("c2_llama2_7b_bf16_b1", LLAMA2_7B,
                       WorkloadRecipe(batch=1, prompt_lens=(128,), prefix_lens=(0,), stop_lens=(256,)), 1002, 2002),
    "c3": DecodeConfig("c3_llama2_7b_bf16_b32_ragged", LLAMA2_7B,
                       WorkloadRecipe(batch=32, prompt_median=200.0, prompt_clip=(16, 1024), prefix_lens=(0, 8, 12),
                                      stop_medians=_DIRECTIVE_STOPS, stop_clip=(1, 1024)), 1003, 2003),
    "c4": DecodeConfig("c4_llama2_13b_bf16_b64_paged", LLAMA2_13B,
                       WorkloadRecipe(batch=64, prompt_median=200.0, prompt_clip=(16, 1024), prefix_lens=(0, 8, 12),
                                      stop_medians=_DIRECTIVE_STOPS, stop_clip=(1, 1024)), 1004, 2004),
    "c5": DecodeConfig("c5_llama2_70b_gqa_bf16_fp32kv_b16", LLAMA2_70B,
                       WorkloadRecipe(batch=16, prompt_median=512.0, prompt_clip=(32, 2048), prefix_lens=(0, 8, 12),
                                      stop_medians=_DIRECTIVE_STOPS, stop_clip=(1, 1024)), 1005, 2005),
}
