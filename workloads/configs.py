"""Layer shapes and run parameters of the synthetic workloads.

The shapes stand in for the vision-language models the paper evaluates
(LLaVA-v1.5 7B/13B and a Qwen2-VL-7B-shaped grouped-query layer, Section 4);
their weights and datasets are not used.  Every tensor is drawn from a seeded
generator in :mod:`workloads.gen`.
"""
from dataclasses import dataclass, field
from typing import Tuple

CACHE_F16, CACHE_I8, CACHE_I4 = 0, 1, 2


@dataclass(frozen=True)
class LayerShape:
    d: int            # embedding dimension E
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    r: int            # joint QKV rank

    @property
    def n_q(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def n_kv(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def N(self) -> int:
        """Columns of the concatenated [W_q | W_k | W_v]."""
        return self.n_q + 2 * self.n_kv


@dataclass(frozen=True)
class Workload:
    cfg_id: int
    name: str
    layer: LayerShape
    spectrum: str                  # "gaussian": iid N(0, w_std^2); "decay": sigma_i ~ i^-decay_exp
    w_bits: int                    # 8: per-output-channel; 4: per-group along the contraction
    w_group: int                   # 0 for per-channel
    a_bits: int                    # per-token activation bits (also latent bits)
    cache_fmt: int                 # CACHE_F16 / CACHE_I8 / CACHE_I4
    prefill_batch: int = 1
    prefill_tokens: Tuple[int, ...] = (64,)   # token counts per sequence segment (image, text)
    outlier_count: int = 4         # channel-wise outliers in X
    outlier_scale: float = 20.0
    decode_batch: int = 1
    decode_ctx: int = 0            # cached tokens before the first decode step
    decode_steps: int = 16
    n_layers: int = 1
    w_std: float = 0.02
    decay_exp: float = 0.7
    beta: float = 0.5

    @property
    def prefill_len(self) -> int:
        return int(sum(self.prefill_tokens))

    @property
    def prefill_M(self) -> int:
        return self.prefill_batch * self.prefill_len


_LLAVA7B = LayerShape(d=4096, n_q_heads=32, n_kv_heads=32, head_dim=128, r=1536)
_QWEN2VL7B = LayerShape(d=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, r=1024)
# 13B-shaped stack layer; r here is nominal, each layer's rank comes from
# gen.stack_ranks (seeded, multiples of 128 in [1024, 3072]).
_LLAVA13B = LayerShape(d=5120, n_q_heads=40, n_kv_heads=40, head_dim=128, r=2048)

WORKLOADS = {
    # Tiny single layer: correctness case the oracle finishes in seconds.
    1: Workload(1, "tiny", LayerShape(d=256, n_q_heads=4, n_kv_heads=4, head_dim=64, r=128),
                spectrum="gaussian", w_bits=8, w_group=0, a_bits=8, cache_fmt=CACHE_F16,
                prefill_batch=1, prefill_tokens=(64,), outlier_count=4, outlier_scale=20.0,
                decode_batch=1, decode_ctx=64, decode_steps=16),
    # LLaVA-1.5-7B-shaped layer, prefill of 4 x (576 image + 64 text) tokens, W8A8.
    2: Workload(2, "llava7b_prefill", _LLAVA7B, spectrum="decay", w_bits=8, w_group=0, a_bits=8,
                cache_fmt=CACHE_F16, prefill_batch=4, prefill_tokens=(576, 64),
                outlier_count=41, outlier_scale=30.0, n_layers=32),
    # Same layer, decode: batch 16 over 4096 cached tokens in an fp16 latent cache.
    3: Workload(3, "llava7b_decode", _LLAVA7B, spectrum="decay", w_bits=8, w_group=0, a_bits=8,
                cache_fmt=CACHE_F16, outlier_count=41, outlier_scale=30.0,
                decode_batch=16, decode_ctx=4096, decode_steps=256, n_layers=32),
    # Qwen2-VL-7B-shaped GQA layer: int8 latent cache, W4A8 (int4 per-group-128 weights).
    4: Workload(4, "qwen2vl7b_gqa_decode", _QWEN2VL7B, spectrum="decay", w_bits=4, w_group=128,
                a_bits=8, cache_fmt=CACHE_I8, outlier_count=36, outlier_scale=30.0,
                decode_batch=32, decode_ctx=8192, decode_steps=64, n_layers=28),
    # LLaVA-1.5-13B-shaped stack of 40 layers with per-layer ranks, W4A4 (int4
    # per-token activations, int4 per-group-128 weights), int4 latent cache;
    # prefill of 8 x (576 image + 128 text) tokens, decode at batch 8 over 4096.
    5: Workload(5, "llava13b_stack", _LLAVA13B, spectrum="decay", w_bits=4, w_group=128, a_bits=4,
                cache_fmt=CACHE_I4, prefill_batch=8, prefill_tokens=(576, 128), outlier_count=51,
                outlier_scale=30.0, decode_batch=8, decode_ctx=4096, decode_steps=64, n_layers=40),
}


def get(cfg_id: int) -> Workload:
    return WORKLOADS[cfg_id]
