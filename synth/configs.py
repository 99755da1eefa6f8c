"""Workload shapes: transformer / MoE weight sets and a paged KV pool.

The paper evaluates engines whose per-GPU model state spans 8 to 124 GiB and
whose shadow runtime keeps a fixed private pool of 4-8 GiB of mutable state
(section 5.3, Shadow memory).  These presets stand in for those models with
synthetic, seeded bf16 contents of the same shapes (weights are never loaded).

Weight-set order follows a decoder-only model:
[embed, per layer (attn_norm, q, k, v, o, ffn_norm, <ffn tensors>), final_norm, lm_head].
"""
from __future__ import annotations

from dataclasses import dataclass
from math import prod

BF16 = 2  # bytes per element


@dataclass(frozen=True)
class TensorSpec:
    name: str
    shape: tuple

    @property
    def numel(self) -> int:
        return prod(self.shape)

    @property
    def nbytes(self) -> int:
        return self.numel * BF16


def _dense(layers, d, q_rows, kv_rows, o_cols, ffn, vocab_rows):
    out = [TensorSpec("embed", (vocab_rows, d))]
    for l in range(layers):
        p = f"l{l}."
        out += [
            TensorSpec(p + "attn_norm", (d,)),
            TensorSpec(p + "q", (q_rows, d)),
            TensorSpec(p + "k", (kv_rows, d)),
            TensorSpec(p + "v", (kv_rows, d)),
            TensorSpec(p + "o", (d, o_cols)),
            TensorSpec(p + "ffn_norm", (d,)),
            TensorSpec(p + "gate", (ffn, d)),
            TensorSpec(p + "up", (ffn, d)),
            TensorSpec(p + "down", (d, ffn)),
        ]
    out += [TensorSpec("final_norm", (d,)), TensorSpec("lm_head", (vocab_rows, d))]
    return out


def _moe(layers, d, q_rows, kv_rows, experts, ffn, vocab_rows):
    out = [TensorSpec("embed", (vocab_rows, d))]
    for l in range(layers):
        p = f"l{l}."
        out += [
            TensorSpec(p + "attn_norm", (d,)),
            TensorSpec(p + "q", (q_rows, d)),
            TensorSpec(p + "k", (kv_rows, d)),
            TensorSpec(p + "v", (kv_rows, d)),
            TensorSpec(p + "o", (d, q_rows)),
            TensorSpec(p + "ffn_norm", (d,)),
            TensorSpec(p + "router", (experts, d)),
        ]
        for e in range(experts):
            out += [
                TensorSpec(p + f"e{e}.gate", (ffn, d)),
                TensorSpec(p + f"e{e}.up", (ffn, d)),
                TensorSpec(p + f"e{e}.down", (d, ffn)),
            ]
    out += [TensorSpec("final_norm", (d,)), TensorSpec("lm_head", (vocab_rows, d))]
    return out


# name -> (seed, builder); seed is the data seed of that workload
WEIGHT_CONFIGS = {
    # 2 layers, d=256, 4 MHA heads of 64, SwiGLU ffn 1024, vocab 4096: 21 tensors, 8.39 MB
    "tiny": (1, lambda: _dense(2, 256, 256, 256, 256, 1024, 4096)),
    # Llama-style 8B: 32 layers, d=4096, GQA 32q/8kv x 128, ffn 14336, vocab 128256: 291 tensors
    "llama8b": (2, lambda: _dense(32, 4096, 4096, 1024, 4096, 14336, 128256)),
    # one rank of an 8-way tensor-parallel 70B: 80 layers, d=8192, 64q/8kv x 128, ffn 28672,
    # q/k/v/gate/up split on output rows, o/down on input columns, vocab split 8 ways
    "llama70b_tp8": (3, lambda: _dense(80, 8192, 8192 // 8, 1024 // 8, 8192 // 8, 28672 // 8, 128256 // 8)),
    # MoE: 48 layers, d=4096, attention as llama8b, 128 experts of ffn 768 each: 18771 tensors
    "moe": (4, lambda: _moe(48, 4096, 4096, 1024, 128, 768, 128256)),
}


def weight_set(name: str):
    """(seed, [TensorSpec]) of a named weight-set workload."""
    seed, build = WEIGHT_CONFIGS[name]
    return seed, build()


@dataclass(frozen=True)
class KVPool:
    """Fixed paged KV pool: per layer [blocks][K,V][block_tokens][kv_heads][head_dim] bf16."""

    layers: int = 32
    blocks: int = 4096
    block_tokens: int = 16
    kv_heads: int = 8
    head_dim: int = 128
    live_frac_num: int = 3
    live_frac_den: int = 5
    seed: int = 5          # data seed of the pool contents (tensor id = layer)
    map_seed: int = 1005   # live-map seed
    map_stream: int = 1
    corrupt_seed: int = 2005
    corrupt_stream: int = 2

    @property
    def unit_bytes(self) -> int:  # one block of one layer: K and V
        return 2 * self.block_tokens * self.kv_heads * self.head_dim * BF16

    @property
    def layer_bytes(self) -> int:
        return self.blocks * self.unit_bytes

    @property
    def n_live(self) -> int:
        return self.blocks * self.live_frac_num // self.live_frac_den


def kv_pool(**kw) -> KVPool:
    return KVPool(**kw)
