"""Model shapes and verify-step workloads.

The five named workloads are the paper's edge-scale model family
(MobileLLaMA-1.4B, Vicuna-7B, Vicuna-13B; Section 5 "Models and testbeds")
plus a tiny fp32 decoder and a 32k-context 7B case.  Shapes are the public
Llama-style architectures; weights are random (the trained checkpoints and
prompt embeddings are not used).  Extra small shapes exist only so parity tests
finish quickly while still spanning several kernel tiles.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    dtype: str                 # "f32" or "bf16": storage type of weights and KV
    n_prompt: int = 3          # prompt tokens (1 EPT each) -- Section 5
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    init_std: float = 0.02

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def layer_params(self) -> int:
        h, f = self.hidden, self.ffn
        return (self.qkv_rows * h + h * self.n_heads * self.head_dim
                + 2 * f * h + h * f + 2 * h)

    def total_params(self) -> int:
        """Decoder parameters excluding the prompt-token table."""
        return (self.n_layers * self.layer_params() + 2 * self.vocab * self.hidden
                + self.hidden)

    def with_layers(self, n: int) -> "ModelShape":
        return replace(self, name=f"{self.name}-{n}L", n_layers=n)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    cache_len: int             # L: tokens already in the KV cache
    tree: str                  # "candidates:<n>" or "total:<T>"
    max_depth: int             # deepest candidate (root = depth 0)
    kv_init: str               # "prefill" (oracle prefill of random ids) or "normal"
    seed_base: int
    max_fanout: int = 4
    capacity_extra: int = 128  # cache slots beyond L (tree staging + growth)

    @property
    def seeds(self):
        c = self.seed_base
        return dict(weights=1000 + c, kv=2000 + c, tree=3000 + c, tokens=4000 + c)

    @property
    def capacity(self) -> int:
        return self.cache_len + self.capacity_extra


TINY = ModelShape("tiny-f32", 2, 256, 4, 4, 64, 688, 1000, "f32")
MLLAMA_1B4 = ModelShape("mobilellama-1.4b", 24, 2048, 16, 16, 128, 5632, 32000, "bf16")
VICUNA_7B = ModelShape("vicuna-7b", 32, 4096, 32, 32, 128, 11008, 32000, "bf16")
VICUNA_13B = ModelShape("vicuna-13b", 40, 5120, 40, 40, 128, 13824, 32000, "bf16")

# small bf16 shapes for fast parity tests (several tiles, ragged vocab/ffn/L)
SMALL_BF16 = ModelShape("small-bf16", 2, 512, 4, 4, 128, 1344, 1000, "bf16")
SMALL_GQA = ModelShape("small-gqa-bf16", 2, 512, 4, 2, 128, 1408, 1000, "bf16")
# narrow hidden, 7B-wide heads and ffn: the QKV and gate/up GEMMs take the
# 7B tilings (256 QKV tiles of 3 row groups; 230 gate/up tiles of 48
# features, the last one ragged) at a size the oracle runs in seconds
WIDE_BF16 = ModelShape("wide-bf16", 1, 512, 32, 32, 128, 11008, 1000, "bf16")
# narrow hidden, 1.4B-wide heads and ffn: QKV and gate/up take the 1.4B
# tilings (split QKV; 176 gate/up tiles of 2 feature groups, each group's
# two k-steps on two waves)
MID_BF16 = ModelShape("mid-bf16", 1, 512, 16, 16, 128, 5632, 1000, "bf16")
# grouped-query heads whose QKV groups (80 x 8 = 640) leave the last 3-group
# QKV tile with one real group
WIDE_GQA = ModelShape("wide-gqa-bf16", 1, 512, 64, 8, 128, 1344, 1000, "bf16")

WORKLOADS = {
    # 0: tiny fp32 decoder, 128-token prefix from a real prefill, 10-candidate tree
    "tiny": Workload("tiny", TINY, 128, "candidates:10", 4, "prefill", 0),
    # 1: MobileLLaMA-1.4B shape, 1k prefix, 32-candidate tree
    "1.4b": Workload("1.4b", MLLAMA_1B4, 1024, "candidates:32", 4, "normal", 1),
    # 2: Vicuna-7B shape, 2k prefix, 64 query tokens in total
    "7b": Workload("7b", VICUNA_7B, 2048, "total:64", 5, "normal", 2),
    # 3: Vicuna-13B shape, 4k prefix, tree-size sweep (T set per run)
    "13b": Workload("13b", VICUNA_13B, 4096, "total:64", 5, "normal", 3),
    # 4: 7B shape with a 32k prefix of N(0,1) keys/values
    "7b-32k": Workload("7b-32k", VICUNA_7B, 32768, "total:64", 5, "normal", 4),
    # test-only shapes
    "small": Workload("small", SMALL_BF16, 300, "total:40", 4, "normal", 10),
    "small-gqa": Workload("small-gqa", SMALL_GQA, 77, "total:29", 4, "normal", 11),
    "wide": Workload("wide", WIDE_BF16, 300, "total:40", 4, "normal", 12),
    "mid": Workload("mid", MID_BF16, 300, "total:40", 4, "normal", 13),
    "wide-gqa": Workload("wide-gqa", WIDE_GQA, 300, "total:40", 4, "normal", 14),
}

T13B_SWEEP = (16, 32, 64, 128)


def workload(name: str, tree: Optional[str] = None, n_layers: Optional[int] = None,
             cache_len: Optional[int] = None) -> Workload:
    w = WORKLOADS[name]
    kw = {}
    if tree is not None:
        kw["tree"] = tree
    if n_layers is not None:
        kw["shape"] = w.shape.with_layers(n_layers)
    if cache_len is not None:
        kw["cache_len"] = cache_len
    if kw:
        w = replace(w, **kw)
    return w
