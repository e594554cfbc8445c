"""Seeded synthetic weights, KV caches and token streams.

All tensors come from `synth.rng` (device-independent), so the same call gives
bit-identical values on the CPU and on the GPU.  Layouts are the ones the C ABI
documents:

  tok_emb     [vocab, hidden]
  prompt_emb  [n_prompt, hidden]
  attn_norm   [hidden]                       (per layer)
  w_qkv       [(n_heads + 2 n_kv_heads) head_dim, hidden]   rows: q | k | v
  w_o         [hidden, n_heads head_dim]
  mlp_norm    [hidden]
  w_gate_up   [2 ffn, hidden]                rows: gate | up
  w_down      [hidden, ffn]
  final_norm  [hidden]
  lm_head     [vocab, hidden]
  K cache     [layer][kv_head][capacity][head_dim]   (keys after RoPE)
  V cache     [layer][kv_head][head_dim][capacity]   (values, position-minor)

Weights are N(0, init_std^2) (approximately; see `synth.rng`).  Norm gains are
1 unless `gain_std` > 0, in which case they are 1 + N(0, gain_std^2), which the
tests use so that a misplaced gain cannot go unnoticed.
"""
from __future__ import annotations

from typing import Dict, List

import torch

from . import rng
from .configs import ModelShape, Workload

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def _w(shape, seed, name, std, dtype, device):
    return rng.normal(shape, seed, name, std, dtype=dtype, device=device)


def _gain(n, seed, name, gain_std, dtype, device):
    if gain_std <= 0:
        return torch.ones(n, dtype=dtype, device=device)
    g = rng.normal((n,), seed, name, gain_std, dtype=torch.float32, device=device)
    return (g + 1.0).to(dtype)


def make_weights(shape: ModelShape, seed: int, device="cpu", gain_std: float = 0.0,
                 layers=None) -> Dict:
    """Weights of `shape`.  `layers` restricts generation to a subset of layer
    indices (others are None); used to build partial copies cheaply."""
    dt = TORCH_DTYPE[shape.dtype]
    s, H, F, std = seed, shape.hidden, shape.ffn, shape.init_std
    nq = shape.n_heads * shape.head_dim
    W: Dict = {
        "tok_emb": _w((shape.vocab, H), s, "tok_emb", std, dt, device),
        "prompt_emb": _w((shape.n_prompt, H), s, "prompt_emb", std, dt, device),
        "final_norm": _gain(H, s, "final_norm", gain_std, dt, device),
        "lm_head": _w((shape.vocab, H), s, "lm_head", std, dt, device),
        "layers": [],
    }
    for l in range(shape.n_layers):
        if layers is not None and l not in layers:
            W["layers"].append(None)
            continue
        W["layers"].append({
            "attn_norm": _gain(H, s, f"L{l}.attn_norm", gain_std, dt, device),
            "w_qkv": _w((shape.qkv_rows, H), s, f"L{l}.w_qkv", std, dt, device),
            "w_o": _w((H, nq), s, f"L{l}.w_o", std, dt, device),
            "mlp_norm": _gain(H, s, f"L{l}.mlp_norm", gain_std, dt, device),
            "w_gate_up": _w((2 * F, H), s, f"L{l}.w_gate_up", std, dt, device),
            "w_down": _w((H, F), s, f"L{l}.w_down", std, dt, device),
        })
    return W


def empty_kv(shape: ModelShape, capacity: int, device="cpu"):
    dt = TORCH_DTYPE[shape.dtype]
    k = torch.zeros((shape.n_layers, shape.n_kv_heads, capacity, shape.head_dim),
                    dtype=dt, device=device)
    v = torch.zeros((shape.n_layers, shape.n_kv_heads, shape.head_dim, capacity),
                    dtype=dt, device=device)
    return k, v


def fill_kv_normal(k: torch.Tensor, v: torch.Tensor, L: int, seed: int,
                   std: float = 1.0):
    """Fill positions [0, L) of every layer/head with N(0, std^2) keys and values.

    Values are drawn in the logical order [layer][kv_head][pos][dim] for both K
    and V (so the V draw does not depend on its transposed storage)."""
    n_layers, nkv, cap, d = k.shape
    assert L <= cap
    per_layer = nkv * L * d
    for l in range(n_layers):
        kl = torch.empty((nkv, L, d), dtype=k.dtype, device=k.device)
        rng.normal_(kl, seed, "kcache", std, offset=l * per_layer)
        k[l, :, :L, :].copy_(kl)
        rng.normal_(kl, seed, "vcache", std, offset=l * per_layer)
        v[l, :, :, :L].copy_(kl.transpose(1, 2))
        del kl


def tokens(n: int, vocab: int, seed: int, name: str = "tokens", device="cpu"):
    return rng.randint(n, vocab, seed, name, device=device)
