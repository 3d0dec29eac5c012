"""Algorithmic byte and FLOP model of one verify step, and MI355X peaks.

"Algorithmic" means what the method has to move or compute, not what a
particular kernel happens to do: each weight byte once, each cached KV byte of
each sequence once, the logits once, the acceptance reads.  Kernel
measurements are divided by these figures to get roofline fractions.
"""
from __future__ import annotations

from typing import Dict, Sequence

HBM_BYTES_PER_S = 8.0e12          # MI355X HBM3E peak
BF16_MFMA_FLOPS = 2.5e15          # dense bf16 matrix peak
FP32_VALU_FLOPS = 157.3e12

_ELT = {"bf16": 2, "f32": 4}


def kv_bytes_per_token(n_layers: int, n_kv_heads: int, head_dim: int, elt_bytes: int = 2) -> int:
    """Cached K and V bytes one token occupies across all layers."""
    return n_layers * 2 * n_kv_heads * head_dim * elt_bytes


def layer_params(shape) -> int:
    s = shape
    return (s.d_model * s.n_heads * s.head_dim + 2 * s.d_model * s.n_kv_heads * s.head_dim
            + s.n_heads * s.head_dim * s.d_model + 3 * s.d_model * s.ffn_dim)


def gemm_shapes(shape, M: int):
    """(name, M, N, K) of every GEMM of the step, per layer first, then the LM head."""
    s = shape
    out = []
    for _ in range(s.n_layers):
        out += [("qkv", M, s.qkv_dim, s.d_model), ("o", M, s.d_model, s.n_heads * s.head_dim),
                ("gate_up", M, 2 * s.ffn_dim, s.d_model), ("down", M, s.d_model, s.ffn_dim)]
    out.append(("lm_head", M, s.vocab, s.d_model))
    return out


def gemm_bytes(M: int, N: int, K: int, elt: int = 2, out_elt: int = 4) -> int:
    """Weight read once, activations read once, output written once."""
    return N * K * elt + M * K * elt + M * N * out_elt


def step_model(shape, B: int, k: int, ctx: Sequence[int]) -> Dict[str, float]:
    """Algorithmic bytes and FLOPs of one verify step at (B, k) with contexts ctx."""
    s = shape
    e = _ELT[s.dtype]
    T = k + 1
    M = B * T
    weights = e * (s.n_layers * layer_params(s) + s.vocab * s.d_model)
    kv_read = sum(int(c) for c in ctx) * kv_bytes_per_token(s.n_layers, s.n_kv_heads, s.head_dim, e)
    window_store = M * kv_bytes_per_token(s.n_layers, s.n_kv_heads, s.head_dim, e)
    logits = M * s.vocab * 4
    accept = 2 * B * s.vocab * 4 + B * k * 4
    gemm_flops = 2 * M * (s.n_layers * layer_params(s) + s.vocab * s.d_model)
    attn_flops = sum(4 * T * s.n_heads * s.head_dim * (int(c) + (k + 2) / 2) * s.n_layers for c in ctx)
    total = weights + kv_read + window_store + logits + accept
    t_roof = max(weights / HBM_BYTES_PER_S, gemm_flops / BF16_MFMA_FLOPS) \
        + (kv_read + window_store) / HBM_BYTES_PER_S + (logits + accept) / HBM_BYTES_PER_S
    return {"M": M, "weight_bytes": weights, "kv_bytes": kv_read, "window_bytes": window_store,
            "logit_bytes": logits, "accept_bytes": accept, "bytes": total,
            "gemm_flops": gemm_flops, "attn_flops": attn_flops, "t_roof_s": t_roof}


def lm_head_bytes(shape, M: int) -> int:
    """LM-head GEMM: weight [V, d] once, activations [M, d], fp32 logits [M, V]."""
    return gemm_bytes(M, shape.vocab, shape.d_model, _ELT[shape.dtype], 4)
