"""Seeded synthetic workloads for the batched speculative verify step.

This module only *builds inputs*: model shapes, random-init weights, a paged
KV cache with a shuffled block table, context lengths, draft tokens with their
draft-model probabilities, and the uniforms that make the acceptance test
deterministic.  It holds none of the verify step's own arithmetic, so both the
CPU oracle and the GPU path can consume the same inputs without sharing code.

Every random quantity comes from its own `numpy.random.SeedSequence` stream,
keyed by (seed, input kind, indices), so changing one input kind never shifts
another.  Storage formats follow the C ABI in ``include/nightjar.h``:

* bf16 tensors are ``numpy.uint16`` bit patterns, rounded to nearest-even
  from fp32 draws; fp32 tensors are ``numpy.float32``.
* K pages: ``[num_blocks][n_kv_heads][block_size][head_dim]``.
* V pages: ``[num_blocks][n_kv_heads][head_dim][block_size]`` (each head's
  block is stored dim-major so that 16 consecutive tokens of one dim are
  contiguous).
* ``block_table[B][max_blocks]`` int32, -1 past the blocks a sequence owns.

The shapes are those of the verify step the paper's planner trades off
(Sec. 2.2 and Sec. 5.1: B sequences, gamma drafts each, one target forward over
B*(gamma+1) tokens); the paper's trained checkpoints and datasets are not
available, so random-init weights of the same architecture and synthetic
context lengths stand in for them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

# Stream keys, one per input kind.
_K_WEIGHT, _K_KV, _K_PERM, _K_CTX, _K_LAST, _K_DLOGIT, _K_DSAMPLE, _K_UNIF, _K_BETA = range(1, 10)


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Llama-style decoder shape (RMSNorm, RoPE, GQA, SwiGLU, untied LM head)."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float
    rope_theta: float
    dtype: str  # "f32" or "bf16"
    block_size: int = 16

    @property
    def qkv_dim(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    def with_layers(self, n_layers: int) -> "ModelShape":
        return dataclasses.replace(self, n_layers=n_layers, name=f"{self.name}-L{n_layers}")


# Tiny fp32 decoder: d 256, 4 MHA heads of 64, FFN 688, vocab 2048.
TINY_F32 = ModelShape("tiny-f32", 1, 256, 4, 4, 64, 688, 2048, 1e-5, 1e4, "f32")
# One Llama-3-8B-shaped layer plus the LM head (GQA 32/8, FFN 14336, vocab 128256).
LLAMA8B_LAYER = ModelShape("llama3-8b-layer", 1, 4096, 32, 8, 128, 14336, 128256, 1e-5, 5e5, "bf16")
LLAMA8B = LLAMA8B_LAYER.with_layers(32)
# Qwen2.5-7B-shaped stack (GQA 28/4, FFN 18944, vocab 152064).
QWEN7B = ModelShape("qwen2.5-7b", 28, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1e6, "bf16")

# Draft model for the 8B target: Llama-3.2-1B-sized (d 2048, 16 layers, FFN 8192,
# the target's vocabulary) with 16 heads of 128 dims (the bf16 path's head size).
LLAMA1B_DRAFT = ModelShape("llama-1b-draft", 16, 2048, 16, 8, 128, 8192, 128256, 1e-5, 5e5, "bf16")

SHAPES = {s.name: s for s in (TINY_F32, LLAMA8B_LAYER, LLAMA8B, QWEN7B, LLAMA1B_DRAFT)}


def _rng(seed: int, *keys: int) -> np.random.Generator:
    return np.random.Generator(np.random.SFC64(np.random.SeedSequence(seed, spawn_key=tuple(keys))))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even) and return the uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return f32_to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    out *= np.float32(std)
    return out


_CHUNK = 1 << 24


def _normal_store(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std^2) draws stored in `dtype`, generated in chunks (no full fp32 copy)."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    buf = np.empty(min(_CHUNK, n), dtype=np.float32)
    for s0 in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s0)
        rng.standard_normal(out=buf[:m], dtype=np.float32)
        buf[:m] *= np.float32(std)
        out[s0: s0 + m] = f32_to_bf16_bits(buf[:m]) if dtype == "bf16" else buf[:m]
    return out.reshape(shape)


def _ones(n: int, dtype: str) -> np.ndarray:
    return _store(np.ones(n, dtype=np.float32), dtype)


# --------------------------------------------------------------------------
# Weights
# --------------------------------------------------------------------------
def make_weights(shape: ModelShape, seed: int = 0, std: float = 0.02) -> Dict:
    """Random-init weights: every matrix and the embedding N(0, std^2); norm gains 1.

    Row-major, reduction dimension contiguous:
      embed [V, d], lm_head [V, d], final_norm [d]; per layer
      attn_norm [d], w_qkv [(H+2Hkv)*D, d] (q rows, then k rows, then v rows),
      w_o [d, H*D], ffn_norm [d], w_gate_up [2F, d] (gate rows, then up rows),
      w_down [d, F].
    """
    s, dt = shape, shape.dtype
    w = {
        "embed": _normal_store(_rng(seed, _K_WEIGHT, 0, 0), (s.vocab, s.d_model), std, dt),
        "lm_head": _normal_store(_rng(seed, _K_WEIGHT, 0, 1), (s.vocab, s.d_model), std, dt),
        "final_norm": _ones(s.d_model, dt),
        "layers": [],
    }
    for l in range(s.n_layers):
        key = 1 + l
        w["layers"].append({
            "attn_norm": _ones(s.d_model, dt),
            "w_qkv": _normal_store(_rng(seed, _K_WEIGHT, key, 0), (s.qkv_dim, s.d_model), std, dt),
            "w_o": _normal_store(_rng(seed, _K_WEIGHT, key, 1), (s.d_model, s.n_heads * s.head_dim), std, dt),
            "ffn_norm": _ones(s.d_model, dt),
            "w_gate_up": _normal_store(_rng(seed, _K_WEIGHT, key, 2), (2 * s.ffn_dim, s.d_model), std, dt),
            "w_down": _normal_store(_rng(seed, _K_WEIGHT, key, 3), (s.d_model, s.ffn_dim), std, dt),
        })
    return w


# --------------------------------------------------------------------------
# Context: paged KV cache and block table
# --------------------------------------------------------------------------
def ctx_lengths(kind: str, B: int, seed: int = 0, **kw) -> np.ndarray:
    """Per-sequence cached context lengths.

    kind "list": the given ``values``; "fixed": all ``value``; "lognormal": clip(rint(exp(N(ln median, sigma^2))),
    lo, hi); "uniform": integers in [lo, hi].
    """
    rng = _rng(seed, _K_CTX, B)
    if kind == "list":
        return np.asarray(kw["values"], dtype=np.int32)[:B].copy()
    if kind == "fixed":
        return np.full(B, int(kw["value"]), dtype=np.int32)
    if kind == "lognormal":
        med, sigma, lo, hi = kw["median"], kw.get("sigma", 0.5), kw["lo"], kw["hi"]
        x = np.exp(rng.normal(math.log(med), sigma, size=B))
        return np.clip(np.rint(x), lo, hi).astype(np.int32)
    if kind == "uniform":
        return rng.integers(kw["lo"], kw["hi"] + 1, size=B).astype(np.int32)
    raise ValueError(kind)


def make_block_table(shape: ModelShape, ctx: Sequence[int], k_max: int, seed: int = 0, spare: float = 0.05):
    """Block table of the paged cache: sequence b owns ceil((ctx_b + k_max + 1)/16)
    physical blocks, taken in order from a shuffled pool of sum(need)*(1+spare)+1
    blocks; unused entries are -1.  Returns (table [B, max_blocks], num_blocks, max_blocks)."""
    ctx = np.asarray(ctx, dtype=np.int32)
    B, bs = len(ctx), shape.block_size
    need = [(int(c) + k_max + 1 + bs - 1) // bs for c in ctx]
    num_blocks = int(math.ceil(sum(need) * (1.0 + spare))) + 1
    perm = _rng(seed, _K_PERM, B).permutation(num_blocks).astype(np.int32)
    max_blocks = max(need)
    table = np.full((B, max_blocks), -1, dtype=np.int32)
    off = 0
    for b in range(B):
        table[b, : need[b]] = perm[off: off + need[b]]
        off += need[b]
    return table, num_blocks, max_blocks


def make_context(shape: ModelShape, ctx: Sequence[int], k_max: int, seed: int = 0,
                 spare: float = 0.05, kv_std: float = 0.5) -> Dict:
    """Paged KV cache holding ``ctx[b]`` cached tokens per sequence.

    Each sequence owns ceil((ctx_b + k_max + 1)/block_size) physical blocks (room
    for the verify window), drawn from a shuffled pool with ``spare`` extra
    blocks.  Every page entry (used or not) is N(0,1)*kv_std.
    """
    s = shape
    ctx = np.asarray(ctx, dtype=np.int32)
    B, bs = len(ctx), s.block_size
    table, num_blocks, max_blocks = make_block_table(shape, ctx, k_max, seed, spare)
    k_pages, v_pages = [], []
    for l in range(s.n_layers):
        kshape = (num_blocks, s.n_kv_heads, bs, s.head_dim)
        vshape = (num_blocks, s.n_kv_heads, s.head_dim, bs)
        k_pages.append(_normal_store(_rng(seed, _K_KV, B, l, 0), kshape, kv_std, s.dtype))
        v_pages.append(_normal_store(_rng(seed, _K_KV, B, l, 1), vshape, kv_std, s.dtype))
    return {"k_pages": k_pages, "v_pages": v_pages, "block_table": table,
            "context_lens": ctx.copy(), "num_blocks": num_blocks, "max_blocks": max_blocks}


# --------------------------------------------------------------------------
# Drafts and uniforms
# --------------------------------------------------------------------------
def _softmax64(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def _sample_rows(q: np.ndarray, u: np.ndarray) -> np.ndarray:
    """Draw one index per row of q (already normalised) with the uniforms u."""
    c = np.cumsum(q, axis=-1)
    idx = np.array([np.searchsorted(c[i], u[i] * c[i, -1], side="right") for i in range(q.shape[0])])
    return np.minimum(idx, q.shape[-1] - 1).astype(np.int32)


def make_drafts(shape: ModelShape, B: int, k: int, seed: int = 0, logit_std: float = 2.0) -> Dict:
    """Last committed tokens, k drafts per sequence with their draft probabilities,
    and the uniforms of the acceptance test.

    Draft distribution: softmax of N(0, logit_std^2) logits (fp32 result).
    uniforms[B, k+1]: columns 0..k-1 are the accept tests, column k the single
    resample / bonus draw.
    """
    V = shape.vocab
    last = _rng(seed, _K_LAST, B, k).integers(0, V, size=B).astype(np.int32)
    if k > 0:
        z = _normal(_rng(seed, _K_DLOGIT, B, k), (B, k, V), logit_std)
        q = _softmax64(z)
        u = _rng(seed, _K_DSAMPLE, B, k).random(B * k)
        toks = _sample_rows(q.reshape(B * k, V), u).reshape(B, k)
        probs = q.astype(np.float32)
    else:
        toks = np.zeros((B, 0), dtype=np.int32)
        probs = np.zeros((B, 0, V), dtype=np.float32)
    unif = _rng(seed, _K_UNIF, B, k).random((B, k + 1), dtype=np.float32)
    return {"last_tokens": last, "draft_tokens": toks, "draft_probs": probs, "uniforms": unif}


def beta_mix_draft_row(target_logits_row: np.ndarray, beta: float, seed: int, *keys: int):
    """One draft position of the beta-mixed draft model.

    q = softmax(beta * target_logits + (1 - beta) * N(0, 4)); the draft token is
    drawn from q.  The caller supplies the target logits (from a pre-pass) and
    drives the position loop, because drafting position i+1 needs the target's
    distribution after draft i.
    """
    rng = _rng(seed, _K_BETA, *keys)
    z = beta * np.asarray(target_logits_row, dtype=np.float64) + (1.0 - beta) * rng.normal(0.0, 2.0, size=len(target_logits_row))
    q = _softmax64(z[None, :])
    tok = _sample_rows(q, np.array([rng.random()]))[0]
    return int(tok), q[0].astype(np.float32)


# --------------------------------------------------------------------------
# Named workloads
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    ctx_kind: str
    ctx_kw: tuple
    grid: tuple  # ((B, k), ...)

    def ctx(self, B: int, seed: int = 0) -> np.ndarray:
        return ctx_lengths(self.ctx_kind, B, seed, **dict(self.ctx_kw))


WORKLOADS = {
    "tiny-f32": Workload("tiny-f32", TINY_F32, "list", (("values", (32, 48)),), ((2, 3),)),
    "llama8b-layer-small-batch": Workload(
        "llama8b-layer-small-batch", LLAMA8B_LAYER, "fixed", (("value", 1024),),
        tuple((B, k) for B in (1, 2, 4, 8) for k in range(6))),
    "llama8b-layer-large-batch": Workload(
        "llama8b-layer-large-batch", LLAMA8B_LAYER, "lognormal",
        (("median", 768), ("sigma", 0.5), ("lo", 128), ("hi", 2048)),
        tuple((B, k) for B in (16, 32, 64, 128) for k in range(6))),
    "llama8b-32layer": Workload(
        "llama8b-32layer", LLAMA8B, "lognormal",
        (("median", 1024), ("sigma", 0.5), ("lo", 128), ("hi", 4096)), ((64, 4),)),
    "qwen7b-28layer": Workload(
        "qwen7b-28layer", QWEN7B, "uniform", (("lo", 1024), ("hi", 4096)),
        tuple((256, k) for k in (0, 2, 4, 7))),
}

TINY_CTX = np.array([32, 48], dtype=np.int32)


def tiny_inputs(seed: int = 0, k: int = 3) -> Dict:
    """The tiny fp32 case: B=2, contexts 32 and 48, k drafts, seed 0."""
    w = make_weights(TINY_F32, seed)
    c = make_context(TINY_F32, TINY_CTX, k, seed)
    d = make_drafts(TINY_F32, 2, k, seed)
    return {"shape": TINY_F32, "weights": w, **c, **d}


# --------------------------------------------------------------------------
# Inputs generated on the device (the 32-layer and Qwen-shaped stacks, whose
# weights and caches take tens of GB): torch's seeded generator, the same
# distributions as the host generators above (not the same bits).
# --------------------------------------------------------------------------
def device_normal_bf16(gen, shape_, std: float, device="cuda"):
    """N(0, std^2) draws rounded to bf16, as int16 bit patterns, generated in
    bounded chunks."""
    import torch
    out = torch.empty(shape_, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    step = 1 << 26
    for i in range(0, flat.numel(), step):
        n = min(step, flat.numel() - i)
        flat[i:i + n] = (torch.randn(n, generator=gen, device=device, dtype=torch.float32) * std).to(torch.bfloat16)
    return out.view(torch.int16)


def device_weights(shape: ModelShape, gen, device="cuda", std: float = 0.02) -> Dict:
    """Random-init weights of `shape` on the device (bf16 bits as int16,
    row-major, the layout of make_weights); norm gains 1."""
    import torch
    ones = torch.ones(shape.d_model, dtype=torch.bfloat16, device=device).view(torch.int16)
    w = {"embed": device_normal_bf16(gen, (shape.vocab, shape.d_model), std, device),
         "lm_head": device_normal_bf16(gen, (shape.vocab, shape.d_model), std, device),
         "final_norm": ones, "layers": []}
    for _ in range(shape.n_layers):
        w["layers"].append({"attn_norm": ones, "ffn_norm": ones,
                            "w_qkv": device_normal_bf16(gen, (shape.qkv_dim, shape.d_model), std, device),
                            "w_o": device_normal_bf16(gen, (shape.d_model, shape.n_heads * shape.head_dim), std, device),
                            "w_gate_up": device_normal_bf16(gen, (2 * shape.ffn_dim, shape.d_model), std, device),
                            "w_down": device_normal_bf16(gen, (shape.d_model, shape.ffn_dim), std, device)})
    return w


def device_pages(shape: ModelShape, num_blocks: int, gen, device="cuda", kv_std: float = 0.5):
    """K and V pages of every layer, N(0,1) * kv_std in bf16 (int16 bits)."""
    kp = [device_normal_bf16(gen, (num_blocks, shape.n_kv_heads, shape.block_size, shape.head_dim), kv_std, device)
          for _ in range(shape.n_layers)]
    vp = [device_normal_bf16(gen, (num_blocks, shape.n_kv_heads, shape.head_dim, shape.block_size), kv_std, device)
          for _ in range(shape.n_layers)]
    return kp, vp
